// Host layer of the C ABI declared in include/tsubame.h: argument
// validation (before anything is enqueued), workspace sizing and carving,
// status strings, and the stage sequence of tsb_step.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include <hip/hip_runtime.h>

#include "tsb_internal.hpp"
#include "tsb_kernels.hpp"

namespace {

thread_local char g_last_error[512] = "";

tsb_status fail(tsb_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
tsb_status fail(tsb_status s, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return s;
}

tsb_status hip_fail(hipError_t e, const char* where) {
    return fail(TSB_E_HIP, "%s: %s (%d)", where, hipGetErrorString(e), (int)e);
}

tsb_status check_config(const tsb_config* c) {
    if (!c) return fail(TSB_E_NULL, "cfg is NULL");
    if (c->R < 1) return fail(TSB_E_SHAPE, "R=%d must be >= 1", c->R);
    if (c->D < 1 || c->D > TSB_MAX_D) return fail(TSB_E_SHAPE, "D=%d must be in [1, %d]", c->D, TSB_MAX_D);
    if (c->K < 1 || c->K > TSB_MAX_K) return fail(TSB_E_SHAPE, "K=%d must be in [1, %d]", c->K, TSB_MAX_K);
    if (c->V < c->K || c->V > (1 << 30)) return fail(TSB_E_SHAPE, "V=%d must be in [K=%d, 2^30]", c->V, c->K);
    if (c->B < 0 || c->B > TSB_MAX_B) return fail(TSB_E_SHAPE, "B=%d must be in [0, %d]", c->B, TSB_MAX_B);
    if ((long long)c->R * (c->B + 1) > (1ll << 31) / 64)
        return fail(TSB_E_SHAPE, "R*(B+1)=%lld too large", (long long)c->R * (c->B + 1));
    if (c->dtype != TSB_F32 && c->dtype != TSB_BF16) return fail(TSB_E_DTYPE, "dtype=%u unknown", c->dtype);
    if (!(isfinite(c->temperature) && c->temperature > 0.f))
        return fail(TSB_E_TEMPERATURE, "temperature=%g must be finite and > 0", (double)c->temperature);
    if ((c->flags & TSB_FLAG_READ_ROWS) && (c->flags & TSB_FLAG_STREAM_ROWS))
        return fail(TSB_E_SHAPE, "flags: TSB_FLAG_READ_ROWS and TSB_FLAG_STREAM_ROWS exclude each other");
    return TSB_OK;
}

tsb_status check_ws(const tsb_config* c, void* ws, size_t bytes) {
    const size_t need = tsb_workspace_bytes(c);
    if (!ws) return fail(TSB_E_NULL, "workspace is NULL");
    if (((uintptr_t)ws & 255) != 0) return fail(TSB_E_WORKSPACE, "workspace not 256-byte aligned");
    if (bytes < need) return fail(TSB_E_WORKSPACE, "workspace has %zu bytes, needs %zu", bytes, need);
    return TSB_OK;
}

tsb_status check_tree(const tsb_tree* t) {
    if (!t) return fail(TSB_E_NULL, "tree is NULL");
    if (!t->parent || !t->depth || !t->rank || !t->n_children || !t->first_child || !t->score || !t->n_nodes ||
        !t->plan_margin)
        return fail(TSB_E_NULL, "a tree array is NULL");
    return TSB_OK;
}

tsb_status check_verdict(const tsb_verdict* o) {
    if (!o) return fail(TSB_E_NULL, "verdict is NULL");
    if (!o->n_acc || !o->acc_node || !o->acc_tok || !o->bonus || !o->req_status)
        return fail(TSB_E_NULL, "a required verdict array is NULL");
    return TSB_OK;
}

tsb_status check_pool(const tsb_config* c, int P, const float* trans) {
    const int pmax = c->V < tsb::kPoolMax ? c->V : tsb::kPoolMax;
    if (P < c->K || P > pmax) return fail(TSB_E_SHAPE, "P=%d must be in [K=%d, %d]", P, c->K, pmax);
    if (c->D > 1 && !trans) return fail(TSB_E_NULL, "trans is NULL with D=%d", c->D);
    return TSB_OK;
}

tsb_status check_pool_ws(const tsb_config* c, int P, void* ws, size_t bytes) {
    const size_t need = tsb::pool_ws_bytes(*c, P);
    if (!ws) return fail(TSB_E_NULL, "workspace is NULL");
    if (((uintptr_t)ws & 255) != 0) return fail(TSB_E_WORKSPACE, "workspace not 256-byte aligned");
    if (bytes < need) return fail(TSB_E_WORKSPACE, "workspace has %zu bytes, needs %zu", bytes, need);
    return TSB_OK;
}

float inv_temperature(float T) {
    volatile float one = 1.0f;  // binary32 division, correctly rounded
    return one / T;
}

#define TRY(x)                              \
    do {                                    \
        const tsb_status s__ = (x);         \
        if (s__ != TSB_OK) return s__;      \
    } while (0)

// Scratch of tsb_step_noalloc: a file-scope device array, one copy per GPU
// the library runs on, held until the process ends. In host code `scratch`
// only names the symbol; its device address on the current GPU comes from
// hipGetSymbolAddress, taken once per device on the first call there.
__device__ __align__(256) unsigned char scratch[TSB_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

tsb_status scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "tsb_step_noalloc/hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(TSB_E_DEVICE, "device %d beyond the %d the library tracks", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "tsb_step_noalloc/hipGetSymbolAddress(scratch)");
        if (!p || ((uintptr_t)p & 255) != 0) return fail(TSB_E_DEVICE, "scratch symbol has no aligned device address");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return TSB_OK;
}

}  // namespace

namespace tsb {
ProfileHook& profile_hook() {
    static thread_local ProfileHook h;
    return h;
}

// The tsb_stats counter block: one per device (a file-scope array; in host
// code its name is not a device address: the address comes from
// hipGetSymbolAddress, taken once per device).
__device__ __align__(256) unsigned long long counters[kStCount];
static_assert(sizeof(tsb_stats) == kStCount * sizeof(unsigned long long), "tsb_stats layout");
thread_local bool g_stats_on = false;
std::mutex g_counters_mu;
void* g_counters_ptr[kMaxDevices];

hipError_t counters_address(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_counters_mu);
    if (!g_counters_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(counters));
        if (e != hipSuccess) return e;
        g_counters_ptr[dev] = p;
    }
    *out = g_counters_ptr[dev];
    return hipSuccess;
}

unsigned long long* stats_ptr() {
    if (!g_stats_on) return nullptr;
    void* p = nullptr;
    return counters_address(&p) == hipSuccess ? (unsigned long long*)p : nullptr;
}
}  // namespace tsb

extern "C" {

size_t tsb_workspace_bytes(const tsb_config* cfg) {
    if (!cfg) return 0;
    char saved[sizeof g_last_error];
    memcpy(saved, g_last_error, sizeof saved);
    const tsb_status s = check_config(cfg);
    memcpy(g_last_error, saved, sizeof saved);
    if (s != TSB_OK) return 0;
    const size_t m = tsb::ws_bytes(*cfg);
    return m < 256 ? 256 : m;
}

tsb_status tsb_plan(const tsb_config* cfg, const void* draft, double* draft_lse, int32_t* topk_tok, float* topk_lp,
                    const tsb_tree* tree, int32_t* req_status, void* workspace, size_t workspace_bytes,
                    hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    if (!draft || !draft_lse || !topk_tok || !topk_lp || !req_status)
        return fail(TSB_E_NULL, "tsb_plan: a required array is NULL");
    TRY(check_tree(tree));
    TRY(check_ws(cfg, workspace, workspace_bytes));
    const hipError_t e = tsb::launch_plan(*cfg, inv_temperature(cfg->temperature), draft, draft_lse, topk_tok,
                                          topk_lp, *tree, req_status, (char*)workspace, stream);
    return e == hipSuccess ? TSB_OK : hip_fail(e, "tsb_plan");
}

tsb_status tsb_plan_ep(const tsb_config* cfg, int32_t frontier, const void* draft, double* draft_lse,
                       int32_t* topk_tok, float* topk_lp, const tsb_tree* tree, int32_t* req_status,
                       void* workspace, size_t workspace_bytes, hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    if (frontier < 1 || frontier > tsb::kEpFrontierLimit)
        return fail(TSB_E_SHAPE, "frontier=%d must be in [1, %d]", frontier, tsb::kEpFrontierLimit);
    if (tsb::ep_generated_bound(*cfg, frontier) < 0)
        return fail(TSB_E_SHAPE, "expand-then-prune with K=%d, D=%d, frontier=%d generates more nodes than a "
                    "workgroup holds", cfg->K, cfg->D, frontier);
    if (!draft || !draft_lse || !topk_tok || !topk_lp || !req_status)
        return fail(TSB_E_NULL, "tsb_plan_ep: a required array is NULL");
    TRY(check_tree(tree));
    TRY(check_ws(cfg, workspace, workspace_bytes));
    const hipError_t e = tsb::launch_plan(*cfg, inv_temperature(cfg->temperature), draft, draft_lse, topk_tok,
                                          topk_lp, *tree, req_status, (char*)workspace, stream, frontier);
    return e == hipSuccess ? TSB_OK : hip_fail(e, "tsb_plan_ep");
}

tsb_status tsb_replay(const tsb_config* cfg, const void* draft, const int32_t* topk_tok, const tsb_tree* tree,
                      uint32_t step, int32_t* node_tok, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    if (!draft || !topk_tok || !node_tok) return fail(TSB_E_NULL, "tsb_replay: a required array is NULL");
    TRY(check_tree(tree));
    TRY(check_ws(cfg, workspace, workspace_bytes));
    const hipError_t e = tsb::launch_replay(*cfg, inv_temperature(cfg->temperature), draft, topk_tok, *tree, step,
                                            node_tok, (char*)workspace, stream);
    return e == hipSuccess ? TSB_OK : hip_fail(e, "tsb_replay");
}

tsb_status tsb_verify(const tsb_config* cfg, const void* draft, const double* draft_lse, const void* target,
                      const tsb_tree* tree, const int32_t* node_tok, uint32_t step, const tsb_verdict* out,
                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    if (!draft || !draft_lse || !target || !node_tok) return fail(TSB_E_NULL, "tsb_verify: a required array is NULL");
    TRY(check_tree(tree));
    TRY(check_verdict(out));
    TRY(check_ws(cfg, workspace, workspace_bytes));
    const hipError_t e = tsb::launch_verify(*cfg, inv_temperature(cfg->temperature), draft, draft_lse, target, *tree,
                                            node_tok, step, *out, (char*)workspace, stream);
    return e == hipSuccess ? TSB_OK : hip_fail(e, "tsb_verify");
}

namespace {

// The stages of a vocabulary-wide round: planner, then the replay scan with
// the target stream in its grid, then the walk. A large target is streamed in
// full only for traversal verification (which needs every row) and for the
// optional normaliser output; otherwise the scan's grid only clears the
// exchange slots and the walk reads the rows of the nodes it enters.
tsb_status step_round(const tsb_config* cfg, const void* draft, const void* target, uint32_t step,
                      double* draft_lse, int32_t* topk_tok, float* topk_lp, const tsb_tree* tree,
                      int32_t* node_tok, const tsb_verdict* out, char* ws, hipStream_t stream, bool traversal,
                      const char* name) {
    char where[64];
    const float invT = inv_temperature(cfg->temperature);
    // a walk that reads the rows it enters gets rows 0 and 1 from the
    // planner's grid
    const tsb::ChainJob cj = tsb::chain_job(*cfg, target, ws);
    hipError_t e = tsb::launch_plan(*cfg, invT, draft, draft_lse, topk_tok, topk_lp, *tree, out->req_status, ws, stream,
                                    0, traversal ? nullptr : &cj);
    if (e != hipSuccess) return hip_fail(e, (snprintf(where, sizeof where, "%s/plan", name), where));
    const tsb::TargetJob tj = tsb::target_job(*cfg, target, *tree, traversal ? nullptr : draft_lse, ws,
                                              traversal || out->target_lse != nullptr ||
                                                  !tsb::walk_reads_rows(*cfg));
    e = tsb::launch_replay(*cfg, invT, draft, topk_tok, *tree, step, node_tok, ws, stream, &tj);
    if (e != hipSuccess) return hip_fail(e, (snprintf(where, sizeof where, "%s/replay+target", name), where));
    e = traversal ? tsb::launch_verify_traversal(*cfg, invT, draft, draft_lse, target, *tree, node_tok, step, *out, ws,
                                                 stream, tsb::kStageWalk)
                  : tsb::launch_verify(*cfg, invT, draft, draft_lse, target, *tree, node_tok, step, *out, ws, stream,
                                       tsb::kStageWalk | tsb::kWalkRecords);
    if (e != hipSuccess) return hip_fail(e, (snprintf(where, sizeof where, "%s/walk", name), where));
    return TSB_OK;
}

}  // namespace

tsb_status tsb_step(const tsb_config* cfg, const void* draft, const void* target, uint32_t step, double* draft_lse,
                    int32_t* topk_tok, float* topk_lp, const tsb_tree* tree, int32_t* node_tok,
                    const tsb_verdict* out, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    if (!draft || !target || !draft_lse || !topk_tok || !topk_lp || !node_tok)
        return fail(TSB_E_NULL, "tsb_step: a required array is NULL");
    TRY(check_tree(tree));
    TRY(check_verdict(out));
    TRY(check_ws(cfg, workspace, workspace_bytes));
    return step_round(cfg, draft, target, step, draft_lse, topk_tok, topk_lp, tree, node_tok, out, (char*)workspace,
                      stream, false, "tsb_step");
}

tsb_status tsb_verify_traversal(const tsb_config* cfg, const void* draft, const double* draft_lse,
                                const void* target, const tsb_tree* tree, const int32_t* node_tok, uint32_t step,
                                const tsb_verdict* out, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    if (!draft || !draft_lse || !target || !node_tok)
        return fail(TSB_E_NULL, "tsb_verify_traversal: a required array is NULL");
    TRY(check_tree(tree));
    TRY(check_verdict(out));
    TRY(check_ws(cfg, workspace, workspace_bytes));
    const hipError_t e = tsb::launch_verify_traversal(*cfg, inv_temperature(cfg->temperature), draft, draft_lse,
                                                      target, *tree, node_tok, step, *out, (char*)workspace, stream);
    return e == hipSuccess ? TSB_OK : hip_fail(e, "tsb_verify_traversal");
}

tsb_status tsb_step_traversal(const tsb_config* cfg, const void* draft, const void* target, uint32_t step,
                              double* draft_lse, int32_t* topk_tok, float* topk_lp, const tsb_tree* tree,
                              int32_t* node_tok, const tsb_verdict* out, void* workspace, size_t workspace_bytes,
                              hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    if (!draft || !target || !draft_lse || !topk_tok || !topk_lp || !node_tok)
        return fail(TSB_E_NULL, "tsb_step_traversal: a required array is NULL");
    TRY(check_tree(tree));
    TRY(check_verdict(out));
    TRY(check_ws(cfg, workspace, workspace_bytes));
    return step_round(cfg, draft, target, step, draft_lse, topk_tok, topk_lp, tree, node_tok, out, (char*)workspace,
                      stream, true, "tsb_step_traversal");
}

tsb_status tsb_step_noalloc(const tsb_config* cfg, const void* draft, const void* target, uint32_t step,
                            double* draft_lse, int32_t* topk_tok, float* topk_lp, const tsb_tree* tree,
                            int32_t* node_tok, const tsb_verdict* out, hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    const size_t need = tsb_workspace_bytes(cfg);
    if (need > (size_t)TSB_NOALLOC_SCRATCH_BYTES)
        return fail(TSB_E_WORKSPACE, "tsb_step_noalloc: this configuration needs %zu bytes of scratch, more than the "
                    "%zu the library holds per device (use tsb_step with a workspace)", need,
                    (size_t)TSB_NOALLOC_SCRATCH_BYTES);
    if (!draft || !target || !draft_lse || !topk_tok || !topk_lp || !node_tok)
        return fail(TSB_E_NULL, "tsb_step_noalloc: a required array is NULL");
    TRY(check_tree(tree));
    TRY(check_verdict(out));
    void* ws = nullptr;
    TRY(scratch_address(&ws));
    return step_round(cfg, draft, target, step, draft_lse, topk_tok, topk_lp, tree, node_tok, out, (char*)ws,
                      stream, false, "tsb_step_noalloc");
}

tsb_status tsb_first_tokens(const tsb_config* cfg, const int32_t* topk_tok, const tsb_tree* tree, int32_t* node_tok,
                            hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    if (!topk_tok || !node_tok) return fail(TSB_E_NULL, "tsb_first_tokens: a required array is NULL");
    TRY(check_tree(tree));
    const hipError_t e = tsb::launch_first_tokens(*cfg, topk_tok, *tree, node_tok, stream);
    return e == hipSuccess ? TSB_OK : hip_fail(e, "tsb_first_tokens");
}

tsb_status tsb_verify_naive(const tsb_config* cfg, const void* target, const tsb_tree* tree, const int32_t* node_tok,
                            uint32_t step, const tsb_verdict* out, void* workspace, size_t workspace_bytes,
                            hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    if (!target || !node_tok) return fail(TSB_E_NULL, "tsb_verify_naive: a required array is NULL");
    TRY(check_tree(tree));
    TRY(check_verdict(out));
    TRY(check_ws(cfg, workspace, workspace_bytes));
    const hipError_t e = tsb::launch_verify_naive(*cfg, inv_temperature(cfg->temperature), target, *tree, node_tok,
                                                  step, *out, (char*)workspace, stream);
    return e == hipSuccess ? TSB_OK : hip_fail(e, "tsb_verify_naive");
}

tsb_status tsb_step_first(const tsb_config* cfg, const void* draft, const void* target, uint32_t step,
                          double* draft_lse, int32_t* topk_tok, float* topk_lp, const tsb_tree* tree,
                          int32_t* node_tok, const tsb_verdict* out, void* workspace, size_t workspace_bytes,
                          hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    if (!draft || !target || !draft_lse || !topk_tok || !topk_lp || !node_tok)
        return fail(TSB_E_NULL, "tsb_step_first: a required array is NULL");
    TRY(check_tree(tree));
    TRY(check_verdict(out));
    TRY(check_ws(cfg, workspace, workspace_bytes));
    const float invT = inv_temperature(cfg->temperature);
    char* ws = (char*)workspace;
    hipError_t e = tsb::launch_plan(*cfg, invT, draft, draft_lse, topk_tok, topk_lp, *tree, out->req_status, ws, stream);
    if (e != hipSuccess) return hip_fail(e, "tsb_step_first/plan");
    e = tsb::launch_first_tokens(*cfg, topk_tok, *tree, node_tok, stream);
    if (e != hipSuccess) return hip_fail(e, "tsb_step_first/first_tokens");
    e = tsb::launch_verify_naive(*cfg, invT, target, *tree, node_tok, step, *out, ws, stream);
    if (e != hipSuccess) return hip_fail(e, "tsb_step_first/verify_naive");
    return TSB_OK;
}

size_t tsb_pool_workspace_bytes(const tsb_config* cfg, int32_t P) {
    if (!cfg) return 0;
    char saved[sizeof g_last_error];
    memcpy(saved, g_last_error, sizeof saved);
    tsb_status s = check_config(cfg);
    if (s == TSB_OK) s = check_pool(cfg, P, (const float*)cfg /* any non-NULL */);
    memcpy(g_last_error, saved, sizeof saved);
    if (s != TSB_OK) return 0;
    const size_t m = tsb::pool_ws_bytes(*cfg, P);
    return m < 256 ? 256 : m;
}

tsb_status tsb_pool_plan(const tsb_config* cfg, int32_t P, const void* draft, const float* trans, int32_t* pool_tok,
                         const tsb_tree* tree, int32_t* plan_tok, int32_t* req_status, void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    TRY(check_pool(cfg, P, trans));
    if (!draft || !pool_tok || !req_status) return fail(TSB_E_NULL, "tsb_pool_plan: a required array is NULL");
    TRY(check_tree(tree));
    TRY(check_pool_ws(cfg, P, workspace, workspace_bytes));
    const hipError_t e = tsb::launch_pool_plan(*cfg, P, inv_temperature(cfg->temperature), draft, trans, pool_tok,
                                               *tree, plan_tok, req_status, (char*)workspace, stream);
    return e == hipSuccess ? TSB_OK : hip_fail(e, "tsb_pool_plan");
}

tsb_status tsb_pool_replay(const tsb_config* cfg, int32_t P, const void* draft, const float* trans,
                           const int32_t* pool_tok, const tsb_tree* tree, uint32_t step, int32_t* node_tok,
                           hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    TRY(check_pool(cfg, P, trans));
    if (!draft || !pool_tok || !node_tok) return fail(TSB_E_NULL, "tsb_pool_replay: a required array is NULL");
    TRY(check_tree(tree));
    const hipError_t e = tsb::launch_pool_replay(*cfg, P, inv_temperature(cfg->temperature), draft, trans, pool_tok,
                                                 *tree, step, node_tok, stream);
    return e == hipSuccess ? TSB_OK : hip_fail(e, "tsb_pool_replay");
}

tsb_status tsb_pool_verify(const tsb_config* cfg, int32_t P, const void* draft, const float* trans,
                           const int32_t* pool_tok, const void* target, const tsb_tree* tree, const int32_t* node_tok,
                           uint32_t step, const tsb_verdict* out, void* workspace, size_t workspace_bytes,
                           hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    TRY(check_pool(cfg, P, trans));
    if (!draft || !pool_tok || !target || !node_tok)
        return fail(TSB_E_NULL, "tsb_pool_verify: a required array is NULL");
    TRY(check_tree(tree));
    TRY(check_verdict(out));
    TRY(check_pool_ws(cfg, P, workspace, workspace_bytes));
    const hipError_t e = tsb::launch_pool_verify(*cfg, P, inv_temperature(cfg->temperature), draft, trans, pool_tok,
                                                 target, *tree, node_tok, step, *out, (char*)workspace, stream);
    return e == hipSuccess ? TSB_OK : hip_fail(e, "tsb_pool_verify");
}

tsb_status tsb_pool_step(const tsb_config* cfg, int32_t P, const void* draft, const float* trans, const void* target,
                         uint32_t step, int32_t* pool_tok, const tsb_tree* tree, int32_t* node_tok,
                         const tsb_verdict* out, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    g_last_error[0] = 0;
    TRY(check_config(cfg));
    TRY(check_pool(cfg, P, trans));
    if (!draft || !target || !pool_tok || !node_tok) return fail(TSB_E_NULL, "tsb_pool_step: a required array is NULL");
    TRY(check_tree(tree));
    TRY(check_verdict(out));
    TRY(check_pool_ws(cfg, P, workspace, workspace_bytes));
    const float invT = inv_temperature(cfg->temperature);
    char* ws = (char*)workspace;
    hipError_t e = tsb::launch_pool_plan(*cfg, P, invT, draft, trans, pool_tok, *tree, nullptr, out->req_status, ws,
                                         stream);
    if (e != hipSuccess) return hip_fail(e, "tsb_pool_step/plan");
    e = tsb::launch_pool_replay(*cfg, P, invT, draft, trans, pool_tok, *tree, step, node_tok, stream);
    if (e != hipSuccess) return hip_fail(e, "tsb_pool_step/replay");
    e = tsb::launch_pool_verify(*cfg, P, invT, draft, trans, pool_tok, target, *tree, node_tok, step, *out, ws,
                                stream);
    if (e != hipSuccess) return hip_fail(e, "tsb_pool_step/verify");
    return TSB_OK;
}

tsb_status tsb_profile_kernel(int32_t kernel_id, hipEvent_t start, hipEvent_t stop) {
    g_last_error[0] = 0;
    tsb::ProfileHook& h = tsb::profile_hook();
    if (kernel_id < 0) {
        h = tsb::ProfileHook();
        return TSB_OK;
    }
    if (kernel_id >= TSB_KERNEL_COUNT) return fail(TSB_E_SHAPE, "kernel_id=%d unknown", kernel_id);
    if (!start || !stop) return fail(TSB_E_NULL, "events are NULL");
    h.kernel = kernel_id;
    h.start = start;
    h.stop = stop;
    return TSB_OK;
}

tsb_status tsb_stats_enable(int32_t on) {
    g_last_error[0] = 0;
    void* p = nullptr;
    const hipError_t e = tsb::counters_address(&p);
    if (e != hipSuccess) return hip_fail(e, "tsb_stats_enable/hipGetSymbolAddress(counters)");
    tsb::g_stats_on = on != 0;
    return TSB_OK;
}

tsb_status tsb_stats_read(tsb_stats* out, int32_t reset) {
    g_last_error[0] = 0;
    if (!out) return fail(TSB_E_NULL, "out is NULL");
    void* p = nullptr;
    hipError_t e = tsb::counters_address(&p);
    if (e != hipSuccess) return hip_fail(e, "tsb_stats_read/hipGetSymbolAddress(counters)");
    if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(e, "tsb_stats_read/hipDeviceSynchronize");
    if ((e = hipMemcpy(out, p, sizeof(tsb_stats), hipMemcpyDeviceToHost)) != hipSuccess)
        return hip_fail(e, "tsb_stats_read/hipMemcpy");
    if (reset) {
        const tsb_stats zero = {};
        if ((e = hipMemcpy(p, &zero, sizeof(tsb_stats), hipMemcpyHostToDevice)) != hipSuccess)
            return hip_fail(e, "tsb_stats_read/hipMemcpy(reset)");
    }
    return TSB_OK;
}

const char* tsb_status_string(tsb_status s) {
    switch (s) {
        case TSB_OK: return "ok";
        case TSB_E_NULL: return "a required pointer is NULL";
        case TSB_E_SHAPE: return "a size is out of range";
        case TSB_E_DTYPE: return "unknown logit dtype";
        case TSB_E_TEMPERATURE: return "temperature must be finite and > 0";
        case TSB_E_WORKSPACE: return "workspace too small or misaligned";
        case TSB_E_HIP: return "HIP runtime error";
        case TSB_E_DEVICE: return "no usable device";
    }
    return "unknown status";
}

const char* tsb_last_error(void) { return g_last_error; }

int32_t tsb_version(void) { return 201; }

}  // extern "C"
