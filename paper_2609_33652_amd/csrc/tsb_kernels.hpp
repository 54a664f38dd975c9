// Launchers of the gfx950 kernels (one per stage of a round). Each returns
// the first HIP error met while enqueueing on `st`.
#pragma once

#include <hip/hip_runtime.h>

#include "tsb_internal.hpp"

namespace tsb {

// Optional event pair around one kernel kind (tsb_profile_kernel).
struct ProfileHook {
    int kernel = -1;
    hipEvent_t start = nullptr, stop = nullptr;
};
ProfileHook& profile_hook();

inline hipError_t hook_before(int kernel, hipStream_t st) {
    const ProfileHook& h = profile_hook();
    return h.kernel == kernel ? hipEventRecord(h.start, st) : hipSuccess;
}
inline hipError_t hook_after(int kernel, hipStream_t st) {
    const ProfileHook& h = profile_hook();
    return h.kernel == kernel ? hipEventRecord(h.stop, st) : hipSuccess;
}

// Device counter block of tsb_stats on the current device while counting is
// enabled on the calling thread, else null (kernels then count nothing).
unsigned long long* stats_ptr();
enum : int {
    kStReplayItems = 0, kStReplayTokens, kStReplayLive, kStReplayKeyed,
    kStWalkRequests, kStWalkNodes, kStWalkTests, kStWalkExchanges,
    kStPlanRequests, kStPlanMergeTicks, kStPlanSearchTicks, kStPlanEmitTicks, kStPlanRounds,
    kStCount = 16
};

// Rows 0 and 1 of every request, streamed beside the planner for a walk that
// reads the other target rows itself (items = 0: none).
struct ChainJob {
    const void* target;
    float* cm;   // partials [R][kChainRows][kChainPieces]: max of a = x invT,
    double* cs;  // sum exp(a - max),
    int* cf;     // non-finite flag
    int items, V, B;
    bool bf16, vec;
};
ChainJob chain_job(const tsb_config& c, const void* target, char* ws);

// frontier > 0: the expand-then-prune first pass with that frontier width;
// 0: the max-heap first pass. With a chain job (max-heap pass only) the
// planner's grid also streams its rows.
hipError_t launch_plan(const tsb_config& c, float invT, const void* draft, double* draft_lse, int32_t* topk_tok,
                       float* topk_lp, const tsb_tree& tree, int32_t* req_status, char* ws, hipStream_t st,
                       int frontier = 0, const ChainJob* cj = nullptr);

// Nodes the expand-then-prune pass generates for this shape and frontier
// width, or -1 if they exceed what a workgroup holds.
int ep_generated_bound(const tsb_config& c, int frontier);
constexpr int kEpFrontierLimit = 64;

// The target stream of verification as a job: ngroups chunks of the flat
// [R (B+1) V] target, each streamed by one workgroup (the target kernel's
// own grid has one workgroup per chunk; the replay scan's grid deals them
// over fewer). The partials do not depend on which workgroup takes a chunk.
struct TargetJob {
    const void* target;
    const int32_t* n_nodes;  // rows at or beyond a request's node count are skipped
    float* tm;               // per-row partials [R (B+1)][P]: max of a = x invT,
    double* ts;              // sum exp(a - max),
    int* tf;                 // non-finite flag
    uint64_t* slots;         // exchange slots and ticket of the walk (cleared by the job)
    long long chunk;
    int nrows, P, ngroups, R;
    bool vec;                // 16-byte loads (row length and base alignment allow them)
    // the walk's node records, written by the replay merge after the job
    // (null: none), and the draft normalisers they copy
    uint32_t* nrec;
    const double* draft_lse;
};
// rows = false: a job that streams nothing and only clears the exchange
// slots of the walk launched after it (the walk then reads the target rows of
// the nodes it enters).
TargetJob target_job(const tsb_config& c, const void* target, const tsb_tree& tree, const double* draft_lse,
                     char* ws, bool rows = true);

// Zeroes the exchange slots of the requests (before a walk that no target
// stream precedes).
hipError_t launch_xchg_clear(const tsb_config& c, uint64_t* slots, hipStream_t st);

// With a target job, the replay scan's grid carries it: ngroups more
// workgroups stream the target while the others scan (one launch).
hipError_t launch_replay(const tsb_config& c, float invT, const void* draft, const int32_t* topk_tok,
                         const tsb_tree& tree, uint32_t step, int32_t* node_tok, char* ws, hipStream_t st,
                         const TargetJob* tj = nullptr);

// Verification is two stages: the target stream (row normaliser partials of
// every row of the tree, for the optional normaliser output, and for the
// verifiers that need every row), or else the clearing of the exchange
// slots, and the walk. A round runs the target stage in the replay scan's
// grid, its merge writes the node records, and then the walk runs alone,
// reading them (kWalkRecords).
enum : int { kStageTarget = 1, kStageWalk = 2, kStagesAll = 3, kWalkRecords = 4 };

hipError_t launch_verify(const tsb_config& c, float invT, const void* draft, const double* draft_lse,
                         const void* target, const tsb_tree& tree, const int32_t* node_tok, uint32_t step,
                         const tsb_verdict& out, char* ws, hipStream_t st, int stages = kStagesAll);

// Traversal verification (sequence-level RRS over the tree) instead of WoR-RRS.
hipError_t launch_verify_traversal(const tsb_config& c, float invT, const void* draft, const double* draft_lse,
                                   const void* target, const tsb_tree& tree, const int32_t* node_tok, uint32_t step,
                                   const tsb_verdict& out, char* ws, hipStream_t st, int stages = kStagesAll);

// Sparse candidate pools of P tokens with context-dependent q_u.
hipError_t launch_pool_partials(const tsb_config& c, int P, float invT, const void* draft, uint64_t* pk, int* pf,
                                int32_t* req_status, hipStream_t st);
hipError_t launch_pool_plan(const tsb_config& c, int P, float invT, const void* draft, const float* trans,
                            int32_t* pool_tok, const tsb_tree& tree, int32_t* plan_tok, int32_t* req_status,
                            char* ws, hipStream_t st);
hipError_t launch_pool_replay(const tsb_config& c, int P, float invT, const void* draft, const float* trans,
                              const int32_t* pool_tok, const tsb_tree& tree, uint32_t step, int32_t* node_tok,
                              hipStream_t st);
hipError_t launch_pool_verify(const tsb_config& c, int P, float invT, const void* draft, const float* trans,
                              const int32_t* pool_tok, const void* target, const tsb_tree& tree,
                              const int32_t* node_tok, uint32_t step, const tsb_verdict& out, char* ws,
                              hipStream_t st, int stages = kStagesAll);

hipError_t launch_first_tokens(const tsb_config& c, const int32_t* topk_tok, const tsb_tree& tree, int32_t* node_tok,
                               hipStream_t st);

hipError_t launch_verify_naive(const tsb_config& c, float invT, const void* target, const tsb_tree& tree,
                               const int32_t* node_tok, uint32_t step, const tsb_verdict& out, char* ws,
                               hipStream_t st);

}  // namespace tsb
