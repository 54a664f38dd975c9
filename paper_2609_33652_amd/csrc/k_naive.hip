// The deterministic first-pass baseline (First) and target-sample matching
// (Naive) on gfx950.
//
// Section 3.1: the first pass builds a deterministic tree from the planning
// candidates; kept with those tokens and verified directly it is the First
// baseline. A node of depth d and rank j carries candidate j of draft
// position d - 1.
//
// Table 2 (Naive), Section 2.3: at node u one token y is drawn from the
// target distribution p_u; the child of u carrying y is accepted and the
// walk continues there, otherwise y is the bonus token. The draw is the
// Gumbel-max sample argmax_v a_v + G_v of the scaled target row a = fl32(x
// invT), G from the BONUS stream of node u (the same draw as a bonus from p_u
// in the RRS walk: a common shift by the normaliser does not move the
// argmax). No normaliser is needed, so only the rows the walk visits are read.
//
//   first_tokens   one thread per (request, node).
//   verify_naive   resident grid, G workgroups per request, each owning a
//                  slice of the vocabulary; per visited node one read of its
//                  slice, the local best key, one exchange of (key, token,
//                  finiteness) through the tagged slots of the request.
#include <math.h>

#include <algorithm>
#include <atomic>

#include "tsb_device.hpp"
#include "tsb_exchange.hpp"
#include "tsb_kernels.hpp"

namespace tsb {

// ------------------------------------------------------------- first_tokens
__global__ __launch_bounds__(kBlock) void first_tokens(int R, int D, int K, int B1, const int32_t* __restrict__ topk_tok,
                                                       tsb_tree tree, int32_t* __restrict__ node_tok) {
    const long long t = (long long)blockIdx.x * kBlock + threadIdx.x;
    if (t >= (long long)R * B1) return;
    const int r = (int)(t / B1);
    const int i = (int)(t - (long long)r * B1);
    const int n = tree.n_nodes[r];
    int tok = -1;
    if (i > 0 && i < n) {
        const int d = tree.depth[t];
        const int j = tree.rank[t];
        if (d >= 1 && d <= D && j >= 0 && j < K) tok = topk_tok[((size_t)r * D + (d - 1)) * K + j];
    }
    node_tok[t] = tok;
}

// ------------------------------------------------------------- naive walk
constexpr int kNaiveThreads = 512;
constexpr int kNaiveBatch = 3;  // groups of four tokens per thread per batch
constexpr int kNaiveBatchTokens = kNaiveBatch * 4 * kNaiveThreads;
constexpr int kNaiveNodes = TSB_MAX_B + 1;

struct NaiveArgs {
    const void* target;
    tsb_tree tree;
    const int32_t* node_tok;
    tsb_verdict out;
    XRegion X;  // exchange slots of the requests
    int V, D, B;
    int R, G;   // requests and workgroups per request of the launch (tickets)
    float invT;
    uint32_t k0, k1, step;
};

// Keys are compared as ordered_bits64(fl32(a) + G) with the low 8 bits
// cleared (an exchanged word carries its tag there): relative resolution
// 2^-44 of the binary64 sum; keys equal after clearing go to the smaller
// token.
__device__ __forceinline__ uint64_t sample_key(float a, float gumbel) {
    return ordered_bits64((double)a + (double)gumbel) & ~kTagMask;
}

// Local result of one slice: best key and its token (smallest id among equal
// keys), plus finiteness of the slice.
struct SliceBest {
    uint64_t key;  // 0: no candidate
    uint32_t tok;  // < 2^31
    int bad;       // a NaN or +inf logit
    int has;       // a finite logit
};

template <int DT, bool VEC>
__device__ __forceinline__ void load_batch(const void* target, size_t trow, int v0, int n, int base,
                                           Raw4<DT> (&a)[kNaiveBatch]) {
#pragma unroll
    for (int j = 0; j < kNaiveBatch; ++j) {
        const int i = (base + j * kNaiveThreads + (int)threadIdx.x) * 4;
        const int valid = max(0, min(4, n - i));
        raw_load4<DT>(target, trow + v0 + (valid ? i : 0), valid, VEC, a[j]);
    }
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t k) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const uint64_t ok = ((uint64_t)__shfl_xor((uint32_t)(k >> 32), o, kWave) << 32) |
                            (uint32_t)__shfl_xor((uint32_t)k, o, kWave);
        k = ok > k ? ok : k;
    }
    return k;
}

// Scores one batch. A group of four tokens whose largest logit, even with
// the largest Gumbel value, stays below the wave's best key so far or below
// the smallest key the largest logit of the batch can get, is skipped
// without drawing its random numbers: its tokens lose strictly to a key the
// wave keeps, so the result is the exact argmax. Groups are scored one at a
// time (scheduling barriers keep the random numbers of one group in flight).
template <int DT>
__device__ __forceinline__ void score_batch(const Raw4<DT> (&raw)[kNaiveBatch], int v0, int n, int base, float invT,
                                            const RngKey& key, uint32_t node, SliceBest& s) {
    float gm[kNaiveBatch], bm = -INFINITY;
#pragma unroll
    for (int j = 0; j < kNaiveBatch; ++j) {
        const int i = (base + j * kNaiveThreads + (int)threadIdx.x) * 4;
        float a[4];
        raw_scaled4<DT>(raw[j], max(0, min(4, n - i)), invT, a);
        gm[j] = -INFINITY;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            s.bad |= (isnan(a[e]) || a[e] == INFINITY) ? 1 : 0;
            s.has |= (a[e] > -INFINITY && a[e] < INFINITY) ? 1 : 0;
            gm[j] = fmaxf(gm[j], a[e]);
        }
        bm = fmaxf(bm, gm[j]);
    }
    bm = wave_max(bm);
    const uint64_t wk = wave_max_u64(s.key);
    const double wave_best = wk ? from_ordered_bits64(wk) : -INFINITY;
    const double thr = fmax(wave_best, bm < INFINITY ? (double)bm + (double)kGumbelMinBound : -INFINITY);
#pragma unroll
    for (int j = 0; j < kNaiveBatch; ++j) {
        __builtin_amdgcn_sched_barrier(0);
        if (!(gm[j] > -INFINITY && (double)gm[j] + (double)kGumbelMaxBound >= thr)) continue;
        const int i = (base + j * kNaiveThreads + (int)threadIdx.x) * 4;
        float a[4];
        raw_scaled4<DT>(raw[j], max(0, min(4, n - i)), invT, a);
        const uint4 w = rng_block(key, node, kStreamBonus, (uint32_t)((v0 + i) >> 2));
        const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (!(a[e] > -INFINITY)) continue;
            const uint64_t k = sample_key(a[e], gumbel_f32(ws[e]));
            const uint32_t v = (uint32_t)(v0 + i + e);
            if (k > s.key || (k == s.key && v < s.tok)) {
                s.key = k;
                s.tok = v;
            }
        }
    }
}

// Workgroup-wide reduction of the per-thread results (key desc, token asc).
__device__ SliceBest reduce_slice(const SliceBest& s) {
    uint64_t k = s.key;
    uint32_t t = s.tok;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const uint64_t ok = ((uint64_t)__shfl_xor((uint32_t)(k >> 32), o, kWave) << 32) |
                            (uint32_t)__shfl_xor((uint32_t)k, o, kWave);
        const uint32_t ot = (uint32_t)__shfl_xor((int)t, o, kWave);
        if (ok > k || (ok == k && ot < t)) {
            k = ok;
            t = ot;
        }
    }
    const int bad = wave_or(s.bad), has = wave_or(s.has);
    __shared__ uint64_t rk[kNaiveThreads / kWave];
    __shared__ uint32_t rt[kNaiveThreads / kWave];
    __shared__ int rf[kNaiveThreads / kWave];
    const int wv = threadIdx.x / kWave;
    if ((threadIdx.x % kWave) == 0) {
        rk[wv] = k;
        rt[wv] = t;
        rf[wv] = bad | (has << 1);
    }
    __syncthreads();
    SliceBest r{rk[0], rt[0], rf[0] & 1, (rf[0] >> 1) & 1};
    for (int i = 1; i < kNaiveThreads / kWave; ++i) {
        if (rk[i] > r.key || (rk[i] == r.key && rt[i] < r.tok)) {
            r.key = rk[i];
            r.tok = rt[i];
        }
        r.bad |= rf[i] & 1;
        r.has |= (rf[i] >> 1) & 1;
    }
    __syncthreads();
    return r;
}

// Round e of request r: publish this workgroup's result, then wave 0 polls
// the G slots (lane h: slots h and h + 64), reduces them in a fixed order
// (key desc, token asc; flags or-ed) and hands the result to the other waves.
// Slot words: key, token << 32 | has << 9 | bad << 8.
__device__ SliceBest naive_round(const NaiveArgs& A, int r, int g, int G, uint32_t e, const SliceBest& mine,
                                 int* timeout) {
    const uint64_t w[2] = {mine.key, xpack_u32(mine.tok) | ((uint64_t)mine.has << 9) | ((uint64_t)mine.bad << 8)};
    xpublish<2>(A.X, r, g, e, w);
    __shared__ SliceBest s_res;
    __shared__ int s_to;
    if (threadIdx.x < kWave) {
        const int lane = threadIdx.x;
        uint64_t k = 0ull;
        uint32_t t = 0xFFFFFFFFu;
        int bad = 0, has = 0, to = 0;
#pragma unroll
        for (int half = 0; half < kWalkGroupsMax / kWave; ++half) {
            const int h = lane + half * kWave;
            if (h < G) {
                uint64_t q[2];
                if (!xpoll<2>(A.X, r, h, e, q)) to = 1;
                const uint64_t kk = q[0] & ~kTagMask;
                const uint32_t tt = xunpack_u32(q[1]);
                bad |= (int)((q[1] >> 8) & 1ull);
                has |= (int)((q[1] >> 9) & 1ull);
                if (kk > k || (kk == k && tt < t)) {
                    k = kk;
                    t = tt;
                }
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const uint64_t ok = ((uint64_t)__shfl_xor((uint32_t)(k >> 32), o, kWave) << 32) |
                                (uint32_t)__shfl_xor((uint32_t)k, o, kWave);
            const uint32_t ot = (uint32_t)__shfl_xor((int)t, o, kWave);
            if (ok > k || (ok == k && ot < t)) {
                k = ok;
                t = ot;
            }
        }
        bad = wave_or(bad);
        has = wave_or(has);
        to = wave_or(to);
        if (lane == 0) {
            s_res = SliceBest{k, t, bad, has};
            s_to = to;
        }
    }
    __syncthreads();
    const SliceBest res = s_res;
    if (s_to) *timeout = 1;
    __syncthreads();  // s_res is rewritten by the next round
    return res;
}

template <int DT, bool VEC>
__global__ __launch_bounds__(kNaiveThreads) void verify_naive(NaiveArgs A) {
    __shared__ int s_nc[kNaiveNodes], s_fc[kNaiveNodes], s_tok[kNaiveNodes];
    const int G = A.G;
    const int ticket = xticket(A.X, A.R);
    const int g = ticket % G;
    const int r = ticket / G;
    const int tid = threadIdx.x;
    const int B1 = A.B + 1;
    const size_t tb = (size_t)r * B1;
    const bool lead = (g == 0 && tid == 0);
    int* status_p = A.out.req_status + r;
    const int n_raw = A.tree.n_nodes[r];
    const bool count_ok = tree_count_ok(n_raw, A.B);
    const int n = count_ok ? n_raw : 0;

    // vocabulary slice (start a multiple of 4; an empty slice is [0, 0))
    const int span = ((A.V + G - 1) / G + 3) & ~3;
    const bool has_slice = (long long)g * span < A.V;
    const int v0 = has_slice ? g * span : 0;
    const int v1 = has_slice ? min(A.V, v0 + span) : 0;
    const int ns = v1 - v0;
    const bool single = ns <= kNaiveBatchTokens;  // the slice is one batch: its loads are issued at once

    const bool plan_bad = (*status_p & TSB_REQ_NONFINITE) != 0;
    int nacc = 0, bonus = -1, add_status = count_ok ? 0 : TSB_REQ_BAD_TREE;
    if (!plan_bad && count_ok) {
        RngKey key;
        key.k0 = A.k0;
        key.k1 = A.k1;
        key.request = (uint32_t)r;
        key.step = A.step;
        int timeout = 0;
        Raw4<DT> cur[kNaiveBatch];
        if (single) load_batch<DT, VEC>(A.target, tb * (size_t)A.V, v0, ns, 0, cur);
        // the request's tree (children and node tokens) in LDS
        for (int i = tid; i < n; i += kNaiveThreads) {
            s_nc[i] = A.tree.n_children[tb + i];
            s_fc[i] = A.tree.first_child[tb + i];
            s_tok[i] = A.node_tok[tb + i];
        }
        __syncthreads();
        int u = 0;
        uint32_t e = 0;
        for (;; ++e) {
            const size_t trow = ((size_t)r * B1 + u) * (size_t)A.V;
            SliceBest mine{0ull, 0xFFFFFFFFu, 0, 0};
            if (single) {
                score_batch<DT>(cur, v0, ns, 0, A.invT, key, (uint32_t)u, mine);
            } else {
                for (int base = 0; base * 4 < ns; base += kNaiveBatch * kNaiveThreads) {
                    load_batch<DT, VEC>(A.target, trow, v0, ns, base, cur);
                    score_batch<DT>(cur, v0, ns, base, A.invT, key, (uint32_t)u, mine);
                }
            }
            // children of u (a well-formed node: m <= TSB_MAX_K, inside the
            // tree after u, and u not deeper than D - 1 on the accepted path)
            const int m = s_nc[u];
            const int fc = s_fc[u];
            const bool well_formed = m == 0 || (m > 0 && m <= TSB_MAX_K && fc > u && fc <= n - m && nacc < A.D);
            const SliceBest all = naive_round(A, r, g, G, e, reduce_slice(mine), &timeout);
            if (all.bad || !all.has) {
                add_status |= TSB_REQ_NONFINITE;
                break;
            }
            if (!well_formed) {
                add_status |= TSB_REQ_BAD_TREE;
                break;
            }
            const int y = (int)all.tok;
            int match = -1;
            for (int j = 0; j < m; ++j)
                if (s_tok[fc + j] == y) {
                    match = fc + j;
                    break;
                }
            if (match < 0) {
                bonus = y;
                break;
            }
            if (lead) {
                A.out.acc_node[(size_t)r * A.D + nacc] = match;
                A.out.acc_tok[(size_t)r * A.D + nacc] = y;
            }
            ++nacc;
            u = match;
            if (single) load_batch<DT, VEC>(A.target, ((size_t)r * B1 + u) * (size_t)A.V, v0, ns, 0, cur);
        }
        if (timeout) add_status |= TSB_REQ_WALK_TIMEOUT;
    } else if (plan_bad) {
        add_status |= TSB_REQ_NONFINITE;
    }
    if (lead) {
        const bool bad = (add_status & (TSB_REQ_NONFINITE | TSB_REQ_BAD_TREE)) != 0;
        if (bad) nacc = 0;
        for (int i = nacc; i < A.D; ++i) {
            A.out.acc_node[(size_t)r * A.D + i] = -1;
            A.out.acc_tok[(size_t)r * A.D + i] = -1;
        }
        A.out.n_acc[r] = bad ? -1 : nacc;
        A.out.bonus[r] = bad ? -1 : bonus;
        *status_p |= add_status;
    }
}

// Zeroes the exchange slots of the requests before a walk that no stream
// kernel precedes.
__global__ __launch_bounds__(kBlock) void xchg_clear(XRegion X, int R) {
    xclear(X, R, (size_t)blockIdx.x * kBlock + threadIdx.x, (size_t)gridDim.x * kBlock);
}

hipError_t launch_xchg_clear(const tsb_config& c, uint64_t* slots, hipStream_t st) {
    XRegion X;
    X.slots = slots;
    const int nclear = (int)std::min<size_t>(1024, (xwords(c.R) + kBlock - 1) / kBlock);
    xchg_clear<<<nclear, kBlock, 0, st>>>(X, c.R);
    return hipGetLastError();
}

// ------------------------------------------------------------------ launch
hipError_t launch_first_tokens(const tsb_config& c, const int32_t* topk_tok, const tsb_tree& tree, int32_t* node_tok,
                               hipStream_t st) {
    const long long n = (long long)c.R * (c.B + 1);
    first_tokens<<<(unsigned)((n + kBlock - 1) / kBlock), kBlock, 0, st>>>(c.R, c.D, c.K, c.B + 1, topk_tok, tree,
                                                                        node_tok);
    return hipGetLastError();
}

// Workgroups of verify_naive resident at once on the current device, queried
// once per (device, kernel instance); every launch stays within it so the
// exchanges of a request complete.
static hipError_t naive_capacity(const void* fn, int dt, int vec, int* cap) {
    constexpr int kDevs = 64;
    static std::atomic<int> cached[kDevs][2][2];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev >= 0 && dev < kDevs) {
        const int v = cached[dev][dt][vec].load(std::memory_order_relaxed);
        if (v > 0) {
            *cap = v;
            return hipSuccess;
        }
    }
    int cus = 0, per_cu = 0;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kNaiveThreads, 0)) != hipSuccess) return e;
    *cap = per_cu * cus;
    if (dev >= 0 && dev < kDevs && *cap > 0) cached[dev][dt][vec].store(*cap, std::memory_order_relaxed);
    return hipSuccess;
}

hipError_t launch_verify_naive(const tsb_config& c, float invT, const void* target, const tsb_tree& tree,
                               const int32_t* node_tok, uint32_t step, const tsb_verdict& out, char* ws,
                               hipStream_t st) {
    NaiveArgs A;
    A.target = target;
    A.tree = tree;
    A.node_tok = node_tok;
    A.out = out;
    A.X.slots = (uint64_t*)(ws + xchg_ws(c).slots);
    A.V = c.V;
    A.D = c.D;
    A.B = c.B;
    A.invT = invT;
    A.k0 = (uint32_t)c.seed;
    A.k1 = (uint32_t)(c.seed >> 32);
    A.step = step;

    const bool vec = c.V % 4 == 0 && ((uintptr_t)target & 15) == 0;
    const void* fn = nullptr;
    if (c.dtype == TSB_BF16)
        fn = vec ? (const void*)verify_naive<TSB_BF16, true> : (const void*)verify_naive<TSB_BF16, false>;
    else
        fn = vec ? (const void*)verify_naive<TSB_F32, true> : (const void*)verify_naive<TSB_F32, false>;
    int cap = 0;
    hipError_t e = naive_capacity(fn, c.dtype == TSB_BF16 ? 1 : 0, vec ? 1 : 0, &cap);
    if (e != hipSuccess) return e;
    if (cap < 1) return hipErrorLaunchOutOfResources;
    // workgroups per request: enough that a slice is one batch, within what
    // keeps the whole batch resident (the launch itself needs only G
    // workgroups to fit at once: tickets)
    const int need = (c.V + kNaiveBatchTokens - 1) / kNaiveBatchTokens;
    int G = cap / c.R;
    if (G > need) G = need;
    if (G > kWalkGroupsMax) G = kWalkGroupsMax;
    if (G < 1) G = 1;
    A.R = c.R;
    A.G = G;

    if ((e = launch_xchg_clear(c, A.X.slots, st)) != hipSuccess) return e;
    if ((e = hook_before(TSB_KERNEL_VERIFY_NAIVE, st)) != hipSuccess) return e;
    void* args[] = {&A};
    e = hipLaunchKernel(fn, dim3((unsigned)(G * c.R)), dim3(kNaiveThreads), args, 0, st);
    if (e != hipSuccess) return e;
    return hook_after(TSB_KERNEL_VERIFY_NAIVE, st);
}

}  // namespace tsb
