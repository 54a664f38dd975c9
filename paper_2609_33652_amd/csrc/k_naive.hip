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
//   naive_clear    zeroes the per-request barrier counters.
//   verify_naive   resident grid, G workgroups per request, each owning a
//                  slice of the vocabulary; per visited node one read of its
//                  slice, the local best key, one exchange of (key, token,
//                  finiteness) through the per-request barrier.
#include <math.h>

#include <atomic>

#include "tsb_device.hpp"
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
constexpr int kNaiveBatch = 4;  // groups of four tokens per thread in flight

__global__ __launch_bounds__(kBlock) void naive_clear(uint32_t* counters, int R) {
    for (int i = blockIdx.x * kBlock + threadIdx.x; i < R; i += gridDim.x * kBlock) counters[i] = 0u;
}

struct NaiveArgs {
    const void* target;
    tsb_tree tree;
    const int32_t* node_tok;
    tsb_verdict out;
    uint32_t* counters;
    double* zpart;  // exchange slots: [R][2][kWalkGroupsMax][4] doubles
    int* bidx;      // [R][2][kWalkGroupsMax]
    int V, D, B, r0;
    float invT;
    uint32_t k0, k1, step;
};

// Local result of one slice: best key (binary64 value of fl32(a) + G) and
// its token (smallest id among equal keys), plus finiteness of the slice.
struct SliceBest {
    double key;
    int tok;
    int bad;  // a NaN or +inf logit
    int has;  // a finite logit
};

// Best (key, token) of the slice [v0, v1) of one target row. A group of
// four tokens whose largest logit cannot reach the wave's best key so far,
// nor the smallest key the wave's largest logit of the batch can get, even
// with the largest Gumbel value, is skipped without drawing its random
// numbers; such tokens lose strictly to a key the wave keeps, so the result
// is the exact argmax.
template <int DT, bool VEC>
__device__ SliceBest slice_sample(const NaiveArgs& A, size_t trow, int v0, int v1, const RngKey& key,
                                  uint32_t node) {
    SliceBest s{-INFINITY, 0x7FFFFFFF, 0, 0};
    const int n = v1 - v0;
    double wave_best = -INFINITY;
    for (int base = 0; base * 4 < n; base += kNaiveBatch * kNaiveThreads) {
        float a[kNaiveBatch][4];
#pragma unroll
        for (int j = 0; j < kNaiveBatch; ++j) {
            const int i = (base + j * kNaiveThreads + (int)threadIdx.x) * 4;
            const int valid = max(0, min(4, n - i));
            float x[4];
            load4<DT>(A.target, trow + v0 + (valid ? i : 0), valid, VEC, x);
#pragma unroll
            for (int e = 0; e < 4; ++e) a[j][e] = e < valid ? x[e] * A.invT : -INFINITY;
        }
        float gm[kNaiveBatch], bm = -INFINITY;
#pragma unroll
        for (int j = 0; j < kNaiveBatch; ++j) {
            gm[j] = -INFINITY;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                s.bad |= (isnan(a[j][e]) || a[j][e] == INFINITY) ? 1 : 0;
                s.has |= (a[j][e] > -INFINITY && a[j][e] < INFINITY) ? 1 : 0;
                gm[j] = fmaxf(gm[j], a[j][e]);
            }
            bm = fmaxf(bm, gm[j]);
        }
        bm = wave_max(bm);
        const double thr = fmax(wave_best, bm < INFINITY ? (double)bm + (double)kGumbelMinBound : -INFINITY);
#pragma unroll
        for (int j = 0; j < kNaiveBatch; ++j) {
            const int i = (base + j * kNaiveThreads + (int)threadIdx.x) * 4;
            if (gm[j] > -INFINITY && (double)gm[j] + (double)kGumbelMaxBound >= thr) {
                const uint4 w = rng_block(key, node, kStreamBonus, (uint32_t)((v0 + i) >> 2));
                const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if (!(a[j][e] > -INFINITY)) continue;
                    const double k = (double)a[j][e] + (double)gumbel_f32(ws[e]);
                    const int v = v0 + i + e;
                    if (k > s.key || (k == s.key && v < s.tok)) {
                        s.key = k;
                        s.tok = v;
                    }
                }
            }
        }
        double b = s.key;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) b = fmax(b, __shfl_xor(b, o, kWave));
        wave_best = b;
    }
    // workgroup argmax (key desc, token asc) and flags
    double k = s.key;
    int t = s.tok;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const double ok = __shfl_xor(k, o, kWave);
        const int ot = __shfl_xor(t, o, kWave);
        if (ok > k || (ok == k && ot < t)) {
            k = ok;
            t = ot;
        }
    }
    const int bad = wave_or(s.bad), has = wave_or(s.has);
    __shared__ double rk[kNaiveThreads / kWave];
    __shared__ int rt[kNaiveThreads / kWave], rb[kNaiveThreads / kWave], rh[kNaiveThreads / kWave];
    const int wv = threadIdx.x / kWave;
    if ((threadIdx.x % kWave) == 0) {
        rk[wv] = k;
        rt[wv] = t;
        rb[wv] = bad;
        rh[wv] = has;
    }
    __syncthreads();
    SliceBest r{rk[0], rt[0], rb[0], rh[0]};
    for (int i = 1; i < kNaiveThreads / kWave; ++i) {
        if (rk[i] > r.key || (rk[i] == r.key && rt[i] < r.tok)) {
            r.key = rk[i];
            r.tok = rt[i];
        }
        r.bad |= rb[i];
        r.has |= rh[i];
    }
    __syncthreads();
    return r;
}

// Exchange of the slice results among the G workgroups of request r; all
// of them get the same reduced result (argmax in a fixed order).
__device__ SliceBest naive_exchange(const NaiveArgs& A, int r, int g, int G, uint32_t* nb, int* timeout,
                                    const SliceBest& mine) {
    const int slot = (r * 2 + (*nb & 1)) * kWalkGroupsMax + g;
    if (threadIdx.x == 0) {
        __hip_atomic_store(&A.zpart[(size_t)slot * 4 + 0], mine.key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&A.zpart[(size_t)slot * 4 + 1], (double)(mine.bad | (mine.has << 1)), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&A.bidx[slot], mine.tok, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    ++*nb;
    request_barrier(&A.counters[r], *nb * (uint32_t)G, timeout);
    __shared__ SliceBest s_res;
    if (threadIdx.x < kWave) {
        const int lane = threadIdx.x;
        double k = -INFINITY;
        int t = 0x7FFFFFFF, fl = 0;
#pragma unroll
        for (int half = 0; half < kWalkGroupsMax / kWave; ++half) {
            const int h = lane + half * kWave;
            if (h < G) {
                const int sl = (r * 2 + ((*nb - 1) & 1)) * kWalkGroupsMax + h;
                const double kk = __hip_atomic_load(&A.zpart[(size_t)sl * 4 + 0], __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
                const double ff = __hip_atomic_load(&A.zpart[(size_t)sl * 4 + 1], __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
                const int tt = __hip_atomic_load(&A.bidx[sl], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                fl |= (int)ff;
                if (kk > k || (kk == k && tt < t)) {
                    k = kk;
                    t = tt;
                }
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const double ok = __shfl_xor(k, o, kWave);
            const int ot = __shfl_xor(t, o, kWave);
            if (ok > k || (ok == k && ot < t)) {
                k = ok;
                t = ot;
            }
        }
        fl = wave_or(fl);
        if (lane == 0) s_res = SliceBest{k, t, fl & 1, (fl >> 1) & 1};
    }
    __syncthreads();
    const SliceBest res = s_res;
    __syncthreads();  // s_res is rewritten by the next exchange
    return res;
}

template <int DT, bool VEC>
__global__ __launch_bounds__(kNaiveThreads) void verify_naive(NaiveArgs A) {
    const int g = blockIdx.x;
    const int G = gridDim.x;
    const int r = A.r0 + blockIdx.y;
    const int tid = threadIdx.x;
    const int B1 = A.B + 1;
    const size_t tb = (size_t)r * B1;
    const bool lead = (g == 0 && tid == 0);
    int* status_p = A.out.req_status + r;
    const int n = A.tree.n_nodes[r];

    // vocabulary slice (start a multiple of 4; an empty slice is [0, 0))
    const int span = ((A.V + G - 1) / G + 3) & ~3;
    const bool has_slice = (long long)g * span < A.V;
    const int v0 = has_slice ? g * span : 0;
    const int v1 = has_slice ? min(A.V, v0 + span) : 0;

    const bool plan_bad = (*status_p & TSB_REQ_NONFINITE) != 0;
    int nacc = 0, bonus = -1, add_status = 0;
    if (!plan_bad && n >= 1 && n <= B1) {
        RngKey key;
        key.k0 = A.k0;
        key.k1 = A.k1;
        key.request = (uint32_t)r;
        key.step = A.step;
        uint32_t nb = 0;
        int timeout = 0;
        int u = 0;
        while (true) {
            const size_t trow = ((size_t)r * B1 + u) * (size_t)A.V;
            const SliceBest mine = slice_sample<DT, VEC>(A, trow, v0, v1, key, (uint32_t)u);
            const SliceBest all = naive_exchange(A, r, g, G, &nb, &timeout, mine);
            if (all.bad || !all.has) {
                add_status |= TSB_REQ_NONFINITE;
                break;
            }
            const int y = all.tok;
            const int m = A.tree.n_children[tb + u];
            const int fc = A.tree.first_child[tb + u];
            int match = -1;
            if (m > 0 && fc > u && fc + m <= n && nacc < A.D)
                for (int j = 0; j < m; ++j)
                    if (A.node_tok[tb + fc + j] == y) {
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
        }
        if (timeout) add_status |= TSB_REQ_WALK_TIMEOUT;
    } else {
        add_status |= TSB_REQ_NONFINITE;
    }
    if (lead) {
        const bool bad = (add_status & TSB_REQ_NONFINITE) != 0;
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
// barriers of a request complete.
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
    const Geometry geo = geometry(c);
    const VerifyWs w = verify_ws(c);
    NaiveArgs A;
    A.target = target;
    A.tree = tree;
    A.node_tok = node_tok;
    A.out = out;
    A.counters = (uint32_t*)(ws + w.counter);
    A.zpart = (double*)(ws + w.zpart);
    A.bidx = (int*)(ws + w.bidx);
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
    int G = geo.G;
    if (G > cap) G = cap;
    const int chunk = cap / G;

    naive_clear<<<(c.R + kBlock - 1) / kBlock < 64 ? (c.R + kBlock - 1) / kBlock : 64, kBlock, 0, st>>>(A.counters,
                                                                                                      c.R);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = hook_before(TSB_KERNEL_VERIFY_NAIVE, st)) != hipSuccess) return e;
    for (int r0 = 0; r0 < c.R; r0 += chunk) {
        A.r0 = r0;
        const int rc = min(chunk, c.R - r0);
        void* args[] = {&A};
        e = hipLaunchKernel(fn, dim3(G, rc), dim3(kNaiveThreads), args, 0, st);
        if (e != hipSuccess) return e;
    }
    return hook_after(TSB_KERNEL_VERIFY_NAIVE, st);
}

}  // namespace tsb
