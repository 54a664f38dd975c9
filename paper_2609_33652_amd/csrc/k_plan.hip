// First pass of a tree-replay round on gfx950 (Section 3.1; Appendix B.3):
//   draft_partials  one workgroup per (draft row, vocabulary segment):
//                   online max / binary64 sum of exp, and the segment's K best
//                   candidates by (logit desc, id asc) kept in a wave-wide
//                   sorted list; one streaming read of the draft logits.
//   draft_merge     one wave per draft row: combine the segments into the
//                   binary64 log-sum-exp, its canonical binary32 rounding and
//                   the planning candidates lp = fl32(a - lse32).
//   plan_tree       one wave per request: lazy best-first expansion of rank
//                   paths under the static order (score desc, depth asc, rank
//                   path lexicographic asc), then BFS canonicalisation.
#include <math.h>

#include "tsb_device.hpp"
#include "tsb_kernels.hpp"

namespace tsb {

// ------------------------------------------------------------------ K1a
template <int DT, bool VEC>
__global__ __launch_bounds__(kBlock) void draft_partials(const void* __restrict__ draft, int V, int D,
                                                         int seg, int S, float invT, int K,
                                                         float* __restrict__ pm, double* __restrict__ ps,
                                                         uint64_t* __restrict__ pk, int* __restrict__ pf,
                                                         int32_t* __restrict__ req_status) {
    const int s = blockIdx.x;
    const int row = blockIdx.y;
    const int tid = threadIdx.x;
    if (s == 0 && (row % D) == 0 && tid == 0) req_status[row / D] = 0;

    const size_t rowbase = (size_t)row * (size_t)V;
    const int lo = s * seg;
    const int hi = min(V, lo + seg);

    __shared__ double s_exp[kExpTable];
    exp64_table_init(s_exp);

    float m = -INFINITY;
    double sum = 0.0;
    int bad = 0;
    WaveTopList top;
    top.init(K);

    for (int base = lo; base < hi; base += kBlock * 8) {
        const int i0 = base + tid * 8;
        float x[8];
        if (VEC && i0 + 8 <= hi) {
            if (DT == TSB_BF16) {
                const uint4 raw = *(const uint4*)((const uint16_t*)draft + rowbase + i0);
                const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    x[2 * j] = __uint_as_float(w[j] << 16);
                    x[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
                }
            } else {
                const float4 a = *(const float4*)((const float*)draft + rowbase + i0);
                const float4 b = *(const float4*)((const float*)draft + rowbase + i0 + 4);
                x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
                x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
            }
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) x[j] = (i0 + j < hi) ? load_logit<DT>(draft, rowbase + i0 + j) : -INFINITY;
        }
        float a[8];
        float cm = -INFINITY;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const bool in = i0 + j < hi;
            a[j] = x[j] * invT;
            if (in && (isnan(a[j]) || a[j] == INFINITY)) bad = 1;
            if (in && a[j] > -INFINITY && a[j] < INFINITY) cm = fmaxf(cm, a[j]);
        }
        if (cm > m) {
            sum = (m == -INFINITY) ? 0.0 : sum * exp64((double)m - (double)cm, s_exp);
            m = cm;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (i0 + j < hi && a[j] > -INFINITY && a[j] < INFINITY) sum += exp64((double)a[j] - (double)m, s_exp);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const bool ok = (i0 + j < hi) && !isnan(x[j]);
            top.offer(cand_key(x[j], (uint32_t)(i0 + j)), ok);
        }
    }

    // combine lanes and waves in a fixed order
    __shared__ float s_m[kBlock / kWave];
    __shared__ double s_s[kBlock / kWave];
    __shared__ int s_bad[kBlock / kWave];
    __shared__ uint64_t s_top[kBlock / kWave][kWave];
    const int wave = tid / kWave, lane = tid % kWave;
    const float wm = wave_max(m);
    double contrib = (m == -INFINITY) ? 0.0 : sum * exp((double)m - (double)wm);
    const double ws = wave_sum(contrib);
    const int wb = wave_or(bad);
    if (lane == 0) {
        s_m[wave] = wm;
        s_s[wave] = ws;
        s_bad[wave] = wb;
    }
    s_top[wave][lane] = top.v;
    __syncthreads();
    if (wave == 0) {
        for (int w = 1; w < kBlock / kWave; ++w) {
            const uint64_t k = s_top[w][lane];
            top.offer(k, lane < K && k != 0);
        }
        if (lane == 0) {
            float M = s_m[0];
            for (int w = 1; w < kBlock / kWave; ++w) M = fmaxf(M, s_m[w]);
            double tot = 0.0;
            int anybad = 0;
            for (int w = 0; w < kBlock / kWave; ++w) {
                if (s_m[w] != -INFINITY) tot += s_s[w] * exp((double)s_m[w] - (double)M);
                anybad |= s_bad[w];
            }
            const size_t o = (size_t)row * S + s;
            pm[o] = M;
            ps[o] = tot;
            pf[o] = anybad;
        }
        if (lane < K) pk[((size_t)row * S + s) * K + lane] = top.v;
    }
}

// ------------------------------------------------------------------ K1b
__global__ __launch_bounds__(kWave) void draft_merge(int D, int S, int K, float invT, const float* __restrict__ pm,
                                                     const double* __restrict__ ps, const uint64_t* __restrict__ pk,
                                                     const int* __restrict__ pf, double* __restrict__ draft_lse,
                                                     int32_t* __restrict__ topk_tok, float* __restrict__ topk_lp,
                                                     int32_t* __restrict__ req_status) {
    const int row = blockIdx.x;
    const int lane = threadIdx.x;
    const size_t o = (size_t)row * S;
    float M = -INFINITY;
    int bad = 0;
    for (int s = lane; s < S; s += kWave) {
        M = fmaxf(M, pm[o + s]);
        bad |= pf[o + s];
    }
    M = wave_max(M);
    bad = wave_or(bad);
    double tot = 0.0;
    for (int s = lane; s < S; s += kWave)
        if (pm[o + s] != -INFINITY) tot += ps[o + s] * exp((double)pm[o + s] - (double)M);
    tot = wave_sum(tot);

    WaveTopList top;
    top.init(K);
    const int n = S * K;
    for (int base = 0; base < n; base += kWave) {
        const int i = base + lane;
        const uint64_t k = i < n ? pk[o * K + i] : 0;
        top.offer(k, i < n && k != 0);
    }

    const bool nonfinite = bad || M == -INFINITY;
    const double l64 = nonfinite ? (double)NAN : (double)M + log(tot);
    const float l32 = (float)l64;
    if (lane == 0) {
        draft_lse[row] = l64;
        if (nonfinite) atomicOr(&req_status[row / D], TSB_REQ_NONFINITE);
    }
    if (lane < K) {
        const uint64_t k = top.v;
        const float x = cand_value(k);
        const float a = x * invT;
        topk_tok[(size_t)row * K + lane] = (int32_t)cand_id(k);
        topk_lp[(size_t)row * K + lane] = a - l32;
    }
}

// ------------------------------------------------------------------ K2
struct PlanShared {
    float lp[TSB_MAX_D * TSB_MAX_K];
    double c_score[TSB_MAX_B + 1];
    int c_parent[TSB_MAX_B + 1];
    int c_rank[TSB_MAX_B + 1];
    int c_depth[TSB_MAX_B + 1];
    union {
        struct {
            double score[TSB_MAX_B + 2];
            int parent[TSB_MAX_B + 2];
            int rank[TSB_MAX_B + 2];
            int depth[TSB_MAX_B + 2];
        } f;  // frontier
        struct {
            int order[TSB_MAX_B + 1];
            int bfs_of[TSB_MAX_B + 1];
            int nch[TSB_MAX_B + 1];
            int fc[TSB_MAX_B + 1];
        } b;  // BFS canonicalisation
    } u;
};

// Frontier order: score desc, depth asc, rank path lexicographic asc.
__device__ __forceinline__ bool plan_better(const PlanShared& sh, int i, int j) {
    const double si = sh.u.f.score[i], sj = sh.u.f.score[j];
    if (si != sj) return si > sj;
    const int di = sh.u.f.depth[i], dj = sh.u.f.depth[j];
    if (di != dj) return di < dj;
    int pa = sh.u.f.parent[i], pb = sh.u.f.parent[j];
    int ra = sh.u.f.rank[i], rb = sh.u.f.rank[j];
    while (pa != pb) {  // equal depth: walk up to the common ancestor
        ra = sh.c_rank[pa];
        rb = sh.c_rank[pb];
        pa = sh.c_parent[pa];
        pb = sh.c_parent[pb];
    }
    return ra < rb;
}

__global__ __launch_bounds__(kWave) void plan_tree(int D, int K, int B, const float* __restrict__ topk_lp,
                                                   tsb_tree tree, int32_t* __restrict__ req_status) {
    __shared__ PlanShared sh;
    const int r = blockIdx.x;
    const int lane = threadIdx.x;
    const bool nonfinite = (req_status[r] & TSB_REQ_NONFINITE) != 0;
    const int Dp = nonfinite ? 0 : D;

    for (int i = lane; i < D * K; i += kWave) sh.lp[i] = topk_lp[(size_t)r * D * K + i];
    if (lane == 0) {
        sh.c_parent[0] = -1;
        sh.c_rank[0] = -1;
        sh.c_depth[0] = 0;
        sh.c_score[0] = 0.0;
    }
    __syncthreads();

    int nf = 0;
    if (Dp > 0 && isfinite(sh.lp[0])) {
        if (lane == 0) {
            sh.u.f.score[0] = 0.0 + (double)sh.lp[0];
            sh.u.f.parent[0] = 0;
            sh.u.f.rank[0] = 0;
            sh.u.f.depth[0] = 1;
        }
        nf = 1;
    }
    int committed = 1;
    __syncthreads();

    while (committed <= B && nf > 0) {
        int best = -1;
        for (int i = lane; i < nf; i += kWave)
            if (best < 0 || plan_better(sh, i, best)) best = i;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const int other = __shfl_xor(best, o, kWave);
            if (other >= 0 && (best < 0 || plan_better(sh, other, best))) best = other;
        }
        const int w = best;
        const double s = sh.u.f.score[w];
        const int par = sh.u.f.parent[w], rk = sh.u.f.rank[w], dep = sh.u.f.depth[w];
        const int c = committed++;
        const bool child = dep < Dp && isfinite(sh.lp[dep * K + 0]);
        const bool sib = rk + 1 < K && isfinite(sh.lp[(dep - 1) * K + rk + 1]);
        __syncthreads();
        if (lane == 0) {
            sh.c_parent[c] = par;
            sh.c_rank[c] = rk;
            sh.c_depth[c] = dep;
            sh.c_score[c] = s;
            int slot_free = 1;
            if (child) {
                sh.u.f.score[w] = s + (double)sh.lp[dep * K + 0];
                sh.u.f.parent[w] = c;
                sh.u.f.rank[w] = 0;
                sh.u.f.depth[w] = dep + 1;
                slot_free = 0;
            }
            if (sib) {
                const int slot = slot_free ? w : nf;
                sh.u.f.score[slot] = sh.c_score[par] + (double)sh.lp[(dep - 1) * K + rk + 1];
                sh.u.f.parent[slot] = par;
                sh.u.f.rank[slot] = rk + 1;
                sh.u.f.depth[slot] = dep;
                slot_free = 0;
            }
            if (slot_free && w != nf - 1) {
                sh.u.f.score[w] = sh.u.f.score[nf - 1];
                sh.u.f.parent[w] = sh.u.f.parent[nf - 1];
                sh.u.f.rank[w] = sh.u.f.rank[nf - 1];
                sh.u.f.depth[w] = sh.u.f.depth[nf - 1];
            }
        }
        nf += (child && sib) ? 1 : ((!child && !sib) ? -1 : 0);
        __syncthreads();
    }
    const int n = committed;

    // margin against the best uncommitted frontier node
    double bestf = -INFINITY;
    for (int i = lane; i < nf; i += kWave) bestf = fmax(bestf, sh.u.f.score[i]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) bestf = fmax(bestf, __shfl_xor(bestf, o, kWave));
    const double margin = (nf > 0 && n > 1) ? sh.c_score[n - 1] - bestf : (double)INFINITY;
    __syncthreads();

    // BFS canonicalisation (the frontier storage is reused)
    for (int i = lane; i < n; i += kWave) sh.u.b.nch[i] = 0;
    __syncthreads();
    for (int c = 1 + lane; c < n; c += kWave) atomicAdd(&sh.u.b.nch[sh.c_parent[c]], 1);
    if (lane == 0) {
        sh.u.b.order[0] = 0;
        sh.u.b.bfs_of[0] = 0;
    }
    __syncthreads();
    int lo = 0, hi = 1, L = 0;
    while (lo < hi) {
        int running = hi;
        for (int base = lo; base < hi; base += kWave) {
            const int i = base + lane;
            const int cnt = i < hi ? sh.u.b.nch[sh.u.b.order[i]] : 0;
            int incl = cnt;
#pragma unroll
            for (int o = 1; o < kWave; o <<= 1) {
                const int t = __shfl_up(incl, o, kWave);
                if (lane >= o) incl += t;
            }
            if (i < hi) sh.u.b.fc[i] = running + incl - cnt;
            running += __shfl(incl, kWave - 1, kWave);
        }
        __syncthreads();
        for (int c = 1 + lane; c < n; c += kWave) {
            if (sh.c_depth[c] == L + 1) {
                const int b = sh.u.b.fc[sh.u.b.bfs_of[sh.c_parent[c]]] + sh.c_rank[c];
                sh.u.b.order[b] = c;
                sh.u.b.bfs_of[c] = b;
            }
        }
        __syncthreads();
        lo = hi;
        hi = running;
        ++L;
    }

    const size_t o = (size_t)r * (B + 1);
    for (int i = lane; i < B + 1; i += kWave) {
        if (i < n) {
            const int c = sh.u.b.order[i];
            tree.parent[o + i] = c == 0 ? -1 : sh.u.b.bfs_of[sh.c_parent[c]];
            tree.depth[o + i] = sh.c_depth[c];
            tree.rank[o + i] = sh.c_rank[c];
            tree.score[o + i] = sh.c_score[c];
            tree.n_children[o + i] = sh.u.b.nch[c];
            tree.first_child[o + i] = sh.u.b.nch[c] ? sh.u.b.fc[i] : -1;
        } else {
            tree.parent[o + i] = -1;
            tree.depth[o + i] = -1;
            tree.rank[o + i] = -1;
            tree.score[o + i] = 0.0;
            tree.n_children[o + i] = 0;
            tree.first_child[o + i] = -1;
        }
    }
    if (lane == 0) {
        tree.n_nodes[r] = n;
        tree.plan_margin[r] = margin;
        if (!nonfinite && n < B + 1) req_status[r] |= TSB_REQ_BUDGET_SHORT;
    }
}

// ------------------------------------------------------------------ launch
hipError_t launch_plan(const tsb_config& c, float invT, const void* draft, double* draft_lse, int32_t* topk_tok,
                       float* topk_lp, const tsb_tree& tree, int32_t* req_status, char* ws, hipStream_t st) {
    const Geometry g = geometry(c);
    const PlanWs w = plan_ws(c);
    float* pm = (float*)(ws + w.pm);
    double* ps = (double*)(ws + w.ps);
    uint64_t* pk = (uint64_t*)(ws + w.pk);
    int* pf = (int*)(ws + w.pf);
    const dim3 grid1(g.S1, c.R * c.D);
    hipError_t e = hook_before(TSB_KERNEL_DRAFT_PARTIALS, st);
    if (e != hipSuccess) return e;
    const bool vec = (c.dtype == TSB_BF16) ? (c.V % 8 == 0 && ((uintptr_t)draft & 15) == 0)
                                           : (c.V % 4 == 0 && ((uintptr_t)draft & 15) == 0);
    if (c.dtype == TSB_BF16) {
        if (vec)
            draft_partials<TSB_BF16, true><<<grid1, kBlock, 0, st>>>(draft, c.V, c.D, g.seg1, g.S1, invT, c.K, pm, ps,
                                                                     pk, pf, req_status);
        else
            draft_partials<TSB_BF16, false><<<grid1, kBlock, 0, st>>>(draft, c.V, c.D, g.seg1, g.S1, invT, c.K, pm, ps,
                                                                      pk, pf, req_status);
    } else {
        if (vec)
            draft_partials<TSB_F32, true><<<grid1, kBlock, 0, st>>>(draft, c.V, c.D, g.seg1, g.S1, invT, c.K, pm, ps,
                                                                    pk, pf, req_status);
        else
            draft_partials<TSB_F32, false><<<grid1, kBlock, 0, st>>>(draft, c.V, c.D, g.seg1, g.S1, invT, c.K, pm, ps,
                                                                     pk, pf, req_status);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((e = hook_after(TSB_KERNEL_DRAFT_PARTIALS, st)) != hipSuccess) return e;
    if ((e = hook_before(TSB_KERNEL_DRAFT_MERGE, st)) != hipSuccess) return e;
    draft_merge<<<c.R * c.D, kWave, 0, st>>>(c.D, g.S1, c.K, invT, pm, ps, pk, pf, draft_lse, topk_tok, topk_lp,
                                             req_status);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((e = hook_after(TSB_KERNEL_DRAFT_MERGE, st)) != hipSuccess) return e;
    if ((e = hook_before(TSB_KERNEL_PLAN_TREE, st)) != hipSuccess) return e;
    plan_tree<<<c.R, kWave, 0, st>>>(c.D, c.K, c.B, topk_lp, tree, req_status);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return hook_after(TSB_KERNEL_PLAN_TREE, st);
}

}  // namespace tsb
