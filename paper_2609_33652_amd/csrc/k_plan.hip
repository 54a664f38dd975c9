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
// Eight consecutive logits of one row as binary32; positions at or past `hi`
// read as -inf.
template <int DT, bool VEC>
__device__ __forceinline__ void load8(const void* __restrict__ draft, size_t rowbase, int i0, int hi, float* x) {
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
            const float4 f0 = *(const float4*)((const float*)draft + rowbase + i0);
            const float4 f1 = *(const float4*)((const float*)draft + rowbase + i0 + 4);
            x[0] = f0.x; x[1] = f0.y; x[2] = f0.z; x[3] = f0.w;
            x[4] = f1.x; x[5] = f1.y; x[6] = f1.z; x[7] = f1.w;
        }
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = (i0 + j < hi) ? load_logit<DT>(draft, rowbase + i0 + j) : -INFINITY;
    }
}

constexpr int kDraftUnroll = 2;  // 8-logit groups per thread per chunk

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
    constexpr int kChunk = kBlock * 8 * kDraftUnroll;

    // the first chunk is in flight while the exp table is built
    float xc[kDraftUnroll][8];
#pragma unroll
    for (int u = 0; u < kDraftUnroll; ++u) load8<DT, VEC>(draft, rowbase, lo + (u * kBlock + tid) * 8, hi, xc[u]);

    __shared__ double s_exp[kExpTable];
    exp64_table_init(s_exp);

    float m = -INFINITY;    // running max of the scaled logits (-inf entries never raise it)
    double sum = 0.0;       // sum of e^(a - m) over this lane's elements
    bool bad = false;       // a NaN or +inf scaled logit
    WaveTopList top;
    top.init(K);
    // Filter (fx, fid): a logit x with id i can still enter the wave's list
    // only if x > fx, or x == fx and i <= fid (the key order is logit desc,
    // id asc). It starts at the K-th largest of the lanes' first-chunk maxima
    // (K distinct logits at or above it exist) with any id, and then follows
    // the list's K-th entry once the list is full.
    float fx;
    uint32_t fid = 0xFFFFFFFFu;
    {
        float lm = -INFINITY;
#pragma unroll
        for (int u = 0; u < kDraftUnroll; ++u)
#pragma unroll
            for (int j = 0; j < 8; ++j) lm = fmaxf(lm, xc[u][j]);
        fx = wave_kth_largest(lm, K);
    }

    for (int base = lo; base < hi; base += kChunk) {
        const int nbase = base + kChunk;
        float xn[kDraftUnroll][8];
        if (nbase < hi) {
#pragma unroll
            for (int u = 0; u < kDraftUnroll; ++u)
                load8<DT, VEC>(draft, rowbase, nbase + (u * kBlock + tid) * 8, hi, xn[u]);
        } else {
#pragma unroll
            for (int u = 0; u < kDraftUnroll; ++u)
#pragma unroll
                for (int j = 0; j < 8; ++j) xn[u][j] = -INFINITY;
        }
#pragma unroll
        for (int u = 0; u < kDraftUnroll; ++u) {
            const int i0 = base + (u * kBlock + tid) * 8;
            float xm = xc[u][0];
#pragma unroll
            for (int j = 1; j < 8; ++j) xm = fmaxf(xm, xc[u][j]);  // NaN is ignored
            float a[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                a[j] = xc[u][j] * invT;
                bad |= __builtin_amdgcn_classf(a[j], 0x203);  // signalling NaN, quiet NaN, +inf
            }
            // rounding is monotone, so the max of the scaled values is the scaled max
            const float am = xm * invT;
            if (am > m && am < INFINITY) {
                sum = (m == -INFINITY) ? 0.0 : sum * exp64((double)m - (double)am, s_exp);
                m = am;
            }
            const double md = (double)m;
#pragma unroll
            for (int j = 0; j < 8; ++j) sum += exp64((double)a[j] - md, s_exp);
            // the group's smallest id is i0
            if (__ballot(xm > fx || (xm == fx && (uint32_t)i0 <= fid))) {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const float xj = xc[u][j];
                    const uint32_t id = (uint32_t)(i0 + j);
                    const bool ok = (i0 + j < hi) && (xj > fx || (xj == fx && id <= fid));  // false for NaN
                    top.offer(cand_key(xj, id), ok);
                }
                if (top.thr) {
                    // the list's K-th key; entering now needs a key above it
                    const float tx = cand_value(top.thr);
                    const uint32_t tid1 = cand_id(top.thr);
                    if (tx > fx || (tx == fx && tid1 <= fid)) {
                        fx = tx;
                        fid = tid1 - 1;  // wraps for id 0 to "any id": looser, and offer re-checks the key
                    }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kDraftUnroll; ++u)
#pragma unroll
            for (int j = 0; j < 8; ++j) xc[u][j] = xn[u][j];
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
// Frontier of the lazy best-first expansion, one wave per request. The best
// (up to) 64 frontier entries are kept sorted across the lanes of the wave
// (lane i holds the i-th best), so a pop is lane 0 and a whole-wave one-lane
// DPP shift, and a push is a ballot for its position and a one-lane shift.
// Entries that fall off the end go to a "cold" list in LDS; every cold entry
// ranks after every hot entry (a push that ranks after the best cold entry
// goes to the cold list too), so the hot head is always the global best.
// When the hot list runs empty, the best cold entries are moved back.
//
// Entry: score (binary64); info = depth << 16 | rank << 10 | parent (pop
// index of the committed parent, root = 0); the parent's score; and the two
// planning log-probabilities the entry needs once popped (its first child's
// and its next sibling's), so a pop reads no memory.
constexpr int kInfoParentBits = 10;
constexpr int kInfoRankBits = 6;

struct PlanShared {
    float lp[TSB_MAX_D * TSB_MAX_K];
    double c_score[TSB_MAX_B + 1];
    int c_parent[TSB_MAX_B + 1];
    int c_rank[TSB_MAX_B + 1];
    int c_depth[TSB_MAX_B + 1];
    union {
        struct {
            double score[TSB_MAX_B + 2];
            double pscore[TSB_MAX_B + 2];
            uint32_t info[TSB_MAX_B + 2];
        } cold;
        struct {
            int order[TSB_MAX_B + 1];
            int bfs_of[TSB_MAX_B + 1];
            int nch[TSB_MAX_B + 1];
            int fc[TSB_MAX_B + 1];
        } b;  // BFS canonicalisation
    } u;
};

__device__ __forceinline__ int info_depth(uint32_t i) { return (int)(i >> 16); }
__device__ __forceinline__ int info_rank(uint32_t i) { return (int)((i >> kInfoParentBits) & ((1u << kInfoRankBits) - 1)); }
__device__ __forceinline__ int info_parent(uint32_t i) { return (int)(i & ((1u << kInfoParentBits) - 1)); }
__device__ __forceinline__ uint32_t make_info(int depth, int rank, int parent) {
    return ((uint32_t)depth << 16) | ((uint32_t)rank << kInfoParentBits) | (uint32_t)parent;
}

// Static order of frontier entries: score desc, depth asc, rank path
// lexicographic asc (equal depth: walk both parents up to their common
// ancestor and compare the ranks just below it). True if a precedes b.
__device__ __forceinline__ bool plan_precedes(const PlanShared& sh, double sa, uint32_t ia, double sb, uint32_t ib) {
    if (sa != sb) return sa > sb;
    const int da = info_depth(ia), db = info_depth(ib);
    if (da != db) return da < db;
    int pa = info_parent(ia), pb = info_parent(ib);
    int ra = info_rank(ia), rb = info_rank(ib);
    for (int guard = 0; pa != pb && guard < TSB_MAX_D; ++guard) {
        ra = sh.c_rank[pa];
        rb = sh.c_rank[pb];
        pa = sh.c_parent[pa];
        pb = sh.c_parent[pb];
    }
    return ra < rb;
}

struct Entry {
    double s, ps;   // score, parent's score
    uint32_t i;     // info
    float lc, lsib; // first child's lp (NaN: none), next sibling's lp (NaN: none)
};

__device__ __forceinline__ Entry shr1(const Entry& e) {
    return Entry{wave_shr1(e.s), wave_shr1(e.ps), wave_shr1(e.i), __uint_as_float(wave_shr1(__float_as_uint(e.lc))),
                 __uint_as_float(wave_shr1(__float_as_uint(e.lsib)))};
}
__device__ __forceinline__ Entry shl1(const Entry& e) {
    return Entry{wave_shl1(e.s), wave_shl1(e.ps), wave_shl1(e.i), __uint_as_float(wave_shl1(__float_as_uint(e.lc))),
                 __uint_as_float(wave_shl1(__float_as_uint(e.lsib)))};
}
__device__ __forceinline__ Entry lane_entry(const Entry& e, int l) {
    return Entry{lane_f64(e.s, l), lane_f64(e.ps, l), lane_u32(e.i, l), lane_f32(e.lc, l), lane_f32(e.lsib, l)};
}

// lp values a new entry (depth dep, rank rk) will need once popped
__device__ __forceinline__ Entry make_entry(const PlanShared& sh, int Dp, int K, double s, double ps, int dep, int rk,
                                            int par) {
    Entry e;
    e.s = s;
    e.ps = ps;
    e.i = make_info(dep, rk, par);
    e.lc = dep < Dp ? sh.lp[dep * K + 0] : (float)NAN;
    e.lsib = rk + 1 < K ? sh.lp[(dep - 1) * K + rk + 1] : (float)NAN;
    return e;
}

struct Frontier {
    Entry h;  // this lane's hot entry
    int nh, ncold;
    double cold_s;  // best cold entry (valid when ncold > 0)
    uint32_t cold_i;
};

__device__ __forceinline__ void frontier_to_cold(PlanShared& sh, Frontier& F, const Entry& e) {
    if (lane_id() == 0) {
        sh.u.cold.score[F.ncold] = e.s;
        sh.u.cold.pscore[F.ncold] = e.ps;
        sh.u.cold.info[F.ncold] = e.i;
    }
    if (F.ncold == 0 || plan_precedes(sh, e.s, e.i, F.cold_s, F.cold_i)) {
        F.cold_s = e.s;
        F.cold_i = e.i;
    }
    ++F.ncold;
}

__device__ __forceinline__ void frontier_push(PlanShared& sh, Frontier& F, const Entry& e) {
    // entries ranking after the best cold entry stay cold (invariant)
    if (F.ncold > 0 && !plan_precedes(sh, e.s, e.i, F.cold_s, F.cold_i)) {
        frontier_to_cold(sh, F, e);
        return;
    }
    const int lane = lane_id();
    const bool before = lane < F.nh && plan_precedes(sh, F.h.s, F.h.i, e.s, e.i);
    const int pos = __popcll(__ballot(before));
    if (F.nh == kWave) {  // the entry that leaves: the old tail, or e if it ranks last
        if (pos == kWave) {
            frontier_to_cold(sh, F, e);
            return;
        }
        frontier_to_cold(sh, F, lane_entry(F.h, kWave - 1));
    }
    const Entry up = shr1(F.h);
    if (lane == pos)
        F.h = e;
    else if (lane > pos)
        F.h = up;
    if (F.nh < kWave) ++F.nh;
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

    Frontier F;
    F.h.s = -INFINITY;
    F.h.ps = 0.0;
    F.h.i = 0;
    F.h.lc = F.h.lsib = (float)NAN;
    F.nh = 0;
    F.ncold = 0;
    F.cold_s = -INFINITY;
    F.cold_i = 0;

    if (Dp > 0 && isfinite(sh.lp[0])) frontier_push(sh, F, make_entry(sh, Dp, K, 0.0 + (double)sh.lp[0], 0.0, 1, 0, 0));
    int committed = 1;

    while (committed <= B && (F.nh > 0 || F.ncold > 0)) {
        if (F.nh == 0) {
            // refill: move the best cold entries back, best first
            __syncthreads();
            const int take = F.ncold < kWave ? F.ncold : kWave;
            for (int t = 0; t < take; ++t) {
                double bs = -INFINITY;
                uint32_t bi = 0;
                int bj = -1;
                for (int j = lane; j < F.ncold; j += kWave) {
                    const double cs = sh.u.cold.score[j];
                    const uint32_t ci = sh.u.cold.info[j];
                    if (bj < 0 || plan_precedes(sh, cs, ci, bs, bi)) {
                        bs = cs;
                        bi = ci;
                        bj = j;
                    }
                }
#pragma unroll
                for (int o = 32; o > 0; o >>= 1) {
                    const double os = __shfl_xor(bs, o, kWave);
                    const uint32_t oi = (uint32_t)__shfl_xor((int)bi, o, kWave);
                    const int oj = __shfl_xor(bj, o, kWave);
                    if (oj >= 0 && (bj < 0 || plan_precedes(sh, os, oi, bs, bi))) {
                        bs = os;
                        bi = oi;
                        bj = oj;
                    }
                }
                const double bps = sh.u.cold.pscore[bj];
                if (lane == t) F.h = make_entry(sh, Dp, K, bs, bps, info_depth(bi), info_rank(bi), info_parent(bi));
                __syncthreads();
                if (lane == 0) {
                    sh.u.cold.score[bj] = sh.u.cold.score[F.ncold - 1];
                    sh.u.cold.pscore[bj] = sh.u.cold.pscore[F.ncold - 1];
                    sh.u.cold.info[bj] = sh.u.cold.info[F.ncold - 1];
                }
                --F.ncold;
                __syncthreads();
            }
            F.nh = take;
            // best remaining cold entry
            if (F.ncold > 0) {
                double bs = -INFINITY;
                uint32_t bi = 0;
                int bj = -1;
                for (int j = lane; j < F.ncold; j += kWave) {
                    const double cs = sh.u.cold.score[j];
                    const uint32_t ci = sh.u.cold.info[j];
                    if (bj < 0 || plan_precedes(sh, cs, ci, bs, bi)) {
                        bs = cs;
                        bi = ci;
                        bj = j;
                    }
                }
#pragma unroll
                for (int o = 32; o > 0; o >>= 1) {
                    const double os = __shfl_xor(bs, o, kWave);
                    const uint32_t oi = (uint32_t)__shfl_xor((int)bi, o, kWave);
                    const int oj = __shfl_xor(bj, o, kWave);
                    if (oj >= 0 && (bj < 0 || plan_precedes(sh, os, oi, bs, bi))) {
                        bs = os;
                        bi = oi;
                        bj = oj;
                    }
                }
                F.cold_s = bs;
                F.cold_i = bi;
            }
        }
        // pop the head
        const Entry top = lane_entry(F.h, 0);
        {
            const Entry dn = shl1(F.h);
            if (lane < F.nh - 1) F.h = dn;
            --F.nh;
        }
        const int dep = info_depth(top.i), rk = info_rank(top.i), par = info_parent(top.i);
        const int c = committed++;
        if (lane == 0) {  // single wave: later LDS reads see these writes in order
            sh.c_parent[c] = par;
            sh.c_rank[c] = rk;
            sh.c_depth[c] = dep;
            sh.c_score[c] = top.s;
        }
        if (!isnan(top.lc) && isfinite(top.lc))
            frontier_push(sh, F, make_entry(sh, Dp, K, top.s + (double)top.lc, top.s, dep + 1, 0, c));
        if (!isnan(top.lsib) && isfinite(top.lsib))
            frontier_push(sh, F, make_entry(sh, Dp, K, top.ps + (double)top.lsib, top.ps, dep, rk + 1, par));
    }
    __syncthreads();
    const int nf = F.nh + F.ncold;
    // best uncommitted: the hot head (the cold list ranks after it), else the best cold entry
    const double bestf = F.nh > 0 ? lane_f64(F.h.s, 0) : F.cold_s;
    const int n = committed;
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
