// Verification of the replayed tree on gfx950 (Section 2.3, eq. (1);
// Appendix A: recursive rejection sampling without replacement; Section 3.3:
// the probabilities are those of the replayed candidates).
//
//   target_partials  grid (segment, request x node): one streaming read of
//                    every target row of the tree; online max and sum of
//                    exp per segment (binary32 terms, binary64 per lane).
//   verify_walk      resident grid (G workgroups per request). All G
//                    workgroups of a request replay the same scalar walk;
//                    every vocabulary-wide reduction of the walk (residual
//                    mass after a rejection, the bonus draw) is split over
//                    them and exchanged through the request's tagged slots
//                    (each workgroup polls the others' slots).
//
// Closed form of WoR-RRS used by the walk (equal to the literal recursion
// of residuals; derived from eq. (1) and the without-replacement update):
// with C_0 = 0, S_0 = 1, Z_0 = 1 at a node, child i with token y is accepted
// iff U < max(p(y) - C_i q(y), 0) / (W_i q(y)), W_i = Z_i / S_i; on
// rejection C_{i+1} = C_i + W_i, S_{i+1} = S_i - q(y),
// Z_{i+1} = sum_v max(p_v - C_{i+1} q_v, 0). The bonus token is
// argmax_v ln max(p_v - C q_v, 0) + G_v (Gumbel-max of the residual; C = 0
// at an accepted leaf).
#include <math.h>

#include <atomic>

#include "tsb_device.hpp"
#include "tsb_exchange.hpp"
#include "tsb_kernels.hpp"
#include "tsb_target.hpp"

namespace tsb {

// ------------------------------------------------------------------ K4
// The target stream on a grid of its own (tsb_verify and the other
// verification entry points; a round runs it inside the replay scan's grid).
template <int DT, bool VEC>
__global__ __launch_bounds__(kBlock) void target_partials(const void* __restrict__ target, int V, int B, int nrows,
                                                          long long chunk, int P, float invT,
                                                          const int32_t* __restrict__ n_nodes,
                                                          float* __restrict__ tm, double* __restrict__ ts,
                                                          int* __restrict__ tf, XRegion X, int R) {
    target_chunk<DT, VEC, kTargetPrefetch>(blockIdx.x, gridDim.x, target, V, B, nrows, chunk, P, invT, n_nodes, tm, ts, tf, X, R);
}

// ------------------------------------------------------------------ K5
struct WalkArgs {
    const void* draft;
    const double* draft_lse;
    const void* target;
    tsb_tree tree;
    const int32_t* node_tok;
    tsb_verdict out;
    const float* tm;
    const double* ts;
    const int* tf;
    XRegion X;  // exchange slots of the requests
    int V, D, B, S4;
    int R, G;   // requests and workgroups per request of the launch (tickets)
    unsigned long long* stats;  // work counters (null: none)
    float invT;
    uint32_t k0, k1, step;
    // pool walk only: pools [R, D, P] and transition scores [R, D-1, P, P]
    const int32_t* pool_tok;
    const float* trans;
    int P;
    // node records (kRecWords per node) when the round's merge wrote them, else null
    const uint32_t* nrec;
    // the RRS walk reads each target row as it enters the node (else the row
    // normalisers come from a stream of every row, through the records or the
    // partials), except rows 0 and 1, streamed before it into their own
    // partials [R][kChainRows][kChainPieces]
    int reads_rows;
    const float* cm;
    const double* cs;
    const int* cf;
};

// binary64 log-sum-exp of target row (r, node) from its segment partials
__device__ double target_lse(const WalkArgs& A, int r, int node, int* bad) {
    return target_row_lse(A.tm, A.ts, A.tf, A.S4, (size_t)r * (A.B + 1) + node, bad);
}

__device__ __forceinline__ double rec_f64(uint32_t lo, uint32_t hi) {
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

struct SplitF {  // binary64 value as binary32 hi + lo
    float hi, lo;
};
__device__ __forceinline__ SplitF split(double v) {
    SplitF s;
    s.hi = (float)v;
    s.lo = (float)(v - (double)s.hi);
    return s;
}

// Block-wide binary64 sum (fixed order: lanes, then waves).
__device__ double block_sum(double v) {
    __shared__ double red[kBlock / kWave];
    const double w = wave_sum(v);
    if ((threadIdx.x % kWave) == 0) red[threadIdx.x / kWave] = w;
    __syncthreads();
    double tot = 0.0;
    for (int i = 0; i < kBlock / kWave; ++i) tot += red[i];
    __syncthreads();
    return tot;
}

// ---------------------------------------------------------------- walk
// A walk workgroup owns the slice [v0, v1) of the vocabulary. At every
// visited node u with children, the first pass over the slice computes, in
// binary64, p~_v = exp(a^t_{u,v} - L0) (L0 the streamed estimate of the
// target normaliser) and q_v = exp(a^d_{depth(u),v} - lse_d), keeps both in
// LDS and returns sum p~ (the exact normaliser is L0 + ln sum_v p~_v over the
// request). The residual passes after rejections and the residual bonus then
// read (p~, q) from LDS. Slices longer than the LDS cache are processed in
// chunks that are recomputed in every pass.
constexpr int kWalkThreads = 512;
constexpr int kWalkCache = kWalkTokensPerGroup;  // tokens of (p~, q) held in LDS

template <int DT>
__device__ __forceinline__ void load4_scaled(const void* base, size_t off, int valid, bool vec, float invT,
                                             float a[4]) {
    float x[4];
    load4<DT>(base, off, valid, vec, x);
#pragma unroll
    for (int e = 0; e < 4; ++e) a[e] = e < valid ? x[e] * invT : -INFINITY;
}

// Block-wide binary64 sum for kWalkThreads threads (fixed order).
__device__ double walk_sum(double v) {
    __shared__ double red[kWalkThreads / kWave];
    const double w = wave_sum(v);
    if ((threadIdx.x % kWave) == 0) red[threadIdx.x / kWave] = w;
    __syncthreads();
    double tot = 0.0;
    for (int i = 0; i < kWalkThreads / kWave; ++i) tot += red[i];
    __syncthreads();
    return tot;
}

// Four block-wide binary64 sums in one reduction (same fixed order as walk_sum).
__device__ void walk_sum4(double (&v)[4]) {
    __shared__ double red4[4][kWalkThreads / kWave];
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = wave_sum(v[k]);
    if ((threadIdx.x % kWave) == 0)
#pragma unroll
        for (int k = 0; k < 4; ++k) red4[k][threadIdx.x / kWave] = v[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        double tot = 0.0;
        for (int i = 0; i < kWalkThreads / kWave; ++i) tot += red4[k][i];
        v[k] = tot;
    }
    __syncthreads();
}

struct WalkSlice {
    int v0, v1, nchunks;
    double* p;  // LDS [kWalkCache]
    double* q;  // LDS [kWalkCache]
};

// First pass at a node: fill (p~, q) for chunk c (into LDS when the slice has
// one chunk) and return sum p~ over the chunk. Groups of four tokens per
// thread; two groups are loaded before either is used.
template <int DT>
__device__ double fill_chunk(const WalkArgs& A, bool vec, const WalkSlice& S, int c, size_t trow, size_t drow,
                             double L0, double Ld, const double* et, bool store) {
    const int c0 = S.v0 + c * kWalkCache;
    const int n = min(kWalkCache, S.v1 - c0);
    double acc = 0.0;
    for (int base = 0; base * 4 < n; base += 2 * kWalkThreads) {
        float at[2][4], ad[2][4];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int i = (base + j * kWalkThreads + (int)threadIdx.x) * 4;
            const int valid = max(0, min(4, n - i));
            load4_scaled<DT>(A.target, trow + c0 + (valid ? i : 0), valid, vec, A.invT, at[j]);
            load4_scaled<DT>(A.draft, drow + c0 + (valid ? i : 0), valid, vec, A.invT, ad[j]);
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int i = (base + j * kWalkThreads + (int)threadIdx.x) * 4;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (i + e >= n) break;
                const double pt = at[j][e] > -INFINITY ? exp64((double)at[j][e] - L0, et) : 0.0;
                const double qd = ad[j][e] > -INFINITY ? exp64((double)ad[j][e] - Ld, et) : 0.0;
                acc += pt;
                if (store) {
                    S.p[i + e] = pt;
                    S.q[i + e] = qd;
                }
            }
        }
    }
    return acc;
}

// Token-wise visit of (p = p~ * inv, q) over the slice: from LDS when cached,
// else recomputed chunk by chunk. f(token, p, q) is called for every token.
template <int DT, typename F>
__device__ void visit_pq(const WalkArgs& A, bool vec, const WalkSlice& S, bool cached, size_t trow, size_t drow,
                         double L0, double inv, double Ld, const double* et, F f) {
    if (cached) {
        const int n = S.v1 - S.v0;
        for (int i = threadIdx.x; i < n; i += kWalkThreads) f(S.v0 + i, S.p[i] * inv, S.q[i]);
        return;
    }
    for (int c = 0; c < S.nchunks; ++c) {
        const int c0 = S.v0 + c * kWalkCache;
        const int n = min(kWalkCache, S.v1 - c0);
        for (int i4 = threadIdx.x; i4 * 4 < n; i4 += kWalkThreads) {
            const int i = i4 * 4;
            const int valid = min(4, n - i);
            float at[4], ad[4];
            load4_scaled<DT>(A.target, trow + c0 + i, valid, vec, A.invT, at);
            load4_scaled<DT>(A.draft, drow + c0 + i, valid, vec, A.invT, ad);
            for (int e = 0; e < valid; ++e) {
                const double pt = at[e] > -INFINITY ? exp64((double)at[e] - L0, et) : 0.0;
                const double qd = ad[e] > -INFINITY ? exp64((double)ad[e] - Ld, et) : 0.0;
                f(c0 + i + e, pt * inv, qd);
            }
        }
    }
}

// (key, token) argmax across the workgroup: key desc, token asc.
__device__ void walk_argmax(float* best, int* bidx) {
    float b = *best;
    int bi = *bidx;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const float ok = __shfl_xor(b, off, kWave);
        const int oi = __shfl_xor(bi, off, kWave);
        if (ok > b || (ok == b && oi < bi)) {
            b = ok;
            bi = oi;
        }
    }
    __shared__ float rk[kWalkThreads / kWave];
    __shared__ int ri[kWalkThreads / kWave];
    if ((threadIdx.x % kWave) == 0) {
        rk[threadIdx.x / kWave] = b;
        ri[threadIdx.x / kWave] = bi;
    }
    __syncthreads();
    b = rk[0];
    bi = ri[0];
    for (int i = 1; i < kWalkThreads / kWave; ++i)
        if (rk[i] > b || (rk[i] == b && ri[i] < bi)) {
            b = rk[i];
            bi = ri[i];
        }
    __syncthreads();
    *best = b;
    *bidx = bi;
}

// Bonus sample from p_u alone (leaf, or empty residual): argmax ln p_v + G_v,
// read straight from the target row.
template <int DT>
__device__ void bonus_from_p(const WalkArgs& A, bool vec, const WalkSlice& S, size_t trow, double Lt,
                             const RngKey& key, uint32_t node, float* bk, int* bi) {
    float best = -INFINITY;
    int bidx = 0x7FFFFFFF;
    const SplitF Ls = split(Lt);
    const int n = S.v1 - S.v0;
    // two groups of four per thread and iteration, both loads issued before
    // either is used
    for (int i4 = threadIdx.x; i4 * 4 < n; i4 += 2 * kWalkThreads) {
        float at[2][4];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int i = (i4 + h * kWalkThreads) * 4;
            const int valid = max(0, min(4, n - i));
            load4_scaled<DT>(A.target, trow + S.v0 + (valid ? i : 0), valid, vec, A.invT, at[h]);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int i = (i4 + h * kWalkThreads) * 4;
            const int valid = max(0, min(4, n - i));
            if (valid == 0) continue;
            const uint4 w = rng_block(key, node, kStreamBonus, (uint32_t)((S.v0 + i) >> 2));
            const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (e >= valid || at[h][e] == -INFINITY) continue;
                const float kv = ((at[h][e] - Ls.hi) - Ls.lo) + gumbel_f32(ws[e]);  // ln p_v + G_v
                const int v = S.v0 + i + e;
                if (kv > best || (kv == best && v < bidx)) {
                    best = kv;
                    bidx = v;
                }
            }
        }
    }
    walk_argmax(&best, &bidx);
    *bk = best;
    *bi = bidx;
}

// Exchange among the G workgroups of a request through the request's
// tagged slots: each contributes up to four binary64 partials (and
// optionally a (key, token) pair); everyone gets the sums (a fixed reduction
// tree over the workgroups, so every run adds in the same order) and the
// best pair. Partials travel with 2^-44 relative resolution.
constexpr int kExVals = 4;

struct Exchange {
    const WalkArgs* A;
    int r, g, G;
    uint32_t nb;  // rounds run
    int timeout;

    template <int NV, bool BEST>
    __device__ void run(const double (&part)[NV], double (&tot)[NV], float bk, int bi, float* fk, int* fi) {
        static_assert(NV <= kExVals, "exchange width");
        constexpr int NW = NV + (BEST ? 2 : 0);
        uint64_t w[NW];
#pragma unroll
        for (int i = 0; i < NV; ++i) w[i] = xpack_f64(part[i]);
        if (BEST) {
            w[NV] = xpack_u32(ordered_bits(bk));
            w[NW - 1] = xpack_u32((uint32_t)bi);
        }
        xpublish<NW>(A->X, r, g, nb, w);
        // wave 0 polls the G slots (lane h: slots h and h + 64), reduces them
        // in a fixed order and hands the result to the others
        __shared__ double s_tot[kExVals];
        __shared__ float s_bk;
        __shared__ int s_bi, s_to;
        if (threadIdx.x < kWave) {
            const int lane = threadIdx.x;
            double v[NV];
            uint32_t kb = 0u, ib = 0xFFFFFFFFu;
            int to = 0;
#pragma unroll
            for (int i = 0; i < NV; ++i) v[i] = 0.0;
#pragma unroll
            for (int half = 0; half < kWalkGroupsMax / kWave; ++half) {
                const int h = lane + half * kWave;
                if (h < G) {
                    uint64_t q[NW];
                    if (!xpoll<NW>(A->X, r, h, nb, q)) to = 1;
#pragma unroll
                    for (int i = 0; i < NV; ++i) v[i] += xunpack_f64(q[i]);
                    if (BEST) {
                        const uint32_t k = xunpack_u32(q[NV]), ix = xunpack_u32(q[NW - 1]);
                        if (k > kb || (k == kb && ix < ib)) {
                            kb = k;
                            ib = ix;
                        }
                    }
                }
            }
#pragma unroll
            for (int i = 0; i < NV; ++i) v[i] = wave_sum(v[i]);
            if (BEST) {
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) {
                    const uint32_t ok = (uint32_t)__shfl_xor((int)kb, off, kWave);
                    const uint32_t oi = (uint32_t)__shfl_xor((int)ib, off, kWave);
                    if (ok > kb || (ok == kb && oi < ib)) {
                        kb = ok;
                        ib = oi;
                    }
                }
            }
            to = wave_or(to);
            if (lane == 0) {
#pragma unroll
                for (int i = 0; i < NV; ++i) s_tot[i] = v[i];
                s_bk = kb ? from_ordered_bits(kb) : -INFINITY;
                s_bi = (int)ib;
                s_to = to;
            }
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < NV; ++i) tot[i] = s_tot[i];
        if (BEST) {
            *fk = s_bk;
            *fi = s_bi;
        }
        if (s_to) timeout = 1;
        ++nb;
        __syncthreads();  // s_tot is rewritten by the next exchange
    }
    template <int NV>
    __device__ void run(const double (&part)[NV], double (&tot)[NV]) {
        run<NV, false>(part, tot, 0.f, 0, nullptr, nullptr);
    }
    __device__ double sum(double part) {
        double p[1] = {part}, t[1];
        run<1>(p, t);
        return t[0];
    }
    __device__ int best(float bk, int bi, double part, double* tot) {
        double p[1] = {part}, t[1];
        float fk;
        int fi;
        run<1, true>(p, t, bk, bi, &fk, &fi);
        *tot = t[0];
        return fk > -INFINITY ? fi : -1;
    }
    // Log-sum-exp of the workgroups' (max a, sum exp(a - max a)) pairs: the
    // largest max, then every sum rescaled to it and added in a fixed order
    // (every workgroup gets the same value). *bad if a workgroup flagged its
    // part, or if no part holds a finite logit.
    __device__ double lse(double mx, double s, bool part_bad, bool* bad) {
        constexpr int NH = kWalkGroupsMax / kWave;
        const uint64_t w[3] = {xpack_f64(mx), xpack_f64(s), xpack_u32(part_bad ? 1u : 0u)};
        xpublish<3>(A->X, r, g, nb, w);
        __shared__ double s_l;
        __shared__ int s_b, s_to;
        if (threadIdx.x < kWave) {
            const int lane = threadIdx.x;
            double hm[NH], hs[NH];
            int b = 0, to = 0;
            double M = -INFINITY;
#pragma unroll
            for (int half = 0; half < NH; ++half) {
                const int h = lane + half * kWave;
                hm[half] = -INFINITY;
                hs[half] = 0.0;
                if (h < G) {
                    uint64_t q[3];
                    if (!xpoll<3>(A->X, r, h, nb, q)) to = 1;
                    hm[half] = xunpack_f64(q[0]);
                    hs[half] = xunpack_f64(q[1]);
                    b |= xunpack_u32(q[2]) != 0u;
                }
                M = fmax(M, hm[half]);
            }
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) M = fmax(M, __shfl_xor(M, off, kWave));
            double t = 0.0;
            if (M > -INFINITY)
#pragma unroll
                for (int half = 0; half < NH; ++half)
                    if (hm[half] > -INFINITY) t += hs[half] * exp(hm[half] - M);
            t = wave_sum(t);
            b = wave_or(b);
            to = wave_or(to);
            if (lane == 0) {
                const bool none = !(M > -INFINITY) || !(t > 0.0);
                s_l = none ? 0.0 : M + log(t);
                s_b = b || none || !isfinite(M) || !isfinite(t);
                s_to = to;
            }
        }
        __syncthreads();
        const double L = s_l;
        *bad = s_b != 0;
        if (s_to) timeout = 1;
        ++nb;
        __syncthreads();  // s_l is rewritten by the next exchange
        return L;
    }
};

// Streamed normaliser of the target row of the node the walk enters (the
// walk reads a target row only when it enters its node): each workgroup
// streams its slice (running maximum m of the raw logits, binary32 terms
// 2^(x c - m c) with c = invT log2(e), added in binary64, as the target
// stream does), then the request's workgroups combine their parts by one
// exchange. Within ~1e-6 of ln sum_v exp(a_v); *bad if the row holds a NaN
// or +inf logit, or no finite one. The slice is read in batches of
// kRowGroups groups of four logits per thread (one batch covers a slice of
// up to 10240 logits).
constexpr int kRowGroups = 5;
template <int DT>
struct RowBatch {
    Raw4<DT> g[kRowGroups];
};

template <int DT>
__device__ __forceinline__ void row_batch_load(const WalkArgs& A, bool vec, const WalkSlice& S, size_t trow, int base,
                                               RowBatch<DT>& rb) {
    const int n = S.v1 - S.v0;
#pragma unroll
    for (int k = 0; k < kRowGroups; ++k) {
        const int i = base + (k * kWalkThreads + (int)threadIdx.x) * 4;
        const int valid = max(0, min(4, n - i));
        raw_load4<DT>(A.target, trow + S.v0 + (valid ? i : 0), valid, vec, rb.g[k]);
    }
}

template <int DT>
__device__ double entered_row_lse(const WalkArgs& A, bool vec, const WalkSlice& S, size_t trow, Exchange& X,
                                  bool* bad) {
    const float c = A.invT * 1.4426950408889634f;
    const int n = S.v1 - S.v0;
    constexpr int kBatch = kRowGroups * 4 * kWalkThreads;
    float m = -INFINITY;
    double sum = 0.0;
    bool nf = false;
    for (int base = 0; base < n; base += kBatch) {
        RowBatch<DT> rb;
        row_batch_load<DT>(A, vec, S, trow, base, rb);
        float x[kRowGroups][4];
#pragma unroll
        for (int k = 0; k < kRowGroups; ++k) {
            if (DT == TSB_BF16) {
                x[k][0] = __uint_as_float(rb.g[k].w[0] << 16);
                x[k][1] = __uint_as_float(rb.g[k].w[0] & 0xFFFF0000u);
                x[k][2] = __uint_as_float(rb.g[k].w[1] << 16);
                x[k][3] = __uint_as_float(rb.g[k].w[1] & 0xFFFF0000u);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) x[k][e] = __uint_as_float(rb.g[k].w[e]);
            }
        }
        float cm = m;
#pragma unroll
        for (int k = 0; k < kRowGroups; ++k)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                nf |= __builtin_amdgcn_classf(x[k][e], 0x203);  // signalling NaN, quiet NaN, +inf
                cm = fmaxf(cm, x[k][e]);                        // NaN is ignored
            }
        if (cm > m) {
            if (m > -INFINITY) sum *= (double)exp2f((m - cm) * c);
            m = cm;
        }
        if (m > -INFINITY && m < INFINITY) {
            const float mc = m * c;
#pragma unroll
            for (int k = 0; k < kRowGroups; ++k) {
                float cs = 0.f;
#pragma unroll
                for (int e = 0; e < 4; ++e) cs += __builtin_amdgcn_exp2f(fmaf(x[k][e], c, -mc));
                sum += (double)cs;
            }
        }
    }
    // the workgroup's part: (max a, sum exp(a - max a)), fixed order
    __shared__ float s_m[kWalkThreads / kWave];
    __shared__ double s_s[kWalkThreads / kWave];
    __shared__ int s_nf;
    if (threadIdx.x == 0) s_nf = 0;
    const float wm = wave_max(m);
    const double ws = wave_sum((m == -INFINITY || m == wm) ? (m == -INFINITY ? 0.0 : sum)
                                                           : sum * (double)exp2f((m - wm) * c));
    const int wnf = wave_or(nf ? 1 : 0);
    __syncthreads();
    if ((threadIdx.x % kWave) == 0) {
        s_m[threadIdx.x / kWave] = wm;
        s_s[threadIdx.x / kWave] = ws;
        if (wnf) s_nf = 1;
    }
    __syncthreads();
    float M = s_m[0];
    for (int w = 1; w < kWalkThreads / kWave; ++w) M = fmaxf(M, s_m[w]);
    double tot = 0.0;
    if (M > -INFINITY && M < INFINITY)
        for (int w = 0; w < kWalkThreads / kWave; ++w)
            if (s_m[w] > -INFINITY) tot += s_s[w] * (double)exp2f((s_m[w] - M) * c);
    const bool part_bad = s_nf != 0 || M == INFINITY || !isfinite(tot);
    return X.lse(M > -INFINITY && !part_bad ? (double)(M * A.invT) : -INFINITY, part_bad ? 0.0 : tot, part_bad, bad);
}

// Relative half-width of the band in which an acceptance test taken with the
// streamed normaliser is recomputed with the exact one (the streamed
// normaliser is within ~1e-6 of it: binary32 terms, binary64 accumulation).
constexpr double kDecisionBand = 1e-4;

// The target and draft logits of a cached slice, loaded ahead of the pass
// that needs them.
constexpr int kFillGroups = (kWalkCache + 4 * kWalkThreads - 1) / (4 * kWalkThreads);
template <int DT>
struct FillRaw {
    Raw4<DT> t[kFillGroups], d[kFillGroups];
};

template <int DT>
__device__ __forceinline__ void fill_prefetch(const WalkArgs& A, bool vec, const WalkSlice& S, size_t trow,
                                              size_t drow, FillRaw<DT>& f) {
    const int n = S.v1 - S.v0;
#pragma unroll
    for (int k = 0; k < kFillGroups; ++k) {
        const int i = (k * kWalkThreads + (int)threadIdx.x) * 4;
        const int valid = max(0, min(4, n - i));
        raw_load4<DT>(A.target, trow + S.v0 + (valid ? i : 0), valid, vec, f.t[k]);
        raw_load4<DT>(A.draft, drow + S.v0 + (valid ? i : 0), valid, vec, f.d[k]);
    }
}

// First exact pass at a node: fills (p~, q) and returns the slice partials of
// sum p~, and, for the first residual (C = 1), sum p~ and sum q over tokens
// with p~ > q (beyond the band where the normaliser could flip the sign) and
// the number of tokens inside that band.
template <int DT>
__device__ void fill_pass(const WalkArgs& A, bool vec, const WalkSlice& S, bool cached, size_t trow, size_t drow,
                          double L0, double Ld, const double* et, double (&out)[4]) {
    double sp = 0.0, pa = 0.0, qa = 0.0, band = 0.0;
    if (cached) {
        // the whole slice fits the LDS cache: every load of the thread is
        // issued before any arithmetic (one memory latency per pass)
        const int n = S.v1 - S.v0;
        FillRaw<DT> pre;
        fill_prefetch<DT>(A, vec, S, trow, drow, pre);
#pragma unroll
        for (int k = 0; k < kFillGroups; ++k) {
            const int i = (k * kWalkThreads + (int)threadIdx.x) * 4;
            const int valid = max(0, min(4, n - i));
            float at[4], ad[4];
            raw_scaled4<DT>(pre.t[k], valid, A.invT, at);
            raw_scaled4<DT>(pre.d[k], valid, A.invT, ad);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const double pt = at[e] > -INFINITY ? exp64((double)at[e] - L0, et) : 0.0;
                const double qd = ad[e] > -INFINITY ? exp64((double)ad[e] - Ld, et) : 0.0;
                sp += pt;
                if (pt > qd * (1.0 + 1e-5)) {
                    pa += pt;
                    qa += qd;
                } else if (pt >= qd * (1.0 - 1e-5) && pt > 0.0) {
                    band += 1.0;
                }
                if (i + e < n) {
                    S.p[i + e] = pt;
                    S.q[i + e] = qd;
                }
            }
        }
    } else {
        for (int c = 0; c < S.nchunks; ++c) {
            const int c0 = S.v0 + c * kWalkCache;
            const int n = min(kWalkCache, S.v1 - c0);
            // one group of four tokens per iteration; the next group's loads are
            // issued before this group's arithmetic
            int i = (int)threadIdx.x * 4;
            float at[4], ad[4];
            {
                const int valid = max(0, min(4, n - i));
                load4_scaled<DT>(A.target, trow + c0 + (valid ? i : 0), valid, vec, A.invT, at);
                load4_scaled<DT>(A.draft, drow + c0 + (valid ? i : 0), valid, vec, A.invT, ad);
            }
            for (; i < n; i += 4 * kWalkThreads) {
                const int inext = i + 4 * kWalkThreads;
                float nt[4], nd[4];
                const int vn = max(0, min(4, n - inext));
                load4_scaled<DT>(A.target, trow + c0 + (vn ? inext : 0), vn, vec, A.invT, nt);
                load4_scaled<DT>(A.draft, drow + c0 + (vn ? inext : 0), vn, vec, A.invT, nd);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const double pt = at[e] > -INFINITY ? exp64((double)at[e] - L0, et) : 0.0;
                    const double qd = ad[e] > -INFINITY ? exp64((double)ad[e] - Ld, et) : 0.0;
                    sp += pt;
                    if (pt > qd * (1.0 + 1e-5)) {
                        pa += pt;
                        qa += qd;
                    } else if (pt >= qd * (1.0 - 1e-5) && pt > 0.0) {
                        band += 1.0;
                    }
                }
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    at[e] = nt[e];
                    ad[e] = nd[e];
                }
            }
        }
    }
    out[0] = sp;
    out[1] = pa;
    out[2] = qa;
    out[3] = band;
    walk_sum4(out);
}

// End of a walk, for every workgroup of the request: the request's outputs,
// and the optional normaliser output (from the target stream's partials,
// which the caller streamed when it asked for it). rows_bad < 0: every target
// row of the tree must be usable (each workgroup checks the partials, so all
// agree); otherwise rows_bad is the walk's own verdict on the rows it entered.
__device__ __forceinline__ void walk_tail(const WalkArgs& A, int r, int g, int G, int n, bool draft_bad, bool invalid, int nacc,
                          int bonus_out, int add_status, int tcount, int rows_bad = -1) {
    __shared__ int s_bad;
    const int tid = threadIdx.x;
    const int B1 = A.B + 1;
    const size_t tb = (size_t)r * B1;
    const bool lead = (g == 0 && tid == 0);
    int* status_p = A.out.req_status + r;
    if (tid == 0) s_bad = 0;
    __syncthreads();
    if (!draft_bad && rows_bad < 0)
        for (int i = tid; i < n; i += kWalkThreads) {
            int b;
            target_lse(A, r, i, &b);
            if (b) atomicOr(&s_bad, 1);
        }
    __syncthreads();
    const bool bad = draft_bad || (rows_bad < 0 ? s_bad != 0 : rows_bad != 0);
    if (A.out.target_lse) {
        // a request rejected by a verifier that reads every row reports no normaliser
        const bool none = draft_bad || (bad && rows_bad < 0);
        for (int i = g * kWalkThreads + tid; i < B1; i += G * kWalkThreads) {
            double l = (double)NAN;
            if (!none && i < n) {
                int b;
                l = target_lse(A, r, i, &b);
                if (b) l = (double)NAN;
            }
            A.out.target_lse[tb + i] = l;
        }
    }
    if (lead) {
        if (bad) {
            nacc = 0;
            bonus_out = -1;
            add_status = (add_status & ~(TSB_REQ_DEGENERATE_RESIDUAL | TSB_REQ_WALK_TIMEOUT)) | TSB_REQ_NONFINITE;
        } else if (invalid) {  // a malformed tree or token: outputs defined, without meaning
            nacc = 0;
            bonus_out = -1;
        }
        for (int i = nacc; i < A.D; ++i) {
            A.out.acc_node[(size_t)r * A.D + i] = -1;
            A.out.acc_tok[(size_t)r * A.D + i] = -1;
        }
        A.out.n_acc[r] = (bad || invalid) ? -1 : nacc;
        A.out.bonus[r] = bonus_out;
        *status_p |= add_status;
        if (A.out.trace)
            for (int i = tcount; i < TSB_TRACE_MAX; ++i)
                for (int f = 0; f < 4; ++f) A.out.trace[((size_t)r * TSB_TRACE_MAX + i) * 4 + f] = -1.0;
    }
}

template <int DT, bool VEC>
__global__ __launch_bounds__(kWalkThreads) void verify_walk(WalkArgs A) {
    extern __shared__ double s_pq[];  // [2 * kWalkCache]: p~ then q
    __shared__ double s_exp[kExpTable];
    __shared__ int s_tok[TSB_MAX_K];
    __shared__ float s_xd[TSB_MAX_K], s_xt[TSB_MAX_K];
    __shared__ double s_u[TSB_MAX_K];
    __shared__ int s_badtok;
    const int G = A.G;
    const int ticket = xticket(A.X, A.R);
    const int g = ticket % G;
    const int r = ticket / G;
    const int tid = threadIdx.x;
    const int B1 = A.B + 1;
    const size_t tb = (size_t)r * B1;
    const bool vec = VEC;
    int* status_p = A.out.req_status + r;
    const int n_raw = A.tree.n_nodes[r];
    const bool count_ok = tree_count_ok(n_raw, A.B);
    const int n = count_ok ? n_raw : 0;
    const bool lead = (g == 0 && tid == 0);
    if (tid == 0) s_badtok = 0;
    exp64_table_init(s_exp);

    // vocabulary slice (start a multiple of 4; an empty slice is [0, 0))
    WalkSlice S;
    {
        const int span = ((A.V + G - 1) / G + 3) & ~3;
        const bool has = (long long)g * span < A.V;
        S.v0 = has ? g * span : 0;
        S.v1 = has ? min(A.V, S.v0 + span) : 0;
        S.nchunks = (S.v1 - S.v0 + kWalkCache - 1) / kWalkCache;
        S.p = s_pq;
        S.q = s_pq + kWalkCache;
    }
    const bool cached = S.nchunks <= 1;
    const bool draft_bad = (*status_p & TSB_REQ_NONFINITE) != 0;

    int tcount = 0;
    int n_entered = 0;  // nodes entered (work counter)
    double* const trace = (lead && A.out.trace) ? A.out.trace + (size_t)r * TSB_TRACE_MAX * 4 : nullptr;

    int bonus_out = -1, add_status = count_ok ? 0 : TSB_REQ_BAD_TREE, nacc = 0;
    bool invalid = !count_ok;
    int rows_bad = 0;  // an entered node's target row is unusable
    if (!draft_bad && count_ok) {
        RngKey key;
        key.k0 = A.k0;
        key.k1 = A.k1;
        key.request = (uint32_t)r;
        key.step = A.step;
        Exchange X{&A, r, g, G, 0u, 0};
        int u = 0;
        while (true) {
            ++n_entered;
            const size_t trow = ((size_t)r * B1 + u) * (size_t)A.V;
            // every workgroup reads the same entries, so all take the same exit
            TreeNode nd;
            double L0 = 0.0, Ld = 0.0;
            bool row_bad = false;  // u's target row is unusable
            uint4 crec = make_uint4(0u, 0u, 0u, 0u);  // child tid's (token, x_d, x_t) from the record
            if (A.nrec) {
                // the node's record: its topology, draft normaliser and
                // children in one round trip
                const uint32_t* rp = A.nrec + (tb + u) * kRecWords;
                const uint4 h0 = *(const uint4*)rp;
                const uint4 h1 = *(const uint4*)(rp + 4);
                if (tid < TSB_MAX_K) crec = *(const uint4*)(rp + 8 + 4 * tid);
                nd.m = (int)h0.x;
                nd.fc = (int)h0.y;
                nd.d = (int)h0.z;
                nd.ok = (h0.w & kRecOk) != 0;
                L0 = rec_f64(h1.x, h1.y);
                row_bad = (h0.w & kRecTargetBad) != 0;
                Ld = rec_f64(h1.z, h1.w);
            } else {
                nd = tree_node(A.tree, tb, u, n, A.D);
                if (!A.reads_rows) {
                    int tbad;
                    L0 = target_lse(A, r, u, &tbad);
                    row_bad = tbad != 0;
                }
            }
            if (!nd.ok || (nd.m > 0 && nacc >= A.D)) {
                add_status |= TSB_REQ_BAD_TREE;
                invalid = true;
                break;
            }
            const int m = nd.m, d = nd.d;
            // or the target row of u, read now that the walk has entered u: its
            // streamed normaliser, and whether it is usable
            if (A.reads_rows) {
                if (u < kChainRows) {  // the root or node 1: streamed before the walk
                    int tbad;
                    L0 = target_row_lse(A.cm, A.cs, A.cf, kChainPieces, (size_t)r * kChainRows + u, &tbad);
                    row_bad = tbad != 0;
                } else {
                    L0 = entered_row_lse<DT>(A, vec, S, trow, X, &row_bad);
                }
            }
            if (row_bad) {
                rows_bad = 1;
                break;
            }
            const size_t drow = ((size_t)r * A.D + (m > 0 ? d : 0)) * (size_t)A.V;
            if (m == 0) {  // accepted leaf: bonus from p_u
                float bk;
                int bi;
                double unused;
                bonus_from_p<DT>(A, vec, S, trow, L0, key, (uint32_t)u, &bk, &bi);
                bonus_out = X.best(bk, bi, 0.0, &unused);
                break;
            }
            if (!A.nrec) Ld = A.draft_lse[(size_t)r * A.D + d];
            // children of u: tokens, their logits and the uniforms, fetched
            // together; a token outside [0, V) is never used as an address
            const int fc = nd.fc;
            if (tid < m) {
                if (A.nrec) {
                    const int y = (int)crec.x;
                    s_tok[tid] = y;
                    s_xd[tid] = __uint_as_float(crec.y);
                    s_xt[tid] = __uint_as_float(crec.z);
                    if (!(y >= 0 && y < A.V)) s_badtok = 1;
                } else {
                    const int y = A.node_tok[tb + fc + tid];
                    const bool yok = y >= 0 && y < A.V;
                    s_tok[tid] = y;
                    s_xd[tid] = yok ? load_logit<DT>(A.draft, drow + y) * A.invT : 0.f;
                    s_xt[tid] = yok ? load_logit<DT>(A.target, trow + y) * A.invT : 0.f;
                    if (!yok) s_badtok = 1;
                }
                s_u[tid] = u24d(rng_word(key, (uint32_t)(fc + tid), kStreamAccept, 0u));
            }
            __syncthreads();
            if (s_badtok) {
                add_status |= TSB_REQ_BAD_TOKEN;
                invalid = true;
                break;
            }

            bool exact = false;
            double Lt = L0, inv = 1.0;
            double C = 0.0, Sq = 1.0, Z = 1.0, Z1 = -1.0;
            bool accepted = false, degenerate = false;
            for (int j = 0; j < m; ++j) {
                const int c = fc + j;
                const int y = s_tok[j];
                const double qy = exp((double)s_xd[j] - Ld);
                const double U = s_u[j];
                const double W = Z / Sq;
                double py = exp((double)s_xt[j] - Lt);
                double num = py - C * qy;
                double ratio = (num > 0.0 ? num : 0.0) / (W * qy);
                if (trace && tcount < TSB_TRACE_MAX) {
                    trace[tcount * 4 + 0] = c;
                    trace[tcount * 4 + 1] = U;
                    trace[tcount * 4 + 3] = -1.0;
                }
                ++tcount;
                // Before the exact pass only the first test of a node is taken, with
                // the streamed normaliser; it stands if U is clear of the ratio by
                // the band. A rejection needs the exact residual anyway.
                if (!exact && (fabs(U - ratio) <= kDecisionBand * ratio || !(U < ratio))) {
                    double part[4], tot[4];
                    fill_pass<DT>(A, vec, S, cached, trow, drow, L0, Ld, s_exp, part);
                    X.run<4>(part, tot);
                    Lt = L0 + log(tot[0]);
                    inv = 1.0 / tot[0];
                    // first residual (C = 1): sum over {p > q} of p - q, exact when no
                    // token lies in the band where the normaliser decides the sign
                    Z1 = tot[3] == 0.0 ? tot[1] * inv - tot[2] : -1.0;
                    exact = true;
                    py = exp((double)s_xt[j] - Lt);
                    num = py - C * qy;
                    ratio = (num > 0.0 ? num : 0.0) / (W * qy);
                }
                if (trace && tcount <= TSB_TRACE_MAX) trace[(tcount - 1) * 4 + 2] = ratio;
                if (U < ratio) {
                    if (lead) {
                        A.out.acc_node[(size_t)r * A.D + nacc] = c;
                        A.out.acc_tok[(size_t)r * A.D + nacc] = y;
                    }
                    ++nacc;
                    u = c;
                    accepted = true;
                    break;
                }
                C = C + W;
                Sq = Sq - qy;
                if (j + 1 == m) break;
                // residual mass at the new C
                if (j == 0 && Z1 >= 0.0) {
                    Z = Z1;
                } else {
                    double zp = 0.0;
                    visit_pq<DT>(A, vec, S, cached, trow, drow, L0, inv, Ld, s_exp, [&](int, double p, double q) {
                        const double rr = p - C * q;
                        zp += rr > 0.0 ? rr : 0.0;
                    });
                    Z = X.sum(walk_sum(zp));
                }
                if (trace && tcount <= TSB_TRACE_MAX) trace[(tcount - 1) * 4 + 3] = Z;
                if (Z <= 0.0 || Sq <= 0.0) {
                    degenerate = true;
                    break;
                }
            }
            __syncthreads();  // s_tok & co. are rewritten at the next node
            if (accepted) continue;
            // every child rejected: bonus from the residual max(p - C q, 0)
            if (!degenerate) {
                float best = -INFINITY;
                int bidx = 0x7FFFFFFF;
                double zp = 0.0;
                const double Cc = C;
                const uint32_t node = (uint32_t)u;
                if (cached) {
                    const int nn = S.v1 - S.v0;
                    for (int i4 = tid; i4 * 4 < nn; i4 += kWalkThreads) {
                        const uint4 w = rng_block(key, node, kStreamBonus, (uint32_t)((S.v0 >> 2) + i4));
                        const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int i = i4 * 4 + e;
                            if (i >= nn) break;
                            const double rr = S.p[i] * inv - Cc * S.q[i];
                            if (rr > 0.0) {
                                zp += rr;
                                const float kv = logf((float)rr) + gumbel_f32(ws[e]);
                                const int v = S.v0 + i;
                                if (kv > best || (kv == best && v < bidx)) {
                                    best = kv;
                                    bidx = v;
                                }
                            }
                        }
                    }
                } else {
                    visit_pq<DT>(A, vec, S, false, trow, drow, L0, inv, Ld, s_exp, [&](int v, double p, double q) {
                        const double rr = p - Cc * q;
                        if (rr > 0.0) {
                            zp += rr;
                            const float kv = logf((float)rr) + gumbel_f32(rng_word(key, node, kStreamBonus, (uint32_t)v));
                            if (kv > best || (kv == best && v < bidx)) {
                                best = kv;
                                bidx = v;
                            }
                        }
                    });
                }
                walk_argmax(&best, &bidx);
                const double zs = walk_sum(zp);
                double mass;
                const int fi = X.best(best, bidx, zs, &mass);
                if (trace && tcount >= 1 && tcount <= TSB_TRACE_MAX) trace[(tcount - 1) * 4 + 3] = mass;
                if (mass > 0.0 && fi >= 0) {
                    bonus_out = fi;
                } else {
                    degenerate = true;
                }
            }
            if (degenerate) {  // empty residual: bonus from p_u
                float bk;
                int bi;
                double unused;
                bonus_from_p<DT>(A, vec, S, trow, Lt, key, (uint32_t)u, &bk, &bi);
                bonus_out = X.best(bk, bi, 0.0, &unused);
                add_status |= TSB_REQ_DEGENERATE_RESIDUAL;
            }
            break;
        }
        if (X.timeout) add_status |= TSB_REQ_WALK_TIMEOUT;
        if (A.stats && lead) {
            atomicAdd(&A.stats[kStWalkRequests], 1ull);
            atomicAdd(&A.stats[kStWalkNodes], (unsigned long long)n_entered);
            atomicAdd(&A.stats[kStWalkTests], (unsigned long long)tcount);
            atomicAdd(&A.stats[kStWalkExchanges], (unsigned long long)X.nb);
        }
    }

    walk_tail(A, r, g, G, n, draft_bad, invalid, nacc, bonus_out, add_status, tcount, rows_bad);
}


// ---------------------------------------------------------------- pool walk
// Verification with pool-restricted, context-dependent q_u (Section 3.1;
// Section 3.3: the probabilities of the replayed candidates, normalised in
// the pool). At node u (depth d, token in slot s_u of pool d - 1) wave 0
// rebuilds q_u over pool d from the draft logits and the transition scores,
// z_j = fl32(a_j + fl32(c[d-1][s_u][j] invT)), q_j = exp(z_j - L_u), and
// reads the target logits at the pool tokens. q vanishes off the pool, so
// after a rejection the residual mass needs no vocabulary pass:
//   Z = sum_{v off pool} p_v + sum_{v in pool} max(p_v - C q_v, 0)
//     = (S~ - sum_{pool} p~_v) / S~ + sum_{pool} max(p~_v / S~ - C q_v, 0)
// with p~_v = exp(a^t_v - L0) and S~ = sum_v p~_v from the one exact pass
// over the target row (L0 the streamed normaliser). The residual bonus is a
// Gumbel-max over the slice with the pool tokens left out (a bitmap of the
// slice in LDS), merged with the pool tokens' residual keys.

// Exact pass over the target row of the slice: sum of exp(a^t_v - L0).
template <int DT>
__device__ double target_pass(const WalkArgs& A, bool vec, const WalkSlice& S, size_t trow, double L0,
                              const double* et) {
    double sp = 0.0;
    const int n = S.v1 - S.v0;
    int i = (int)threadIdx.x * 4;
    float at[4];
    {
        const int valid = max(0, min(4, n - i));
        load4_scaled<DT>(A.target, trow + S.v0 + (valid ? i : 0), valid, vec, A.invT, at);
    }
    for (; i < n; i += 4 * kWalkThreads) {
        const int inext = i + 4 * kWalkThreads;
        float nt[4];
        const int vn = max(0, min(4, n - inext));
        load4_scaled<DT>(A.target, trow + S.v0 + (vn ? inext : 0), vn, vec, A.invT, nt);
#pragma unroll
        for (int e = 0; e < 4; ++e) sp += at[e] > -INFINITY ? exp64((double)at[e] - L0, et) : 0.0;
#pragma unroll
        for (int e = 0; e < 4; ++e) at[e] = nt[e];
    }
    return walk_sum(sp);
}

// Gumbel-max of ln p_v over the slice's tokens outside the pool.
template <int DT>
__device__ void bonus_off_pool(const WalkArgs& A, bool vec, const WalkSlice& S, size_t trow, double Lt,
                               const RngKey& key, uint32_t node, const uint32_t* bits, float* bk, int* bi) {
    float best = -INFINITY;
    int bidx = 0x7FFFFFFF;
    const SplitF Ls = split(Lt);
    const int n = S.v1 - S.v0;
    for (int i4 = threadIdx.x; i4 * 4 < n; i4 += kWalkThreads) {
        const int i = i4 * 4;
        const int valid = min(4, n - i);
        float at[4];
        load4_scaled<DT>(A.target, trow + S.v0 + i, valid, vec, A.invT, at);
        const uint4 w = rng_block(key, node, kStreamBonus, (uint32_t)((S.v0 + i) >> 2));
        const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (e >= valid || at[e] == -INFINITY) continue;
            if ((bits[(i + e) >> 5] >> ((i + e) & 31)) & 1u) continue;  // a pool token
            const float kv = ((at[e] - Ls.hi) - Ls.lo) + gumbel_f32(ws[e]);
            const int v = S.v0 + i + e;
            if (kv > best || (kv == best && v < bidx)) {
                best = kv;
                bidx = v;
            }
        }
    }
    *bk = best;
    *bi = bidx;
}

template <int DT, bool VEC>
__global__ __launch_bounds__(kWalkThreads) void verify_pool_walk(WalkArgs A) {
    extern __shared__ uint32_t s_bits[];  // pool membership over the slice
    __shared__ double s_exp[kExpTable];
    __shared__ int s_ptok[kPoolMax];
    __shared__ double s_q[kPoolMax], s_pp[kPoolMax];
    __shared__ float s_pat[kPoolMax];
    __shared__ int s_tok[TSB_MAX_K], s_cslot[TSB_MAX_K];
    __shared__ float s_xt[TSB_MAX_K];
    __shared__ double s_u[TSB_MAX_K];
    __shared__ double s_z;
    __shared__ int s_badtok;
    const int G = A.G;
    const int ticket = xticket(A.X, A.R);
    const int g = ticket % G;
    const int r = ticket / G;
    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int B1 = A.B + 1;
    const int P = A.P;
    const size_t tb = (size_t)r * B1;
    const bool vec = VEC;
    const int n_raw = A.tree.n_nodes[r];
    const bool count_ok = tree_count_ok(n_raw, A.B);
    const int n = count_ok ? n_raw : 0;
    const bool lead = (g == 0 && tid == 0);
    exp64_table_init(s_exp);
    if (tid == 0) s_badtok = 0;

    WalkSlice S;
    {
        const int span = ((A.V + G - 1) / G + 3) & ~3;
        const bool has = (long long)g * span < A.V;
        S.v0 = has ? g * span : 0;
        S.v1 = has ? min(A.V, S.v0 + span) : 0;
        S.nchunks = 1;
        S.p = nullptr;
        S.q = nullptr;
    }
    const int nwords = (S.v1 - S.v0 + 31) / 32;
    const bool draft_bad = (A.out.req_status[r] & TSB_REQ_NONFINITE) != 0;

    int tcount = 0;
    double* const trace = (lead && A.out.trace) ? A.out.trace + (size_t)r * TSB_TRACE_MAX * 4 : nullptr;

    int bonus_out = -1, add_status = count_ok ? 0 : TSB_REQ_BAD_TREE, nacc = 0;
    bool invalid = !count_ok;
    int rows_bad = 0;  // an entered node's target row is unusable
    if (!draft_bad && count_ok) {
        RngKey key;
        key.k0 = A.k0;
        key.k1 = A.k1;
        key.request = (uint32_t)r;
        key.step = A.step;
        Exchange X{&A, r, g, G, 0u, 0};
        int u = 0, su = 0;
        while (true) {
            // every workgroup reads the same entries, so all take the same exit
            const TreeNode nd = tree_node(A.tree, tb, u, n, A.D);
            if (!nd.ok || (nd.m > 0 && nacc >= A.D)) {
                add_status |= TSB_REQ_BAD_TREE;
                invalid = true;
                break;
            }
            const int m = nd.m, d = nd.d;
            const size_t trow = ((size_t)r * B1 + u) * (size_t)A.V;
            int tbad;
            const double L0 = target_lse(A, r, u, &tbad);
            if (m == 0) {  // accepted leaf: bonus from p_u
                float bk;
                int bi;
                double unused;
                bonus_from_p<DT>(A, vec, S, trow, L0, key, (uint32_t)u, &bk, &bi);
                bonus_out = X.best(bk, bi, 0.0, &unused);
                break;
            }
            // q_u over pool d, target logits at the pool tokens
            if (tid < kWave) {
                float z = -INFINITY, at = -INFINITY;
                int tok = -1;
                if (lane < P) {
                    tok = A.pool_tok[((size_t)r * A.D + d) * P + lane];
                    if (tok >= 0 && tok < A.V) {
                        z = load_logit<DT>(A.draft, ((size_t)r * A.D + d) * A.V + tok) * A.invT;
                        if (d > 0) {
                            const float c = A.trans[(((size_t)r * (A.D - 1) + (d - 1)) * P + su) * (size_t)P + lane];
                            const float cs = c * A.invT;
                            z = z + cs;
                        }
                        at = load_logit<DT>(A.target, trow + tok) * A.invT;
                    }
                }
                const float zm = wave_max(z);
                double q = 0.0;
                if (zm > -INFINITY) {
                    const double e = z > -INFINITY ? exp64((double)z - (double)zm, s_exp) : 0.0;
                    const double Lz = (double)zm + log(wave_sum(e));
                    q = z > -INFINITY ? exp64((double)z - Lz, s_exp) : 0.0;
                }
                if (lane < P) {
                    s_ptok[lane] = tok;
                    s_q[lane] = q;
                    s_pat[lane] = at;
                }
            }
            const int fc = nd.fc;
            if (tid < m) {
                const int y = A.node_tok[tb + fc + tid];
                s_tok[tid] = y;
                s_xt[tid] = (y >= 0 && y < A.V) ? load_logit<DT>(A.target, trow + y) * A.invT : -INFINITY;
                s_u[tid] = u24d(rng_word(key, (uint32_t)(fc + tid), kStreamAccept, 0u));
            }
            __syncthreads();
            if (tid < m) {  // pool slot of each child's token
                const int y = s_tok[tid];
                int sl = -1;
                for (int j = 0; j < P; ++j)
                    if (s_ptok[j] == y) {
                        sl = j;
                        break;
                    }
                s_cslot[tid] = sl;
                if (sl < 0) s_badtok = 1;
            }
            __syncthreads();

            bool exact = false;
            double Lt = L0, inv = 1.0, Stot = 1.0;
            double C = 0.0, Sq = 1.0, Z = 1.0;
            bool accepted = false, degenerate = false;
            for (int j = 0; j < m; ++j) {
                const int c = fc + j;
                const int y = s_tok[j];
                const int sl = s_cslot[j];
                const double qy = sl >= 0 ? s_q[sl] : 0.0;
                const double U = s_u[j];
                const double W = Z / Sq;
                double py = s_xt[j] > -INFINITY ? exp((double)s_xt[j] - Lt) : 0.0;
                double num = py - C * qy;
                double ratio = qy > 0.0 ? (num > 0.0 ? num : 0.0) / (W * qy) : (py > 0.0 ? INFINITY : 0.0);
                if (trace && tcount < TSB_TRACE_MAX) {
                    trace[tcount * 4 + 0] = c;
                    trace[tcount * 4 + 1] = U;
                    trace[tcount * 4 + 3] = -1.0;
                }
                ++tcount;
                if (!exact && (fabs(U - ratio) <= kDecisionBand * ratio || !(U < ratio))) {
                    Stot = X.sum(target_pass<DT>(A, vec, S, trow, L0, s_exp));
                    Lt = L0 + log(Stot);
                    inv = 1.0 / Stot;
                    exact = true;
                    // pool probabilities p~_v with the same exponential as the pass
                    if (tid < kWave) {
                        const double pp = lane < P && s_pat[lane] > -INFINITY ? exp64((double)s_pat[lane] - L0, s_exp)
                                                                              : 0.0;
                        if (lane < P) s_pp[lane] = pp;
                    }
                    __syncthreads();
                    py = s_xt[j] > -INFINITY ? exp((double)s_xt[j] - Lt) : 0.0;
                    num = py - C * qy;
                    ratio = qy > 0.0 ? (num > 0.0 ? num : 0.0) / (W * qy) : (py > 0.0 ? INFINITY : 0.0);
                }
                if (trace && tcount <= TSB_TRACE_MAX) trace[(tcount - 1) * 4 + 2] = ratio;
                if (U < ratio) {
                    if (lead) {
                        A.out.acc_node[(size_t)r * A.D + nacc] = c;
                        A.out.acc_tok[(size_t)r * A.D + nacc] = y;
                    }
                    ++nacc;
                    u = c;
                    su = sl >= 0 ? sl : 0;
                    accepted = true;
                    break;
                }
                C = C + W;
                Sq = Sq - qy;
                // residual mass at the new C, from the pool alone
                if (tid < kWave) {
                    double pin = 0.0, res = 0.0;
                    if (lane < P) {
                        pin = s_pp[lane];
                        const double rr = s_pp[lane] * inv - C * s_q[lane];
                        res = rr > 0.0 ? rr : 0.0;
                    }
                    pin = wave_sum(pin);
                    res = wave_sum(res);
                    if (lane == 0) s_z = (Stot - pin) * inv + res;
                }
                __syncthreads();
                Z = s_z;
                __syncthreads();
                if (trace && tcount <= TSB_TRACE_MAX) trace[(tcount - 1) * 4 + 3] = Z;
                if (Z <= 0.0 || (j + 1 < m && Sq <= 0.0)) {
                    degenerate = true;
                    break;
                }
            }
            __syncthreads();  // s_tok & co. are rewritten at the next node
            if (accepted) continue;
            // every child rejected: bonus from the residual max(p - C q, 0)
            if (!degenerate) {
                for (int w = tid; w < nwords; w += kWalkThreads) s_bits[w] = 0u;
                __syncthreads();
                if (tid < P) {
                    const int t = s_ptok[tid];
                    if (t >= S.v0 && t < S.v1) atomicOr(&s_bits[(t - S.v0) >> 5], 1u << ((t - S.v0) & 31));
                }
                __syncthreads();
                float best;
                int bidx;
                bonus_off_pool<DT>(A, vec, S, trow, Lt, key, (uint32_t)u, s_bits, &best, &bidx);
                if (tid < P) {
                    const int t = s_ptok[tid];
                    if (t >= S.v0 && t < S.v1) {
                        const double rr = s_pp[tid] * inv - C * s_q[tid];
                        if (rr > 0.0) {
                            const float kv = logf((float)rr) +
                                             gumbel_f32(rng_word(key, (uint32_t)u, kStreamBonus, (uint32_t)t));
                            if (kv > best || (kv == best && t < bidx)) {
                                best = kv;
                                bidx = t;
                            }
                        }
                    }
                }
                walk_argmax(&best, &bidx);
                double unused;
                const int fi = X.best(best, bidx, 0.0, &unused);
                if (fi >= 0) {
                    bonus_out = fi;
                } else {
                    degenerate = true;
                }
            }
            if (degenerate) {  // empty residual: bonus from p_u
                float bk;
                int bi;
                double unused;
                bonus_from_p<DT>(A, vec, S, trow, Lt, key, (uint32_t)u, &bk, &bi);
                bonus_out = X.best(bk, bi, 0.0, &unused);
                add_status |= TSB_REQ_DEGENERATE_RESIDUAL;
            }
            break;
        }
        if (X.timeout) add_status |= TSB_REQ_WALK_TIMEOUT;
        __syncthreads();
        if (s_badtok) add_status |= TSB_REQ_BAD_TOKEN;
    }
    walk_tail(A, r, g, G, n, draft_bad, invalid, nacc, bonus_out, add_status, tcount);
}

// ---------------------------------------------------------- traversal walk
// Traversal verification (Appendix A; Table 2): sequence-level recursive
// rejection sampling over the replayed tree. All G workgroups of a request
// replay the same scalar traversal over a stack of the current path (in
// LDS); every vocabulary-wide quantity is split over their slices and
// exchanged:
//   * the binary64 target normaliser of an internal node when the traversal
//     first descends from it (its children's acceptance probabilities need
//     p_u);
//   * the residual mass T = sum_v max(A' p_v - C' q_v, 0) at a node after one
//     of its children was rejected;
//   * the bonus draw at the node that ends the round.
// Closed form of a node's state (equal to the literal updates): Mb_u =
// max(A p - C q, 0) / Z is the bonus distribution at u, Ms_u = q / S over
// the tokens not yet removed the draft distribution of its remaining
// children; a node enters with alpha from its parent and (A, C, Z, S) =
// (1, 0, 1, 1). The child of u with token y has
//   alpha_c = min(1, alpha_u max(A p(y) - C q(y), 0) / Z * S / q(y));
// rejecting it maps u's state to A' = alpha A / Z, C' = alpha C / Z + 1 / S,
// Z' = T, alpha' = T / (T + 1 - alpha), S' = S - q(y).
// The traversal is post-order (the first remaining child first, down to a
// node with none left, which is tested with U < alpha); the root has
// alpha = 1 and is accepted once its children are all rejected. One
// (p~, q) slice is kept in LDS: that of the node the last pass was over, so
// consecutive rejections among the children of one node reuse it.
struct TravEntry {
    int node, left;
    double alpha, A, C, Z, S, L;  // L: binary64 log normaliser of the node's target row, NaN until computed
};
constexpr int kTravStack = TSB_MAX_D + 1;  // root .. depth D

// (p~, q) of a node's slice into the LDS cache when the slice fits, and the
// block sum of p~ = exp(a^t - L0) over the slice.
template <int DT>
__device__ double trav_fill(const WalkArgs& A, bool vec, const WalkSlice& S, bool cached, size_t trow, size_t drow,
                            double L0, double Ld, const double* et) {
    double acc = 0.0;
    for (int c = 0; c < S.nchunks; ++c) acc += fill_chunk<DT>(A, vec, S, c, trow, drow, L0, Ld, et, cached);
    return walk_sum(acc);
}

template <int DT, bool VEC>
__global__ __launch_bounds__(kWalkThreads) void verify_traversal(WalkArgs A) {
    extern __shared__ double s_pq[];  // [2 * kWalkCache]: p~ then q of the cached node
    __shared__ double s_exp[kExpTable];
    __shared__ TravEntry s_stk[kTravStack];
    __shared__ int s_cache;  // node whose slice is in the cache, -1 for none
    const int G = A.G;
    const int ticket = xticket(A.X, A.R);
    const int g = ticket % G;
    const int r = ticket / G;
    const int tid = threadIdx.x;
    const int B1 = A.B + 1;
    const size_t tb = (size_t)r * B1;
    const bool vec = VEC;
    int* status_p = A.out.req_status + r;
    const int n_raw = A.tree.n_nodes[r];
    const bool count_ok = tree_count_ok(n_raw, A.B);
    const int n = count_ok ? n_raw : 0;
    const bool lead = (g == 0 && tid == 0);
    if (tid == 0) s_cache = -1;
    exp64_table_init(s_exp);

    WalkSlice S;
    {
        const int span = ((A.V + G - 1) / G + 3) & ~3;
        const bool has = (long long)g * span < A.V;
        S.v0 = has ? g * span : 0;
        S.v1 = has ? min(A.V, S.v0 + span) : 0;
        S.nchunks = (S.v1 - S.v0 + kWalkCache - 1) / kWalkCache;
        S.p = s_pq;
        S.q = s_pq + kWalkCache;
    }
    const bool cached = S.nchunks <= 1;
    const bool draft_bad = (*status_p & TSB_REQ_NONFINITE) != 0;

    int tcount = 0;
    double* const trace = (lead && A.out.trace) ? A.out.trace + (size_t)r * TSB_TRACE_MAX * 4 : nullptr;
    int bonus_out = -1, add_status = count_ok ? 0 : TSB_REQ_BAD_TREE, nacc = 0;
    bool invalid = !count_ok;
    int rows_bad = 0;  // an entered node's target row is unusable
    if (!draft_bad && count_ok) {
        RngKey key;
        key.k0 = A.k0;
        key.k1 = A.k1;
        key.request = (uint32_t)r;
        key.step = A.step;
        Exchange X{&A, r, g, G, 0u, 0};
        if (tid == 0) s_stk[0] = TravEntry{0, 0, 1.0, 1.0, 0.0, 1.0, 1.0, (double)NAN};
        __syncthreads();
        int top = 0;
        // end of the round at the node on top of the stack: bonus from Mb (or
        // from p on an empty residual) and the accepted path = stack[1 .. top]
        int end_kind = 0;  // 1: bonus from Mb of the top node, 2: degenerate (bonus from p)
        while (true) {
            const TravEntry E = s_stk[top];
            const int u = E.node;
            // every workgroup reads the same entries, so all take the same exits
            const TreeNode nd = tree_node(A.tree, tb, u, n, A.D);
            if (!nd.ok) {
                add_status |= TSB_REQ_BAD_TREE;
                invalid = true;
                break;
            }
            const size_t trow = ((size_t)r * B1 + u) * (size_t)A.V;
            if (E.left < nd.m) {  // descend to the next remaining child of u
                if (top + 1 > A.D) {
                    add_status |= TSB_REQ_BAD_TREE;
                    invalid = true;
                    break;
                }
                const size_t drow = ((size_t)r * A.D + nd.d) * (size_t)A.V;
                const double Ld = A.draft_lse[(size_t)r * A.D + nd.d];
                double L = E.L;
                if (isnan(L)) {  // first descent from u: binary64 normaliser of its target row
                    int tbad;
                    const double L0 = target_lse(A, r, u, &tbad);
                    const double tot = X.sum(trav_fill<DT>(A, vec, S, cached, trow, drow, L0, Ld, s_exp));
                    L = L0 + log(tot);
                    if (tid == 0) {
                        s_stk[top].L = L;
                        s_cache = cached ? u : -1;
                    }
                }
                const int c = nd.fc + E.left;
                const int y = A.node_tok[tb + c];
                if (y < 0 || y >= A.V) {
                    add_status |= TSB_REQ_BAD_TOKEN;
                    invalid = true;
                    break;
                }
                const double py = exp((double)(load_logit<DT>(A.target, trow + y) * A.invT) - L);
                const double qy = exp((double)(load_logit<DT>(A.draft, drow + y) * A.invT) - Ld);
                const double num = E.A * py - E.C * qy;  // Z Mb_u(y) before the max
                const double ms = qy / E.S;             // Ms_u(y)
                double ac;
                if (!(ms > 0.0))
                    ac = (num > 0.0 && E.alpha > 0.0) ? 1.0 : 0.0;
                else
                    ac = num > 0.0 ? fmin(1.0, E.alpha * (num / E.Z) / ms) : 0.0;
                __syncthreads();  // every thread has read s_stk[top] and s_cache
                if (tid == 0) s_stk[top + 1] = TravEntry{c, 0, ac, 1.0, 0.0, 1.0, 1.0, (double)NAN};
                __syncthreads();
                ++top;
                continue;
            }
            if (top == 0) {  // every child of the root rejected: the root is accepted
                end_kind = 1;
                break;
            }
            // test u: accept the path root .. u with probability alpha_u
            const double U = u24d(rng_word(key, (uint32_t)u, kStreamAccept, 0u));
            if (trace && tcount < TSB_TRACE_MAX) {
                trace[tcount * 4 + 0] = u;
                trace[tcount * 4 + 1] = U;
                trace[tcount * 4 + 2] = E.alpha;
                trace[tcount * 4 + 3] = -1.0;
            }
            ++tcount;
            if (U < E.alpha) {
                end_kind = 1;
                break;
            }
            // u rejected: update its parent w with the quantities u was drawn from
            const TravEntry W = s_stk[top - 1];
            const int w = W.node;
            const TreeNode nw = tree_node(A.tree, tb, w, n, A.D);  // checked when it was descended from
            const size_t trow_w = ((size_t)r * B1 + w) * (size_t)A.V;
            const size_t drow_w = ((size_t)r * A.D + nw.d) * (size_t)A.V;
            const double Ld = A.draft_lse[(size_t)r * A.D + nw.d];
            int tbad;
            const double L0 = target_lse(A, r, w, &tbad);
            const int yu = A.node_tok[tb + u];
            const double qy = exp((double)(load_logit<DT>(A.draft, drow_w + yu) * A.invT) - Ld);
            const double A2 = W.alpha * W.A / W.Z;
            const double C2 = W.alpha * W.C / W.Z + 1.0 / W.S;
            const bool hit = cached && s_cache == w;
            __syncthreads();  // every thread has read s_stk and s_cache
            if (cached && !hit) {
                trav_fill<DT>(A, vec, S, true, trow_w, drow_w, L0, Ld, s_exp);
                if (tid == 0) s_cache = w;
            }
            const double inv = exp(L0 - W.L);
            double zp = 0.0;
            visit_pq<DT>(A, vec, S, cached, trow_w, drow_w, L0, inv, Ld, s_exp, [&](int, double p, double q) {
                const double rr = A2 * p - C2 * q;
                zp += rr > 0.0 ? rr : 0.0;
            });
            const double T = X.sum(walk_sum(zp));
            if (trace && tcount <= TSB_TRACE_MAX) trace[(tcount - 1) * 4 + 3] = T;
            const int left = W.left + 1;
            const double S2 = W.S - qy;
            --top;
            if ((T <= 0.0 && W.alpha >= 1.0) || (S2 <= 0.0 && left < nw.m)) {
                end_kind = 2;
                break;
            }
            if (tid == 0) {
                TravEntry& e = s_stk[top];
                e.left = left;
                e.S = S2;
                if (T > 0.0) {
                    e.alpha = T / (T + (1.0 - W.alpha));
                    e.A = A2;
                    e.C = C2;
                    e.Z = T;
                } else {
                    e.alpha = 0.0;
                    e.A = 0.0;
                    e.C = 0.0;
                    e.Z = 1.0;
                }
            }
            __syncthreads();
        }
        if (end_kind != 0) {
            const TravEntry E = s_stk[top];
            const int u = E.node;
            const TreeNode nd = tree_node(A.tree, tb, u, n, A.D);
            const size_t trow = ((size_t)r * B1 + u) * (size_t)A.V;
            int tbad;
            const double L0 = target_lse(A, r, u, &tbad);
            bool from_p = end_kind == 2 || E.left == 0;  // a node whose residual was never formed: Mb = p
            if (!from_p) {
                // Gumbel-max of ln max(p - (C / A) q, 0) (the positive factor A and the normaliser Z shift
                // every key alike)
                const size_t drow = ((size_t)r * A.D + nd.d) * (size_t)A.V;
                const double Ld = A.draft_lse[(size_t)r * A.D + nd.d];
                const double lam = E.C / E.A;
                const bool hit = cached && s_cache == u;
                __syncthreads();
                if (cached && !hit) trav_fill<DT>(A, vec, S, true, trow, drow, L0, Ld, s_exp);
                const double inv = exp(L0 - E.L);
                float best = -INFINITY;
                int bidx = 0x7FFFFFFF;
                const uint32_t node = (uint32_t)u;
                if (cached) {
                    const int nn = S.v1 - S.v0;
                    for (int i4 = tid; i4 * 4 < nn; i4 += kWalkThreads) {
                        const uint4 wv = rng_block(key, node, kStreamBonus, (uint32_t)((S.v0 >> 2) + i4));
                        const uint32_t ws[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int i = i4 * 4 + e;
                            if (i >= nn) break;
                            const double rr = S.p[i] * inv - lam * S.q[i];
                            if (rr > 0.0) {
                                const float kv = logf((float)rr) + gumbel_f32(ws[e]);
                                const int v = S.v0 + i;
                                if (kv > best || (kv == best && v < bidx)) {
                                    best = kv;
                                    bidx = v;
                                }
                            }
                        }
                    }
                } else {
                    visit_pq<DT>(A, vec, S, false, trow, drow, L0, inv, Ld, s_exp, [&](int v, double p, double q) {
                        const double rr = p - lam * q;
                        if (rr > 0.0) {
                            const float kv = logf((float)rr) + gumbel_f32(rng_word(key, node, kStreamBonus, (uint32_t)v));
                            if (kv > best || (kv == best && v < bidx)) {
                                best = kv;
                                bidx = v;
                            }
                        }
                    });
                }
                walk_argmax(&best, &bidx);
                double unused;
                const int fi = X.best(best, bidx, 0.0, &unused);
                if (fi >= 0) {
                    bonus_out = fi;
                } else {
                    from_p = true;
                    end_kind = 2;
                }
            }
            if (from_p) {
                float bk;
                int bi;
                double unused;
                bonus_from_p<DT>(A, vec, S, trow, isnan(E.L) ? L0 : E.L, key, (uint32_t)u, &bk, &bi);
                bonus_out = X.best(bk, bi, 0.0, &unused);
            }
            if (end_kind == 2) add_status |= TSB_REQ_DEGENERATE_RESIDUAL;
            nacc = top;
            if (lead)
                for (int i = 1; i <= top; ++i) {
                    const int c = s_stk[i].node;
                    A.out.acc_node[(size_t)r * A.D + i - 1] = c;
                    A.out.acc_tok[(size_t)r * A.D + i - 1] = A.node_tok[tb + c];
                }
        }
        if (X.timeout) add_status |= TSB_REQ_WALK_TIMEOUT;
    }
    walk_tail(A, r, g, G, n, draft_bad, invalid, nacc, bonus_out, add_status, tcount);
}

// ------------------------------------------------------------------ launch
// Workgroups of the walk that are resident at once on the current device
// (one per CU: the LDS cache fills a CU). Every launch of the walk stays
// within this, in order of requests, so all workgroups of a launch run
// together and every exchange completes; the bounded polling of an exchange
// turns a device shared with other work (workgroups kept waiting) into
// TSB_REQ_WALK_TIMEOUT instead of a hang. Queried once per (device,
// kernel instance).
static hipError_t walk_capacity(const void* fn, int kind, int dt, int vec, size_t lds, int* cap) {
    constexpr int kDevs = 64;
    static std::atomic<int> cached[kDevs][3][2][2];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev >= 0 && dev < kDevs) {
        const int v = cached[dev][kind][dt][vec].load(std::memory_order_relaxed);
        if (v > 0) {
            *cap = v;
            return hipSuccess;
        }
    }
    int cus = 0, per_cu = 0;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    if ((e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds)) != hipSuccess) return e;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kWalkThreads, lds)) != hipSuccess) return e;
    *cap = per_cu * cus;
    if (dev >= 0 && dev < kDevs && *cap > 0) cached[dev][kind][dt][vec].store(*cap, std::memory_order_relaxed);
    return hipSuccess;
}

TargetJob target_job(const tsb_config& c, const void* target, const tsb_tree& tree, const double* draft_lse,
                     char* ws, bool rows) {
    const Geometry g = geometry(c);
    const VerifyWs w = verify_ws(c);
    TargetJob j;
    j.target = target;
    j.n_nodes = tree.n_nodes;
    j.tm = (float*)(ws + w.tm);
    j.ts = (double*)(ws + w.ts);
    j.tf = (int*)(ws + w.tf);
    j.slots = (uint64_t*)(ws + xchg_ws(c).slots);
    j.chunk = g.chunk4;
    j.nrows = c.R * (c.B + 1);
    j.P = g.S4;
    j.ngroups = g.G4;
    j.R = c.R;
    j.vec = (c.dtype == TSB_BF16) ? (c.V % 8 == 0 && ((uintptr_t)target & 15) == 0)
                                  : (c.V % 4 == 0 && ((uintptr_t)target & 15) == 0);
    j.nrec = draft_lse ? (uint32_t*)(ws + w.nrec) : nullptr;
    j.draft_lse = draft_lse;
    if (!rows) {
        // no row: the job's workgroups only clear the exchange slots
        j.nrows = 0;
        j.ngroups = kClearWorkgroups;
    }
    return j;
}

static hipError_t launch_target_partials(const tsb_config& c, float invT, const void* target, const tsb_tree& tree,
                                         const VerifyWs& w, char* ws, hipStream_t st) {
    TargetJob j = target_job(c, target, tree, nullptr, ws);
    j.tm = (float*)(ws + w.tm);
    j.ts = (double*)(ws + w.ts);
    j.tf = (int*)(ws + w.tf);
    XRegion X;
    X.slots = j.slots;
    hipError_t e = hook_before(TSB_KERNEL_TARGET_PARTIALS, st);
    if (e != hipSuccess) return e;
    auto fn = c.dtype == TSB_BF16 ? (j.vec ? target_partials<TSB_BF16, true> : target_partials<TSB_BF16, false>)
                                  : (j.vec ? target_partials<TSB_F32, true> : target_partials<TSB_F32, false>);
    fn<<<j.ngroups, kBlock, 0, st>>>(target, c.V, c.B, j.nrows, j.chunk, j.P, invT, j.n_nodes, j.tm, j.ts, j.tf, X,
                                     c.R);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return hook_after(TSB_KERNEL_TARGET_PARTIALS, st);
}

// Rows 0 and 1 of every request for a walk that reads the other rows itself
// (tsb_verify; a round streams them beside the planner), and the clearing of
// the walk's exchange slots. No profiling id: tsb_profile_kernel's target
// stream is target_partials alone.
template <int DT, bool VEC>
__global__ __launch_bounds__(kChainThreads) void chain_rows(ChainJob cj, XRegion X, int R, float invT) {
    xclear(X, R, (size_t)blockIdx.x * kChainThreads + threadIdx.x, (size_t)gridDim.x * kChainThreads);
    for (int g = blockIdx.x; g < cj.items; g += gridDim.x)
        chain_piece<DT, VEC>(g, cj.target, cj.V, cj.B, invT, cj.cm, cj.cs, cj.cf);
}

static hipError_t launch_chain_rows(const tsb_config& c, float invT, const void* target, char* ws, hipStream_t st) {
    const ChainJob j = chain_job(c, target, ws);
    XRegion X;
    X.slots = (uint64_t*)(ws + xchg_ws(c).slots);
    const int grid = std::max(kClearWorkgroups, std::min(j.items, 1024));
    auto fn = c.dtype == TSB_BF16 ? (j.vec ? chain_rows<TSB_BF16, true> : chain_rows<TSB_BF16, false>)
                                  : (j.vec ? chain_rows<TSB_F32, true> : chain_rows<TSB_F32, false>);
    fn<<<grid, kChainThreads, 0, st>>>(j, X, c.R, invT);
    return hipGetLastError();
}

// Walk arguments shared by both walks.
static WalkArgs walk_args(const tsb_config& c, float invT, const void* draft, const double* draft_lse,
                          const void* target, const tsb_tree& tree, const int32_t* node_tok, uint32_t step,
                          const tsb_verdict& out, const VerifyWs& w, char* ws) {
    const Geometry g = geometry(c);
    WalkArgs A;
    A.draft = draft;
    A.draft_lse = draft_lse;
    A.target = target;
    A.tree = tree;
    A.node_tok = node_tok;
    A.out = out;
    A.tm = (const float*)(ws + w.tm);
    A.ts = (const double*)(ws + w.ts);
    A.tf = (const int*)(ws + w.tf);
    A.X.slots = (uint64_t*)(ws + xchg_ws(c).slots);
    A.V = c.V;
    A.D = c.D;
    A.B = c.B;
    A.S4 = g.S4;
    A.R = c.R;
    A.G = 1;
    A.stats = stats_ptr();
    A.invT = invT;
    A.k0 = (uint32_t)c.seed;
    A.k1 = (uint32_t)(c.seed >> 32);
    A.step = step;
    A.pool_tok = nullptr;
    A.trans = nullptr;
    A.P = 0;
    A.nrec = nullptr;
    A.reads_rows = 0;
    const XchgWs x = xchg_ws(c);
    A.cm = (const float*)(ws + x.cm);
    A.cs = (const double*)(ws + x.cs);
    A.cf = (const int*)(ws + x.cf);
    return A;
}

// One launch of a walk grid: G workgroups per request, each taking its
// (request, slice) from a ticket (xticket), so only G workgroups need to fit
// on the device at once (cap: resident workgroups of this kernel).
static hipError_t launch_walk_grid(const void* fn, WalkArgs& A, int R, int G0, int cap, size_t lds, hipStream_t st) {
    A.R = R;
    A.G = G0 < cap ? G0 : cap;
    void* args[] = {&A};
    return hipLaunchKernel(fn, dim3((unsigned)(A.G * R)), dim3(kWalkThreads), args, lds, st);
}

hipError_t launch_verify(const tsb_config& c, float invT, const void* draft, const double* draft_lse,
                         const void* target, const tsb_tree& tree, const int32_t* node_tok, uint32_t step,
                         const tsb_verdict& out, char* ws, hipStream_t st, int stages) {
    const VerifyWs w = verify_ws(c);
    hipError_t e = hipSuccess;
    // a walk that reads the rows of the nodes it enters needs every row
    // streamed only for the optional normaliser output
    const bool reads = walk_reads_rows(c);
    if (stages & kStageTarget) {
        if ((out.target_lse || !reads) && (e = launch_target_partials(c, invT, target, tree, w, ws, st)) != hipSuccess)
            return e;
        if (reads && (e = launch_chain_rows(c, invT, target, ws, st)) != hipSuccess) return e;
    }
    if (!(stages & kStageWalk)) return hipSuccess;
    WalkArgs A = walk_args(c, invT, draft, draft_lse, target, tree, node_tok, step, out, w, ws);
    A.reads_rows = reads ? 1 : 0;
    if (stages & kWalkRecords) A.nrec = (const uint32_t*)(ws + w.nrec);
    const bool vec4 = c.V % 4 == 0 && ((uintptr_t)target & 15) == 0 && ((uintptr_t)draft & 15) == 0;
    const void* fn = nullptr;
    if (c.dtype == TSB_BF16)
        fn = vec4 ? (const void*)verify_walk<TSB_BF16, true> : (const void*)verify_walk<TSB_BF16, false>;
    else
        fn = vec4 ? (const void*)verify_walk<TSB_F32, true> : (const void*)verify_walk<TSB_F32, false>;
    const size_t lds = 2 * (size_t)kWalkCache * sizeof(double);
    int cap = 0;
    if ((e = walk_capacity(fn, 0, c.dtype == TSB_BF16 ? 1 : 0, vec4 ? 1 : 0, lds, &cap)) != hipSuccess) return e;
    if (cap < 1) return hipErrorLaunchOutOfResources;
    if ((e = hook_before(TSB_KERNEL_VERIFY_WALK, st)) != hipSuccess) return e;
    if ((e = launch_walk_grid(fn, A, c.R, geometry(c).G, cap, lds, st)) != hipSuccess) return e;
    return hook_after(TSB_KERNEL_VERIFY_WALK, st);
}

hipError_t launch_verify_traversal(const tsb_config& c, float invT, const void* draft, const double* draft_lse,
                                   const void* target, const tsb_tree& tree, const int32_t* node_tok, uint32_t step,
                                   const tsb_verdict& out, char* ws, hipStream_t st, int stages) {
    const VerifyWs w = verify_ws(c);
    hipError_t e = hipSuccess;
    if ((stages & kStageTarget) && (e = launch_target_partials(c, invT, target, tree, w, ws, st)) != hipSuccess)
        return e;
    if (!(stages & kStageWalk)) return hipSuccess;
    WalkArgs A = walk_args(c, invT, draft, draft_lse, target, tree, node_tok, step, out, w, ws);
    const bool vec4 = c.V % 4 == 0 && ((uintptr_t)target & 15) == 0 && ((uintptr_t)draft & 15) == 0;
    const void* fn = nullptr;
    if (c.dtype == TSB_BF16)
        fn = vec4 ? (const void*)verify_traversal<TSB_BF16, true> : (const void*)verify_traversal<TSB_BF16, false>;
    else
        fn = vec4 ? (const void*)verify_traversal<TSB_F32, true> : (const void*)verify_traversal<TSB_F32, false>;
    const size_t lds = 2 * (size_t)kWalkCache * sizeof(double);
    int cap = 0;
    if ((e = walk_capacity(fn, 2, c.dtype == TSB_BF16 ? 1 : 0, vec4 ? 1 : 0, lds, &cap)) != hipSuccess) return e;
    if (cap < 1) return hipErrorLaunchOutOfResources;
    if ((e = hook_before(TSB_KERNEL_TRAVERSAL_WALK, st)) != hipSuccess) return e;
    if ((e = launch_walk_grid(fn, A, c.R, geometry(c).G, cap, lds, st)) != hipSuccess) return e;
    return hook_after(TSB_KERNEL_TRAVERSAL_WALK, st);
}

hipError_t launch_pool_verify(const tsb_config& c, int P, float invT, const void* draft, const float* trans,
                              const int32_t* pool_tok, const void* target, const tsb_tree& tree,
                              const int32_t* node_tok, uint32_t step, const tsb_verdict& out, char* ws,
                              hipStream_t st, int stages) {
    const VerifyWs w = pool_verify_ws(c);
    hipError_t e = hipSuccess;
    if ((stages & kStageTarget) && (e = launch_target_partials(c, invT, target, tree, w, ws, st)) != hipSuccess)
        return e;
    if (!(stages & kStageWalk)) return hipSuccess;
    WalkArgs A = walk_args(c, invT, draft, nullptr, target, tree, node_tok, step, out, w, ws);
    A.pool_tok = pool_tok;
    A.trans = trans;
    A.P = P;
    const bool vec4 = c.V % 4 == 0 && ((uintptr_t)target & 15) == 0;
    const void* fn = nullptr;
    if (c.dtype == TSB_BF16)
        fn = vec4 ? (const void*)verify_pool_walk<TSB_BF16, true> : (const void*)verify_pool_walk<TSB_BF16, false>;
    else
        fn = vec4 ? (const void*)verify_pool_walk<TSB_F32, true> : (const void*)verify_pool_walk<TSB_F32, false>;
    // the slice bitmap: one bit per token of the widest slice at the fewest
    // workgroups per request the capacity allows
    const size_t lds_max = kPoolBitmapBytes;
    int cap = 0;
    if ((e = walk_capacity(fn, 1, c.dtype == TSB_BF16 ? 1 : 0, vec4 ? 1 : 0, lds_max, &cap)) != hipSuccess) return e;
    if (cap < 1) return hipErrorLaunchOutOfResources;
    int G = geometry(c).G;
    if (G > cap) G = cap;
    const long long span = (((long long)c.V + G - 1) / G + 3) & ~3ll;
    const size_t lds = (size_t)((span + 31) / 32) * sizeof(uint32_t);
    if (lds > lds_max) return hipErrorInvalidConfiguration;  // vocabulary too wide for the slice bitmap
    if ((e = hook_before(TSB_KERNEL_POOL_WALK, st)) != hipSuccess) return e;
    if ((e = launch_walk_grid(fn, A, c.R, G, cap, lds, st)) != hipSuccess) return e;
    return hook_after(TSB_KERNEL_POOL_WALK, st);
}

}  // namespace tsb
