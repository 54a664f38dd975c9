// Target stream of verification (Section 2.3, eq. (1): the target row
// normalisers the walk starts from), shared by the target kernel and by the
// replay scan, whose grid can carry it beside the scan.
#pragma once

#include "tsb_device.hpp"
#include "tsb_exchange.hpp"

namespace tsb {

// The target kernel's own grid loads a chunk's next step during this one
// (82 VGPRs: 5 waves per SIMD, 3% faster than 8 waves without it); the
// replay scan's grid does not (it would drop the scan to 5 waves per SIMD).
constexpr bool kTargetPrefetch = true;

// Streamed estimate of every target row's normaliser: per thread, four
// 16-byte loads in flight, a running maximum of the raw logits and
// sum 2^(x c - m c) with c = invT log2(e) (one FMA and one v_exp_f32 per
// logit; partial sums of 8 terms in binary32, accumulated in binary64).
// The estimate only has to be within ~1e-6 of ln sum exp(a): the walk uses it
// to take acceptance tests that are clear of U by a wide band, and computes
// the exact normaliser (binary64 terms) for every other node it tests.
// A NaN or +inf logit surfaces as a non-finite maximum or sum.
//
// Loads are non-temporal: the rows stream through once, and keeping them out
// of the caches' normal allocation was measured ~11% faster on this part.
//
// Layout: the target is one flat array of R (B+1) V logits cut into equal
// chunks (at least kTargetMinChunk logits, at most kTargetWorkgroups of
// them). The target kernel's own grid has one workgroup per chunk, all
// resident at once, so none trails the others; the replay scan's grid deals
// the chunks over fewer workgroups. A chunk covers pieces of one or more
// rows; the k-th chunk that meets row t gives partial slot k of the row, and
// the chunk holding the row's first logit marks the slots no piece uses as
// empty, so the partials depend on the chunking only, never on the grid.
// The chunks also zero the exchange slots of the walk launched after them.
template <int DT, bool VEC, bool PREF, int NT = kBlock>
__device__ __forceinline__ void stream_piece(const void* __restrict__ target, size_t rowbase, int lo, int hi,
                                             float c, float& m_out, double& sum_out) {
    constexpr int kEl = 8;      // logits per 16-byte load (bf16); fp32 loads are 2 x 16 bytes
    constexpr int kLoads = 4;   // loads in flight per thread
    constexpr int kW = DT == TSB_BF16 ? 1 : 2;  // 16-byte loads per eight logits
    const int tid = threadIdx.x;
    float m = -INFINITY;   // running max of the raw logits
    double sum = 0.0;      // sum of 2^(x c - m c)
    constexpr int kStep = NT * kEl * kLoads;
    // a whole step in range (uniform over the workgroup) has every load
    // issued before the first is used; with PREF the next whole step's loads
    // are issued before this step's arithmetic
    uint4 nxt[kLoads][kW];
    auto issue = [&](int b) {
#pragma unroll
        for (int l = 0; l < kLoads; ++l) {
            const int i0 = b + (l * NT + tid) * kEl;
            if (DT == TSB_BF16) {
                nxt[l][0] = load_stream16((const uint16_t*)target + rowbase + i0);
            } else {
                nxt[l][0] = load_stream16((const float*)target + rowbase + i0);
                nxt[l][kW - 1] = load_stream16((const float*)target + rowbase + i0 + 4);
            }
        }
    };
    if (PREF && VEC && lo + kStep <= hi) issue(lo);
    for (int base = lo; base < hi; base += kStep) {
        float x[kLoads][kEl];
        if (VEC && base + kStep <= hi) {
            if (!PREF) issue(base);
            uint4 raw[kLoads][kW];
#pragma unroll
            for (int l = 0; l < kLoads; ++l)
#pragma unroll
                for (int q = 0; q < kW; ++q) raw[l][q] = nxt[l][q];
            if (PREF && base + 2 * kStep <= hi) issue(base + kStep);
#pragma unroll
            for (int l = 0; l < kLoads; ++l) {
                if (DT == TSB_BF16) {
                    const uint32_t w[4] = {raw[l][0].x, raw[l][0].y, raw[l][0].z, raw[l][0].w};
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        x[l][2 * j] = __uint_as_float(w[j] << 16);
                        x[l][2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
                    }
                } else {
                    const uint4 a = raw[l][0], b = raw[l][kW - 1];
                    x[l][0] = __uint_as_float(a.x); x[l][1] = __uint_as_float(a.y);
                    x[l][2] = __uint_as_float(a.z); x[l][3] = __uint_as_float(a.w);
                    x[l][4] = __uint_as_float(b.x); x[l][5] = __uint_as_float(b.y);
                    x[l][6] = __uint_as_float(b.z); x[l][7] = __uint_as_float(b.w);
                }
            }
        } else {
#pragma unroll
        for (int l = 0; l < kLoads; ++l) {
            const int i0 = base + (l * NT + tid) * kEl;
            if (VEC && i0 + kEl <= hi) {
                if (DT == TSB_BF16) {
                    const uint4 raw = load_stream16((const uint16_t*)target + rowbase + i0);
                    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        x[l][2 * j] = __uint_as_float(w[j] << 16);
                        x[l][2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
                    }
                } else {
                    const uint4 a = load_stream16((const float*)target + rowbase + i0);
                    const uint4 b = load_stream16((const float*)target + rowbase + i0 + 4);
                    x[l][0] = __uint_as_float(a.x); x[l][1] = __uint_as_float(a.y);
                    x[l][2] = __uint_as_float(a.z); x[l][3] = __uint_as_float(a.w);
                    x[l][4] = __uint_as_float(b.x); x[l][5] = __uint_as_float(b.y);
                    x[l][6] = __uint_as_float(b.z); x[l][7] = __uint_as_float(b.w);
                }
            } else {
#pragma unroll
                for (int j = 0; j < kEl; ++j)
                    x[l][j] = (i0 + j < hi) ? load_logit<DT>(target, rowbase + i0 + j) : -INFINITY;
            }
        }
        }
        float cm = m;
#pragma unroll
        for (int l = 0; l < kLoads; ++l)
#pragma unroll
            for (int j = 0; j < kEl; ++j) cm = fmaxf(cm, x[l][j]);
        if (cm > m) {
            if (m > -INFINITY) sum *= (double)exp2f((m - cm) * c);
            m = cm;
        }
        if (m > -INFINITY) {
            const float mc = m * c;
#pragma unroll
            for (int l = 0; l < kLoads; ++l) {
                float cs = __builtin_amdgcn_exp2f(fmaf(x[l][0], c, -mc));
#pragma unroll
                for (int j = 1; j < kEl; ++j) cs += __builtin_amdgcn_exp2f(fmaf(x[l][j], c, -mc));
                sum += (double)cs;
            }
        }
    }
    m_out = m;
    sum_out = sum;
}

// Chunk g of ngroups, by one workgroup (rows at or beyond n_nodes[r] are
// skipped).
template <int DT, bool VEC, bool PREF>
__device__ __forceinline__ void target_chunk(int g, int ngroups, const void* __restrict__ target, int V, int B,
                                             int nrows, long long chunk, int P, float invT,
                                             const int32_t* __restrict__ n_nodes, float* __restrict__ tm,
                                             double* __restrict__ ts, int* __restrict__ tf, const XRegion& X, int R) {
    const int tid = threadIdx.x;
    // the walk that follows starts from cleared exchange slots
    xclear(X, R, (size_t)g * kBlock + tid, (size_t)ngroups * kBlock);
    const long long N = (long long)nrows * V;
    const long long e0 = (long long)g * chunk;
    if (e0 >= N) return;
    const long long e1 = min(e0 + chunk, N);
    const int t0 = (int)(e0 / V), t1 = (int)((e1 - 1) / V);
    const float c = invT * 1.4426950408889634f;  // invT * log2(e)
    __shared__ float s_m[kBlock / kWave];
    __shared__ double s_s[kBlock / kWave];
    const int wave = tid / kWave, lane = tid % kWave;
    for (int t = t0; t <= t1; ++t) {
        const int r = t / (B + 1);
        const int node = t % (B + 1);
        const long long rb = (long long)t * V;
        const int gf = (int)(rb / chunk);            // the row's first chunk
        const int gl = (int)((rb + V - 1) / chunk);  // and its last
        const size_t o = (size_t)t * P;
        if (g == gf && tid == 0) {
            for (int q = gl - gf + 1; q < P; ++q) {
                tm[o + q] = -INFINITY;
                ts[o + q] = 0.0;
                tf[o + q] = 0;
            }
        }
        if (node >= n_nodes[r]) continue;  // uniform over the workgroup
        const int lo = (int)max(e0 - rb, 0LL);
        const int hi = (int)min(e1 - rb, (long long)V);
        float m;
        double sum;
        stream_piece<DT, VEC, PREF>(target, (size_t)rb, lo, hi, c, m, sum);
        const float wm = wave_max(m);
        const double contrib = (m == -INFINITY) ? 0.0 : sum * (double)exp2f((m - wm) * c);
        const double wsum = wave_sum(contrib);
        if (lane == 0) {
            s_m[wave] = wm;
            s_s[wave] = wsum;
        }
        __syncthreads();
        if (tid == 0) {
            float M = s_m[0];
            for (int w = 1; w < kBlock / kWave; ++w) M = fmaxf(M, s_m[w]);
            double tot = 0.0;
            for (int w = 0; w < kBlock / kWave; ++w)
                if (s_m[w] != -INFINITY) tot += s_s[w] * (double)exp2f((s_m[w] - M) * c);
            const size_t q = o + (size_t)(g - gf);
            // partial as (max of a, sum exp(a - max a)), a = x invT; non-finite input
            // leaves a NaN or infinite max/sum
            tm[q] = M * invT;
            ts[q] = tot;
            tf[q] = (isnan(M) || M == INFINITY || !isfinite(tot)) ? 1 : 0;
        }
        __syncthreads();
    }
}

// Rows 0 and 1 of every request (the root, and its first child in BFS
// order; neither depends on the topology), for a walk that reads the other
// target rows itself: item g of R * kChainRows * kChainPieces is (request,
// row, piece), one workgroup of kChainThreads threads streams that equal
// piece of the row (multiples of 8 logits) with the target stream's
// arithmetic and writes its partial slot. Row 1 exists only when B >= 1.
constexpr int kChainThreads = 1024;
template <int DT, bool VEC>
__device__ __forceinline__ void chain_piece(int g, const void* __restrict__ target, int V, int B, float invT,
                                            float* __restrict__ cm, double* __restrict__ cs,
                                            int* __restrict__ cf) {
    constexpr int P = kChainPieces;
    const int r = g / (kChainRows * P), k = (g / P) % kChainRows, q = g % P;
    if (k > B) return;
    const int seg = ((V + P - 1) / P + 7) / 8 * 8;
    const int lo = min(V, q * seg), hi = min(V, lo + seg);
    const float c = invT * 1.4426950408889634f;
    float m;
    double sum;
    stream_piece<DT, VEC, false, kChainThreads>(target, ((size_t)r * (B + 1) + k) * (size_t)V, lo, hi, c, m, sum);
    __shared__ float s_m[kChainThreads / kWave];
    __shared__ double s_s[kChainThreads / kWave];
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const float wm = wave_max(m);
    const double contrib = (m == -INFINITY) ? 0.0 : sum * (double)exp2f((m - wm) * c);
    const double wsum = wave_sum(contrib);
    if (lane == 0) {
        s_m[wave] = wm;
        s_s[wave] = wsum;
    }
    __syncthreads();
    if (tid == 0) {
        float M = s_m[0];
        for (int w = 1; w < kChainThreads / kWave; ++w) M = fmaxf(M, s_m[w]);
        double tot = 0.0;
        for (int w = 0; w < kChainThreads / kWave; ++w)
            if (s_m[w] != -INFINITY) tot += s_s[w] * (double)exp2f((s_m[w] - M) * c);
        const size_t o = ((size_t)r * kChainRows + k) * P + q;
        cm[o] = M * invT;
        cs[o] = tot;
        cf[o] = (isnan(M) || M == INFINITY || !isfinite(tot)) ? 1 : 0;
    }
    __syncthreads();
}

// binary64 log-sum-exp of one target row from its P partial slots (fixed
// order), and whether the row held a non-finite logit (or none finite).
__device__ __forceinline__ double target_row_lse(const float* __restrict__ tm, const double* __restrict__ ts,
                                                 const int* __restrict__ tf, int P, size_t row, int* bad) {
    const size_t o = row * (size_t)P;
    float M = -INFINITY;
    int b = 0;
    for (int s = 0; s < P; ++s) {
        M = fmaxf(M, tm[o + s]);
        b |= tf[o + s];
    }
    double tot = 0.0;
    for (int s = 0; s < P; ++s)
        if (tm[o + s] != -INFINITY) tot += ts[o + s] * exp((double)tm[o + s] - (double)M);
    *bad = b || M == -INFINITY;
    return (double)M + log(tot);
}

// Node records for the walk, written by the replay merge of a whole round:
// everything the walk reads when it enters node u, in one record of
// kRecWords 32-bit words, so that entering a node costs one memory round
// trip (besides its target row, when the walk reads rows as it enters their
// nodes). Words: 0 m (children; 0 for a leaf), 1 first child, 2 depth,
// 3 flags (kRecOk: the node passed the topology checks; kRecTargetBad: its
// target row is unusable), 4-5 the row's streamed normaliser L0 (binary64;
// both only when every row was streamed before the merge, else 0), 6-7 the
// draft normaliser of the children's row, then per child j (up to
// TSB_MAX_K) four words at 8 + 4 j: token, draft logit x invT and target
// logit x invT (binary32 bits; 0 for a token outside [0, V)), unused.
constexpr uint32_t kRecOk = 1u, kRecTargetBad = 2u;

}  // namespace tsb
