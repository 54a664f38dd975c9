// Device-side building blocks shared by the gfx950 kernels of the
// tree-replay library: counter-based RNG, uniform and Gumbel maps, logit
// loads, order-preserving keys and wave64 reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tsb_internal.hpp"

namespace tsb {

constexpr int kWave = 64;

// ---------------------------------------------------------------- Philox
// Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC'11): each round
// multiplies counter words 0 and 2 by fixed 32-bit constants and mixes the
// high halves with the other words and the key; the key advances by two Weyl
// increments between rounds.
constexpr uint32_t kPhiloxM0 = 0xD2511F53u;
constexpr uint32_t kPhiloxM1 = 0xCD9E8D57u;
constexpr uint32_t kPhiloxW0 = 0x9E3779B9u;
constexpr uint32_t kPhiloxW1 = 0xBB67AE85u;

// a ^ b ^ c in one instruction (v_bitop3_b32, truth table 0x96)
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

__device__ __forceinline__ uint4 philox10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = (uint64_t)kPhiloxM0 * c.x;
        const uint64_t p1 = (uint64_t)kPhiloxM1 * c.z;
        const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        c = make_uint4(xor3(hi1, c.y, k0), lo1, xor3(hi0, c.w, k1), lo0);
        k0 += kPhiloxW0;
        k1 += kPhiloxW1;
    }
    return c;
}

// Counter layout: (draw >> 2, node | stream << 16, request, step); key =
// (seed lo, seed hi); the draw uses output word draw & 3.
struct RngKey {
    uint32_t k0, k1;
    uint32_t request, step;
};

__device__ __forceinline__ uint4 rng_block(const RngKey& key, uint32_t node, uint32_t stream,
                                           uint32_t block) {
    return philox10(make_uint4(block, (node & 0xFFFFu) | (stream << 16), key.request, key.step),
                    key.k0, key.k1);
}

__device__ __forceinline__ uint32_t rng_word(const RngKey& key, uint32_t node, uint32_t stream,
                                             uint32_t draw) {
    const uint4 w = rng_block(key, node, stream, draw >> 2);
    const uint32_t s = draw & 3u;
    return s == 0 ? w.x : (s == 1 ? w.y : (s == 2 ? w.z : w.w));
}

// Uniform (2 * (w >> 9) + 1) * 2^-24 in (0, 1): exact in binary32.
__device__ __forceinline__ float u24f(uint32_t w) {
    return (float)(((w >> 9) << 1) | 1u) * 0x1p-24f;
}
__device__ __forceinline__ double u24d(uint32_t w) {
    return (double)(((w >> 9) << 1) | 1u) * 0x1p-24;
}

// Standard Gumbel -ln(-ln u) in binary32 via base-2 logarithms:
// -ln u = ln2 * (-log2 u);  G = -ln2 * log2(-log2 u) - ln(ln 2).
__device__ __forceinline__ float gumbel_f32(uint32_t w) {
    const float u = u24f(w);
    const float e2 = -__log2f(u);  // > 0
    return fmaf(-0.69314718055994531f, __log2f(e2), 0.36651292058166432f);
}

// Bounds of gumbel_f32 over all 2^23 uniforms, with slack for rounding
// (the extremes are about 16.63 at u = 1 - 2^-24 and -2.81 at u = 2^-24).
constexpr float kGumbelMaxBound = 16.75f;
constexpr float kGumbelMinBound = -2.85f;

// ---------------------------------------------------------------- exp (binary64)
// Table-driven exponential (P. T. P. Tang, "Table-driven implementation of
// the exponential function in IEEE floating-point arithmetic", ACM TOMS
// 15(2), 1989): x = (256 m + j) ln2/256 + r with |r| <= ln2/512, so
// e^x = 2^m * 2^(j/256) * e^r, e^r - 1 by its degree-4 Taylor polynomial.
// The reduction uses one FMA against fl64(ln2)/256, whose error (9.1e-20)
// times |n| stays below 1.3e-15 for every x >= -36, i.e. for every term that
// is not already below 2^-52 of the largest one; the truncation is below
// 4e-17 relative. The 256 table entries 2^(j/256) live in LDS
// (exp64_table_init). Inputs below -746 give 0; -inf gives 0; NaN gives 0.
constexpr int kExpTable = 256;

__device__ __forceinline__ void exp64_table_init(double* t) {
    for (int j = threadIdx.x; j < kExpTable; j += blockDim.x) t[j] = exp2((double)j / (double)kExpTable);
    __syncthreads();
}

__device__ __forceinline__ double exp64(double x, const double* t) {
    constexpr double kInvL = 369.3299304675746;            // 256 / ln2
    constexpr double kL = 0.0027076061740622863;           // fl64(ln2) / 256
    x = fmax(x, -746.0);                                   // e^-746 rounds to 0
    const double n = rint(x * kInvL);
    const double r = fma(-n, kL, x);
    const int ni = (int)n;
    const int j = ni & (kExpTable - 1);
    const int m = ni >> 8;                                 // floor(ni / 256)
    double p = fma(r, 1.0 / 24.0, 1.0 / 6.0);
    p = fma(r, p, 0.5);
    p = fma(r, p, 1.0);
    p = p * r;                                             // e^r - 1
    const double s = t[j];
    return ldexp(fma(s, p, s), m);
}

// ---------------------------------------------------------------- logits
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

template <int DT>
__device__ __forceinline__ float load_logit(const void* base, size_t i) {
    if (DT == TSB_BF16)
        return bf16_to_f32(((const uint16_t*)base)[i]);
    else
        return ((const float*)base)[i];
}

// 16-byte load with the non-temporal hint, for data read exactly once.
typedef unsigned int tsb_u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_stream16(const void* p) {
    const tsb_u32x4 v = __builtin_nontemporal_load((const tsb_u32x4*)p);
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Order-preserving map of a binary32 value to uint32 (larger float -> larger
// key); -0 is folded onto +0 so equal values give equal keys.
__device__ __forceinline__ uint32_t ordered_bits(float x) {
    uint32_t u = __float_as_uint(x);
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float from_ordered_bits(uint32_t k) {
    const uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
    return __uint_as_float(u);
}

// Order-preserving map of a binary64 value to uint64 (-0 folded onto +0).
__device__ __forceinline__ uint64_t ordered_bits64(double x) {
    uint64_t u = (uint64_t)__double_as_longlong(x);
    if (u == 0x8000000000000000ull) u = 0ull;
    return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Inverse of ordered_bits64 (for a key with cleared low bits: a value at
// most that of the full key).
__device__ __forceinline__ double from_ordered_bits64(uint64_t k) {
    const uint64_t u = (k >> 63) ? (k & 0x7FFFFFFFFFFFFFFFull) : ~k;
    return __longlong_as_double((long long)u);
}

// Candidate key: logit desc, then token id asc.
__device__ __forceinline__ uint64_t cand_key(float x, uint32_t id) {
    return ((uint64_t)ordered_bits(x) << 32) | (uint32_t)(~id);
}
__device__ __forceinline__ uint32_t cand_id(uint64_t k) { return ~(uint32_t)k; }
__device__ __forceinline__ float cand_value(uint64_t k) { return from_ordered_bits((uint32_t)(k >> 32)); }

// ---------------------------------------------------------------- caller trees
// One node of a caller-supplied topology, checked before any of its entries
// becomes an address. A node with m > 0 children is well formed when
// m <= TSB_MAX_K, its children occupy [fc, fc + m) with u < fc and
// fc + m <= n (so every descent moves to a larger index and stays inside the
// tree) and its depth d lies in [0, D) (its children read draft row d). A
// node with m == 0 is a leaf whatever its other entries hold.
struct TreeNode {
    int m, fc, d;
    bool ok;
};

__device__ __forceinline__ TreeNode tree_node(const tsb_tree& t, size_t tb, int u, int n, int D) {
    TreeNode v;
    v.m = t.n_children[tb + u];
    v.fc = t.first_child[tb + u];
    v.d = t.depth[tb + u];
    v.ok = v.m == 0 || (v.m > 0 && v.m <= TSB_MAX_K && v.fc > u && v.fc <= n - v.m && v.d >= 0 && v.d < D);
    if (!v.ok || v.m == 0) v.m = 0;
    return v;
}

// n_nodes of a caller-supplied topology is usable when it lies in [1, B + 1].
__device__ __forceinline__ bool tree_count_ok(int n, int B) { return n >= 1 && n <= B + 1; }

// ---------------------------------------------------------------- wave ops
__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }

// The value of lane (lane ^ j). Distances 1 and 2 are DPP quad permutations
// ([1, 0, 3, 2] and [2, 3, 0, 1]); 16 and 32 are the row and half swaps of
// v_permlane16_swap / v_permlane32_swap applied to two copies of the value
// (the first result holds the partner's value in the odd rows / upper half,
// the second in the even rows / lower half); none of them goes through LDS.
// 4 and 8 use ds_swizzle in bit-mask mode (no address operand); other
// distances ds_bpermute. j is a compile-time constant wherever the sorts
// unroll.
__device__ __forceinline__ uint32_t xor_lane_u32(uint32_t x, int j) {
    if (j == 1) return (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0xB1, 0xF, 0xF, false);
    if (j == 2) return (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x4E, 0xF, 0xF, false);
    // bit-mask swizzle within 32 lanes: and 0x1F, or 0, xor j
    if (j == 4) return (uint32_t)__builtin_amdgcn_ds_swizzle((int)x, 0x1F | (4 << 10));
    if (j == 8) return (uint32_t)__builtin_amdgcn_ds_swizzle((int)x, 0x1F | (8 << 10));
    if (j == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
        return (lane_id() & 16) ? r[0] : r[1];
    }
    if (j == 32) {
        const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
        return (lane_id() & 32) ? r[0] : r[1];
    }
    return (uint32_t)__shfl_xor((int)x, j, kWave);
}

// As xor_lane_u32 for the butterfly reductions, with distances 16 and 32 on
// ds_bpermute (the permlane swaps measured slower there).
__device__ __forceinline__ uint32_t xor_lane_red_u32(uint32_t x, int j) {
    return (j >= 16) ? (uint32_t)__shfl_xor((int)x, j, kWave) : xor_lane_u32(x, j);
}

// Butterfly reductions over the wave (partners lane ^ 32, ^ 16, ..., ^ 1:
// every lane ends with the same value, added in the same order).
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __uint_as_float(xor_lane_red_u32(__float_as_uint(v), o)));
    return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const uint64_t u = (uint64_t)__double_as_longlong(v);
        const uint64_t p = ((uint64_t)xor_lane_red_u32((uint32_t)(u >> 32), o) << 32) | xor_lane_red_u32((uint32_t)u, o);
        v += __longlong_as_double((long long)p);
    }
    return v;
}
__device__ __forceinline__ int wave_or(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v |= (int)xor_lane_red_u32((uint32_t)v, o);
    return v;
}
// Whole-wave one-lane shifts through DPP (lane i receives lane i-1, resp.
// i+1; the edge lane keeps its own value) and reads of one lane's value
// (the lane index must be wave-uniform).
__device__ __forceinline__ uint32_t wave_shr1(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x138, 0xf, 0xf, false);
}
__device__ __forceinline__ uint32_t wave_shl1(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x130, 0xf, 0xf, false);
}
__device__ __forceinline__ uint64_t wave_shr1(uint64_t v) {
    return ((uint64_t)wave_shr1((uint32_t)(v >> 32)) << 32) | wave_shr1((uint32_t)v);
}
__device__ __forceinline__ uint64_t wave_shl1(uint64_t v) {
    return ((uint64_t)wave_shl1((uint32_t)(v >> 32)) << 32) | wave_shl1((uint32_t)v);
}
__device__ __forceinline__ double wave_shr1(double v) {
    return __longlong_as_double((long long)wave_shr1((uint64_t)__double_as_longlong(v)));
}
__device__ __forceinline__ double wave_shl1(double v) {
    return __longlong_as_double((long long)wave_shl1((uint64_t)__double_as_longlong(v)));
}
__device__ __forceinline__ uint32_t lane_u32(uint32_t v, int l) { return (uint32_t)__builtin_amdgcn_readlane((int)v, l); }
__device__ __forceinline__ float lane_f32(float v, int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l)); }
__device__ __forceinline__ uint64_t lane_u64(uint64_t v, int l) {
    return ((uint64_t)lane_u32((uint32_t)(v >> 32), l) << 32) | lane_u32((uint32_t)v, l);
}
__device__ __forceinline__ double lane_f64(double v, int l) {
    return __longlong_as_double((long long)lane_u64((uint64_t)__double_as_longlong(v), l));
}

// ---------------------------------------------------------------- walk support
template <int DT>
__device__ __forceinline__ void load4(const void* base, size_t off, int valid, bool vec, float x[4]) {
    if (vec && valid == 4) {
        if (DT == TSB_BF16) {
            const uint2 raw = *(const uint2*)((const uint16_t*)base + off);
            x[0] = __uint_as_float(raw.x << 16);
            x[1] = __uint_as_float(raw.x & 0xFFFF0000u);
            x[2] = __uint_as_float(raw.y << 16);
            x[3] = __uint_as_float(raw.y & 0xFFFF0000u);
        } else {
            const float4 a = *(const float4*)((const float*)base + off);
            x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
        }
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = e < valid ? load_logit<DT>(base, off + e) : -INFINITY;
    }
}

// Four logits as loaded (bf16 pairs or binary32), so the loads of a pass can
// be issued early and converted later.
template <int DT>
struct Raw4 {
    uint32_t w[DT == TSB_BF16 ? 2 : 4];
};

template <int DT>
__device__ __forceinline__ void raw_load4(const void* base, size_t off, int valid, bool vec, Raw4<DT>& g) {
    if (vec && valid == 4) {
        if (DT == TSB_BF16) {
            const uint2 raw = *(const uint2*)((const uint16_t*)base + off);
            g.w[0] = raw.x;
            g.w[1] = raw.y;
        } else {
            const uint4 raw = *(const uint4*)((const float*)base + off);
            g.w[0] = raw.x;
            g.w[1] = raw.y;
            g.w[2] = raw.z;
            g.w[3] = raw.w;
        }
    } else {
        float x[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = e < valid ? load_logit<DT>(base, off + e) : -INFINITY;
        if (DT == TSB_BF16) {  // a bf16 value is the top half of its binary32 value
            g.w[0] = (__float_as_uint(x[0]) >> 16) | (__float_as_uint(x[1]) & 0xFFFF0000u);
            g.w[1] = (__float_as_uint(x[2]) >> 16) | (__float_as_uint(x[3]) & 0xFFFF0000u);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) g.w[e] = __float_as_uint(x[e]);
        }
    }
}

template <int DT>
__device__ __forceinline__ void raw_scaled4(const Raw4<DT>& g, int valid, float invT, float a[4]) {
    float x[4];
    if (DT == TSB_BF16) {
        x[0] = __uint_as_float(g.w[0] << 16);
        x[1] = __uint_as_float(g.w[0] & 0xFFFF0000u);
        x[2] = __uint_as_float(g.w[1] << 16);
        x[3] = __uint_as_float(g.w[1] & 0xFFFF0000u);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = __uint_as_float(g.w[e]);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) a[e] = e < valid ? x[e] * invT : -INFINITY;
}

// A descending list of the `k` (<= 64) largest uint64 keys seen so far,
// one entry per lane (lane i holds the i-th largest; lanes >= k hold 0).
// Key 0 is reserved as "empty". An insertion is a ballot for the position
// and a one-lane shift of the tail.
struct WaveTopList {
    uint64_t v;    // this lane's entry
    uint64_t thr;  // smallest kept key (entry of lane k-1), uniform
    int k;

    __device__ void init(int kk) {
        k = kk;
        v = 0;
        thr = 0;
    }
    // Insert the key held by every lane whose `want` is set (lanes may hold
    // different keys). Keys <= thr are ignored.
    __device__ void offer(uint64_t key, bool want) {
        want = want && key > thr;
        uint64_t ballot = __ballot(want);
        const int lane = lane_id();
        while (ballot) {
            const int src = __ffsll((unsigned long long)ballot) - 1;
            ballot &= ballot - 1;
            const uint64_t c = lane_u64(key, src);
            if (c <= thr) continue;
            const int pos = __popcll(__ballot(lane < k && v > c));
            const uint64_t up = wave_shr1(v);
            if (lane < k) {
                if (lane == pos)
                    v = c;
                else if (lane > pos)
                    v = up;
            }
            thr = lane_u64(v, k - 1);
        }
    }
    // As offer, for candidates given as (logit, id): the key is formed only
    // for the one candidate being inserted (from wave-uniform values).
    __device__ void offer_xid(float x, uint32_t id, bool want) {
        uint64_t ballot = __ballot(want);
        const int lane = lane_id();
        while (ballot) {
            const int src = __ffsll((unsigned long long)ballot) - 1;
            ballot &= ballot - 1;
            const uint64_t c = cand_key(lane_f32(x, src), lane_u32(id, src));
            if (c <= thr) continue;
            const int pos = __popcll(__ballot(lane < k && v > c));
            const uint64_t up = wave_shr1(v);
            if (lane < k) {
                if (lane == pos)
                    v = c;
                else if (lane > pos)
                    v = up;
            }
            thr = lane_u64(v, k - 1);
        }
    }
};

// Orders a wave's LDS accesses before and after this point (for lanes that
// read what other lanes of the same wave wrote).
__device__ __forceinline__ void wave_lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int j) {
    return ((uint64_t)xor_lane_u32((uint32_t)(v >> 32), j) << 32) | xor_lane_u32((uint32_t)v, j);
}

// Sorts the NR * 64 keys held NR per lane in descending order (element
// r * 64 + lane in v[r]): a bitonic network, lane exchanges for distances
// below 64 and register exchanges above. Cheaper than K selection rounds
// once K is large.
template <int NR>
__device__ __forceinline__ void wave_sort_desc(uint64_t (&v)[NR]) {
    const int lane = lane_id();
    constexpr int N = NR * kWave;
#pragma unroll
    for (int k = 2; k <= N; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            if (j >= kWave) {
                const int rj = j / kWave;
#pragma unroll
                for (int r = 0; r < NR; ++r) {
                    if (r & rj) continue;  // each register pair (r, r | rj) once
                    const bool desc = ((r * kWave + lane) & k) == 0;
                    const uint64_t a = v[r], b = v[r | rj];
                    const bool sw = desc ? (a < b) : (a > b);  // the lower element keeps the max when descending
                    v[r] = sw ? b : a;
                    v[r | rj] = sw ? a : b;
                }
            } else {
#pragma unroll
                for (int r = 0; r < NR; ++r) {
                    const uint64_t o = shfl_xor_u64(v[r], j);
                    const bool lower = (lane & j) == 0;
                    const bool desc = ((r * kWave + lane) & k) == 0;
                    const bool keep_max = lower == desc;
                    v[r] = keep_max ? (v[r] > o ? v[r] : o) : (v[r] < o ? v[r] : o);
                }
            }
        }
    }
}

// Number of lanes below this one whose bit is set in b.
__device__ __forceinline__ int lanes_below_u64(uint64_t b) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0u));
}

// Exclusive prefix sum over the lanes of small non-negative counts
// (< 2^NB), one ballot per bit; `total` receives the wave sum.
template <int NB>
__device__ __forceinline__ int wave_excl_scan(int c, int& total) {
    int off = 0;
    total = 0;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const uint64_t m = __ballot((c >> b) & 1);
        const int below = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                         __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        off += below << b;
        total += __popcll(m) << b;
    }
    return off;
}

// The k-th largest (1 <= k <= 64) of the values held by the 64 lanes, NaN
// counted as -inf; wave-uniform.
__device__ __forceinline__ float wave_kth_largest(float x, int k) {
    x = isnan(x) ? -INFINITY : x;
    const int lane = lane_id();
    int rank = 0;
    for (int l = 0; l < kWave; ++l) {
        const float o = lane_f32(x, l);
        rank += (o > x || (o == x && l < lane)) ? 1 : 0;
    }
    const uint64_t b = __ballot(rank == k - 1);
    return lane_f32(x, __ffsll((unsigned long long)b) - 1);
}

}  // namespace tsb
