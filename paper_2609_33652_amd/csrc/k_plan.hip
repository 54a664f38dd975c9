// First pass of a tree-replay round on gfx950 (Section 3.1; Appendix B.3):
//   draft_partials  one workgroup per (draft row, vocabulary segment):
//                   online max / binary64 sum of exp, and the segment's K best
//                   candidates by (logit desc, id asc) kept in a wave-wide
//                   sorted list; one streaming read of the draft logits.
//   plan_tree       one workgroup per request: merge of the segment partials
//                   into the binary64 log-sum-exp, its canonical binary32
//                   rounding and lp = fl32(a - lse32); then the first B rank
//                   paths under the static order (score desc, depth asc, rank
//                   path lexicographic asc) by a parallel threshold search,
//                   emitted in BFS order.
#include <math.h>

#include <algorithm>

#include "tsb_device.hpp"
#include "tsb_kernels.hpp"
#include "tsb_target.hpp"

namespace tsb {

// ------------------------------------------------------------------ K1a
// Row statistics of the draft: one workgroup of kDraftThreads threads per
// (draft row, vocabulary segment), one streaming read of the segment. The
// next chunk's loads are issued before the current chunk is processed, and
// chunks stay raw words until then.
//
// Normaliser. For bf16 logits at a temperature whose scaled logits stay in
// range, e^a is looked up per logit instead of evaluated: a = fl32(x invT)
// depends only on the 16-bit pattern of x, so a binary64 table of e^a over
// every pattern with 2^-16 <= |x| < 64 (22 binades, both signs) is built in
// LDS per workgroup and the segment sum is a binary64 sum of table entries
// (no running maximum: the entries stay within binary64's normal range).
// Logits outside the table (zero, tiny, large, non-finite) and every logit of
// binary32 rows take the evaluated path: a running maximum m per lane and a
// binary64 sum of e^(a - m) by the table-driven exp64. The two parts of a
// lane (reference 0 and reference m) are combined at the end.
//
// Candidates. A group of 8 logits whose maximum passes a filter (x > fx, or
// x == fx with id <= fid) is only recorded (its offset, in a short per-lane
// list in LDS); the stream does no other candidate work. When some lane's
// list is full, and at the end, the wave re-reads the recorded groups, one
// per lane per round, and appends the logits that pass to its LDS buffer; a
// buffer that runs full keeps its K best keys and the filter rises to the
// K-th of them (shared with the other waves of the workgroup through an LDS
// maximum). The filter starts at the K-th largest of the first chunk's
// column maxima: K distinct logits at least that large exist, so nothing
// below it can be among the segment's K best. At the end one wave selects
// the K best of all buffers.
constexpr int kDraftThreads = 512;
constexpr int kDraftWaves = kDraftThreads / kWave;
constexpr int kDraftU = 4;     // 8-logit groups per thread per chunk
// candidate buffer entries per wave (the pool selection, with no table in
// LDS, keeps more: its K reaches 64)
template <bool STATS>
constexpr int cand_cap() { return STATS ? 128 : 256; }
constexpr int kDraftChunk = kDraftThreads * 8 * kDraftU;
// recorded groups per lane before the wave flushes (the pool selection, with
// no table in LDS and a weaker first filter at K = 64, keeps more)
template <bool STATS>
constexpr int rec_slots() { return STATS ? 8 : 24; }
constexpr int kRecBatch = 4;   // recorded groups re-read at once

// Exponential table over bf16 patterns with biased exponent field in
// [kTabExpLo, kTabExpLo + kTabBinades) (2^-16 <= |x| < 64): the entry of
// magnitude index t = (pattern & 0x7FFF) - kTabBase and sign bit s sits at
// byte offset 8 t + 32768 s, so that the offsets of both halves of a word of
// two patterns come from one shift of the clamped indices and one OR of the
// sign bits. Index kTabHalf holds 0.0 for both signs: patterns outside the
// table are clamped onto it. The gap between the positive half and the
// negative half holds other LDS data of the workgroup.
constexpr uint32_t kTabExpLo = 111;  // 2^-16
constexpr int kTabBinades = 22;      // up to 2^6 (exclusive)
constexpr int kTabHalf = kTabBinades * 128;
constexpr uint32_t kTabBase = kTabExpLo << 7;
constexpr int kTabNeg = 32768 / 8;               // first binary64 slot of the negative half
constexpr int kTabDoubles = kTabNeg + kTabHalf + 1;
constexpr int kTabGap = kTabHalf + 1;            // first free slot of the gap
constexpr int kSpecialCap = 256;                 // deferred out-of-table patterns per wave
static_assert(8 * kTabHalf < 32768, "the positive half must end below the sign bit of an offset");

// Whether the table may be used at this inverse temperature: every entry
// e^(fl32(x invT)), |x| < 64, is a normal binary64 number (and a sum of up
// to 2^31 of them stays finite).
inline bool draft_table_ok(float invT) { return 63.75f * invT < 680.0f; }
// Segments shorter than this evaluate every exponential (the table would
// cost more to build than it saves).
constexpr int kTableMinSeg = 8192;

// Raw words of one 8-logit group: four words of bf16 pairs, or eight binary32.
template <int DT>
struct Raw8 {
    uint32_t w[DT == TSB_BF16 ? 4 : 8];
};

// Loads one group; positions at or past `hi` read as -inf. Issues the loads
// only: nothing here waits for them.
template <int DT, bool VEC>
__device__ __forceinline__ void load_raw8(const void* __restrict__ draft, size_t rowbase, int i0, int hi,
                                          Raw8<DT>& g) {
    if (VEC && i0 + 8 <= hi) {
        if (DT == TSB_BF16) {
            const uint4 r = load_stream16((const uint16_t*)draft + rowbase + i0);
            g.w[0] = r.x; g.w[1] = r.y; g.w[2] = r.z; g.w[3] = r.w;
        } else {
            const uint4 r0 = load_stream16((const float*)draft + rowbase + i0);
            const uint4 r1 = load_stream16((const float*)draft + rowbase + i0 + 4);
            g.w[0] = r0.x; g.w[1] = r0.y; g.w[2] = r0.z; g.w[3] = r0.w;
            g.w[4] = r1.x; g.w[5] = r1.y; g.w[6] = r1.z; g.w[7] = r1.w;
        }
    } else {
        if (DT == TSB_BF16) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t a = (i0 + 2 * j < hi) ? (uint32_t)((const uint16_t*)draft)[rowbase + i0 + 2 * j] : 0xFF80u;
                const uint32_t b = (i0 + 2 * j + 1 < hi) ? (uint32_t)((const uint16_t*)draft)[rowbase + i0 + 2 * j + 1]
                                                         : 0xFF80u;
                g.w[j] = a | (b << 16);
            }
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                g.w[j] = (i0 + j < hi) ? __float_as_uint(((const float*)draft)[rowbase + i0 + j]) : 0xFF800000u;
        }
    }
}

// A chunk (kDraftU groups per thread) that lies inside the segment: vector
// loads with no bounds test.
template <int DT>
__device__ __forceinline__ void load_chunk(const void* __restrict__ draft, size_t rowbase, int base, int tid,
                                           Raw8<DT> (&r)[kDraftU]) {
#pragma unroll
    for (int u = 0; u < kDraftU; ++u) {
        const size_t i0 = rowbase + (size_t)(base + (u * kDraftThreads + tid) * 8);
        if (DT == TSB_BF16) {
            const uint4 v = load_stream16((const uint16_t*)draft + i0);
            r[u].w[0] = v.x; r[u].w[1] = v.y; r[u].w[2] = v.z; r[u].w[3] = v.w;
        } else {
            const uint4 v0 = load_stream16((const float*)draft + i0);
            const uint4 v1 = load_stream16((const float*)draft + i0 + 4);
            r[u].w[0] = v0.x; r[u].w[1] = v0.y; r[u].w[2] = v0.z; r[u].w[3] = v0.w;
            r[u].w[4] = v1.x; r[u].w[5] = v1.y; r[u].w[6] = v1.z; r[u].w[7] = v1.w;
        }
    }
}

// A chunk that may reach past `hi` (positions there read as -inf).
template <int DT, bool VEC>
__device__ __forceinline__ void load_chunk_masked(const void* __restrict__ draft, size_t rowbase, int base, int hi,
                                                  int tid, Raw8<DT> (&r)[kDraftU]) {
#pragma unroll
    for (int u = 0; u < kDraftU; ++u) load_raw8<DT, VEC>(draft, rowbase, base + (u * kDraftThreads + tid) * 8, hi, r[u]);
}

template <int DT>
__device__ __forceinline__ void raw8_values(const Raw8<DT>& g, float* x) {
    if (DT == TSB_BF16) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            x[2 * j] = __uint_as_float(g.w[j] << 16);
            x[2 * j + 1] = __uint_as_float(g.w[j] & 0xFFFF0000u);
        }
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = __uint_as_float(g.w[j]);
    }
}

// The k-th largest (1 <= k <= 64) of the values held by the 64 lanes (NaN
// counted as -inf), wave-uniform: a bitonic sort across the lanes.
__device__ __forceinline__ float wave_kth_largest_sorted(float x, int k) {
    x = isnan(x) ? -INFINITY : x;
    const int lane = lane_id();
#pragma unroll
    for (int kk = 2; kk <= kWave; kk <<= 1) {
#pragma unroll
        for (int j = kk >> 1; j > 0; j >>= 1) {
            const float o = __shfl_xor(x, j, kWave);
            const bool keep_max = ((lane & j) == 0) == ((lane & kk) == 0);  // descending overall
            x = keep_max ? fmaxf(x, o) : fminf(x, o);
        }
    }
    return lane_f32(x, k - 1);
}

// One step of a wave maximum through DPP: lanes of the rows in ROWMASK take
// the larger of their key and the key DPP control CTRL moves to them.
template <int CTRL, int ROWMASK>
__device__ __forceinline__ uint64_t dpp_max_step(uint64_t v) {
    const int h = (int)(uint32_t)(v >> 32), l = (int)(uint32_t)v;
    const uint32_t oh = (uint32_t)__builtin_amdgcn_update_dpp(h, h, CTRL, ROWMASK, 0xf, false);
    const uint32_t ol = (uint32_t)__builtin_amdgcn_update_dpp(l, l, CTRL, ROWMASK, 0xf, false);
    const uint64_t o = ((uint64_t)oh << 32) | ol;
    return o > v ? o : v;
}

// Wave-uniform maximum of a uint64 key: within quads, half rows and rows by
// DPP permutations, then row broadcasts carry the running maximum to lane 63.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
    v = dpp_max_step<0xB1, 0xF>(v);   // quad_perm [1, 0, 3, 2]
    v = dpp_max_step<0x4E, 0xF>(v);   // quad_perm [2, 3, 0, 1]
    v = dpp_max_step<0x141, 0xF>(v);  // row_half_mirror
    v = dpp_max_step<0x140, 0xF>(v);  // row_mirror
    v = dpp_max_step<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
    v = dpp_max_step<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
    return lane_u64(v, kWave - 1);
}

// The K (<= 64) largest of the NR * 64 keys held NR per lane (0 = empty;
// keys are distinct): lane r receives the r-th largest, lanes >= K and lanes
// past the number of non-empty keys receive 0. Destroys v.
template <int NR>
__device__ __forceinline__ uint64_t wave_select_top(uint64_t (&v)[NR], int K) {
    const int lane = lane_id();
    uint64_t out = 0;
    for (int r = 0; r < K; ++r) {
        uint64_t m = v[0];
#pragma unroll
        for (int i = 1; i < NR; ++i) m = v[i] > m ? v[i] : m;
        const uint64_t w = wave_max_u64(m);
        if (w == 0) break;
        if (lane == r) out = w;
#pragma unroll
        for (int i = 0; i < NR; ++i)
            if (v[i] == w) v[i] = 0;
    }
    return out;
}

// The K (<= 64) largest keys in lanes 0..K-1 (sorted; 0 past them), by
// selection rounds for small K and by a sort for large K. Destroys v.
template <int NR>
__device__ __forceinline__ uint64_t wave_top(uint64_t (&v)[NR], int K) {
    if (K <= 16) return wave_select_top<NR>(v, K);
    wave_sort_desc<NR>(v);
    return lane_id() < K ? v[0] : 0ull;
}

// Per-wave candidate buffer with its filter.
template <int CAP>
struct CandBuf {
    uint64_t* buf;  // CAP entries in LDS
    int n;          // entries in use (wave-uniform)
    float fx;       // filter value
    uint32_t fid;   // filter id bound for x == fx

    __device__ bool pass(float x, uint32_t id) const { return x > fx || (x == fx && id <= fid); }
    // Tighten the filter to key k (the K-th best of some set of distinct
    // logits): entering needs a larger key.
    __device__ void raise_to(uint64_t k) {
        const float tx = cand_value(k);
        const uint32_t ti = cand_id(k);
        if (tx > fx || (tx == fx && ti <= fid)) {
            fx = tx;
            fid = ti - 1;  // wraps for id 0 to "any id": looser, and the keys still order correctly
        }
    }
    // Keep the K best keys at the front; when K keys are kept, raise the
    // filter to the K-th and publish it to s_key.
    __device__ __forceinline__ void compact(int K, unsigned long long* s_key) {
        const int lane = lane_id();
        wave_lds_fence();
        uint64_t v[CAP / kWave];
#pragma unroll
        for (int i = 0; i < CAP / kWave; ++i) {
            const int j = i * kWave + lane;
            v[i] = j < n ? buf[j] : 0ull;
        }
        const uint64_t t = wave_top<CAP / kWave>(v, K);
        wave_lds_fence();
        if (lane < K) buf[lane] = t;
        wave_lds_fence();
        n = __popcll(__ballot(t != 0ull));
        if (n == K) {
            const uint64_t kth = lane_u64(t, K - 1);
            raise_to(kth);
            if (lane == 0) atomicMax(s_key, (unsigned long long)kth);
        }
    }
    // Append the logits of one group (lane's x[0..8) with ids i0..i0+7)
    // that pass, one per lane per round.
    __device__ __forceinline__ void offer8(const float* x, int i0, int hi, bool live, int K, unsigned long long* s_key) {
        uint32_t mask = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (live && i0 + j < hi && pass(x[j], (uint32_t)(i0 + j))) mask |= 1u << j;
        for (;;) {
            const uint64_t b = __ballot(mask != 0u);
            if (!b) break;
            if (n + kWave > CAP) compact(K, s_key);
            const int j = mask ? (int)__builtin_ctz(mask) : 0;
            // x[j] by a select tree on the bits of j (no indexed register access)
            const bool b0 = j & 1, b1 = j & 2, b2 = j & 4;
            const float t0 = b0 ? x[1] : x[0], t1 = b0 ? x[3] : x[2];
            const float t2 = b0 ? x[5] : x[4], t3 = b0 ? x[7] : x[6];
            const float u0 = b1 ? t1 : t0, u1 = b1 ? t3 : t2;
            const float xv = b2 ? u1 : u0;
            const int pos = n + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32),
                                                               __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0u));
            if (mask) buf[pos] = cand_key(xv, (uint32_t)(i0 + j));
            n += __popcll(b);
            mask &= mask - 1u;
        }
    }
};

// Re-reads the groups this wave's lanes recorded (nrec per lane, offsets in
// s_rec[.][tid]) and offers their logits, one group per lane per round.
template <int DT, bool VEC, int CAP, int BATCH = kRecBatch>
__device__ __forceinline__ void flush_recorded(CandBuf<CAP>& cb, const void* __restrict__ draft, size_t rowbase, int hi, int K,
                               int (*s_rec)[kDraftThreads], int nrec, unsigned long long* s_key) {
    const int tid = threadIdx.x;
    int rounds = nrec;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) rounds = max(rounds, __shfl_xor(rounds, o, kWave));
    for (int r0 = 0; r0 < rounds; r0 += BATCH) {
        Raw8<DT> g[BATCH];
        int off[BATCH];
#pragma unroll
        for (int r = 0; r < BATCH; ++r) {
            off[r] = r0 + r < nrec ? s_rec[r0 + r][tid] : 0;
            if (r0 + r < nrec) load_raw8<DT, VEC>(draft, rowbase, off[r], hi, g[r]);
        }
#pragma unroll
        for (int r = 0; r < BATCH; ++r) {
            if (r0 + r >= rounds) break;
            float x[8];
            raw8_values<DT>(g[r], x);
            cb.offer8(x, off[r], hi, r0 + r < nrec, K, s_key);
        }
    }
}

// Evaluated path of the normaliser for one logit (scaled value a): running
// maximum m and sum of e^(a - m); NaN and +inf set bad, -inf adds nothing.
__device__ __forceinline__ void eval_term(float a, float& m, double& sum, bool& bad, const double* et) {
    if (__builtin_amdgcn_classf(a, 0x203)) {  // signalling NaN, quiet NaN, +inf
        bad = true;
        return;
    }
    if (a == -INFINITY) return;
    if (a > m) {
        sum = (m == -INFINITY) ? 1.0 : sum * exp64((double)m - (double)a, et) + 1.0;
        m = a;
    } else {
        sum += exp64((double)a - (double)m, et);
    }
}

// Table part of the normaliser for the two bf16 patterns of a word, with
// packed 16-bit arithmetic: adds their entries to s0 and s1 (0.0 outside the
// table) and keeps the running packed maximum of the unclamped indices
// (a half at or above kTabHalf is a pattern outside the table; patterns below
// it wrap to large indices). Clamped indices stay below 2^12, so one 32-bit
// shift by 3 scales both halves.
typedef unsigned short tsb_u16x2 __attribute__((ext_vector_type(2)));
typedef short tsb_i16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void tab_word(uint32_t w, const double* tab, double& s0, double& s1, tsb_u16x2& tmax) {
    const tsb_u16x2 base = {(unsigned short)kTabBase, (unsigned short)kTabBase};
    const tsb_u16x2 lim = {(unsigned short)kTabHalf, (unsigned short)kTabHalf};
    const tsb_u16x2 t = __builtin_bit_cast(tsb_u16x2, w & 0x7FFF7FFFu) - base;
    tmax = __builtin_elementwise_max(tmax, t);
    const tsb_u16x2 tc = __builtin_elementwise_min(t, lim);
    const uint32_t off = (__builtin_bit_cast(uint32_t, tc) << 3) | (w & 0x80008000u);
    s0 += *(const double*)((const char*)tab + (off & 0xFFFFu));
    s1 += *(const double*)((const char*)tab + (off >> 16));
}

// Order-preserving signed 16-bit keys of the two bf16 patterns of a word
// (a larger value has a larger key; -0 sits just below +0; NaN patterns sit
// above +inf or below -inf by their sign).
__device__ __forceinline__ tsb_i16x2 bf16_keys(uint32_t w) {
    const tsb_i16x2 v = __builtin_bit_cast(tsb_i16x2, w);
    const tsb_i16x2 sgn = v >> (tsb_i16x2){15, 15};  // 0 or -1 per half
    return v ^ (sgn & (tsb_i16x2){0x7FFF, 0x7FFF});
}

// Key of the smallest bf16 value at least x (x not NaN): the pattern of a
// positive x rounded up, of a negative x truncated toward zero.
__device__ __forceinline__ int bf16_key_at_least(float x) {
    const uint32_t b = __float_as_uint(x);
    const uint32_t p = (b >> 31) ? (b >> 16) : ((b + 0xFFFFu) >> 16);
    const int v = (int)(short)(uint16_t)p;
    return v < 0 ? v ^ 0x7FFF : v;
}

// Whether some logit of the group (four words of bf16 pairs) has a key above
// kf (k2 = kf in both halves).
__device__ __forceinline__ bool group_reaches(const uint32_t (&w)[4], tsb_i16x2 k2) {
    const tsb_i16x2 a = __builtin_elementwise_max(bf16_keys(w[0]), bf16_keys(w[1]));
    const tsb_i16x2 b = __builtin_elementwise_max(bf16_keys(w[2]), bf16_keys(w[3]));
    const tsb_i16x2 m = __builtin_elementwise_max(__builtin_elementwise_max(a, b), k2);
    return __builtin_bit_cast(uint32_t, m) != __builtin_bit_cast(uint32_t, k2);
}

// Per-workgroup-lane state of the draft stream: candidate buffer, recorded
// groups, normaliser parts and the LDS tables.
template <int CAP>
struct DraftState {
    CandBuf<CAP>& cb;
    const void* draft;
    size_t rowbase;
    int hi, K;
    float invT;
    bool use_tab;
    const double* tab_lds;
    const double* exp_lds;
    int (*rec)[kDraftThreads];
    unsigned long long* key;
    uint16_t* special;      // table path: the wave's deferred patterns outside the table
    int nrec = 0;           // groups recorded by this lane
    int nspecial = 0;       // deferred patterns (wave-uniform; past kSpecialCap: the list overflowed)
    bool rec_full = false;  // table path: a group passed with this lane's list full
    double sumF = 0.0;      // sum of table entries (reference 0)
    float m = -INFINITY;    // evaluated path: running maximum of the scaled logits
    double sum = 0.0;       // evaluated path: sum of e^(a - m)
    bool bad = false;       // a NaN or +inf scaled logit
};

// Records a candidate group in this lane's list. With the normaliser the
// stream never flushes (the stream's registers are taken): a lane whose list
// is full marks itself and offers its part of the segment again at the end.
// The pool selection flushes between chunks instead (its first filter is
// weak, so its lists fill).
template <bool STATS, int CAP>
__device__ __forceinline__ void record_group(DraftState<CAP>& St, int i0) {
    if (!STATS || St.nrec < rec_slots<STATS>()) {
        St.rec[St.nrec][threadIdx.x] = i0;
        ++St.nrec;
    } else {
        St.rec_full = true;
    }
}

// One chunk held in r, starting at base: normaliser terms, finiteness and
// the recording of candidate groups.
template <int DT, bool VEC, bool STATS, bool TAB, int CAP>
__device__ __forceinline__ void draft_chunk(const Raw8<DT> (&r)[kDraftU], int base, DraftState<CAP>& St) {
    if constexpr (TAB) {
      {
        // table sum on packed pairs, four independent binary64 chains
        tsb_u16x2 tmax = {0, 0};
        double s4[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int u = 0; u < kDraftU; ++u)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int c = 2 * ((u * 4 + j) & 1);
                tab_word(r[u].w[j], St.tab_lds, s4[c], s4[c + 1], tmax);
                // eight table lookups in flight at a time (a whole chunk's
                // would not fit the registers)
                if (j == 3) __builtin_amdgcn_sched_barrier(0);
            }
        St.sumF += (s4[0] + s4[1]) + (s4[2] + s4[3]);
        // patterns outside the table (rare; -inf adds nothing) are deferred
        // to the wave's list and evaluated after the stream
        const bool slow = (uint32_t)__builtin_elementwise_max(tmax.x, tmax.y) >= (uint32_t)kTabHalf;
        if (__ballot(slow)) {
#pragma unroll
            for (int q = 0; q < 4 * kDraftU; ++q)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const uint32_t p = (r[q >> 2].w[q & 3] >> (16 * h)) & 0xFFFFu;
                    const bool out = ((p & 0x7FFFu) - kTabBase) >= (uint32_t)kTabHalf && p != 0xFF80u;
                    const uint64_t b = __ballot(out);
                    if (b) {
                        if (out && St.nspecial + __popcll(b) <= kSpecialCap)
                            St.special[St.nspecial + lanes_below_u64(b)] = (uint16_t)p;
                        St.nspecial = min(St.nspecial + __popcll(b), kSpecialCap + 1);
                    }
                }
        }
        // candidates: a group is recorded when one of its logits reaches the
        // filter, by order-preserving 16-bit keys
        const int kf = bf16_key_at_least(St.cb.fx) - 1;
        const tsb_i16x2 k2 = {(short)kf, (short)kf};
#pragma unroll
        for (int u = 0; u < kDraftU; ++u)
            if (group_reaches(r[u].w, k2)) record_group<STATS>(St, base + (u * kDraftThreads + (int)threadIdx.x) * 8);
        return;
      }
    }
#pragma unroll
    for (int u = 0; u < kDraftU; ++u) {
        const int i0 = base + (u * kDraftThreads + (int)threadIdx.x) * 8;
        float x[8];
        raw8_values<DT>(r[u], x);
        if (STATS) {
            // evaluated path for every logit: rescale once per group
            float a[8];
            float am = -INFINITY;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                a[j] = x[j] * St.invT;
                St.bad |= __builtin_amdgcn_classf(a[j], 0x203);
                am = fmaxf(am, a[j]);  // NaN is ignored
            }
            if (am > St.m && am < INFINITY) {
                St.sum = (St.m == -INFINITY) ? 0.0 : St.sum * exp64((double)St.m - (double)am, St.exp_lds);
                St.m = am;
            }
            const double md = (double)St.m;
            double s2[2] = {0.0, 0.0};
#pragma unroll
            for (int j = 0; j < 8; ++j) s2[j & 1] += exp64((double)a[j] - md, St.exp_lds);
            St.sum += s2[0] + s2[1];
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) St.bad |= __builtin_amdgcn_classf(x[j] * St.invT, 0x203);
        }
        // candidates: record the group if its maximum passes (its
        // smallest id is i0)
        float xm = x[0];
#pragma unroll
        for (int j = 1; j < 8; ++j) xm = fmaxf(xm, x[j]);  // NaN is ignored
        if (St.cb.pass(xm, (uint32_t)i0)) record_group<STATS>(St, i0);
    }
}

// Per chunk, after draft_chunk: the filter shared by the other waves and the
// flush of the recorded groups when some lane's list is nearly full.
template <int DT, bool VEC, bool STATS, bool TAB, int CAP>
__device__ __forceinline__ void draft_chunk_tail(DraftState<CAP>& St) {
    {
        // an LDS load (a generic volatile load would also wait for the
        // chunks in flight)
        const uint64_t sk = __hip_atomic_load(St.key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (sk) St.cb.raise_to(sk);
    }
    if constexpr (!STATS) {
        if (__ballot(St.nrec > rec_slots<STATS>() - kDraftU)) {
            flush_recorded<DT, VEC, CAP>(St.cb, St.draft, St.rowbase, St.hi, St.K, St.rec, St.nrec, St.key);
            St.nrec = 0;
        }
    }
}

// Issues the loads of the chunk at `base` (nothing at or past hi): a chunk
// that lies wholly inside the segment is read with unconditional vector loads
// (a wave-uniform choice), a last partial chunk with per-position bounds.
template <int DT, bool VEC>
__device__ __forceinline__ void issue_chunk(const void* __restrict__ draft, size_t rowbase, int base, int hi, int tid,
                                            Raw8<DT> (&r)[kDraftU]) {
    if (VEC && base + kDraftChunk <= hi)
        load_chunk<DT>(draft, rowbase, base, tid, r);
    else if (base < hi)
        load_chunk_masked<DT, VEC>(draft, rowbase, base, hi, tid, r);
}

// Number of keys of a descending list of n (<= 64) distinct keys in LDS that
// are larger than k.
__device__ __forceinline__ int count_larger(const uint64_t* list, int n, uint64_t k) {
    int pos = 0;
#pragma unroll
    for (int step = 64; step > 0; step >>= 1)
        if (pos + step <= n && list[pos + step - 1] > k) pos += step;
    return pos;
}

// STATS = false is the pool selection: the same candidate lists (K = pool
// size) and finiteness flags without the normaliser (pm, ps unused).
template <int DT, bool VEC, bool STATS, bool TAB>
__global__ __launch_bounds__(kDraftThreads) __attribute__((amdgpu_waves_per_eu(4))) void draft_partials(const void* __restrict__ draft, int V, int D,
                                                                int seg, int S, float invT, int K,
                                                                float* __restrict__ pm, double* __restrict__ ps,
                                                                uint64_t* __restrict__ pk, int* __restrict__ pf,
                                                                int32_t* __restrict__ req_status) {
    const int s = blockIdx.x;
    const int row = blockIdx.y;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    if (s == 0 && (row % D) == 0 && tid == 0) req_status[row / D] = 0;

    const size_t rowbase = (size_t)row * (size_t)V;
    const int lo = s * seg;
    const int hi = min(V, lo + seg);
    static_assert(!TAB || (DT == TSB_BF16 && STATS), "the table path is for bf16 rows with the normaliser");

    // the first chunk is in flight before anything else is done
    Raw8<DT> rA[kDraftU];
    issue_chunk<DT, VEC>(draft, rowbase, lo, hi, tid, rA);

    // bf16 rows with the normaliser: the exponential table, with the exp64
    // table and the column maxima in its gap; otherwise the exp64 table and
    // the column maxima on their own. One LDS block with the table first, so
    // that table offsets fit the immediate offset of an LDS load.
    constexpr bool kTabbed = TAB;
    constexpr int CAP = cand_cap<STATS>();
    static_assert(!kTabbed || kTabGap + kExpTable + kDraftThreads / 2 + kDraftWaves * kSpecialCap / 4 <= kTabNeg,
                  "the gap holds the exp64 table, the column maxima and the deferred patterns");
    struct Lds {
        double tab[kTabbed ? kTabDoubles : kExpTable + kDraftThreads / 2];
        uint64_t buf[kDraftWaves][CAP];
        int rec[rec_slots<STATS>()][kDraftThreads];
        int n[kDraftWaves];
        float m[kDraftWaves];
        double s[kDraftWaves];
        int bad[kDraftWaves];
        unsigned long long key;
    };
    __shared__ Lds L;
    double* const s_tab = L.tab;
    double* const s_exp = kTabbed ? s_tab + kTabGap : s_tab;
    float (*const s_lm)[kWave] = (float (*)[kWave])(s_exp + kExpTable);
    // (the table path only: its deferred out-of-table patterns, in the gap)
    uint16_t* const s_special = (uint16_t*)(s_exp + kExpTable + kDraftThreads / 2) + wave * kSpecialCap;
    if (STATS) {
        for (int j = tid; j < kExpTable; j += kDraftThreads) s_exp[j] = exp2((double)j / (double)kExpTable);
        __syncthreads();
        if (TAB) {
            for (int i = tid; i < 2 * (kTabHalf + 1); i += kDraftThreads) {
                const int sg = i >= kTabHalf + 1;
                const int t = i - sg * (kTabHalf + 1);
                const uint32_t h = (kTabBase + (uint32_t)t) | ((uint32_t)sg << 15);
                s_tab[sg * kTabNeg + t] = t < kTabHalf ? exp64((double)(__uint_as_float(h << 16) * invT), s_exp) : 0.0;
            }
        }
    }

    CandBuf<CAP> cb;
    cb.buf = L.buf[wave];
    cb.n = 0;
    cb.fid = 0xFFFFFFFFu;
    {
        // the first filter, from the first chunk's column maxima (the barrier
        // also orders the tables before their first use)
        float lm = -INFINITY;
#pragma unroll
        for (int u = 0; u < kDraftU; ++u) {
            float x[8];
            raw8_values<DT>(rA[u], x);
#pragma unroll
            for (int j = 0; j < 8; ++j) lm = fmaxf(lm, x[j]);
        }
        s_lm[wave][lane] = isnan(lm) ? -INFINITY : lm;
        if (tid == 0) L.key = 0ull;
        __syncthreads();
        if (K <= 16) {
            float cm = s_lm[0][lane];
#pragma unroll
            for (int w = 1; w < kDraftWaves; ++w) cm = fmaxf(cm, s_lm[w][lane]);
            cb.fx = wave_kth_largest_sorted(cm, K);
        } else {
            // large K: the K-th largest of the 512 lane maxima (each over
            // distinct logits), by a radix selection on their ordered bits
            uint32_t kb[kDraftWaves];
#pragma unroll
            for (int w = 0; w < kDraftWaves; ++w) kb[w] = ordered_bits(s_lm[w][lane]);
            uint32_t t = 0;
            for (int bit = 31; bit >= 0; --bit) {
                const uint32_t cand = t | (1u << bit);
                int cnt = 0;
#pragma unroll
                for (int w = 0; w < kDraftWaves; ++w) cnt += __popcll(__ballot(kb[w] >= cand));
                if (cnt >= K) t = cand;
            }
            cb.fx = from_ordered_bits(t);
        }
    }

    DraftState<CAP> St{cb, draft, rowbase, hi, K, invT, TAB, s_tab, s_exp, L.rec, &L.key, s_special};
    for (int base = lo; base < hi; base += kDraftChunk) {
        // the next chunk's loads are issued before this one is processed
        Raw8<DT> rB[kDraftU];
        issue_chunk<DT, VEC>(draft, rowbase, base + kDraftChunk, hi, tid, rB);
        draft_chunk<DT, VEC, STATS, TAB, CAP>(rA, base, St);
        draft_chunk_tail<DT, VEC, STATS, TAB, CAP>(St);
#pragma unroll
        for (int u = 0; u < kDraftU; ++u) rA[u] = rB[u];
    }
    flush_recorded<DT, VEC, CAP, STATS ? 8 : kRecBatch>(St.cb, draft, rowbase, hi, K, L.rec, St.nrec, &L.key);
    if constexpr (STATS) {
        if (__ballot(St.rec_full)) {
            // a lane whose list ran full offers every group of its part of
            // the segment again (the filter only rose since)
            for (int base = lo; base < hi; base += kDraftChunk) {
#pragma unroll
                for (int u = 0; u < kDraftU; ++u) {
                    const int i0 = base + (u * kDraftThreads + tid) * 8;
                    Raw8<DT> g;
                    const bool live = St.rec_full && i0 < hi;
                    if (live) {
                        load_raw8<DT, VEC>(draft, rowbase, i0, hi, g);
                    } else {
#pragma unroll
                        for (int j = 0; j < (DT == TSB_BF16 ? 4 : 8); ++j)
                            g.w[j] = DT == TSB_BF16 ? 0xFF80FF80u : 0xFF800000u;
                    }
                    float x[8];
                    raw8_values<DT>(g, x);
                    St.cb.offer8(x, i0, hi, live, K, &L.key);
                }
            }
        }
        if (TAB && St.nspecial > 0) {
            // the deferred patterns, one per lane at a time; a wave whose list
            // overflowed reads its part of the segment again instead
            wave_lds_fence();
            if (St.nspecial <= kSpecialCap) {
                for (int i = lane; i < St.nspecial; i += kWave)
                    eval_term(__uint_as_float((uint32_t)s_special[i] << 16) * invT, St.m, St.sum, St.bad, s_exp);
            } else {
                for (int base = lo; base < hi; base += kDraftChunk) {
                    Raw8<DT> rr[kDraftU];
                    issue_chunk<DT, VEC>(draft, rowbase, base, hi, tid, rr);
#pragma unroll
                    for (int u = 0; u < kDraftU; ++u)
#pragma unroll
                        for (int j = 0; j < 8; ++j) {
                            const uint32_t p = (rr[u].w[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
                            const bool out = ((p & 0x7FFFu) - kTabBase) >= (uint32_t)kTabHalf && p != 0xFF80u &&
                                             base + (u * kDraftThreads + tid) * 8 + j < hi;
                            if (out) eval_term(__uint_as_float(p << 16) * invT, St.m, St.sum, St.bad, s_exp);
                        }
                }
            }
        }
    }

    // lane partial: reference Ml (0 for the table part) and the sum relative
    // to it; exponentials only where references differ
    const bool anyF = St.sumF > 0.0;  // table entries are positive
    float Ml;
    double sl;
    if (St.m == -INFINITY) {
        Ml = anyF ? 0.0f : -INFINITY;
        sl = St.sumF;
    } else if (!anyF) {
        Ml = St.m;
        sl = St.sum;
    } else {
        Ml = fmaxf(0.0f, St.m);
        sl = (Ml == 0.0f ? St.sumF : St.sumF * exp(-(double)Ml)) +
             (St.m == Ml ? St.sum : St.sum * exp((double)St.m - (double)Ml));
    }
    const float wm = wave_max(Ml);
    double contrib = 0.0;
    if (Ml != -INFINITY) {
        if (Ml == wm)
            contrib = sl;
        else
            contrib = sl * exp((double)Ml - (double)wm);
    }
    const double wsum = STATS ? wave_sum(contrib) : 0.0;
    const int wb = wave_or(St.bad);

    const int n = cb.n;
    if (lane == 0) {
        L.n[wave] = n;
        L.m[wave] = wm;
        L.s[wave] = wsum;
        L.bad[wave] = wb;
    }
    __syncthreads();
    int total = 0;
#pragma unroll
    for (int w = 0; w < kDraftWaves; ++w) total += L.n[w];
    const size_t o = (size_t)row * S + s;
    if (total <= 2 * kWave) {
        // few entries: the rank of a key is the number of larger keys over
        // all the buffers; the segment's K best go to their slots
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int i = h * kWave + lane;
            if (i < n) {
                const uint64_t mine = cb.buf[i];
                int rank = 0;
                for (int w = 0; w < kDraftWaves; ++w) {
                    const int nw = L.n[w];
                    for (int j = 0; j < nw; ++j) rank += L.buf[w][j] > mine ? 1 : 0;
                }
                if (rank < K) pk[o * K + rank] = mine;
            }
        }
    } else {
        // every wave keeps its K best, sorted; a key's rank is its place in
        // its own list plus the number of larger keys in every other list
        uint64_t v[CAP / kWave];
#pragma unroll
        for (int i = 0; i < CAP / kWave; ++i) v[i] = i * kWave + lane < n ? cb.buf[i * kWave + lane] : 0ull;
        wave_sort_desc<CAP / kWave>(v);
        const uint64_t top = v[0];
        const int c = min(n, K);
        __syncthreads();
        if (lane < c) cb.buf[lane] = top;
        if (lane == 0) L.n[wave] = c;
        __syncthreads();
        if (lane < c) {
            int rank = lane;
#pragma unroll
            for (int w = 0; w < kDraftWaves; ++w)
                if (w != wave) rank += count_larger(L.buf[w], L.n[w], top);
            if (rank < K) pk[o * K + rank] = top;
        }
        total = 0;
#pragma unroll
        for (int w = 0; w < kDraftWaves; ++w) total += L.n[w];
    }
    // empty slots get 0
    if (tid >= total && tid < K) pk[o * K + tid] = 0ull;
    if (wave == 0) {
        // segment normaliser: lanes w < kDraftWaves hold wave w's partial
        const float mw = lane < kDraftWaves ? L.m[lane] : -INFINITY;
        const float M = wave_max(mw);
        double sw = 0.0;
        if (lane < kDraftWaves && mw != -INFINITY) {
            if (mw == M)
                sw = L.s[lane];
            else
                sw = L.s[lane] * exp((double)mw - (double)M);
        }
        const double tot = STATS ? wave_sum(sw) : 0.0;
        const int anybad = wave_or(lane < kDraftWaves ? L.bad[lane] : 0);
        if (lane == 0) {
            if (STATS) {
                pm[o] = M;
                ps[o] = tot;
            }
            pf[o] = anybad;
        }
    }
}

// ------------------------------------------------------------------ K2
// One workgroup of kPlanWaves waves per request.
//
// 1. Merge: each wave combines the segment partials of some draft rows into
//    the binary64 log-sum-exp, its canonical binary32 rounding and the K
//    planning candidates lp = fl32(a - lse32), kept in LDS.
// 2. Threshold search. The topology is the first B rank paths under the
//    static order (score desc, depth asc, rank path lexicographic asc), which
//    is what lazy best-first expansion commits (Section 3.1; Appendix B.3).
//    With t* the (B+1)-th largest path score, it is every node scoring above
//    t* plus the first B - #(above t*) nodes scoring exactly t*, taken in
//    (depth, rank path) order. Path scores never increase from a node to its
//    children or younger siblings (lp <= 0, sorted by rank), so the nodes
//    scoring at least a threshold form a subtree that a level-by-level count
//    enumerates. Each wave counts one candidate threshold per round:
//      - hi: a threshold with count(hi) <= B, and m(hi), the largest node
//        score below hi (count(m(hi)) > count(hi));
//      - wave 0 counts at m(hi); if that reaches B + 1, t* = m(hi);
//      - the other waves count at thresholds spread below m(hi); a count in
//        [B + 1, cap] has every node scoring at least its threshold in LDS,
//        and t* is selected among them;
//      - otherwise hi moves to the lowest threshold that counted <= B (its
//        count grows by at least one per round, so rounds end).
// 3. Emission: one wave enumerates the admitted nodes level by level in
//    (depth, rank path) order, which is the BFS canonical order: parents in
//    order, children by rank. Chosen children form a prefix of each parent's
//    children.
constexpr int kPlanWaves = 16;
constexpr int kPlanThreads = kPlanWaves * kWave;
static_assert(kPlanThreads == kChainThreads, "the chain rows run on the planner's workgroups");
constexpr int kChainGridMax = 1024;  // workgroups for the chain rows beside the planner
constexpr int kPlanBuf = 12288;  // binary64 slots shared by the counting waves

struct PlanShared {
    float lp[TSB_MAX_D * TSB_MAX_K];
    int kfin[TSB_MAX_D];  // finite candidates per row (a prefix: -inf sorts last)
    int bad;
    double piv[kPlanWaves];
    double mval[kPlanWaves];
    int cnt[kPlanWaves];
    double tstar;
    int g;
    union {
        double buf[kPlanBuf];
        struct {
            double score[TSB_MAX_B + 1];
            int par[TSB_MAX_B + 1];
            int rank[TSB_MAX_B + 1];
            int depth[TSB_MAX_B + 1];
            int nch[TSB_MAX_B + 1];
            int fc[TSB_MAX_B + 1];
        } t;
    } u;
};

__device__ __forceinline__ double wave_max_f64(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, kWave));
    return v;
}
__device__ __forceinline__ double wave_min_f64(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmin(v, __shfl_xor(v, o, kWave));
    return v;
}

// Merge of one draft row (one wave): log-sum-exp from the segment partials
// in a fixed order, candidates from the segment lists.
template <typename SH>
__device__ void merge_row(SH& sh, int row, int rrow, int S, int K, float invT, const float* __restrict__ pm,
                          const double* __restrict__ ps, const uint64_t* __restrict__ pk,
                          const int* __restrict__ pf, double* __restrict__ draft_lse,
                          int32_t* __restrict__ topk_tok, float* __restrict__ topk_lp) {
    const int lane = lane_id();
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

    const int n = S * K;
    uint64_t best;  // lane j < K: the j-th best candidate of the row
    if (n <= kWave) {
        // one candidate per lane: its rank is the number of larger keys (keys
        // are distinct, empty slots are 0); all lanes in parallel
        const uint64_t mine = lane < n ? pk[o * K + lane] : 0;
        int rank = 0;
        for (int j = 0; j < n; ++j) rank += lane_u64(mine, j) > mine ? 1 : 0;
        __shared__ uint64_t s_rank[kPlanWaves][kWave];
        uint64_t* sr = s_rank[threadIdx.x / kWave];
        sr[lane] = 0;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        if (mine != 0 && rank < K) sr[rank] = mine;
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        best = sr[lane];
    } else {
        WaveTopList top;
        top.init(K);
        for (int base = 0; base < n; base += kWave) {
            const int i = base + lane;
            const uint64_t k = i < n ? pk[o * K + i] : 0;
            top.offer(k, i < n && k != 0);
        }
        best = top.v;
    }

    const bool nonfinite = bad || M == -INFINITY;
    const double l64 = nonfinite ? (double)NAN : (double)M + log(tot);
    const float l32 = (float)l64;
    float lp = -INFINITY;
    if (lane < K) {
        const uint64_t k = best;
        const float a = cand_value(k) * invT;
        lp = a - l32;
        topk_tok[(size_t)row * K + lane] = (int32_t)cand_id(k);
        topk_lp[(size_t)row * K + lane] = lp;
        sh.lp[rrow * K + lane] = lp;
    }
    const int nfin = __popcll(__ballot(lane < K && lp > -INFINITY && lp < INFINITY));
    if (lane == 0) {
        draft_lse[row] = l64;
        sh.kfin[rrow] = nfin;
        if (nonfinite) atomicOr(&sh.bad, 1);
    }
}

// Number of nodes (root excluded) scoring at least tau, level by level, with
// their scores stored in buf; cap + 1 once more than cap. m_out: the largest
// node score below tau (-inf if none; meaningful without overflow). Lane l
// takes candidate l % K of parent l / K, so a pass covers 64 / K parents and
// one ballot compacts the children that reach tau in (parent, rank) order.
__device__ __forceinline__ int lanes_below(uint64_t b) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0u));
}

__device__ int plan_count(const PlanShared& sh, int Dp, int K, double tau, int cap, double* buf, double& m_out) {
    const int lane = lane_id();
    const int per = kWave / K;  // parents per pass
    const int pp = lane / K, pj = lane - pp * K;
    int total = 0;
    int plo = 0, phi = 0;  // parents of the current level in buf; level 0: the root
    double m = -INFINITY;
    for (int k = 0; k < Dp; ++k) {
        const int kk = sh.kfin[k];
        const bool cand = pp < per && pj < kk;
        const double lpj = cand ? (double)sh.lp[k * K + pj] : -INFINITY;
        const int np = k == 0 ? 1 : phi - plo;
        const int nstart = total;
        for (int base = 0; base < np; base += per) {
            const int i = base + pp;
            const bool valid = cand && i < np;
            const double s = (valid && k > 0) ? buf[plo + i] : 0.0;
            const double cs = s + lpj;
            const bool ok = valid && cs >= tau;
            if (valid && !ok) m = fmax(m, cs);  // children below tau (the best of them counts)
            const uint64_t b = __ballot(ok);
            const int cnt = __popcll(b);
            if (total + cnt > cap) {
                m_out = -INFINITY;
                return cap + 1;
            }
            if (ok) buf[total + lanes_below(b)] = cs;
            total += cnt;
        }
        __threadfence_block();  // the next level reads these scores from other lanes
        plo = nstart;
        phi = total;
        if (phi == plo) break;
    }
    m_out = wave_max_f64(m);
    return total;
}

__global__ __launch_bounds__(kPlanThreads) void plan_tree(int D, int S, int K, int B, float invT,
                                                          const float* __restrict__ pm,
                                                          const double* __restrict__ ps,
                                                          const uint64_t* __restrict__ pk,
                                                          const int* __restrict__ pf, double* __restrict__ draft_lse,
                                                          int32_t* __restrict__ topk_tok,
                                                          float* __restrict__ topk_lp, tsb_tree tree,
                                                          int32_t* __restrict__ req_status,
                                                          unsigned long long* __restrict__ stats, int R,
                                                          ChainJob cj) {
    if ((int)blockIdx.x >= R) {
        // the chain rows, on the workgroups after the requests'
        for (int g = (int)blockIdx.x - R; g < cj.items; g += (int)gridDim.x - R) {
            if (cj.bf16)
                cj.vec ? chain_piece<TSB_BF16, true>(g, cj.target, cj.V, cj.B, invT, cj.cm, cj.cs, cj.cf)
                       : chain_piece<TSB_BF16, false>(g, cj.target, cj.V, cj.B, invT, cj.cm, cj.cs, cj.cf);
            else
                cj.vec ? chain_piece<TSB_F32, true>(g, cj.target, cj.V, cj.B, invT, cj.cm, cj.cs, cj.cf)
                       : chain_piece<TSB_F32, false>(g, cj.target, cj.V, cj.B, invT, cj.cm, cj.cs, cj.cf);
        }
        return;
    }
    __shared__ PlanShared sh;
    const int r = blockIdx.x;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    unsigned long long t_start = 0, t_merge = 0, t_search = 0;  // work counters (thread 0)
    int n_rounds = 0;
    if (stats && tid == 0) t_start = __builtin_amdgcn_s_memrealtime();

    if (tid == 0) sh.bad = 0;
    __syncthreads();
    for (int d = wave; d < D; d += kPlanWaves)
        merge_row(sh, r * D + d, d, S, K, invT, pm, ps, pk, pf, draft_lse, topk_tok, topk_lp);
    __syncthreads();
    if (stats && tid == 0) t_merge = __builtin_amdgcn_s_memrealtime();
    const bool nonfinite = sh.bad != 0;
    const int Dp = nonfinite ? 0 : D;

    // ---- threshold search (uniform control flow across the workgroup)
    // a count succeeds when it lands in [B + 1, cap]: a narrow window keeps
    // every count short (measured best at 1.25 (B + 1) over the workloads),
    // at the price of a round more now and then
    const int cap = (5 * (B + 1) + 3) / 4;
    const int ns = min(kPlanWaves, kPlanBuf / cap);
    double hi_m = (Dp > 0 && sh.kfin[0] > 0) ? (double)sh.lp[0] : -INFINITY;  // the best node's score
    int hi_cnt = 0;
    double lo = -INFINITY;
    int mode = 3;  // 1: t* = hi_m; 2: t* selected in a wave's buffer; 3: every node is chosen
    int src = -1;
    // every round raises count(hi) by at least one (at most B + 1 rounds); the
    // guard only bounds the loop
    for (int round = 0; hi_m > -INFINITY; ++round) {
        n_rounds = round + 1;
        if (round > B + 1) {
            mode = 1;
            break;
        }
        if (wave < ns) {
            const double tau = wave == 0 ? hi_m
                               : (lo > -INFINITY ? hi_m - (hi_m - lo) * ((double)wave / (double)ns)
                                                 : hi_m - 0.25 * exp2(0.5 * (double)(wave - 1)));
            double m;
            const int c = plan_count(sh, Dp, K, tau, cap, sh.u.buf + wave * cap, m);
            if (lane == 0) {
                sh.piv[wave] = tau;
                sh.cnt[wave] = c;
                sh.mval[wave] = m;
            }
        }
        __syncthreads();
        if (sh.cnt[0] >= B + 1) {
            mode = 1;
            break;
        }
        int best = -1;
        for (int w = 1; w < ns; ++w)
            if (sh.cnt[w] >= B + 1 && sh.cnt[w] <= cap && (best < 0 || sh.piv[w] > sh.piv[best])) best = w;
        if (best >= 0) {
            mode = 2;
            src = best;
            break;
        }
        int nh = 0;  // count(piv[0]) <= B here
        double nlo = lo;
        for (int w = 1; w < ns; ++w) {
            if (sh.cnt[w] <= B && sh.piv[w] < sh.piv[nh]) nh = w;
            if (sh.cnt[w] > cap && sh.piv[w] > nlo) nlo = sh.piv[w];
        }
        hi_cnt = sh.cnt[nh];
        hi_m = sh.mval[nh];
        lo = nlo;
        __syncthreads();
    }
    if (mode == 1) {
        if (tid == 0) {
            sh.tstar = hi_m;
            sh.g = hi_cnt;
        }
    } else if (mode == 2) {
        const int c = sh.cnt[src];
        const double* b = sh.u.buf + src * cap;
        for (int i = tid; i < c; i += kPlanThreads) {
            const double v = b[i];
            int gt = 0, ge = 0;
            for (int j = 0; j < c; ++j) {
                const double w = b[j];
                gt += w > v ? 1 : 0;
                ge += w >= v ? 1 : 0;
            }
            if (gt <= B && ge >= B + 1) {  // every such thread holds the same value
                sh.tstar = v;
                sh.g = gt;
            }
        }
    } else if (tid == 0) {
        sh.tstar = -INFINITY;  // every node scores above it
        sh.g = 0;
    }
    __syncthreads();
    if (wave != 0) return;
    if (stats && tid == 0) t_search = __builtin_amdgcn_s_memrealtime();

    // ---- emission in BFS order (wave 0)
    const double tstar = sh.tstar;
    int quota = mode == 3 ? 0 : B - sh.g;  // nodes scoring exactly t* still admitted
    bool tie_admitted = false;
    double minsc = INFINITY;
    if (lane == 0) {
        sh.u.t.score[0] = 0.0;
        sh.u.t.par[0] = -1;
        sh.u.t.rank[0] = -1;
        sh.u.t.depth[0] = 0;
    }
    // lane l takes candidate l % K of parent l / K (as in plan_count); the
    // admitted children of a parent are a prefix of its candidates
    const int per = kWave / K;
    const int pp = lane / K, pj = lane - pp * K;
    int n = 1, plo = 0, phi = 1;
    for (int k = 0; k < Dp && plo < phi; ++k) {
        const int kk = sh.kfin[k];
        const bool cand = pp < per && pj < kk;
        const double lpj = cand ? (double)sh.lp[k * K + pj] : -INFINITY;
        for (int base = plo; base < phi; base += per) {
            const int i = base + pp;
            const bool par_ok = pp < per && i < phi;
            const bool valid = cand && i < phi;
            const double s = par_ok ? sh.u.t.score[i] : 0.0;
            const double cs = s + lpj;
            const bool gt = valid && cs > tstar;
            const bool eq = valid && cs == tstar;
            // nodes scoring exactly t* are admitted in (depth, rank path) order,
            // which is lane order here
            const uint64_t beq = __ballot(eq);
            const int etot = __popcll(beq);
            const bool adm = gt || (eq && lanes_below(beq) < quota);
            if (etot > 0 && quota > 0) tie_admitted = true;
            quota -= min(etot, quota);
            const uint64_t b = __ballot(adm);
            if (adm) {
                const int x = n + lanes_below(b);
                if (x <= B) {  // always true: the admitted nodes number at most B
                    sh.u.t.score[x] = cs;
                    sh.u.t.par[x] = i;
                    sh.u.t.rank[x] = pj;
                    sh.u.t.depth[x] = k + 1;
                    minsc = fmin(minsc, cs);
                }
            }
            if (par_ok && pj == 0) {
                const uint64_t seg = (K >= 64 ? ~0ull : ((1ull << K) - 1ull)) << (pp * K);
                const int c = __popcll(b & seg);
                sh.u.t.nch[i] = c;
                sh.u.t.fc[i] = c ? n + __popcll(b & ((1ull << (pp * K)) - 1ull)) : -1;
            }
            n = min(n + __popcll(b), B + 1);
        }
        __threadfence_block();
        plo = phi;
        phi = n;
    }
    for (int i = plo + lane; i < phi; i += kWave) {  // the last level has no children
        sh.u.t.nch[i] = 0;
        sh.u.t.fc[i] = -1;
    }
    minsc = wave_min_f64(minsc);

    const size_t o = (size_t)r * (B + 1);
    for (int i = lane; i < B + 1; i += kWave) {
        if (i < n) {
            tree.parent[o + i] = sh.u.t.par[i];
            tree.depth[o + i] = sh.u.t.depth[i];
            tree.rank[o + i] = sh.u.t.rank[i];
            tree.score[o + i] = sh.u.t.score[i];
            tree.n_children[o + i] = sh.u.t.nch[i];
            tree.first_child[o + i] = sh.u.t.fc[i];
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
        // margin: score of the B-th node in the order minus that of the (B+1)-th
        double margin = (double)INFINITY;
        if (mode != 3 && n > 1) margin = (tie_admitted ? tstar : minsc) - tstar;
        tree.n_nodes[r] = n;
        tree.plan_margin[r] = margin;
        int st = req_status[r];
        if (nonfinite) st |= TSB_REQ_NONFINITE;
        else if (n < B + 1) st |= TSB_REQ_BUDGET_SHORT;
        req_status[r] = st;
        if (stats) {
            const unsigned long long t_end = __builtin_amdgcn_s_memrealtime();
            atomicAdd(&stats[kStPlanRequests], 1ull);
            atomicAdd(&stats[kStPlanMergeTicks], t_merge - t_start);
            atomicAdd(&stats[kStPlanSearchTicks], t_search - t_merge);
            atomicAdd(&stats[kStPlanEmitTicks], t_end - t_search);
            atomicAdd(&stats[kStPlanRounds], (unsigned long long)n_rounds);
        }
    }
}

// ------------------------------------------------------------------ K2b
// Expand-then-prune first pass (Section 3.1; Appendix B.3), one workgroup of
// kPlanWaves waves per request. Layer 1 is the root's children; the frontier
// of a layer is its W best nodes (score desc, rank path lex asc); the next
// layer holds every child of every frontier node; the tree is the first B of
// all generated nodes (score desc, depth asc, rank path lex asc).
//
// Layers are stored one after another, each in rank-path lexicographic order
// (a child of the frontier node that is f-th in lexicographic order, rank j,
// sits at f * K_d + j), so the storage order is the order of (depth, path):
// ties on score are resolved by storage index, and the chosen nodes in
// storage order are the BFS order of the tree.
constexpr int kEpMax = 6144;  // generated nodes held in LDS

struct EpShared {
    float lp[TSB_MAX_D * TSB_MAX_K];
    int kfin[TSB_MAX_D];
    int bad;
    double score[kEpMax];
    int16_t par[kEpMax];  // storage index of the parent, -1 for the root
    int16_t pos[kEpMax];  // scratch positions, then BFS index
    int16_t nch[kEpMax];
    int16_t fc[kEpMax];
    uint8_t rank[kEpMax];
    uint8_t depth[kEpMax];
    uint8_t flag[kEpMax];
    int16_t front[kEpFrontierLimit];
    int lstart[TSB_MAX_D + 1];
    uint64_t lists[kPlanWaves][kWave];
    uint32_t hist[256];
    int wsum[kPlanWaves];
    double wmax[kPlanWaves];
    int cnt;
    uint64_t tkey;
    int root_nch, root_fc;
};

constexpr uint8_t kEpFront = 1, kEpTie = 2, kEpChosen = 4, kEpAbove = 8;

// Positions of the elements of [lo, hi) whose flag has `bit`, in index order
// (pos[i] for those elements); returns their number. Called by all threads.
__device__ int ep_scan(EpShared& sh, uint8_t bit, int lo, int hi) {
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int per = (hi - lo + kPlanThreads - 1) / kPlanThreads;
    const int b = lo + tid * per, e = min(hi, b + per);
    int c = 0;
    for (int i = b; i < e; ++i) c += (sh.flag[i] & bit) ? 1 : 0;
    int incl = c;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int t = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += t;
    }
    if (lane == kWave - 1) sh.wsum[wave] = incl;
    __syncthreads();
    int base = 0, total = 0;
    for (int w = 0; w < kPlanWaves; ++w) {
        base += w < wave ? sh.wsum[w] : 0;
        total += sh.wsum[w];
    }
    int run = base + incl - c;
    for (int i = b; i < e; ++i)
        if (sh.flag[i] & bit) sh.pos[i] = (int16_t)run++;
    __syncthreads();
    return total;
}

// Number of elements of [lo, hi) whose flag has `bit` (all threads).
__device__ int ep_count(EpShared& sh, uint8_t bit, int lo, int hi) {
    int c = 0;
    for (int i = lo + (int)threadIdx.x; i < hi; i += kPlanThreads) c += (sh.flag[i] & bit) ? 1 : 0;
    if (threadIdx.x == 0) sh.cnt = 0;
    __syncthreads();
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, kWave);
    if ((threadIdx.x % kWave) == 0 && c) atomicAdd(&sh.cnt, c);
    __syncthreads();
    const int t = sh.cnt;
    __syncthreads();
    return t;
}

__global__ __launch_bounds__(kPlanThreads) void plan_ep(int D, int S, int K, int B, int W, float invT,
                                                        const float* __restrict__ pm, const double* __restrict__ ps,
                                                        const uint64_t* __restrict__ pk, const int* __restrict__ pf,
                                                        double* __restrict__ draft_lse, int32_t* __restrict__ topk_tok,
                                                        float* __restrict__ topk_lp, tsb_tree tree,
                                                        int32_t* __restrict__ req_status) {
    __shared__ EpShared sh;
    const int r = blockIdx.x;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;

    if (tid == 0) sh.bad = 0;
    __syncthreads();
    for (int d = wave; d < D; d += kPlanWaves)
        merge_row(sh, r * D + d, d, S, K, invT, pm, ps, pk, pf, draft_lse, topk_tok, topk_lp);
    __syncthreads();
    const bool nonfinite = sh.bad != 0;
    const int Dp = nonfinite ? 0 : D;

    // layer of depth 1: the root's candidates
    const int k0 = Dp > 0 ? sh.kfin[0] : 0;
    for (int i = tid; i < k0; i += kPlanThreads) {
        sh.score[i] = (double)sh.lp[i];
        sh.par[i] = -1;
        sh.rank[i] = (uint8_t)i;
        sh.depth[i] = 1;
        sh.flag[i] = 0;
    }
    if (tid == 0) {
        sh.lstart[0] = 0;
        sh.lstart[1] = k0;
    }
    int ntot = k0, layers = k0 > 0 ? 1 : 0;
    __syncthreads();

    // expansion (wave 0 alone: a layer holds at most frontier * K nodes):
    // frontier of each layer, then its children
    if (wave == 0) {
        for (int d = 1; d < Dp; ++d) {
            const int lb = sh.lstart[d - 1], le = sh.lstart[d], nl = le - lb, kd = sh.kfin[d];
            if (nl == 0 || kd == 0) break;
            int f = 0;  // frontier nodes, listed in lexicographic (storage) order
            if (nl <= W) {
                for (int base = lb; base < le; base += kWave) {
                    const int i = base + lane;
                    if (i < le) sh.front[i - lb] = (int16_t)i;
                }
                f = nl;
            } else {
                // the W-th largest score of the layer (with multiplicity): a
                // sort of the layer's keys when it holds at most 128 nodes
                uint64_t tk;
                if (nl <= 2 * kWave && W <= kWave) {
                    uint64_t v[2];
#pragma unroll
                    for (int q = 0; q < 2; ++q) {
                        const int i = lb + q * kWave + lane;
                        v[q] = i < le ? ordered_bits64(sh.score[i]) : 0ull;
                    }
                    wave_sort_desc<2>(v);
                    tk = lane_u64(v[0], W - 1);
                } else {  // inserts (measured no slower than a 256-key sort)
                    WaveTopList tl;
                    tl.init(W);
                    for (int base = lb; base < le; base += kWave) {
                        const int i = base + lane;
                        tl.offer(i < le ? ordered_bits64(sh.score[i]) : 0ull, i < le);
                    }
                    tk = lane_u64(tl.v, W - 1);
                }
                int above = 0;
                for (int base = lb; base < le; base += kWave) {
                    const int i = base + lane;
                    above += __popcll(__ballot(i < le && ordered_bits64(sh.score[i]) > tk));
                }
                // nodes above the W-th score, then ties in lexicographic order
                int ties = 0;
                for (int base = lb; base < le; base += kWave) {
                    const int i = base + lane;
                    const uint64_t k = i < le ? ordered_bits64(sh.score[i]) : 0ull;
                    const bool tie = i < le && k == tk;
                    const uint64_t tb = __ballot(tie);
                    const int trank = ties + __popcll(tb & ((1ull << lane) - 1ull));
                    const bool in = (i < le && k > tk) || (tie && trank < W - above);
                    const uint64_t ib = __ballot(in);
                    if (in) sh.front[f + __popcll(ib & ((1ull << lane) - 1ull))] = (int16_t)i;
                    f += __popcll(ib);
                    ties += __popcll(tb);
                }
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            if (le + f * kd > kEpMax) break;  // the host bounds the generated nodes; never taken
            for (int t = lane; t < f * kd; t += kWave) {
                const int p = sh.front[t / kd], j = t % kd;
                const int c = le + t;
                sh.score[c] = sh.score[p] + (double)sh.lp[d * K + j];
                sh.par[c] = (int16_t)p;
                sh.rank[c] = (uint8_t)j;
                sh.depth[c] = (uint8_t)(d + 1);
                sh.flag[c] = 0;
            }
            if (lane == 0) sh.lstart[d + 1] = le + f * kd;
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            ntot = le + f * kd;
            layers = d + 1;
        }
        if (lane == 0) sh.cnt = ntot;
    }
    __syncthreads();
    ntot = sh.cnt;
    __syncthreads();
    for (int i = tid; i < ntot; i += kPlanThreads) sh.flag[i] &= (uint8_t)~(kEpFront | kEpTie);
    __syncthreads();

    // prune: the first B generated nodes
    double margin = (double)INFINITY;
    if (ntot <= B || B == 0) {
        if (B > 0)
            for (int i = tid; i < ntot; i += kPlanThreads) sh.flag[i] = kEpChosen;
        __syncthreads();
    } else {
        // t* = the B-th largest score, by radix selection on the ordered keys
        uint64_t prefix = 0ull;
        int remaining = B;
        for (int shift = 56; shift >= 0; shift -= 8) {
            for (int b = tid; b < 256; b += kPlanThreads) sh.hist[b] = 0u;
            __syncthreads();
            for (int i = tid; i < ntot; i += kPlanThreads) {
                const uint64_t k = ordered_bits64(sh.score[i]);
                if (shift == 56 || (k >> (shift + 8)) == prefix) atomicAdd(&sh.hist[(k >> shift) & 255u], 1u);
            }
            __syncthreads();
            if (wave == 0) {
                // lane l holds bins 255 - 4l .. 252 - 4l: counts from the top
                int c4[4], ls = 0;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    c4[q] = (int)sh.hist[255 - 4 * lane - q];
                    ls += c4[q];
                }
                int incl = ls;
#pragma unroll
                for (int o = 1; o < kWave; o <<= 1) {
                    const int t = __shfl_up(incl, o, kWave);
                    if (lane >= o) incl += t;
                }
                const uint64_t hit = __ballot(incl >= remaining);
                const int l0 = hit ? __ffsll((unsigned long long)hit) - 1 : kWave - 1;
                if (lane == l0) {
                    int acc = incl - ls, q = 0;
                    for (; q < 3; ++q) {
                        if (acc + c4[q] >= remaining) break;
                        acc += c4[q];
                    }
                    sh.cnt = remaining - acc;
                    sh.tkey = (prefix << 8) | (uint64_t)(255 - 4 * lane - q);
                }
            }
            __syncthreads();
            remaining = sh.cnt;
            prefix = sh.tkey;
            __syncthreads();
        }
        const uint64_t tk = prefix;
        double below = -INFINITY;
        for (int i = tid; i < ntot; i += kPlanThreads) {
            const uint64_t k = ordered_bits64(sh.score[i]);
            sh.flag[i] = k > tk ? (uint8_t)(kEpChosen | kEpAbove) : (k == tk ? kEpTie : 0);
            if (k < tk) below = fmax(below, sh.score[i]);
        }
        below = wave_max_f64(below);
        if (lane == 0) sh.wmax[wave] = below;
        __syncthreads();
        const int above = ep_count(sh, kEpAbove, 0, ntot);
        const int ties = ep_scan(sh, kEpTie, 0, ntot);
        const int need = B - above;
        for (int i = tid; i < ntot; i += kPlanThreads)
            if ((sh.flag[i] & kEpTie) && sh.pos[i] < need) sh.flag[i] |= kEpChosen;
        double bmax = -INFINITY;
        for (int w = 0; w < kPlanWaves; ++w) bmax = fmax(bmax, sh.wmax[w]);
        // the last chosen node scores t*; the next one ties or is the best below
        margin = ties > need ? 0.0 : from_ordered_bits64(tk) - bmax;
        __syncthreads();
    }

    // BFS positions: the chosen nodes in storage order
    const int n = ep_scan(sh, kEpChosen, 0, ntot) + 1;
    if (tid == 0) {
        sh.root_nch = 0;
        sh.root_fc = -1;
    }
    __syncthreads();
    // children of a node are a rank prefix stored together: the rank-0 child
    // gives the first child, the last chosen one the count
    for (int i = tid; i < ntot; i += kPlanThreads) {
        sh.nch[i] = 0;
        sh.fc[i] = -1;
    }
    __syncthreads();
    for (int i = tid; i < ntot; i += kPlanThreads) {
        if (!(sh.flag[i] & kEpChosen)) continue;
        const int p = sh.par[i];
        const int j = sh.rank[i];
        const int kd = sh.kfin[sh.depth[i] - 1];
        const bool last = j + 1 >= kd || !(sh.flag[i + 1] & kEpChosen);
        if (p >= 0) {
            if (j == 0) sh.fc[p] = (int16_t)(sh.pos[i] + 1);
            if (last) sh.nch[p] = (int16_t)(j + 1);
        } else {
            if (j == 0) sh.root_fc = sh.pos[i] + 1;
            if (last) sh.root_nch = j + 1;
        }
    }
    __syncthreads();

    const size_t o = (size_t)r * (B + 1);
    for (int i = tid; i < ntot; i += kPlanThreads) {
        if (!(sh.flag[i] & kEpChosen)) continue;
        const size_t x = o + sh.pos[i] + 1;
        const int p = sh.par[i];
        tree.parent[x] = p >= 0 ? sh.pos[p] + 1 : 0;
        tree.depth[x] = sh.depth[i];
        tree.rank[x] = sh.rank[i];
        tree.score[x] = sh.score[i];
        tree.n_children[x] = sh.nch[i];
        tree.first_child[x] = sh.fc[i];
    }
    for (int i = n + tid; i < B + 1; i += kPlanThreads) {
        tree.parent[o + i] = -1;
        tree.depth[o + i] = -1;
        tree.rank[o + i] = -1;
        tree.score[o + i] = 0.0;
        tree.n_children[o + i] = 0;
        tree.first_child[o + i] = -1;
    }
    if (tid == 0) {
        tree.parent[o] = -1;
        tree.depth[o] = 0;
        tree.rank[o] = -1;
        tree.score[o] = 0.0;
        tree.n_children[o] = sh.root_nch;
        tree.first_child[o] = sh.root_fc;
        tree.n_nodes[r] = n;
        tree.plan_margin[r] = n > 1 ? margin : (double)INFINITY;
        int st = req_status[r];
        if (nonfinite) st |= TSB_REQ_NONFINITE;
        else if (n < B + 1) st |= TSB_REQ_BUDGET_SHORT;
        req_status[r] = st;
    }
    (void)layers;
}

// ------------------------------------------------------------------ launch
template <bool STATS>
hipError_t launch_draft_partials(const tsb_config& c, int K, float invT, const void* draft, float* pm, double* ps,
                                 uint64_t* pk, int* pf, int32_t* req_status, hipStream_t st) {
    const Geometry g = geometry(c);
    const dim3 grid1(g.S1, c.R * c.D);
    const bool vec = (c.dtype == TSB_BF16) ? (c.V % 8 == 0 && ((uintptr_t)draft & 15) == 0)
                                           : (c.V % 4 == 0 && ((uintptr_t)draft & 15) == 0);
    const bool tab = STATS && c.dtype == TSB_BF16 && draft_table_ok(invT) && g.seg1 >= kTableMinSeg;
#define TSB_DRAFT_LAUNCH(DT, VEC, TAB)                                                                          \
    draft_partials<DT, VEC, STATS, (TAB) && STATS><<<grid1, kDraftThreads, 0, st>>>(draft, c.V, c.D, g.seg1, g.S1, \
                                                                                invT, K, pm, ps, pk, pf,       \
                                                                                req_status)
    if (c.dtype == TSB_BF16) {
        if (tab) {
            if (vec)
                TSB_DRAFT_LAUNCH(TSB_BF16, true, true);
            else
                TSB_DRAFT_LAUNCH(TSB_BF16, false, true);
        } else {
            if (vec)
                TSB_DRAFT_LAUNCH(TSB_BF16, true, false);
            else
                TSB_DRAFT_LAUNCH(TSB_BF16, false, false);
        }
    } else {
        if (vec)
            TSB_DRAFT_LAUNCH(TSB_F32, true, false);
        else
            TSB_DRAFT_LAUNCH(TSB_F32, false, false);
    }
#undef TSB_DRAFT_LAUNCH
    return hipGetLastError();
}

ChainJob chain_job(const tsb_config& c, const void* target, char* ws) {
    const XchgWs x = xchg_ws(c);
    ChainJob j;
    j.target = target;
    j.cm = (float*)(ws + x.cm);
    j.cs = (double*)(ws + x.cs);
    j.cf = (int*)(ws + x.cf);
    j.items = walk_reads_rows(c) ? c.R * kChainRows * kChainPieces : 0;
    j.V = c.V;
    j.B = c.B;
    j.bf16 = c.dtype == TSB_BF16;
    j.vec = (c.dtype == TSB_BF16) ? (c.V % 8 == 0 && ((uintptr_t)target & 15) == 0)
                                  : (c.V % 4 == 0 && ((uintptr_t)target & 15) == 0);
    return j;
}

hipError_t launch_plan(const tsb_config& c, float invT, const void* draft, double* draft_lse, int32_t* topk_tok,
                       float* topk_lp, const tsb_tree& tree, int32_t* req_status, char* ws, hipStream_t st,
                       int frontier, const ChainJob* cj) {
    const Geometry g = geometry(c);
    const PlanWs w = plan_ws(c);
    float* pm = (float*)(ws + w.pm);
    double* ps = (double*)(ws + w.ps);
    uint64_t* pk = (uint64_t*)(ws + w.pk);
    int* pf = (int*)(ws + w.pf);
    hipError_t e = hook_before(TSB_KERNEL_DRAFT_PARTIALS, st);
    if (e != hipSuccess) return e;
    if ((e = launch_draft_partials<true>(c, c.K, invT, draft, pm, ps, pk, pf, req_status, st)) != hipSuccess) return e;
    if ((e = hook_after(TSB_KERNEL_DRAFT_PARTIALS, st)) != hipSuccess) return e;
    if ((e = hook_before(TSB_KERNEL_PLAN_TREE, st)) != hipSuccess) return e;
    if (frontier > 0)
        plan_ep<<<c.R, kPlanThreads, 0, st>>>(c.D, g.S1, c.K, c.B, frontier, invT, pm, ps, pk, pf, draft_lse,
                                              topk_tok, topk_lp, tree, req_status);
    else {
        ChainJob none{};
        const ChainJob& j = cj ? *cj : none;
        plan_tree<<<c.R + std::min(j.items, kChainGridMax), kPlanThreads, 0, st>>>(
            c.D, g.S1, c.K, c.B, invT, pm, ps, pk, pf, draft_lse, topk_tok, topk_lp, tree, req_status, stats_ptr(),
            c.R, j);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return hook_after(TSB_KERNEL_PLAN_TREE, st);
}

hipError_t launch_pool_partials(const tsb_config& c, int P, float invT, const void* draft, uint64_t* pk, int* pf,
                                int32_t* req_status, hipStream_t st) {
    hipError_t e = hook_before(TSB_KERNEL_POOL_PARTIALS, st);
    if (e != hipSuccess) return e;
    if ((e = launch_draft_partials<false>(c, P, invT, draft, nullptr, nullptr, pk, pf, req_status, st)) != hipSuccess)
        return e;
    return hook_after(TSB_KERNEL_POOL_PARTIALS, st);
}

int ep_generated_bound(const tsb_config& c, int frontier) {
    long long n = c.K, layer = c.K;
    for (int d = 1; d < c.D; ++d) {
        layer = (layer < frontier ? layer : frontier) * (long long)c.K;
        n += layer;
        if (n > (1ll << 30)) break;
    }
    return n > kEpMax ? -1 : (int)n;
}

}  // namespace tsb
