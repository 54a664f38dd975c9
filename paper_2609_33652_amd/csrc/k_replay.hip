// Second pass of a tree-replay round on gfx950 (Section 3.2, eq. (2);
// Appendix A): every parent u at depth d refills its m_u child slots with the
// m_u largest Gumbel keys a_{d,v} + G(u, v) over the whole vocabulary
// (Gumbel-top-k = ordered sampling without replacement).
//
//   replay_threshold  one wave per parent: a lower bound of its m-th key
//                 from its planning candidates; one more workgroup writes
//                 the flat list of the parents of the batch (request-major,
//                 BFS order, so a depth's parents are contiguous).
//   replay_scan   one wave per (parent, vocabulary tile) item, dealt
//                 grid-stride over a persistent grid (parents of one (request,
//                 depth) are adjacent, so their tiles of draft row d meet in
//                 cache). Per item, tokens whose key cannot reach the
//                 parent's threshold (a lower bound of its m-th key, taken
//                 from its planning candidates) are skipped before any random
//                 number is drawn; the survivors are compacted within the
//                 wave and only they pay for Philox and two logarithms; the
//                 wave keeps the parent's m best keys of the tile in a sorted
//                 wave-wide list.
//   replay_scan_target
//                 the scan of a whole round (tsb_step and its variants): one
//                 grid whose first workgroups stream the target's row
//                 normalisers for verification (target_chunk) while the
//                 others scan, so the HBM-bound stream and the VALU-bound
//                 scan share the compute units.
//   replay_merge  one wave per parent: merge the per-tile lists, keep the m
//                 best (key desc, token asc) in slot order.
//
// Keys are binary32 and relative to the row's largest logit c_d:
// key = fl32(a_v - c_d) + G_v (the offset is common to all tokens of the
// row, so the order is that of a_v + G_v).
#include <math.h>

#include <algorithm>

#include "tsb_device.hpp"
#include "tsb_kernels.hpp"
#include "tsb_target.hpp"

namespace tsb {

constexpr int kTileGroups = kReplayTile / 4;  // groups of four tokens per tile
constexpr int kPassGroups = kTileGroups / 4;  // groups per compaction pass
constexpr int kScanWaves = kBlock / kWave;
constexpr int kScanWorkgroups = 1536;  // resident at 6 waves per SIMD
// Workgroups of replay_scan_target: the target's (about 2.7 waves per SIMD,
// three chunks each of the 2048 of a large target) and the scan's beside
// them (they fill the rest as they fit, and start as workgroups finish).
// Measured with inputs rotated over four sets: 683 target workgroups beat
// 1024 (two chunks each) by 7% and 512 (four each) by 2% at the batched
// workload, where the scan ends last. The scan's workgroups grow with the
// tree's node count, from 2048 (batched: 1536 was 4% slower, 3072 even) to
// 4096 (the 64-request large-budget workload: 3% faster than 2048).
constexpr int kFusedTargetWorkgroups = 683;
constexpr bool kFusedTargetPrefetch = false;  // see kTargetPrefetch
constexpr int kFusedScanWorkgroupsMin = 2048, kFusedScanWorkgroupsMax = 4096;

// A parent that replay fills: a well-formed node of the caller's topology
// (entries in range, see tree_node) with 1 <= m <= K children. Malformed
// parents, and every node of a request whose n_nodes lies outside
// [1, B + 1], are skipped: their child slots are not written.
__device__ __forceinline__ bool replay_parent(const tsb_tree& tree, int r, int u, int B, int D, int K, TreeNode* nd) {
    const int nn = tree.n_nodes[r];
    const int n = tree_count_ok(nn, B) ? nn : 0;
    if (u >= n) return false;
    *nd = tree_node(tree, (size_t)r * (B + 1), u, n, D);
    return nd->ok && nd->m > 0 && nd->m <= K;
}

// Flat list of every parent, request-major, BFS order within a request (so
// parents of one (request, depth) are contiguous): plist[i] =
// r * (B + 1) + u; ptotal[0] = list length. One workgroup of kBlock threads:
// a thread takes eight consecutive nodes of a chunk (their loads in flight
// together) and a block scan places them.
__device__ void prep_list(int R, int B, int D, int K, const tsb_tree& tree, int* __restrict__ plist,
                          int* __restrict__ ptotal) {
    constexpr int kPer = 8;
    __shared__ int s_w[kBlock / kWave];
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const int total_nodes = R * (B + 1);
    int out = 0;
    for (int c0 = 0; c0 < total_nodes; c0 += kBlock * kPer) {
        // every entry of the thread's nodes is loaded before any is tested
        // (replay_parent's conditions, without its dependent loads)
        int nn[kPer], nm[kPer], nfc[kPer], nd[kPer];
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int i = c0 + tid * kPer + k;
            const bool in = i < total_nodes;
            const int r = in ? i / (B + 1) : 0;
            const size_t e = in ? (size_t)i : 0;
            nn[k] = in ? tree.n_nodes[r] : 0;
            nm[k] = tree.n_children[e];
            nfc[k] = tree.first_child[e];
            nd[k] = tree.depth[e];
        }
        int flags = 0;  // bit k: node c0 + tid * kPer + k has children
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int i = c0 + tid * kPer + k;
            const int u = i % (B + 1);
            const int n = tree_count_ok(nn[k], B) ? nn[k] : 0;
            const int m = nm[k], fc = nfc[k], d = nd[k];
            const bool ok = m == 0 || (m > 0 && m <= TSB_MAX_K && fc > u && fc <= n - m && d >= 0 && d < D);
            if (i < total_nodes && u < n && ok && m > 0 && m <= K) flags |= 1 << k;
        }
        int wt;
        const int off = wave_excl_scan<4>(__popc(flags), wt);
        if (lane == 0) s_w[wave] = wt;
        __syncthreads();
        int o = out, tot = 0;
        for (int w = 0; w < kBlock / kWave; ++w) {
            const int x = s_w[w];
            o += w < wave ? x : 0;
            tot += x;
        }
        o += off;
#pragma unroll
        for (int k = 0; k < kPer; ++k)
            if ((flags >> k) & 1) plist[o++] = c0 + tid * kPer + k;
        out += tot;
        __syncthreads();  // s_w is rewritten by the next chunk
    }
    if (tid == 0) ptotal[0] = out;
}

__device__ __forceinline__ bool key_better(float ka, int ia, float kb, int ib) {
    return ka > kb || (ka == kb && ia < ib);
}

// Per parent u (one wave each): the m_u-th largest key among the keys of
// its planning candidates, a lower bound of its m_u-th largest key over the
// vocabulary (the same key arithmetic as the scan; -inf without pruning),
// stored with what the scan needs of the parent in one record
// (c_d, thr, depth, m_u). The grid's last workgroup builds the parent list
// instead.
template <int DT>
__global__ __launch_bounds__(kBlock) void replay_threshold(const void* __restrict__ draft, int R, int V, int D, int B,
                                                           int K, float invT, const int32_t* __restrict__ topk_tok,
                                                           tsb_tree tree, uint32_t k0, uint32_t k1, uint32_t step,
                                                           int prune, float4* __restrict__ rec,
                                                           int* __restrict__ plist, int* __restrict__ ptotal) {
    if (blockIdx.x == gridDim.x - 1) {
        prep_list(R, B, D, K, tree, plist, ptotal);
        return;
    }
    const int lane = threadIdx.x % kWave;
    const int node = blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave;
    if (node >= R * (B + 1)) return;
    const int r = node / (B + 1), u = node % (B + 1);
    TreeNode nd;
    if (!replay_parent(tree, r, u, B, D, K, &nd)) return;
    const int m = nd.m, d = nd.d;
    const size_t rowbase = ((size_t)r * D + d) * (size_t)V;
    const int32_t* tk = topk_tok + ((size_t)r * D + d) * K;
    // candidate tokens are checked before they become addresses; the
    // threshold is a lower bound of the m-th key only over K distinct tokens
    // of the row, so an out-of-range or repeated candidate turns pruning off
    const int t0 = tk[0];
    const float cd = (t0 >= 0 && t0 < V) ? load_logit<DT>(draft, rowbase + t0) * invT : 0.f;
    RngKey key;
    key.k0 = k0;
    key.k1 = k1;
    key.request = (uint32_t)r;
    key.step = step;
    float kj = -INFINITY;
    int tj = 0x7FFFFFFF;
    bool tok_ok = true;
    if (lane < K) {
        tj = tk[lane];
        tok_ok = tj >= 0 && tj < V;
        const float a = tok_ok ? load_logit<DT>(draft, rowbase + tj) * invT : -INFINITY;
        const float bj = a - cd;
        kj = bj + gumbel_f32(rng_word(key, (uint32_t)u, kStreamReplay, (uint32_t)tj));
    }
    int above = 0;
    for (int j = 0; j < K; ++j) {
        const float kk = __shfl(kj, j, kWave);
        const int tt = __shfl(tj, j, kWave);
        above += key_better(kk, tt, kj, tj) ? 1 : 0;
        tok_ok = tok_ok && !(lane < K && j < lane && tt == tj);
    }
    const bool cands_ok = __ballot(!tok_ok) == 0ull && t0 >= 0 && t0 < V;
    const uint64_t at = __ballot(lane < K && above == m - 1);  // one lane for distinct finite keys
    const float thr = (prune && cands_ok && at != 0ull) ? lane_f32(kj, (int)__ffsll((unsigned long long)at) - 1)
                                                        : -INFINITY;
    if (lane == 0) rec[node] = make_float4(cd, thr, __int_as_float(d), __int_as_float(m));
}

// Four logits of the draft row as b = fl32(a - c_d); positions at or past
// `tn` (relative to the tile) read as -inf.
template <int DT, bool VEC>
__device__ __forceinline__ void load_b4(const void* __restrict__ draft, size_t base, int e0, int tn, float invT,
                                        float cd, float b[4]) {
    float x[4];
    if (VEC && e0 + 4 <= tn) {
        if (DT == TSB_BF16) {
            const uint2 raw = *(const uint2*)((const uint16_t*)draft + base + e0);
            x[0] = __uint_as_float(raw.x << 16);
            x[1] = __uint_as_float(raw.x & 0xFFFF0000u);
            x[2] = __uint_as_float(raw.y << 16);
            x[3] = __uint_as_float(raw.y & 0xFFFF0000u);
        } else {
            const float4 a = *(const float4*)((const float*)draft + base + e0);
            x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
        }
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = (e0 + e < tn) ? load_logit<DT>(draft, base + e0 + e) : -INFINITY;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) b[e] = (e0 + e < tn) ? x[e] * invT - cd : -INFINITY;
}

// Raw logits of four consecutive tokens of a tile; positions at or past `tn`
// read as -inf. FULL: the whole tile exists and rows are vector-aligned, so
// the four are one unconditional load.
template <int DT, bool VEC, bool FULL>
__device__ __forceinline__ void load_x4(const void* __restrict__ draft, size_t base, int e0, int tn, float x[4]) {
    if (FULL || (VEC && e0 + 4 <= tn)) {
        if (DT == TSB_BF16) {
            const uint2 raw = *(const uint2*)((const uint16_t*)draft + base + e0);
            x[0] = __uint_as_float(raw.x << 16);
            x[1] = __uint_as_float(raw.x & 0xFFFF0000u);
            x[2] = __uint_as_float(raw.y << 16);
            x[3] = __uint_as_float(raw.y & 0xFFFF0000u);
        } else {
            const float4 a = *(const float4*)((const float*)draft + base + e0);
            x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
        }
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = (e0 + e < tn) ? load_logit<DT>(draft, base + e0 + e) : -INFINITY;
    }
}

// Smallest raw Philox word a token may hold for its key to reach thr when its
// b = fl32(a - c_d) is at most `bmax`: a necessary condition only (words
// below it are certain misses, words at or above it are evaluated exactly).
// With x = thr - bmax, the key can reach thr only if G(u) >= x - s for a
// slack s that covers the rounding of the binary32 Gumbel map and of the key
// sum; G(u) >= y means -ln u <= e^-y, and -ln u >= 1 - u, so it needs
// 1 - u <= e^(s - x), i.e. k = w >> 9 >= 2^23 (1 - e^(s - x)) - 1/2 for
// u = (2k + 1) 2^-24. s = 1/4 plus a few units in the last place of thr
// (far above the Gumbel map's error, which stays near 1e-6). e^(s - x) comes
// from the hardware base-2 exponential (about one unit in the last place;
// a result flushed to zero only drops the bound by less than the margin);
// the floor and the margin of two keep the result below the exact bound
// despite the rounding of the binary32 arithmetic here. An infinite or NaN
// gap gives 0 (every word is evaluated exactly).
__device__ __forceinline__ uint32_t gumbel_word_floor(float thr, float bmax, float slack) {
    const float E = __builtin_amdgcn_exp2f((slack - (thr - bmax)) * 1.44269504088896341f);
    const float k = floorf(8388608.0f - E * 8388608.0f) - 2.0f;
    return (uint32_t)fmaxf(k, 0.0f) << 9;
}

struct ScanArgs {
    const void* draft;
    int V, D, B, T;
    float invT;
    const int* plist;
    const float4* rec;
    uint32_t k0, k1, step;
    uint64_t* out_cand;
    int* out_cnt;
};
// Work counters of one wave in LDS (items, tokens, live groups, keyed
// groups), kept only while counting is on; lane 0 updates them.
struct ScanCounters {
    unsigned long long* c;  // null: not counting
    __device__ void add(int k, unsigned long long v, int lane) const {
        if (c && lane == 0) c[k] += v;
    }
    __device__ void flush(unsigned long long* stats, int lane) const {
        if (c && lane == 0 && c[0]) {
            atomicAdd(&stats[kStReplayItems], c[0]);
            atomicAdd(&stats[kStReplayTokens], c[1]);
            atomicAdd(&stats[kStReplayLive], c[2]);
            atomicAdd(&stats[kStReplayKeyed], c[3]);
        }
    }
};
__device__ __forceinline__ ScanCounters scan_counters(unsigned long long (*s)[4], int wave, int lane,
                                                      const unsigned long long* stats) {
    ScanCounters C;
    C.c = stats ? s[wave] : nullptr;
    if (C.c && lane < 4) C.c[lane] = 0;
    return C;
}

// One (parent, tile) item, by one wave; `queue` is the wave's LDS queue.
template <int DT, bool VEC>
__device__ __forceinline__ void scan_item(const ScanArgs& A, long long it, int lane, uint4* queue, const ScanCounters& C) {
    const void* __restrict__ draft = A.draft;
    const int V = A.V, D = A.D, B = A.B, T = A.T;
    const float invT = A.invT;
    const int pi = (int)(it / T);
    const int t = (int)(it - (long long)pi * T);
    const int node = A.plist[pi];
    const float4 pr = A.rec[node];  // (c_d, thr, depth, m) of the parent
    const int r = node / (B + 1);
    const int u = node - r * (B + 1);
    const int d = __float_as_int(pr.z);
    const int m = __float_as_int(pr.w);
    const size_t rowbase = ((size_t)r * D + d) * (size_t)V;
    const float cd = pr.x;
    const float thr = pr.y;
    const float bound = thr - kGumbelMaxBound;
    const int t0 = t * kReplayTile;
    const int tn = min(kReplayTile, V - t0);
    const size_t tbase = rowbase + t0;
    const bool full = VEC && tn == kReplayTile;
    const float slack = 0.25f + fabsf(thr) * 0x1p-20f;
    RngKey key;
    key.k0 = A.k0;
    key.k1 = A.k1;
    key.request = (uint32_t)r;
    key.step = A.step;
    const uint32_t blk0 = (uint32_t)(t0 >> 2);
    WaveTopList top;
    top.init(m);
    constexpr int kPer = kPassGroups / kWave;  // groups per lane and pass
#pragma unroll 1
    for (int g0 = 0; g0 < kTileGroups; g0 += kPassGroups) {
        // 1. largest b of each group of four (b = fl32(x invT - c_d) is
        // non-decreasing in x, so it is that of the largest raw logit);
        // groups whose largest b cannot reach thr are dropped, the rest
        // are compacted within the wave
        float x[kPer][4];
        uint32_t xw[kPer][2];  // bf16: the group's logits as two words
        if (full) {
#pragma unroll
            for (int k = 0; k < kPer; ++k) {
                const int e0 = (g0 + k * kWave + lane) * 4;
                if (DT == TSB_BF16) {
                    // the loaded words are kept for the queue
                    const uint2 raw = *(const uint2*)((const uint16_t*)draft + tbase + e0);
                    xw[k][0] = raw.x;
                    xw[k][1] = raw.y;
                    x[k][0] = __uint_as_float(raw.x << 16);
                    x[k][1] = __uint_as_float(raw.x & 0xFFFF0000u);
                    x[k][2] = __uint_as_float(raw.y << 16);
                    x[k][3] = __uint_as_float(raw.y & 0xFFFF0000u);
                } else {
                    load_x4<DT, VEC, true>(draft, tbase, e0, tn, x[k]);
                }
            }
        } else {
#pragma unroll
            for (int k = 0; k < kPer; ++k) {
                load_x4<DT, VEC, false>(draft, tbase, (g0 + k * kWave + lane) * 4, tn, x[k]);
                // a bf16 logit is the top half of its binary32 value (-inf past tn included)
                xw[k][0] = (__float_as_uint(x[k][0]) >> 16) | (__float_as_uint(x[k][1]) & 0xFFFF0000u);
                xw[k][1] = (__float_as_uint(x[k][2]) >> 16) | (__float_as_uint(x[k][3]) & 0xFFFF0000u);
            }
        }
        int qn = 0;
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const float gx = fmaxf(fmaxf(x[k][0], x[k][1]), fmaxf(x[k][2], x[k][3]));
            const float bmax = gx * invT - cd;
            const bool live = bmax >= bound && bmax > -INFINITY;
            const uint64_t bal = __ballot(live);
            if (live) {
                const uint32_t w0 = xw[k][0], w1 = xw[k][1];
                queue[qn + __popcll(bal & ((1ull << lane) - 1ull))] =
                    make_uint4((uint32_t)(g0 + k * kWave + lane), w0, w1, __float_as_uint(bmax));
            }
            qn += __popcll(bal);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        C.add(2, (unsigned)qn, lane);

        // 2. Philox for the survivors; a word below its group's floor is a
        // certain miss; groups holding a word at or above it get their
        // exact keys, and the m best keys >= thr are kept
        for (int base = 0; base < qn; base += kWave) {
            const int q = base + lane;
            const bool valid = q < qn;
            const uint4 ent = queue[valid ? q : 0];
            const int gl = (int)ent.x;
            const uint4 w = rng_block(key, (uint32_t)u, kStreamReplay, blk0 + (uint32_t)gl);
            const uint32_t wf = gumbel_word_floor(thr, __uint_as_float(ent.w), slack);
            const bool pass = valid && max(max(w.x, w.y), max(w.z, w.w)) >= wf;
            const uint64_t pb = __ballot(pass);
            C.add(3, (unsigned)__popcll(pb), lane);
            if (pb == 0) continue;
            float bv[4];
            if constexpr (DT == TSB_BF16) {
                // the group's logits come from the queue (no second read)
                const float xq[4] = {__uint_as_float(ent.y << 16), __uint_as_float(ent.y & 0xFFFF0000u),
                                     __uint_as_float(ent.z << 16), __uint_as_float(ent.z & 0xFFFF0000u)};
#pragma unroll
                for (int e = 0; e < 4; ++e) bv[e] = (pass && gl * 4 + e < tn) ? xq[e] * invT - cd : -INFINITY;
            } else {
                load_b4<DT, VEC>(draft, tbase, gl * 4, pass ? tn : 0, invT, cd, bv);
            }
            const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
            float kv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const bool in = bv[e] >= bound && bv[e] > -INFINITY;
                kv[e] = in ? bv[e] + gumbel_f32(ws[e]) : -INFINITY;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e)
                top.offer(cand_key(kv[e], (uint32_t)(t0 + gl * 4 + e)), kv[e] >= thr && kv[e] > -INFINITY);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");  // the queue is rewritten by the next pass
    }
    const size_t o = (size_t)node * (size_t)T + t;
    const int cnt = __popcll(__ballot(lane < m && top.v != 0));
    if (lane < cnt) A.out_cand[o * TSB_MAX_K + lane] = top.v;
    if (lane == 0) A.out_cnt[o] = cnt;
    C.add(0, 1, lane);
    C.add(1, (unsigned)tn, lane);
}

template <int DT, bool VEC>
__global__ __launch_bounds__(kBlock) void replay_scan(ScanArgs A, const int* __restrict__ ptotal,
                                                      unsigned long long* __restrict__ stats) {
    // surviving groups of the current pass, per wave: (group, its four bf16
    // logits as two words, largest b); binary32 rows keep (group, largest b)
    // and read the group again
    __shared__ uint4 s_queue[kScanWaves][kPassGroups];
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const long long items = (long long)ptotal[0] * A.T;
    const long long nw = (long long)gridDim.x * kScanWaves;
    __shared__ unsigned long long s_cnt[kScanWaves][4];
    const ScanCounters C = scan_counters(s_cnt, wave, lane, stats);
    for (long long it = (long long)blockIdx.x * kScanWaves + wave; it < items; it += nw)
        scan_item<DT, VEC>(A, it, lane, s_queue[wave], C);
    C.flush(stats, lane);
}

// The scan and the target stream of verification in one grid: the first nt
// workgroups stream the target (the job's chunks dealt over them) and the
// others scan (items dealt grid-stride over the scan's workgroups, as in
// replay_scan). The target's workgroups come first, so they are dispatched
// first and every compute unit mixes the target's HBM stream with the
// scan's VALU work; the scan's workgroups beyond what fits start as others
// finish.
template <int DT, bool VEC, bool TVEC>
__global__ __launch_bounds__(kBlock) void replay_scan_target(ScanArgs A, const int* __restrict__ ptotal,
                                                             unsigned long long* __restrict__ stats, TargetJob job,
                                                             int nt) {
    if ((int)blockIdx.x < nt) {
        // chunks blockIdx.x, blockIdx.x + nt, ... of the job
        XRegion X;
        X.slots = job.slots;
        for (int g = blockIdx.x; g < job.ngroups; g += nt)
            target_chunk<DT, TVEC, kFusedTargetPrefetch>(g, job.ngroups, job.target, A.V, A.B, job.nrows, job.chunk, job.P, A.invT,
                                   job.n_nodes, job.tm, job.ts, job.tf, X, job.R);
        return;
    }
    __shared__ uint4 s_queue[kScanWaves][kPassGroups];
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const long long items = (long long)ptotal[0] * A.T;
    const int sb = (int)blockIdx.x - nt;
    const long long nw = (long long)((int)gridDim.x - nt) * kScanWaves;
    __shared__ unsigned long long s_cnt[kScanWaves][4];
    const ScanCounters C = scan_counters(s_cnt, wave, lane, stats);
    for (long long it = (long long)sb * kScanWaves + wave; it < items; it += nw)
        scan_item<DT, VEC>(A, it, lane, s_queue[wave], C);
    C.flush(stats, lane);
}

// The walk's node record of u (a whole round: job.nrec set), from the same
// loads and arithmetic as the walk would do. The parts that do not depend
// on the children's tokens are read first (NodeHead), so their loads overlap
// the merge; tok is child lane's token.
struct NodeHead {
    TreeNode t;
    double L0, Ld;
    int bad;
};
__device__ __forceinline__ NodeHead node_head(const TargetJob& job, const tsb_tree& tree, int r, int u, int n,
                                              size_t tb, int D) {
    NodeHead h;
    h.t = tree_node(tree, tb, u, n, D);
    h.L0 = 0.0;
    h.bad = 0;
    if (job.nrows > 0) h.L0 = target_row_lse(job.tm, job.ts, job.tf, job.P, tb + u, &h.bad);
    h.Ld = (h.t.ok && h.t.m > 0) ? job.draft_lse[(size_t)r * D + h.t.d] : 0.0;
    return h;
}

template <int DT>
__device__ void write_record(const TargetJob& job, const NodeHead& h, const void* __restrict__ draft, int V, int D,
                             float invT, int r, int u, size_t tb, int tok) {
    const int lane = threadIdx.x;
    const TreeNode& t = h.t;
    uint32_t* rp = job.nrec + (tb + u) * kRecWords;
    const int m = t.ok ? t.m : 0;
    if (lane == 0) {
        const uint64_t l0 = (uint64_t)__double_as_longlong(h.L0), ld = (uint64_t)__double_as_longlong(h.Ld);
        *(uint4*)rp = make_uint4((uint32_t)m, (uint32_t)t.fc, (uint32_t)t.d,
                                 (t.ok ? kRecOk : 0u) | (h.bad ? kRecTargetBad : 0u));
        *(uint4*)(rp + 4) = make_uint4((uint32_t)l0, (uint32_t)(l0 >> 32), (uint32_t)ld, (uint32_t)(ld >> 32));
    }
    if (lane < m) {
        const size_t trow = (tb + u) * (size_t)V;
        const size_t drow = ((size_t)r * D + t.d) * (size_t)V;
        const bool yok = tok >= 0 && tok < V;
        const float xd = yok ? load_logit<DT>(draft, drow + tok) * invT : 0.f;
        const float xt = yok ? load_logit<DT>(job.target, trow + tok) * invT : 0.f;
        *(uint4*)(rp + 8 + 4 * lane) = make_uint4((uint32_t)tok, __float_as_uint(xd), __float_as_uint(xt), 0u);
    }
}

template <int DT>
__global__ __launch_bounds__(kWave) void replay_merge(int B, int D, int K, int T, tsb_tree tree,
                                                      const uint64_t* __restrict__ cand, const int* __restrict__ cc,
                                                      int32_t* __restrict__ node_tok, const void* __restrict__ draft,
                                                      int V, float invT, TargetJob job) {
    const int r = blockIdx.y;
    const int u = blockIdx.x;
    const int lane = threadIdx.x;
    const size_t tb = (size_t)r * (B + 1);
    const int nn = tree.n_nodes[r];
    const int n = tree_count_ok(nn, B) ? nn : 0;
    if (u == 0 || u >= n) {
        if (lane == 0) node_tok[tb + u] = -1;
    }
    NodeHead head;
    if (job.nrec && u < n) head = node_head(job, tree, r, u, n, tb, D);
    TreeNode nd;
    if (!replay_parent(tree, r, u, B, D, K, &nd)) {
        if (job.nrec && u < n) {
            // a leaf, or a node replay leaves alone: its children (if any) keep
            // the tokens the caller's topology gave them
            const TreeNode& t = head.t;
            const int tok = (t.ok && lane < t.m) ? node_tok[tb + t.fc + lane] : -1;
            write_record<DT>(job, head, draft, V, D, invT, r, u, tb, tok);
        }
        return;
    }
    const int m = nd.m;
    const int fc = nd.fc;
    // the children's tokens (lane j < m: child j), then the node record
    auto finish = [&](int tok) {
        if (lane < m) node_tok[tb + fc + lane] = tok;
        if (job.nrec) write_record<DT>(job, head, draft, V, D, invT, r, u, tb, tok);
    };
    const size_t o = (tb + u) * (size_t)T;
    if (T <= kWave) {
        // lane t holds tile t's count; the keys of all lists are gathered
        // contiguously, rank-major (every tile's best key, then every second
        // best, ...: each list is sorted, so the best keys come first), their
        // indices placed through LDS. At most 64 keys: one per lane, sorted,
        // and the first m are the children. More: in batches of 64 against
        // the running list, a batch sorted first when more than m of its keys
        // beat the list's smallest, so that at most m are inserted
        __shared__ int s_idx[kWave * TSB_MAX_K];
        const int ct = lane < T ? cc[o + lane] : 0;
        int nv = 0;
        for (int j = 0;; ++j) {
            const uint64_t bj = __ballot(j < ct);
            if (!bj) break;
            if (j < ct) s_idx[nv + lanes_below_u64(bj)] = lane * TSB_MAX_K + j;
            nv += __popcll(bj);
        }
        wave_lds_fence();
        const uint64_t* cb = cand + o * TSB_MAX_K;
        if (nv <= kWave) {
            uint64_t v[1];
            v[0] = lane < nv ? cb[s_idx[lane]] : 0ull;
            wave_sort_desc<1>(v);
            finish((int32_t)cand_id(v[0]));
            return;
        }
        WaveTopList top;
        top.init(m);
        constexpr int kMergeBatches = 8;  // batches whose loads are in flight together
        const int nb = (nv + kWave - 1) / kWave;
        for (int b0 = 0; b0 < nb; b0 += kMergeBatches) {
            uint64_t kb[kMergeBatches];
#pragma unroll
            for (int q = 0; q < kMergeBatches; ++q) {
                const int e = (b0 + q) * kWave + lane;
                kb[q] = e < nv ? cb[s_idx[e]] : 0ull;
            }
#pragma unroll
            for (int q = 0; q < kMergeBatches; ++q) {
                if (b0 + q >= nb) break;
                const bool want = kb[q] > top.thr;
                if (__popcll(__ballot(want)) > m) {
                    uint64_t v[1];
                    v[0] = want ? kb[q] : 0ull;
                    wave_sort_desc<1>(v);
                    top.offer(v[0], lane < m && v[0] != 0);
                } else {
                    top.offer(kb[q], want);
                }
            }
        }
        finish((int32_t)cand_id(top.v));
        return;
    }
    WaveTopList top;
    top.init(m);
    // the tiles' lists (at most m entries each), all loads of a batch in flight together
    const int ne = T * m;
    for (int base = 0; base < ne; base += kWave) {
        const int i = base + lane;
        const int tt = i / m, j = i - tt * m;
        uint64_t k = 0;
        if (i < ne && j < cc[o + tt]) k = cand[(o + tt) * TSB_MAX_K + j];
        top.offer(k, k != 0);
    }
    finish((int32_t)cand_id(top.v));
}

hipError_t launch_replay(const tsb_config& c, float invT, const void* draft, const int32_t* topk_tok,
                         const tsb_tree& tree, uint32_t step, int32_t* node_tok, char* ws, hipStream_t st,
                         const TargetJob* tj) {
    const Geometry g = geometry(c);
    const ReplayWs w = replay_ws(c);
    uint64_t* cand = (uint64_t*)(ws + w.cand);
    int* cc = (int*)(ws + w.cnt);
    int* plist = (int*)(ws + w.plist);
    int* ptotal = (int*)(ws + w.ptotal);
    const uint32_t k0 = (uint32_t)c.seed, k1 = (uint32_t)(c.seed >> 32);
    const int prune = (c.flags & TSB_FLAG_NO_PRUNE) ? 0 : 1;
    const bool vec = c.V % 4 == 0 && ((uintptr_t)draft & 15) == 0;
    float4* rec = (float4*)(ws + w.thr);
    // one workgroup per four nodes, and one more for the parent list
    const int nthr = (c.R * (c.B + 1) + kBlock / kWave - 1) / (kBlock / kWave) + 1;
    if (c.dtype == TSB_BF16)
        replay_threshold<TSB_BF16><<<nthr, kBlock, 0, st>>>(draft, c.R, c.V, c.D, c.B, c.K, invT, topk_tok, tree, k0,
                                                            k1, step, prune, rec, plist, ptotal);
    else
        replay_threshold<TSB_F32><<<nthr, kBlock, 0, st>>>(draft, c.R, c.V, c.D, c.B, c.K, invT, topk_tok, tree, k0,
                                                           k1, step, prune, rec, plist, ptotal);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int scan_id = tj ? TSB_KERNEL_SCAN_TARGET : TSB_KERNEL_REPLAY_SCAN;
    if ((e = hook_before(scan_id, st)) != hipSuccess) return e;
    unsigned long long* const stats = stats_ptr();
    ScanArgs A{draft, c.V, c.D, c.B, g.T, invT, plist, rec, k0, k1, step, cand, cc};
    if (tj) {
        const int nt = std::min(tj->ngroups, kFusedTargetWorkgroups);
        const int nscan = std::min(kFusedScanWorkgroupsMax, std::max(kFusedScanWorkgroupsMin, c.R * (c.B + 1) / 4));
        const int grid = nt + nscan;
        const bool tv = tj->vec;
        if (c.dtype == TSB_BF16) {
            auto fn = vec ? (tv ? replay_scan_target<TSB_BF16, true, true> : replay_scan_target<TSB_BF16, true, false>)
                          : (tv ? replay_scan_target<TSB_BF16, false, true> : replay_scan_target<TSB_BF16, false, false>);
            fn<<<grid, kBlock, 0, st>>>(A, ptotal, stats, *tj, nt);
        } else {
            auto fn = vec ? (tv ? replay_scan_target<TSB_F32, true, true> : replay_scan_target<TSB_F32, true, false>)
                          : (tv ? replay_scan_target<TSB_F32, false, true> : replay_scan_target<TSB_F32, false, false>);
            fn<<<grid, kBlock, 0, st>>>(A, ptotal, stats, *tj, nt);
        }
    } else {
        // a persistent grid: the item count is only known on the device
        const long long max_items = (long long)c.R * c.B * g.T;
        const int grid = (int)std::max<long long>(1, std::min<long long>(kScanWorkgroups,
                                                                         (max_items + kScanWaves - 1) / kScanWaves));
        auto fn = c.dtype == TSB_BF16 ? (vec ? replay_scan<TSB_BF16, true> : replay_scan<TSB_BF16, false>)
                                      : (vec ? replay_scan<TSB_F32, true> : replay_scan<TSB_F32, false>);
        fn<<<grid, kBlock, 0, st>>>(A, ptotal, stats);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((e = hook_after(scan_id, st)) != hipSuccess) return e;
    if ((e = hook_before(TSB_KERNEL_REPLAY_MERGE, st)) != hipSuccess) return e;
    TargetJob none{};
    const TargetJob& rj = tj ? *tj : none;  // node records only in a whole round
    if (c.dtype == TSB_BF16)
        replay_merge<TSB_BF16><<<dim3(c.B + 1, c.R), kWave, 0, st>>>(c.B, c.D, c.K, g.T, tree, cand, cc, node_tok,
                                                                     draft, c.V, invT, rj);
    else
        replay_merge<TSB_F32><<<dim3(c.B + 1, c.R), kWave, 0, st>>>(c.B, c.D, c.K, g.T, tree, cand, cc, node_tok,
                                                                    draft, c.V, invT, rj);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return hook_after(TSB_KERNEL_REPLAY_MERGE, st);
}

}  // namespace tsb
