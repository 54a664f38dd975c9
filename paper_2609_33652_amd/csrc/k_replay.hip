// Second pass of a tree-replay round on gfx950 (Section 3.2, eq. (2);
// Appendix A): every parent u at depth d refills its m_u child slots with the
// m_u largest Gumbel keys a_{d,v} + G(u, v) over the whole vocabulary
// (Gumbel-top-k = ordered sampling without replacement).
//
//   replay_prep   one workgroup: flat list of the parents of the batch
//                 (request-major, BFS order, so a depth's parents are
//                 contiguous).
//   replay_scan   grid (vocabulary tile, 64 rows); a row takes a contiguous
//                 chunk of the parent list and stages the tile of draft row d
//                 once for consecutive parents of the same (request, depth)
//                 (they share q_d). Per parent, tokens whose key cannot reach the
//                 parent's threshold (a lower bound of its m-th key, taken
//                 from its planning candidates) are skipped before any
//                 random number is drawn; the survivors are compacted per
//                 wave and only they pay for Philox and two logarithms. Each
//                 (parent, tile) emits its best m keys.
//   replay_merge  one wave per parent: merge the per-tile lists, keep the m
//                 best (key desc, token asc) in slot order.
//
// Keys are binary32 and relative to the row's largest logit c_d:
// key = fl32(a_v - c_d) + G_v (the offset is common to all tokens of the
// row, so the order is that of a_v + G_v).
#include <math.h>

#include "tsb_device.hpp"
#include "tsb_kernels.hpp"

namespace tsb {

constexpr int kTileGroups = kReplayTile / 4;  // groups of four tokens per tile
constexpr int kTileOut = kReplayTileOut;       // candidates a (parent, tile) may hand to the merge

struct ReplayShared {
    float b[kReplayTile];                         // fl32(a_v - c_d) of the tile
    int queue[kBlock / kWave][kTileGroups / (kBlock / kWave)];
    float ckey[kReplayTile];                      // candidates of the current parent
    int cidx[kReplayTile];
    int ccount;
    float thr;
};

constexpr int kPrepThreads = 1024;
constexpr int kScanRows = 256;  // workgroup rows of the scan grid (each takes a chunk of parents)

// Flat list of every node with children, request-major, BFS order within a
// request (so parents of one (request, depth) are contiguous): plist[i] =
// r * (B + 1) + u; ptotal[0] = list length.
__global__ __launch_bounds__(kPrepThreads) void replay_prep(int R, int B, tsb_tree tree, int* __restrict__ plist,
                                                            int* __restrict__ ptotal) {
    __shared__ int s_wave[kPrepThreads / kWave];
    __shared__ int s_base;
    const int tid = threadIdx.x;
    const int lane = tid % kWave, wave = tid / kWave;
    if (tid == 0) s_base = 0;
    __syncthreads();
    const int total_nodes = R * (B + 1);
    for (int base = 0; base < total_nodes; base += kPrepThreads) {
        const int i = base + tid;
        int flag = 0;
        if (i < total_nodes) {
            const int r = i / (B + 1), u = i % (B + 1);
            flag = (u < tree.n_nodes[r] && tree.n_children[i] > 0) ? 1 : 0;
        }
        const uint64_t bal = __ballot(flag);
        const int before = __popcll(bal & ((1ull << lane) - 1ull));
        if (lane == 0) s_wave[wave] = __popcll(bal);
        __syncthreads();
        int off = s_base;
        for (int w = 0; w < wave; ++w) off += s_wave[w];
        if (flag) plist[off + before] = i;
        __syncthreads();
        if (tid == 0) {
            int t = 0;
            for (int w = 0; w < kPrepThreads / kWave; ++w) t += s_wave[w];
            s_base += t;
        }
        __syncthreads();
    }
    if (tid == 0) ptotal[0] = s_base;
}

__device__ __forceinline__ bool key_better(float ka, int ia, float kb, int ib) {
    return ka > kb || (ka == kb && ia < ib);
}

// Per parent u (one wave each): the m_u-th largest key among the keys of
// its planning candidates, a lower bound of its m_u-th largest key over the
// vocabulary (the same key arithmetic as the scan). -inf without pruning.
template <int DT>
__global__ __launch_bounds__(kBlock) void replay_threshold(const void* __restrict__ draft, int R, int V, int D, int B,
                                                           int K, float invT, const int32_t* __restrict__ topk_tok,
                                                           tsb_tree tree, uint32_t k0, uint32_t k1, uint32_t step,
                                                           int prune, float* __restrict__ thr) {
    const int lane = threadIdx.x % kWave;
    const int node = blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave;
    if (node >= R * (B + 1)) return;
    const int r = node / (B + 1), u = node % (B + 1);
    if (u >= tree.n_nodes[r]) return;
    const int m = tree.n_children[node];
    if (m == 0) return;
    const int d = tree.depth[node];
    const size_t rowbase = ((size_t)r * D + d) * (size_t)V;
    const int32_t* tk = topk_tok + ((size_t)r * D + d) * K;
    const float cd = load_logit<DT>(draft, rowbase + tk[0]) * invT;
    RngKey key;
    key.k0 = k0;
    key.k1 = k1;
    key.request = (uint32_t)r;
    key.step = step;
    float kj = -INFINITY;
    int tj = 0x7FFFFFFF;
    if (lane < K) {
        tj = tk[lane];
        const float a = load_logit<DT>(draft, rowbase + tj) * invT;
        const float bj = a - cd;
        kj = bj + gumbel_f32(rng_word(key, (uint32_t)u, kStreamReplay, (uint32_t)tj));
    }
    int above = 0;
    for (int j = 0; j < K; ++j) {
        const float kk = __shfl(kj, j, kWave);
        const int tt = __shfl(tj, j, kWave);
        above += key_better(kk, tt, kj, tj) ? 1 : 0;
    }
    if (lane < K && above == m - 1) thr[node] = prune ? kj : -INFINITY;
}

template <int DT, bool VEC>
__global__ __launch_bounds__(kBlock) void replay_scan(const void* __restrict__ draft, int V, int D, int B, int K,
                                                      int T, float invT, const int32_t* __restrict__ topk_tok,
                                                      tsb_tree tree, const int* __restrict__ plist,
                                                      const int* __restrict__ ptotal, const float* __restrict__ thr_in,
                                                      uint32_t k0, uint32_t k1, uint32_t step,
                                                      float* __restrict__ out_key, int* __restrict__ out_idx,
                                                      int* __restrict__ out_cnt) {
    __shared__ ReplayShared sh;
    const int t = blockIdx.x;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    const int total = ptotal[0];
    const int chunk = (total + kScanRows - 1) / kScanRows;
    const int p0 = blockIdx.y * chunk;
    const int p1 = min(total, p0 + chunk);
    if (p0 >= p1) return;
    const int t0 = t * kReplayTile;
    const int tn = min(kReplayTile, V - t0);
    const uint32_t blk0 = (uint32_t)(t0 >> 2);
    int staged = -1;  // r * D + d of the staged tile

    for (int pi = p0; pi < p1; ++pi) {
        const int node = plist[pi];
        const int r = node / (B + 1);
        const int u = node % (B + 1);
        const size_t tb = (size_t)r * (B + 1);
        const int d = tree.depth[tb + u];
        const int m = tree.n_children[tb + u];
        const size_t rowbase = ((size_t)r * D + d) * (size_t)V;
        const int tok0 = topk_tok[((size_t)r * D + d) * K];
        const float cd = load_logit<DT>(draft, rowbase + tok0) * invT;
        if (staged != r * D + d) {
            // stage b_v = fl32(a_v - c_d) for the tile
            __syncthreads();
            for (int g = tid; g < kTileGroups; g += kBlock) {
                const int e0 = g * 4;
                float x[4];
                if (VEC && e0 + 4 <= tn) {
                    if (DT == TSB_BF16) {
                        const uint2 raw = *(const uint2*)((const uint16_t*)draft + rowbase + t0 + e0);
                        x[0] = __uint_as_float(raw.x << 16);
                        x[1] = __uint_as_float(raw.x & 0xFFFF0000u);
                        x[2] = __uint_as_float(raw.y << 16);
                        x[3] = __uint_as_float(raw.y & 0xFFFF0000u);
                    } else {
                        const float4 a = *(const float4*)((const float*)draft + rowbase + t0 + e0);
                        x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        x[e] = (e0 + e < tn) ? load_logit<DT>(draft, rowbase + t0 + e0 + e) : -INFINITY;
                }
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float a = x[e] * invT;
                    sh.b[e0 + e] = (e0 + e < tn) ? a - cd : -INFINITY;
                }
            }
            __syncthreads();
            staged = r * D + d;
        }

        RngKey key;
        key.k0 = k0;
        key.k1 = k1;
        key.request = (uint32_t)r;
        key.step = step;
        if (tid == 0) {
            sh.thr = thr_in[node];
            sh.ccount = 0;
        }
        __syncthreads();
        const float thr = sh.thr;
        const float bound = thr - kGumbelMaxBound;

        // compact surviving groups of this wave
        int qn = 0;
        const int gpw = kTileGroups / (kBlock / kWave);  // groups per wave
        for (int base = 0; base < gpw; base += kWave) {
            const int gl = wave * gpw + base + lane;
            const float* bb = &sh.b[gl * 4];
            const bool live = (bb[0] >= bound) | (bb[1] >= bound) | (bb[2] >= bound) | (bb[3] >= bound);
            const uint64_t bal = __ballot(live);
            const int pos = qn + __popcll(bal & ((1ull << lane) - 1ull));
            if (live) sh.queue[wave][pos] = gl;
            qn += __popcll(bal);
        }
        __syncthreads();
        for (int q = lane; q < qn; q += kWave) {
            const int gl = sh.queue[wave][q];
            const uint4 w = rng_block(key, (uint32_t)u, kStreamReplay, blk0 + (uint32_t)gl);
            const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float bv = sh.b[gl * 4 + e];
                if (bv >= bound && bv > -INFINITY) {
                    const float kv = bv + gumbel_f32(ws[e]);
                    if (kv >= thr) {
                        const int slot = atomicAdd(&sh.ccount, 1);
                        sh.ckey[slot] = kv;
                        sh.cidx[slot] = t0 + gl * 4 + e;
                    }
                }
            }
        }
        __syncthreads();

        // candidates of this tile (at most kTileOut; beyond that the tile's best
        // m are selected here); the merge settles the order
        const int c = sh.ccount;
        const size_t o = (tb + u) * (size_t)T + t;
        if (c <= kTileOut) {
            for (int j = tid; j < c; j += kBlock) {
                out_key[o * kTileOut + j] = sh.ckey[j];
                out_idx[o * kTileOut + j] = sh.cidx[j];
            }
        } else {
            for (int j = 0; j < m; ++j) {
                float bk = -INFINITY;
                int bi = 0x7FFFFFFF, bs = -1;
                for (int i = tid; i < c; i += kBlock) {
                    if (sh.cidx[i] >= 0 && (bs < 0 || key_better(sh.ckey[i], sh.cidx[i], bk, bi))) {
                        bk = sh.ckey[i];
                        bi = sh.cidx[i];
                        bs = i;
                    }
                }
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) {
                    const float ok = __shfl_xor(bk, off, kWave);
                    const int oi = __shfl_xor(bi, off, kWave);
                    const int os = __shfl_xor(bs, off, kWave);
                    if (os >= 0 && (bs < 0 || key_better(ok, oi, bk, bi))) {
                        bk = ok;
                        bi = oi;
                        bs = os;
                    }
                }
                __shared__ float wk[kBlock / kWave];
                __shared__ int wi[kBlock / kWave], wsl[kBlock / kWave];
                if (lane == 0) {
                    wk[wave] = bk;
                    wi[wave] = bi;
                    wsl[wave] = bs;
                }
                __syncthreads();
                if (tid == 0) {
                    float fk = wk[0];
                    int fi = wi[0], fs = wsl[0];
                    for (int w2 = 1; w2 < kBlock / kWave; ++w2)
                        if (wsl[w2] >= 0 && (fs < 0 || key_better(wk[w2], wi[w2], fk, fi))) {
                            fk = wk[w2];
                            fi = wi[w2];
                            fs = wsl[w2];
                        }
                    out_key[o * kTileOut + j] = fk;
                    out_idx[o * kTileOut + j] = fi;
                    sh.cidx[fs] = -1;  // taken
                }
                __syncthreads();
            }
        }
        if (tid == 0) out_cnt[o] = c <= kTileOut ? c : m;
        __syncthreads();
    }
}

__global__ __launch_bounds__(kWave) void replay_merge(int B, int K, int T, tsb_tree tree,
                                                      const float* __restrict__ ck, const int* __restrict__ ci,
                                                      const int* __restrict__ cc, int32_t* __restrict__ node_tok) {
    const int r = blockIdx.y;
    const int u = blockIdx.x;
    const int lane = threadIdx.x;
    const size_t tb = (size_t)r * (B + 1);
    const int n = tree.n_nodes[r];
    if (u == 0 || u >= n) {
        if (lane == 0) node_tok[tb + u] = -1;
    }
    if (u >= n) return;
    const int m = tree.n_children[tb + u];
    if (m == 0) return;
    WaveTopList top;
    top.init(m);
    const size_t o = (tb + u) * (size_t)T;
    for (int t = 0; t < T; ++t) {
        const int c = cc[o + t];
        for (int base = 0; base < c; base += kWave) {
            const int j = base + lane;
            uint64_t k = 0;
            if (j < c) k = cand_key(ck[(o + t) * kTileOut + j], (uint32_t)ci[(o + t) * kTileOut + j]);
            top.offer(k, j < c);
        }
    }
    if (lane < m) node_tok[tb + tree.first_child[tb + u] + lane] = (int32_t)cand_id(top.v);
}

hipError_t launch_replay(const tsb_config& c, float invT, const void* draft, const int32_t* topk_tok,
                         const tsb_tree& tree, uint32_t step, int32_t* node_tok, char* ws, hipStream_t st) {
    const Geometry g = geometry(c);
    const ReplayWs w = replay_ws(c);
    float* ck = (float*)(ws + w.key);
    int* ci = (int*)(ws + w.idx);
    int* cc = (int*)(ws + w.cnt);
    int* plist = (int*)(ws + w.plist);
    int* ptotal = (int*)(ws + w.ptotal);
    const uint32_t k0 = (uint32_t)c.seed, k1 = (uint32_t)(c.seed >> 32);
    const int prune = (c.flags & TSB_FLAG_NO_PRUNE) ? 0 : 1;
    const bool vec = c.V % 4 == 0 && ((uintptr_t)draft & 15) == 0;
    hipError_t e = hook_before(TSB_KERNEL_REPLAY_SCAN, st);
    if (e != hipSuccess) return e;
    replay_prep<<<1, kPrepThreads, 0, st>>>(c.R, c.B, tree, plist, ptotal);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    float* thr = (float*)(ws + w.thr);
    const int nthr = (c.R * (c.B + 1) + kBlock / kWave - 1) / (kBlock / kWave);
    if (c.dtype == TSB_BF16)
        replay_threshold<TSB_BF16><<<nthr, kBlock, 0, st>>>(draft, c.R, c.V, c.D, c.B, c.K, invT, topk_tok, tree, k0,
                                                            k1, step, prune, thr);
    else
        replay_threshold<TSB_F32><<<nthr, kBlock, 0, st>>>(draft, c.R, c.V, c.D, c.B, c.K, invT, topk_tok, tree, k0,
                                                           k1, step, prune, thr);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const dim3 grid(g.T, kScanRows);
    if (c.dtype == TSB_BF16) {
        if (vec)
            replay_scan<TSB_BF16, true><<<grid, kBlock, 0, st>>>(draft, c.V, c.D, c.B, c.K, g.T, invT, topk_tok, tree,
                                                                 plist, ptotal, thr, k0, k1, step, ck, ci, cc);
        else
            replay_scan<TSB_BF16, false><<<grid, kBlock, 0, st>>>(draft, c.V, c.D, c.B, c.K, g.T, invT, topk_tok,
                                                                  tree, plist, ptotal, thr, k0, k1, step, ck, ci,
                                                                  cc);
    } else {
        if (vec)
            replay_scan<TSB_F32, true><<<grid, kBlock, 0, st>>>(draft, c.V, c.D, c.B, c.K, g.T, invT, topk_tok, tree,
                                                                plist, ptotal, thr, k0, k1, step, ck, ci, cc);
        else
            replay_scan<TSB_F32, false><<<grid, kBlock, 0, st>>>(draft, c.V, c.D, c.B, c.K, g.T, invT, topk_tok, tree,
                                                                 plist, ptotal, thr, k0, k1, step, ck, ci, cc);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((e = hook_after(TSB_KERNEL_REPLAY_SCAN, st)) != hipSuccess) return e;
    if ((e = hook_before(TSB_KERNEL_REPLAY_MERGE, st)) != hipSuccess) return e;
    replay_merge<<<dim3(c.B + 1, c.R), kWave, 0, st>>>(c.B, c.K, g.T, tree, ck, ci, cc, node_tok);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return hook_after(TSB_KERNEL_REPLAY_MERGE, st);
}

}  // namespace tsb
