// Second pass of a tree-replay round on gfx950 (Section 3.2, eq. (2);
// Appendix A): every parent u at depth d refills its m_u child slots with the
// m_u largest Gumbel keys a_{d,v} + G(u, v) over the whole vocabulary
// (Gumbel-top-k = ordered sampling without replacement).
//
//   replay_scan   grid (vocabulary tile, request x depth). One read of the
//                 tile of draft row d serves every parent at depth d (they
//                 share q_d). Per parent, tokens whose key cannot reach the
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

struct ReplayShared {
    float b[kReplayTile];                         // fl32(a_v - c_d) of the tile
    int queue[kBlock / kWave][kTileGroups / (kBlock / kWave)];
    float ckey[kReplayTile];                      // candidates of the current parent
    int cidx[kReplayTile];
    int parents[TSB_MAX_B + 1];
    int ccount;
    int nparents;
    int lo, hi;
    float thr;
    float sel_key;
    int sel_idx;
};

__device__ __forceinline__ bool key_better(float ka, int ia, float kb, int ib) {
    return ka > kb || (ka == kb && ia < ib);
}

template <int DT, bool VEC>
__global__ __launch_bounds__(kBlock) void replay_scan(const void* __restrict__ draft, int V, int D, int B, int K,
                                                      int T, float invT, const int32_t* __restrict__ topk_tok,
                                                      tsb_tree tree, uint32_t k0, uint32_t k1, uint32_t step,
                                                      int prune, float* __restrict__ out_key,
                                                      int* __restrict__ out_idx, int* __restrict__ out_cnt) {
    __shared__ ReplayShared sh;
    const int t = blockIdx.x;
    const int r = blockIdx.y / D;
    const int d = blockIdx.y % D;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    const size_t tb = (size_t)r * (B + 1);
    const int n = tree.n_nodes[r];

    // parents at depth d: contiguous BFS range with depth == d, having children
    if (tid == 0) {
        sh.lo = n;
        sh.hi = 0;
        sh.nparents = 0;
    }
    __syncthreads();
    for (int i = tid; i < n; i += kBlock) {
        const int di = tree.depth[tb + i];
        if (di == d) {
            atomicMin(&sh.lo, i);
            atomicMax(&sh.hi, i + 1);
        }
    }
    __syncthreads();
    if (tid == 0) {
        int np = 0;
        for (int i = sh.lo; i < sh.hi; ++i)
            if (tree.n_children[tb + i] > 0) sh.parents[np++] = i;
        sh.nparents = np;
    }
    __syncthreads();
    const int P = sh.nparents;
    if (P == 0) return;

    const size_t rowbase = ((size_t)r * D + d) * (size_t)V;
    const int tok0 = topk_tok[((size_t)r * D + d) * K];
    const float cd = load_logit<DT>(draft, rowbase + tok0) * invT;
    const int t0 = t * kReplayTile;
    const int tn = min(kReplayTile, V - t0);

    // stage b_v = fl32(a_v - c_d) for the tile
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
            for (int e = 0; e < 4; ++e) x[e] = (e0 + e < tn) ? load_logit<DT>(draft, rowbase + t0 + e0 + e) : -INFINITY;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float a = x[e] * invT;
            sh.b[e0 + e] = (e0 + e < tn) ? a - cd : -INFINITY;
        }
    }
    __syncthreads();

    RngKey key;
    key.k0 = k0;
    key.k1 = k1;
    key.request = (uint32_t)r;
    key.step = step;
    const uint32_t blk0 = (uint32_t)(t0 >> 2);

    for (int p = 0; p < P; ++p) {
        const int u = sh.parents[p];
        const int m = tree.n_children[tb + u];
        // threshold: m-th largest key among the planning candidates (a lower
        // bound of the m-th largest key over the vocabulary)
        if (wave == 0) {
            float kj = -INFINITY;
            int tj = 0x7FFFFFFF;
            if (lane < K) {
                tj = topk_tok[((size_t)r * D + d) * K + lane];
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
            if (lane < K && above == m - 1) sh.thr = prune ? kj : -INFINITY;
            if (lane == 0) sh.ccount = 0;
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

        // keep this tile's best m (slot order is settled by the merge)
        const int c = sh.ccount;
        const size_t o = (tb + u) * (size_t)T + t;
        if (c <= m) {
            for (int j = tid; j < c; j += kBlock) {
                out_key[o * K + j] = sh.ckey[j];
                out_idx[o * K + j] = sh.cidx[j];
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
                    out_key[o * K + j] = fk;
                    out_idx[o * K + j] = fi;
                    sh.cidx[fs] = -1;  // taken
                }
                __syncthreads();
            }
        }
        if (tid == 0) out_cnt[o] = c < m ? c : m;
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
            if (j < c) k = cand_key(ck[(o + t) * K + j], (uint32_t)ci[(o + t) * K + j]);
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
    const uint32_t k0 = (uint32_t)c.seed, k1 = (uint32_t)(c.seed >> 32);
    const int prune = (c.flags & TSB_FLAG_NO_PRUNE) ? 0 : 1;
    const bool vec = c.V % 4 == 0 && ((uintptr_t)draft & 15) == 0;
    const dim3 grid(g.T, c.R * c.D);
    hipError_t e = hook_before(TSB_KERNEL_REPLAY_SCAN, st);
    if (e != hipSuccess) return e;
    if (c.dtype == TSB_BF16) {
        if (vec)
            replay_scan<TSB_BF16, true><<<grid, kBlock, 0, st>>>(draft, c.V, c.D, c.B, c.K, g.T, invT, topk_tok, tree,
                                                                 k0, k1, step, prune, ck, ci, cc);
        else
            replay_scan<TSB_BF16, false><<<grid, kBlock, 0, st>>>(draft, c.V, c.D, c.B, c.K, g.T, invT, topk_tok, tree,
                                                                  k0, k1, step, prune, ck, ci, cc);
    } else {
        if (vec)
            replay_scan<TSB_F32, true><<<grid, kBlock, 0, st>>>(draft, c.V, c.D, c.B, c.K, g.T, invT, topk_tok, tree,
                                                                k0, k1, step, prune, ck, ci, cc);
        else
            replay_scan<TSB_F32, false><<<grid, kBlock, 0, st>>>(draft, c.V, c.D, c.B, c.K, g.T, invT, topk_tok, tree,
                                                                 k0, k1, step, prune, ck, ci, cc);
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
