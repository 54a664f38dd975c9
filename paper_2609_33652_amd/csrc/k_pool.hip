// Sparse candidate pools with context-dependent draft distributions on
// gfx950 (Section 3.1: pools of the backbone's top-scoring tokens, corrections
// and normalisation inside the pool, max-heap planning for drafters that look
// their conditionals up; Section 3.2, eq. (2): replay under the replayed
// prefix with the same pools; Section 3.3).
//
// The correction is a transition-score lookup: c[d-1][i][j] scores pool slot
// j of position d after a token in pool slot i of position d - 1.
//   z_u(j) = fl32(a_{d,j} + fl32(c[d-1][s_u][j] invT)),  a_{d,j} = fl32(x invT)
//   q_u = softmax of z_u over the pool (binary64 normaliser L_u)
//   lp_u(j) = fl32(z_u(j) - fl32(L_u)); candidates by (lp desc, slot asc)
//
//   pool_lists   one workgroup per draft row (request, position d): merges
//                the segment lists of the pool selection into pool d, then
//                builds the candidate list of every context that draws from
//                pool d (the root's for d = 0, one per parent slot otherwise).
//   pool_plan    one workgroup per request: best-first expansion over the
//                per-node candidate lists. One wave pops: the fringe (every
//                uncommitted node whose predecessor is committed) sits in
//                LDS and every pop is a wave-wide argmax over it; then the
//                committed nodes are laid out in BFS order level by level.
//   pool_replay  one workgroup per request: layer by layer, one wave per
//                parent, lane j scores pool slot j; the children get the m
//                largest Gumbel keys in rank order.
#include <math.h>

#include "tsb_device.hpp"
#include "tsb_kernels.hpp"

namespace tsb {

constexpr int kPoolThreads = 1024;
constexpr int kPoolWaves = kPoolThreads / kWave;

__device__ __forceinline__ uint64_t pack_entry(float lp, int slot) {
    return ((uint64_t)__float_as_uint(lp) << 32) | (uint32_t)slot;
}
__device__ __forceinline__ float entry_lp(uint64_t e) { return __uint_as_float((uint32_t)(e >> 32)); }
__device__ __forceinline__ int entry_slot(uint64_t e) { return (int)(uint32_t)e; }

// fl32(a + fl32(c invT)): both roundings where written (contraction is off).
__device__ __forceinline__ float corrected_logit(float a, float c, float invT) {
    const float cs = c * invT;
    return a + cs;
}

__device__ __forceinline__ size_t trans_row(int r, int D, int d, int slot, int P) {
    return (((size_t)r * (D - 1) + (d - 1)) * P + slot) * (size_t)P;
}

// ------------------------------------------------------------------ lists
// Candidate list of one context from z (lane j < P holds z_j, -inf beyond):
// binary64 log-sum-exp over the pool (lanes summed in a fixed order), lp,
// and the rank of each slot under (lp desc, slot asc).
__device__ void build_list(float z, int P, int K, const double* et, uint64_t* out, int* nfin_out) {
    const int lane = lane_id();
    const float m = wave_max(z);
    int nf = 0;
    if (m > -INFINITY) {
        const double e = z > -INFINITY ? exp64((double)z - (double)m, et) : 0.0;
        const double L = (double)m + log(wave_sum(e));
        const float L32 = (float)L;
        const float lp = (float)((double)z - (double)L32);
        const bool valid = lane < P && lp > -INFINITY;
        const uint64_t key = valid ? ((uint64_t)ordered_bits(lp) << 32) | (uint32_t)(~lane) : 0ull;
        int rank = 0;
        for (int k = 0; k < kWave; ++k) rank += lane_u64(key, k) > key ? 1 : 0;
        if (valid && rank < K) out[rank] = pack_entry(lp, lane);
        nf = __popcll(__ballot(valid));
    }
    if (lane == 0) *nfin_out = nf < K ? nf : K;
}

__global__ __launch_bounds__(kPoolThreads) void pool_lists(int D, int S, int P, int K, float invT,
                                                           const uint64_t* __restrict__ pk, const int* __restrict__ pf,
                                                           const float* __restrict__ trans, int32_t* __restrict__ pool_tok,
                                                           uint64_t* __restrict__ lists, int* __restrict__ nfin,
                                                           int32_t* __restrict__ req_status) {
    const int d = blockIdx.x, r = blockIdx.y;
    const int row = r * D + d;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    __shared__ double s_exp[kExpTable];
    __shared__ float s_a[kPoolMax];
    exp64_table_init(s_exp);

    if (wave == 0) {
        // merge of the row's segment lists into the pool (keys are distinct;
        // empty slots are 0)
        const size_t o = (size_t)row * S;
        int bad = 0;
        for (int s = lane; s < S; s += kWave) bad |= pf[o + s];
        bad = wave_or(bad);
        const int n = S * P;
        uint64_t best;
        if (n <= kWave) {
            const uint64_t mine = lane < n ? pk[o * P + lane] : 0ull;
            int rank = 0;
            for (int j = 0; j < n; ++j) rank += lane_u64(mine, j) > mine ? 1 : 0;
            best = 0ull;
            for (int j = 0; j < n; ++j) {
                const uint64_t kj = lane_u64(mine, j);
                const int rj = __builtin_amdgcn_readlane(rank, j);
                if (kj != 0ull && rj == lane) best = kj;
            }
        } else {
            WaveTopList top;
            top.init(P);
            for (int base = 0; base < n; base += kWave) {
                const int i = base + lane;
                const uint64_t k = i < n ? pk[o * P + i] : 0ull;
                top.offer(k, i < n && k != 0ull);
            }
            best = top.v;
        }
        float a = -INFINITY;
        if (lane < P) {
            a = cand_value(best) * invT;
            pool_tok[(size_t)row * P + lane] = (int32_t)cand_id(best);
            s_a[lane] = a;
        }
        // a row without a finite logit has -inf at slot 0
        if (lane == 0 && (bad || !(a > -INFINITY))) atomicOr(&req_status[r], TSB_REQ_NONFINITE);
    }
    __syncthreads();

    const int NL = 1 + (D - 1) * P;
    uint64_t* L = lists + (size_t)r * NL * K;
    int* F = nfin + (size_t)r * NL;
    if (d == 0) {
        if (wave == 0) build_list(lane < P ? s_a[lane] : -INFINITY, P, K, s_exp, L, F);
        return;
    }
    int tbad = 0;
    for (int i = wave; i < P; i += kPoolWaves) {
        float z = -INFINITY;
        if (lane < P) {
            const float c = trans[trans_row(r, D, d, i, P) + lane];
            tbad |= !isfinite(c);
            z = corrected_logit(s_a[lane], c, invT);
        }
        const int li = 1 + (d - 1) * P + i;
        build_list(z, P, K, s_exp, L + (size_t)li * K, F + li);
    }
    tbad = wave_or(tbad);
    if (lane == 0 && tbad) atomicOr(&req_status[r], TSB_REQ_NONFINITE);
}

// ------------------------------------------------------------------ plan
// Lists held in LDS by the planner (entries beyond are read from the
// workspace).
constexpr int kPoolListLds = 16384;
constexpr int kPoolListsMax = 1 + (TSB_MAX_D - 1) * kPoolMax;
constexpr int kFringeMax = TSB_MAX_B + 2;
constexpr int kPlanPoolThreads = 256;

struct PoolPlanShared {
    float llp[kPoolListLds];
    uint8_t lslot[kPoolListLds];
    uint8_t lnf[kPoolListsMax];
    // committed nodes by pop index (0 = root)
    double cscore[TSB_MAX_B + 1];
    int16_t cpar[TSB_MAX_B + 1];
    uint8_t crank[TSB_MAX_B + 1], cdepth[TSB_MAX_B + 1], cslot[TSB_MAX_B + 1], cnch[TSB_MAX_B + 1];
    // fringe: (score, depth, parent pop index, rank)
    double fscore[kFringeMax];
    int16_t fpar[kFringeMax];
    uint8_t frank[kFringeMax], fdepth[kFringeMax];
    // BFS layout
    int16_t order[TSB_MAX_B + 1], bfs_of_pop[TSB_MAX_B + 1], fcb[TSB_MAX_B + 1], bucket[TSB_MAX_B + 1];
    int dcnt[TSB_MAX_D + 2], dstart[TSB_MAX_D + 2];
};

struct ListView {
    const PoolPlanShared* sh;
    const uint64_t* g;  // this request's lists in the workspace
    int K, P;
    __device__ float lp(int li, int k) const {
        const int i = li * K + k;
        return i < kPoolListLds ? sh->llp[i] : entry_lp(g[i]);
    }
    __device__ int slot(int li, int k) const {
        const int i = li * K + k;
        return i < kPoolListLds ? (int)sh->lslot[i] : entry_slot(g[i]);
    }
    // list of the children of a committed node
    __device__ int of(int depth, int slot) const { return depth == 0 ? 0 : 1 + (depth - 1) * P + slot; }
};

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

// Rank paths of two fringe entries at the same depth, lexicographically:
// true if entry a comes first. Walks up the committed parents to the first
// common one.
__device__ bool fringe_lex_less(const PoolPlanShared& sh, int a, int b) {
    int pa = sh.fpar[a], pb = sh.fpar[b];
    if (pa == pb) return sh.frank[a] < sh.frank[b];
    while (sh.cpar[pa] != sh.cpar[pb]) {
        pa = sh.cpar[pa];
        pb = sh.cpar[pb];
    }
    return sh.crank[pa] < sh.crank[pb];
}

__device__ __forceinline__ double wave_max_d(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, kWave));
    return v;
}
__device__ __forceinline__ int wave_min_i(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, kWave));
    return v;
}

__global__ __launch_bounds__(kPlanPoolThreads) void pool_plan(int D, int P, int K, int B,
                                                              const uint64_t* __restrict__ lists,
                                                              const int* __restrict__ nfin,
                                                              const int32_t* __restrict__ pool_tok, tsb_tree tree,
                                                              int32_t* __restrict__ plan_tok,
                                                              int32_t* __restrict__ req_status) {
    __shared__ PoolPlanShared sh;
    const int r = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave;
    const int NL = 1 + (D - 1) * P;
    const uint64_t* G = lists + (size_t)r * NL * K;
    const bool bad = (req_status[r] & TSB_REQ_NONFINITE) != 0;

    // lists into LDS (all threads)
    const int nent = min(NL * K, kPoolListLds);
    for (int i = tid; i < nent; i += kPlanPoolThreads) {
        const int li = i / K, k = i % K;
        const uint64_t e = k < nfin[(size_t)r * NL + li] ? G[i] : 0ull;
        sh.llp[i] = entry_lp(e);
        sh.lslot[i] = (uint8_t)entry_slot(e);
    }
    for (int i = tid; i < NL; i += kPlanPoolThreads) sh.lnf[i] = (uint8_t)nfin[(size_t)r * NL + i];
    __syncthreads();
    if (tid >= kWave) return;

    const ListView LV{&sh, G, K, P};
    // root committed; its first child enters the fringe
    int ncom = 1, nf = 0;
    if (lane == 0) {
        sh.cscore[0] = 0.0;
        sh.cpar[0] = -1;
        sh.crank[0] = 0;
        sh.cdepth[0] = 0;
        sh.cslot[0] = 0;
        sh.cnch[0] = 0;
    }
    if (!bad && D > 0 && B > 0 && sh.lnf[0] > 0) {
        if (lane == 0) {
            sh.fscore[0] = 0.0 + (double)LV.lp(0, 0);
            sh.fpar[0] = 0;
            sh.frank[0] = 0;
            sh.fdepth[0] = 1;
        }
        nf = 1;
    }
    wave_lds_sync();

    while (ncom - 1 < B && nf > 0) {
        // best fringe entry: score desc, depth asc, rank path asc
        double bs = -INFINITY;
        int bd = 255, bi = -1, bc = 0;
        for (int i = lane; i < nf; i += kWave) {
            const double s = sh.fscore[i];
            const int dd = sh.fdepth[i];
            if (bi < 0 || s > bs || (s == bs && dd < bd)) {
                bs = s;
                bd = dd;
                bi = i;
                bc = 1;
            } else if (s == bs && dd == bd) {
                ++bc;
            }
        }
        const double ws = wave_max_d(bi >= 0 ? bs : -INFINITY);
        const int wd = wave_min_i(bi >= 0 && bs == ws ? bd : 255);
        const bool mine = bi >= 0 && bs == ws && bd == wd;
        const uint64_t m1 = __ballot(mine), m2 = __ballot(mine && bc >= 2);
        int b;
        if (__popcll(m1) == 1 && m2 == 0) {
            b = __builtin_amdgcn_readlane(bi, __ffsll((unsigned long long)m1) - 1);
        } else {  // equal score and depth: the lexicographically smaller rank path
            int best = -1;
            if (lane == 0)
                for (int i = 0; i < nf; ++i)
                    if (sh.fscore[i] == ws && sh.fdepth[i] == wd && (best < 0 || fringe_lex_less(sh, i, best)))
                        best = i;
            b = __builtin_amdgcn_readlane(best, 0);
        }
        // commit entry b
        const double s = sh.fscore[b];
        const int dd = sh.fdepth[b], p = sh.fpar[b], k = sh.frank[b];
        const int lip = LV.of(sh.cdepth[p], sh.cslot[p]);
        const int slot = LV.slot(lip, k);
        const int c = ncom++;
        // successors: c's first child, then its next younger sibling
        bool has_a = false, has_b = false;
        double sa = 0.0, sb = 0.0;
        if (dd < D) {
            const int lic = LV.of(dd, slot);
            if (sh.lnf[lic] > 0) {
                has_a = true;
                sa = s + (double)LV.lp(lic, 0);
            }
        }
        if (k + 1 < sh.lnf[lip]) {
            has_b = true;
            sb = sh.cscore[p] + (double)LV.lp(lip, k + 1);
        }
        wave_lds_sync();
        if (lane == 0) {
            sh.cscore[c] = s;
            sh.cpar[c] = (int16_t)p;
            sh.crank[c] = (uint8_t)k;
            sh.cdepth[c] = (uint8_t)dd;
            sh.cslot[c] = (uint8_t)slot;
            sh.cnch[c] = 0;
            sh.cnch[p] = (uint8_t)(k + 1);  // children are committed in rank order
            int at = b;
            if (has_a) {
                sh.fscore[at] = sa;
                sh.fpar[at] = (int16_t)c;
                sh.frank[at] = 0;
                sh.fdepth[at] = (uint8_t)(dd + 1);
                at = nf;
            }
            if (has_b) {
                sh.fscore[at] = sb;
                sh.fpar[at] = (int16_t)p;
                sh.frank[at] = (uint8_t)(k + 1);
                sh.fdepth[at] = (uint8_t)dd;
                at = nf;
            }
            if (!has_a && !has_b && b != nf - 1) {  // fill the hole with the last entry
                sh.fscore[b] = sh.fscore[nf - 1];
                sh.fpar[b] = sh.fpar[nf - 1];
                sh.frank[b] = sh.frank[nf - 1];
                sh.fdepth[b] = sh.fdepth[nf - 1];
            }
        }
        nf += (has_a && has_b) ? 1 : ((!has_a && !has_b) ? -1 : 0);
        wave_lds_sync();
    }

    // plan margin: last committed score - best uncommitted score
    double margin = INFINITY;
    {
        double m = -INFINITY;
        for (int i = lane; i < nf; i += kWave) m = fmax(m, sh.fscore[i]);
        m = wave_max_d(m);
        if (ncom > 1 && nf > 0) margin = sh.cscore[ncom - 1] - m;
    }

    // BFS layout: nodes bucketed by depth, then level by level the first
    // child of every node (prefix sums of the children counts in BFS order)
    const int n = ncom;
    for (int d = lane; d < TSB_MAX_D + 2; d += kWave) sh.dcnt[d] = 0;
    wave_lds_sync();
    for (int c = lane; c < n; c += kWave) atomicAdd(&sh.dcnt[sh.cdepth[c]], 1);
    wave_lds_sync();
    if (lane == 0) {
        int acc = 0;
        for (int d = 0; d <= D; ++d) {
            sh.dstart[d] = acc;
            acc += sh.dcnt[d];
            sh.dcnt[d] = 0;
        }
    }
    wave_lds_sync();
    for (int c = lane; c < n; c += kWave) {
        const int d = sh.cdepth[c];
        const int pos = atomicAdd(&sh.dcnt[d], 1);
        sh.bucket[sh.dstart[d] + pos] = (int16_t)c;
    }
    if (lane == 0) {
        sh.order[0] = 0;
        sh.bfs_of_pop[0] = 0;
    }
    wave_lds_sync();
    int lo = 0, hi = 1;
    for (int d = 0; d < D && hi > lo; ++d) {
        int next = hi;
        for (int base = lo; base < hi; base += kWave) {
            const int i = base + lane;
            const int cnt = i < hi ? (int)sh.cnch[sh.order[i]] : 0;
            int tot;
            const int off = wave_excl_scan<6>(cnt, tot);
            if (i < hi) sh.fcb[i] = (int16_t)(cnt > 0 ? next + off : -1);
            next += tot;
        }
        wave_lds_sync();
        const int b0 = sh.dstart[d + 1], b1 = b0 + (next - hi);
        for (int j = b0 + lane; j < b1; j += kWave) {
            const int c = sh.bucket[j];
            const int bp = sh.bfs_of_pop[sh.cpar[c]];
            const int bc = sh.fcb[bp] + sh.crank[c];
            sh.order[bc] = (int16_t)c;
            sh.bfs_of_pop[c] = (int16_t)bc;
        }
        wave_lds_sync();
        lo = hi;
        hi = next;
    }
    for (int i = lo + lane; i < hi; i += kWave) sh.fcb[i] = -1;  // the deepest level has no children
    wave_lds_sync();

    const size_t tb = (size_t)r * (B + 1);
    for (int i = lane; i <= B; i += kWave) {
        if (i < n) {
            const int c = sh.order[i];
            tree.parent[tb + i] = i == 0 ? -1 : (int32_t)sh.bfs_of_pop[sh.cpar[c]];
            tree.depth[tb + i] = sh.cdepth[c];
            tree.rank[tb + i] = i == 0 ? -1 : (int32_t)sh.crank[c];
            tree.n_children[tb + i] = sh.cnch[c];
            tree.first_child[tb + i] = sh.fcb[i];
            tree.score[tb + i] = sh.cscore[c];
            if (plan_tok)
                plan_tok[tb + i] = i == 0 ? -1
                                          : pool_tok[((size_t)r * D + (sh.cdepth[c] - 1)) * P + sh.cslot[c]];
        } else {
            tree.parent[tb + i] = -1;
            tree.depth[tb + i] = -1;
            tree.rank[tb + i] = -1;
            tree.n_children[tb + i] = -1;
            tree.first_child[tb + i] = -1;
            tree.score[tb + i] = 0.0;
            if (plan_tok) plan_tok[tb + i] = -1;
        }
    }
    if (lane == 0) {
        tree.n_nodes[r] = n;
        tree.plan_margin[r] = margin;
        if (!bad && n < B + 1) req_status[r] |= TSB_REQ_BUDGET_SHORT;
    }
}

// ------------------------------------------------------------------ replay
__device__ __forceinline__ double gumbel_f64(uint32_t w) { return -log(-log(u24d(w))); }

template <int DT>
__global__ __launch_bounds__(kPoolThreads) void pool_replay(int D, int V, int P, int B, float invT, const void* draft,
                                                            const float* __restrict__ trans,
                                                            const int32_t* __restrict__ pool_tok, tsb_tree tree,
                                                            uint32_t k0, uint32_t k1, uint32_t step,
                                                            int32_t* __restrict__ node_tok) {
    __shared__ int s_tok[TSB_MAX_D * kPoolMax];
    __shared__ float s_a[TSB_MAX_D * kPoolMax];
    __shared__ int16_t s_slot[TSB_MAX_B + 1];
    __shared__ int s_lvl[TSB_MAX_D + 2];
    const int r = blockIdx.x;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const size_t tb = (size_t)r * (B + 1);
    const int n = tree.n_nodes[r];

    for (int i = tid; i < D * P; i += kPoolThreads) {
        const int d = i / P;
        const int t = pool_tok[((size_t)r * D) * P + i];
        s_tok[i] = t;
        s_a[i] = (t >= 0 && t < V) ? load_logit<DT>(draft, ((size_t)r * D + d) * V + t) * invT : -INFINITY;
    }
    for (int d = tid; d < TSB_MAX_D + 2; d += kPoolThreads) s_lvl[d] = n;
    if (tid == 0) {
        s_lvl[0] = 0;
        s_slot[0] = -1;
    }
    __syncthreads();
    for (int i = 1 + tid; i < n; i += kPoolThreads) {
        const int di = tree.depth[tb + i];
        if (di != tree.depth[tb + i - 1]) s_lvl[di] = i;
    }
    for (int i = tid; i <= B; i += kPoolThreads) node_tok[tb + i] = -1;
    __syncthreads();

    RngKey key;
    key.k0 = k0;
    key.k1 = k1;
    key.request = (uint32_t)r;
    key.step = step;
    for (int d = 0; d < D; ++d) {
        const int lo = s_lvl[d], hi = s_lvl[d + 1];
        if (lo >= hi) break;
        for (int u = lo + wave; u < hi; u += kPoolWaves) {
            const int m = tree.n_children[tb + u];
            if (m <= 0) continue;
            const int fc = tree.first_child[tb + u];
            float z = -INFINITY;
            int tok = 0x7FFFFFFF;
            if (lane < P) {
                tok = s_tok[d * P + lane];
                z = s_a[d * P + lane];
                if (d > 0) z = corrected_logit(z, trans[trans_row(r, D, d, s_slot[u], P) + lane], invT);
            }
            const bool valid = lane < P && z > -INFINITY;
            const double kv =
                valid ? (double)z + gumbel_f64(rng_word(key, (uint32_t)u, kStreamReplay, (uint32_t)tok)) : -INFINITY;
            // rank under (key desc, token asc) among valid lanes
            int rank = 0;
            for (int k = 0; k < kWave; ++k) {
                const double ok = lane_f64(kv, k);
                const int ot = __builtin_amdgcn_readlane(tok, k);
                rank += (ok > kv || (ok == kv && ot < tok)) ? 1 : 0;
            }
            if (valid && rank < m) {
                node_tok[tb + fc + rank] = tok;
                s_slot[fc + rank] = (int16_t)lane;
            }
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------ launch
hipError_t launch_pool_plan(const tsb_config& c, int P, float invT, const void* draft, const float* trans,
                            int32_t* pool_tok, const tsb_tree& tree, int32_t* plan_tok, int32_t* req_status,
                            char* ws, hipStream_t st) {
    const Geometry g = geometry(c);
    const PoolWs w = pool_ws(c, P);
    uint64_t* pk = (uint64_t*)(ws + w.pk);
    int* pf = (int*)(ws + w.pf);
    uint64_t* lists = (uint64_t*)(ws + w.lists);
    int* nfin = (int*)(ws + w.nfin);
    hipError_t e = launch_pool_partials(c, P, invT, draft, pk, pf, req_status, st);
    if (e != hipSuccess) return e;
    if ((e = hook_before(TSB_KERNEL_POOL_LISTS, st)) != hipSuccess) return e;
    pool_lists<<<dim3(c.D, c.R), kPoolThreads, 0, st>>>(c.D, g.S1, P, c.K, invT, pk, pf, trans, pool_tok, lists,
                                                         nfin, req_status);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = hook_after(TSB_KERNEL_POOL_LISTS, st)) != hipSuccess) return e;
    if ((e = hook_before(TSB_KERNEL_POOL_PLAN, st)) != hipSuccess) return e;
    pool_plan<<<c.R, kPlanPoolThreads, 0, st>>>(c.D, P, c.K, c.B, lists, nfin, pool_tok, tree, plan_tok, req_status);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return hook_after(TSB_KERNEL_POOL_PLAN, st);
}

hipError_t launch_pool_replay(const tsb_config& c, int P, float invT, const void* draft, const float* trans,
                              const int32_t* pool_tok, const tsb_tree& tree, uint32_t step, int32_t* node_tok,
                              hipStream_t st) {
    hipError_t e = hook_before(TSB_KERNEL_POOL_REPLAY, st);
    if (e != hipSuccess) return e;
    const uint32_t k0 = (uint32_t)c.seed, k1 = (uint32_t)(c.seed >> 32);
    if (c.dtype == TSB_BF16)
        pool_replay<TSB_BF16><<<c.R, kPoolThreads, 0, st>>>(c.D, c.V, P, c.B, invT, draft, trans, pool_tok, tree, k0,
                                                             k1, step, node_tok);
    else
        pool_replay<TSB_F32><<<c.R, kPoolThreads, 0, st>>>(c.D, c.V, P, c.B, invT, draft, trans, pool_tok, tree, k0,
                                                            k1, step, node_tok);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return hook_after(TSB_KERNEL_POOL_REPLAY, st);
}

}  // namespace tsb
