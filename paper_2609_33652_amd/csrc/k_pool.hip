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
//   pool_plan    one workgroup per request: the first B rank paths under the
//                static order over the per-node candidate lists, found by
//                the threshold search of the vocabulary-wide planner (path
//                scores never grow toward children or younger siblings, so
//                the nodes scoring at least a threshold form a subtree that
//                a level-by-level count enumerates; here a node's children
//                come from its own list, and nodes carry their pool slot),
//                then emitted in BFS order.
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
// and the slots in (lp desc, slot asc) order by a sort of the 64 keys.
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
        uint64_t v[1];
        v[0] = valid ? ((uint64_t)ordered_bits(lp) << 32) | (uint32_t)(~lane) : 0ull;
        wave_sort_desc<1>(v);
        // lane k holds the k-th slot; its lp bits are taken from that slot's lane
        const int slot = (int)(~(uint32_t)v[0]) & (kWave - 1);
        const float lps = __shfl(lp, slot, kWave);
        if (lane < K && v[0] != 0ull) out[lane] = pack_entry(lps, slot);
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
    // the transition rows of this wave's lists are fetched before the merge
    constexpr int kListsPerWave = (kPoolMax + kPoolWaves - 1) / kPoolWaves;
    float cv[kListsPerWave];
#pragma unroll
    for (int q = 0; q < kListsPerWave; ++q) {
        const int i = wave + q * kPoolWaves;
        cv[q] = (d > 0 && i < P && lane < P) ? trans[trans_row(r, D, d, i, P) + lane] : 0.0f;
    }

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
        } else if (n <= 2 * kWave) {
            uint64_t v[2];
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const int i = q * kWave + lane;
                v[q] = i < n ? pk[o * P + i] : 0ull;
            }
            wave_sort_desc<2>(v);
            best = lane < P ? v[0] : 0ull;
        } else if (n <= 4 * kWave) {
            // a bitonic sort of up to 256 keys: the pool is the first P
            uint64_t v[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int i = q * kWave + lane;
                v[q] = i < n ? pk[o * P + i] : 0ull;
            }
            wave_sort_desc<4>(v);
            best = lane < P ? v[0] : 0ull;
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
#pragma unroll
    for (int q = 0; q < kListsPerWave; ++q) {
        const int i = wave + q * kPoolWaves;
        if (i >= P) break;
        float z = -INFINITY;
        if (lane < P) {
            const float c = cv[q];
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
constexpr int kPlanPoolWaves = 16;
constexpr int kPlanPoolThreads = kPlanPoolWaves * kWave;
constexpr int kPoolPlanBuf = 6144;  // (score, slot) records shared by the counting waves

struct PoolPlanShared {
    float llp[kPoolListLds];
    uint8_t lslot[kPoolListLds];
    uint8_t lnf[kPoolListsMax];
    double piv[kPlanPoolWaves];
    double mval[kPlanPoolWaves];
    int cnt[kPlanPoolWaves];
    double tstar;
    int g;
    union {
        struct {
            double score[kPoolPlanBuf];
            uint8_t slot[kPoolPlanBuf];
        } b;
        struct {
            double score[TSB_MAX_B + 1];
            int par[TSB_MAX_B + 1];
            int rank[TSB_MAX_B + 1];
            int depth[TSB_MAX_B + 1];
            int nch[TSB_MAX_B + 1];
            int fc[TSB_MAX_B + 1];
            uint8_t slot[TSB_MAX_B + 1];
        } t;
    } u;
};

// Entry k of list li (LDS, or the workspace beyond the LDS copy).
__device__ __forceinline__ float list_lp(const PoolPlanShared& sh, const uint64_t* g, int K, int li, int k) {
    const int i = li * K + k;
    return i < kPoolListLds ? sh.llp[i] : entry_lp(g[i]);
}
__device__ __forceinline__ int list_slot(const PoolPlanShared& sh, const uint64_t* g, int K, int li, int k) {
    const int i = li * K + k;
    return i < kPoolListLds ? (int)sh.lslot[i] : entry_slot(g[i]);
}
// list of the children of a node at `depth` whose token holds `slot`
__device__ __forceinline__ int list_of(int P, int depth, int slot) { return depth == 0 ? 0 : 1 + (depth - 1) * P + slot; }

__device__ __forceinline__ int lanes_below(uint64_t b) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0u));
}

__device__ __forceinline__ double wave_max_d(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, kWave));
    return v;
}
__device__ __forceinline__ double wave_min_d(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmin(v, __shfl_xor(v, o, kWave));
    return v;
}

// Number of nodes (root excluded) scoring at least tau, level by level, with
// their (score, slot) stored in (bs, bsl); cap + 1 once more than cap.
// m_out: the largest node score below tau (-inf if none; meaningful without
// overflow). Lane l takes candidate l % K of parent l / K.
__device__ int pool_count(const PoolPlanShared& sh, const uint64_t* G, int P, int Dp, int K, double tau, int cap,
                          double* bs, uint8_t* bsl, double& m_out) {
    const int lane = lane_id();
    const int per = kWave / K;
    const int pp = lane / K, pj = lane - pp * K;
    int total = 0;
    int plo = 0, phi = 0;  // parents of the current level in the buffer; level 0: the root
    double m = -INFINITY;
    for (int k = 0; k < Dp; ++k) {
        const int np = k == 0 ? 1 : phi - plo;
        const int nstart = total;
        for (int base = 0; base < np; base += per) {
            const int i = base + pp;
            const bool par_ok = pp < per && i < np;
            const double s = (par_ok && k > 0) ? bs[plo + i] : 0.0;
            const int li = list_of(P, k, (par_ok && k > 0) ? (int)bsl[plo + i] : 0);
            const bool valid = par_ok && pj < (int)sh.lnf[li];
            const double cs = valid ? s + (double)list_lp(sh, G, K, li, pj) : -INFINITY;
            const bool ok = valid && cs >= tau;
            if (valid && !ok) m = fmax(m, cs);  // children below tau (the best of them counts)
            const uint64_t b = __ballot(ok);
            const int cnt = __popcll(b);
            if (total + cnt > cap) {
                m_out = -INFINITY;
                return cap + 1;
            }
            if (ok) {
                const int x = total + lanes_below(b);
                bs[x] = cs;
                bsl[x] = (uint8_t)list_slot(sh, G, K, li, pj);
            }
            total += cnt;
        }
        __threadfence_block();  // the next level reads these records from other lanes
        plo = nstart;
        phi = total;
        if (phi == plo) break;
    }
    m_out = wave_max_d(m);
    return total;
}

__global__ __launch_bounds__(kPlanPoolThreads) void pool_plan(int D, int P, int K, int B,
                                                              const uint64_t* __restrict__ lists,
                                                              const int* __restrict__ nfin,
                                                              const int32_t* __restrict__ pool_tok, tsb_tree tree,
                                                              int32_t* __restrict__ plan_tok,
                                                              int32_t* __restrict__ req_status) {
    __shared__ PoolPlanShared sh;
    const int r = blockIdx.x;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    const int NL = 1 + (D - 1) * P;
    const uint64_t* G = lists + (size_t)r * NL * K;
    const bool bad = (req_status[r] & TSB_REQ_NONFINITE) != 0;

    // lists into LDS
    const int nent = min(NL * K, kPoolListLds);
    for (int i = tid; i < nent; i += kPlanPoolThreads) {
        const int li = i / K, k = i % K;
        const uint64_t e = k < nfin[(size_t)r * NL + li] ? G[i] : 0ull;
        sh.llp[i] = entry_lp(e);
        sh.lslot[i] = (uint8_t)entry_slot(e);
    }
    for (int i = tid; i < NL; i += kPlanPoolThreads) sh.lnf[i] = (uint8_t)nfin[(size_t)r * NL + i];
    __syncthreads();
    const int Dp = (bad || B == 0) ? 0 : D;

    // ---- threshold search (uniform control flow across the workgroup), as
    // in the vocabulary-wide planner
    // a count succeeds when it lands in [B + 1, cap]: a narrow window keeps
    // every count short (measured best at 1.25 (B + 1) over the workloads),
    // at the price of a round more now and then
    const int cap = (5 * (B + 1) + 3) / 4;
    const int ns = min(kPlanPoolWaves, kPoolPlanBuf / cap);
    double hi_m = (Dp > 0 && sh.lnf[0] > 0) ? (double)sh.llp[0] : -INFINITY;  // the best node's score
    int hi_cnt = 0;
    double lo = -INFINITY;
    int mode = 3;  // 1: t* = hi_m; 2: t* selected in a wave's buffer; 3: every node is chosen
    int src = -1;
    for (int round = 0; hi_m > -INFINITY; ++round) {
        if (round > B + 1) {
            mode = 1;
            break;
        }
        if (wave < ns) {
            const double tau = wave == 0 ? hi_m
                               : (lo > -INFINITY ? hi_m - (hi_m - lo) * ((double)wave / (double)ns)
                                                 : hi_m - 0.25 * exp2(0.5 * (double)(wave - 1)));
            double m;
            const int c = pool_count(sh, G, P, Dp, K, tau, cap, sh.u.b.score + wave * cap, sh.u.b.slot + wave * cap, m);
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
        const double* b = sh.u.b.score + src * cap;
        for (int i = tid; i < c; i += kPlanPoolThreads) {
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

    // ---- emission in BFS order (wave 0): lane l takes candidate l % K of
    // parent l / K; the admitted children of a parent are a prefix of its list
    const double tstar = sh.tstar;
    int quota = mode == 3 ? 0 : B - sh.g;  // nodes scoring exactly t* still admitted
    bool tie_admitted = false;
    double minsc = INFINITY;
    if (lane == 0) {
        sh.u.t.score[0] = 0.0;
        sh.u.t.par[0] = -1;
        sh.u.t.rank[0] = -1;
        sh.u.t.depth[0] = 0;
        sh.u.t.slot[0] = 0;
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    const int per = kWave / K;
    const int pp = lane / K, pj = lane - pp * K;
    int n = 1, plo = 0, phi = 1;
    for (int k = 0; k < Dp && plo < phi; ++k) {
        for (int base = plo; base < phi; base += per) {
            const int i = base + pp;
            const bool par_ok = pp < per && i < phi;
            const double s = par_ok ? sh.u.t.score[i] : 0.0;
            const int li = list_of(P, k, par_ok ? (int)sh.u.t.slot[i] : 0);
            const bool valid = par_ok && pj < (int)sh.lnf[li];
            const double cs = valid ? s + (double)list_lp(sh, G, K, li, pj) : -INFINITY;
            const bool gt = valid && cs > tstar;
            const bool eq = valid && cs == tstar;
            // nodes scoring exactly t* are admitted in (depth, rank path)
            // order, which is lane order here
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
                    sh.u.t.slot[x] = (uint8_t)list_slot(sh, G, K, li, pj);
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
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        plo = phi;
        phi = n;
    }
    for (int i = plo + lane; i < phi; i += kWave) {  // the last level has no children
        sh.u.t.nch[i] = 0;
        sh.u.t.fc[i] = -1;
    }
    minsc = wave_min_d(minsc);
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");

    const size_t tb = (size_t)r * (B + 1);
    for (int i = lane; i <= B; i += kWave) {
        if (i < n) {
            tree.parent[tb + i] = sh.u.t.par[i];
            tree.depth[tb + i] = sh.u.t.depth[i];
            tree.rank[tb + i] = sh.u.t.rank[i];
            tree.n_children[tb + i] = sh.u.t.nch[i];
            tree.first_child[tb + i] = sh.u.t.fc[i];
            tree.score[tb + i] = sh.u.t.score[i];
            if (plan_tok)
                plan_tok[tb + i] = i == 0 ? -1 : pool_tok[((size_t)r * D + (sh.u.t.depth[i] - 1)) * P + sh.u.t.slot[i]];
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
        // margin: score of the B-th node in the order minus that of the (B+1)-th
        double margin = (double)INFINITY;
        if (mode != 3 && n > 1) margin = (tie_admitted ? tstar : minsc) - tstar;
        tree.n_nodes[r] = n;
        tree.plan_margin[r] = margin;
        if (!bad && n < B + 1) req_status[r] |= TSB_REQ_BUDGET_SHORT;
    }
}

// ------------------------------------------------------------------ replay
__device__ __forceinline__ double gumbel_f64(uint32_t w) { return -log(-log(u24d(w))); }

// Internal nodes whose Gumbel draws are computed before the layer walk.
constexpr int kReplayGCap = 128;

// Exact rank of lane's key under (key desc, token asc) among the wave's 64
// keys (invalid lanes carry -inf); used when two valid keys are equal.
__device__ __forceinline__ int rank_exact(double kv, int tok) {
    int rank = 0;
    for (int k = 0; k < kWave; ++k) {
        const double ok = lane_f64(kv, k);
        const int ot = __builtin_amdgcn_readlane(tok, k);
        rank += (ok > kv || (ok == kv && ot < tok)) ? 1 : 0;
    }
    return rank;
}

constexpr int kReplayMatRegs = (kPoolMax * kPoolMax) / kPoolThreads;

// LDS state of the pool replay walk.
struct PoolReplayLds {
    const int* tok;        // [D][P] pool tokens
    const float* a;        // [D][P] tempered draft logits
    const double* g;       // [kReplayGCap][kPoolMax] Gumbel draws of internal nodes
    const uint16_t* in;    // internal nodes: node | depth << 10
    const int16_t* m;      // child count of internal node q
    const int16_t* fc;     // first child of internal node q
    int16_t* slot;         // pool slot of every node's replayed token
    int* ntok;             // replayed token of every node
    uint64_t* key;         // [waves][64] keys of a wave's parent
    int8_t* pos;           // [waves][64] rank claims
};

// Transition matrix j of a request into registers; every thread loads every
// time (the index is clamped into the matrix, entries past its end land in
// the unused tail of the LDS buffer), so the loads are issued unconditionally.
__device__ __forceinline__ void fetch_matrix(float (&v)[kReplayMatRegs], const float* src, size_t base, int mat,
                                             int tid) {
#pragma unroll
    for (int k = 0; k < kReplayMatRegs; ++k) v[k] = src[base + min(tid + k * kPoolThreads, mat - 1)];
}
__device__ __forceinline__ void store_matrix(float* buf, const float (&v)[kReplayMatRegs], int tid) {
#pragma unroll
    for (int k = 0; k < kReplayMatRegs; ++k) buf[tid + k * kPoolThreads] = v[k];
}

// The parents of layer d (internal nodes lo..hi-1), one wave each: lane j
// scores pool slot j under the parent's replayed slot (matrix tr of position
// d - 1), and the m largest keys give the children in rank order.
__device__ __forceinline__ void replay_parents(const PoolReplayLds& L, int d, int lo, int hi, int P, float invT,
                                               const float* tr, const RngKey& key, int wave, int lane) {
    for (int g = lo + wave; g < hi; g += kPoolWaves) {
        const int u = L.in[g] & 1023;
        const int m = L.m[g], fc = L.fc[g];
        float z = -INFINITY;
        int tok = 0x7FFFFFFF;
        if (lane < P) {
            tok = L.tok[d * P + lane];
            z = L.a[d * P + lane];
            if (d > 0) z = corrected_logit(z, tr[L.slot[u] * P + lane], invT);
        }
        const bool valid = lane < P && z > -INFINITY;
        double kv = -INFINITY;
        if (valid) {
            const double G = g < kReplayGCap ? L.g[g * kPoolMax + lane]
                                             : gumbel_f64(rng_word(key, (uint32_t)u, kStreamReplay, (uint32_t)tok));
            kv = (double)z + G;
        }
        const uint64_t kb = valid ? ordered_bits64(kv) : 0ull;
        uint64_t* wk = L.key + wave * kWave;
        wk[lane] = kb;
        wave_lds_fence();
        int rank = 0;
#pragma unroll 16
        for (int k = 0; k < kWave; ++k) rank += wk[k] > kb ? 1 : 0;
        // equal keys among the first m share a count: each claims its
        // position, and a lane that lost its claim sends the wave to the exact
        // ranking
        wave_lds_fence();
        int8_t* wp = L.pos + wave * kWave;
        const bool top = valid && rank < m;
        if (top) wp[rank] = (int8_t)lane;
        wave_lds_fence();
        if (__ballot(top && wp[rank] != lane)) rank = rank_exact(kv, valid ? tok : 0x7FFFFFFF);
        wave_lds_fence();
        if (valid && rank < m) {
            L.ntok[fc + rank] = tok;
            L.slot[fc + rank] = (int16_t)lane;
        }
    }
}

// One workgroup per request. Set-up, all waves at once: the pool tokens and
// their tempered draft logits, the internal nodes in BFS order with their
// depth, first child and child count, and the Gumbel draws of the first
// kReplayGCap internal nodes (the draws depend on the node and the pool token
// only). Then layer by layer, one wave per parent: the transition matrix of
// the layer sits in LDS, fetched into registers two layers ahead (two
// register sets, the walk unrolled by two), and a lane's rank is the count of
// larger keys, read back from LDS. Replayed tokens stay in LDS until the end.
template <int DT>
__global__ __launch_bounds__(kPoolThreads) void pool_replay(int D, int V, int P, int B, float invT, const void* draft,
                                                            const float* __restrict__ trans,
                                                            const int32_t* __restrict__ pool_tok, tsb_tree tree,
                                                            uint32_t k0, uint32_t k1, uint32_t step,
                                                            int32_t* __restrict__ node_tok) {
    __shared__ int s_tok[TSB_MAX_D * kPoolMax];
    __shared__ float s_a[TSB_MAX_D * kPoolMax];
    __shared__ float s_tr[2][kPoolMax * kPoolMax];
    __shared__ double s_g[kReplayGCap * kPoolMax];
    __shared__ uint64_t s_key[kPoolWaves][kWave];
    __shared__ int8_t s_pos[kPoolWaves][kWave];
    __shared__ int16_t s_slot[TSB_MAX_B + 1];
    __shared__ int s_ntok[TSB_MAX_B + 1];
    __shared__ uint16_t s_int[TSB_MAX_B + 1];  // node | depth << 10
    __shared__ int16_t s_fc[TSB_MAX_B + 1];
    __shared__ int16_t s_m[TSB_MAX_B + 1];
    __shared__ int s_ilvl[TSB_MAX_D + 2];
    __shared__ int s_wcnt[kPoolWaves];
    static_assert(TSB_MAX_B + 1 <= kPoolThreads, "one thread per node");
    static_assert(TSB_MAX_B + 1 <= 1024 && TSB_MAX_D <= 64, "node | depth << 10 fits 16 bits");
    static_assert(kReplayMatRegs * kPoolThreads == kPoolMax * kPoolMax, "matrix split over the threads");
    const int r = blockIdx.x;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const size_t tb = (size_t)r * (B + 1);
    const int nn = tree.n_nodes[r];
    const int n = tree_count_ok(nn, B) ? nn : 0;  // a request with an unusable count is not replayed
    // transition matrices of the request (with D = 1 there are none: the
    // fetches then read pool_tok[0] and their values are never used)
    const bool has_t = D > 1;
    const float* tsrc = has_t ? trans : (const float*)pool_tok;
    const int mat = has_t ? P * P : 1;
    const size_t trb = has_t ? (size_t)r * (D - 1) * mat : 0;
    const int jmax = has_t ? D - 2 : 0;

    for (int i = tid; i < D * P; i += kPoolThreads) {
        const int d = i / P;
        const int t = pool_tok[((size_t)r * D) * P + i];
        s_tok[i] = t;
        s_a[i] = (t >= 0 && t < V) ? load_logit<DT>(draft, ((size_t)r * D + d) * V + t) * invT : -INFINITY;
    }
    for (int i = tid; i <= B; i += kPoolThreads) {
        s_ntok[i] = -1;
        s_slot[i] = 0;  // every node below the root gets its slot from its parent's layer
    }
    // internal nodes in BFS order (their depths are contiguous from 0); a
    // malformed node (entries out of range, see tree_node) is not replayed
    TreeNode nd{0, 0, 0, false};
    if (tid < n) nd = tree_node(tree, tb, tid, n, D);
    const bool internal = nd.ok && nd.m > 0;
    const uint64_t bal = __ballot(internal);
    const int below = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
    if (lane == 0) s_wcnt[wave] = __popcll(bal);
    __syncthreads();
    int q = below, n_int = 0;
    for (int w = 0; w < kPoolWaves; ++w) {
        const int c = s_wcnt[w];
        q += w < wave ? c : 0;
        n_int += c;
    }
    if (internal) {
        s_int[q] = (uint16_t)(tid | (nd.d << 10));
        s_fc[q] = (int16_t)nd.fc;
        s_m[q] = (int16_t)nd.m;
    }
    for (int d = tid; d < TSB_MAX_D + 2; d += kPoolThreads) s_ilvl[d] = n_int;
    __syncthreads();
    if (tid < n_int) {
        const int dep = s_int[tid] >> 10;
        if (tid == 0 || (s_int[tid - 1] >> 10) != dep) s_ilvl[dep] = tid;
    }

    RngKey key;
    key.k0 = k0;
    key.k1 = k1;
    key.request = (uint32_t)r;
    key.step = step;
    float ra[kReplayMatRegs], rb[kReplayMatRegs];
    fetch_matrix(rb, tsrc, trb, mat, tid);  // position 0, stored after layer 0
    const int ng = n_int < kReplayGCap ? n_int : kReplayGCap;
    for (int g = wave; g < ng; g += kPoolWaves) {
        const int u = s_int[g] & 1023, d = s_int[g] >> 10;
        if (lane < P) s_g[g * kPoolMax + lane] = gumbel_f64(rng_word(key, (uint32_t)u, kStreamReplay,
                                                                       (uint32_t)s_tok[d * P + lane]));
    }
    __syncthreads();

    PoolReplayLds L;
    L.tok = s_tok;
    L.a = s_a;
    L.g = s_g;
    L.in = s_int;
    L.m = s_m;
    L.fc = s_fc;
    L.slot = s_slot;
    L.ntok = s_ntok;
    L.key = &s_key[0][0];
    L.pos = &s_pos[0][0];
    // layer d reads the matrix of position d - 1 from buffer (d - 1) & 1 and
    // stores that of position d (fetched during layer d - 1) into buffer d & 1
    for (int d = 0; d < D; d += 2) {
        int lo = s_ilvl[d], hi = s_ilvl[d + 1];
        if (lo >= hi) break;
        fetch_matrix(ra, tsrc, trb + (size_t)min(d + 1, jmax) * mat, mat, tid);
        replay_parents(L, d, lo, hi, P, invT, s_tr[1], key, wave, lane);
        store_matrix(s_tr[0], rb, tid);
        __syncthreads();
        if (d + 1 >= D) break;
        lo = s_ilvl[d + 1];
        hi = s_ilvl[d + 2];
        if (lo >= hi) break;
        fetch_matrix(rb, tsrc, trb + (size_t)min(d + 2, jmax) * mat, mat, tid);
        replay_parents(L, d + 1, lo, hi, P, invT, s_tr[0], key, wave, lane);
        store_matrix(s_tr[1], ra, tid);
        __syncthreads();
    }
    for (int i = tid; i <= B; i += kPoolThreads) node_tok[tb + i] = s_ntok[i];
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
