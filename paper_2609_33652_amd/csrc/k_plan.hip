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

constexpr int kDraftUnroll = 1;  // 8-logit groups per thread per chunk

// STATS = false is the pool selection: the same candidate lists (K = pool
// size) and finiteness flags without the normaliser (pm, ps unused).
template <int DT, bool VEC, bool STATS>
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
    if (STATS) exp64_table_init(s_exp);

    float m = -INFINITY;    // running max of the scaled logits (-inf entries never raise it)
    double sum = 0.0;       // sum of e^(a - m) over this lane's elements
    bool bad = false;       // a NaN or +inf scaled logit
    WaveTopList top;
    top.init(K);
    // Filter (fx, fid): a logit x with id i can still be among the row's K best
    // only if x > fx, or x == fx and i <= fid (the key order is logit desc,
    // id asc). It starts at the K-th largest of the workgroup's column maxima
    // over its first chunk (K distinct logits at or above it exist) with any
    // id; then every wave whose list is full publishes its K-th key to s_key
    // (an LDS maximum) and all waves filter against the best published key.

    const int wave = tid / kWave, lane = tid % kWave;
    __shared__ float s_lm[kBlock / kWave][kWave];
    __shared__ unsigned long long s_key;
    float fx;
    uint32_t fid = 0xFFFFFFFFu;
    {
        float lm = -INFINITY;
#pragma unroll
        for (int u = 0; u < kDraftUnroll; ++u)
#pragma unroll
            for (int j = 0; j < 8; ++j) lm = fmaxf(lm, xc[u][j]);
        s_lm[wave][lane] = isnan(lm) ? -INFINITY : lm;
        if (tid == 0) s_key = 0ull;
        __syncthreads();
        float cm = s_lm[0][lane];
#pragma unroll
        for (int w = 1; w < kBlock / kWave; ++w) cm = fmaxf(cm, s_lm[w][lane]);
        fx = wave_kth_largest(cm, K);
    }
    uint64_t pub = 0;  // the key this wave last published

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
        // row statistics first, as one straight-line block (the exps of all
        // groups interleave), then the candidate filter
        float xm[kDraftUnroll];
        float a[kDraftUnroll][8];
        float am = -INFINITY;
#pragma unroll
        for (int u = 0; u < kDraftUnroll; ++u) {
            xm[u] = xc[u][0];
#pragma unroll
            for (int j = 1; j < 8; ++j) xm[u] = fmaxf(xm[u], xc[u][j]);  // NaN is ignored
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                a[u][j] = xc[u][j] * invT;
                bad |= __builtin_amdgcn_classf(a[u][j], 0x203);  // signalling NaN, quiet NaN, +inf
            }
            am = fmaxf(am, xm[u] * invT);  // rounding is monotone: the scaled max is the max of the scaled
        }
        if (STATS && am > m && am < INFINITY) {
            sum = (m == -INFINITY) ? 0.0 : sum * exp64((double)m - (double)am, s_exp);
            m = am;
        }
        if (STATS) {
            const double md = (double)m;
            double s2[2] = {0.0, 0.0};
#pragma unroll
            for (int u = 0; u < kDraftUnroll; ++u)
#pragma unroll
                for (int j = 0; j < 8; ++j) s2[j & 1] += exp64((double)a[u][j] - md, s_exp);
            sum += s2[0] + s2[1];
        }
#pragma unroll
        for (int u = 0; u < kDraftUnroll; ++u) {
            const int i0 = base + (u * kBlock + tid) * 8;
            // the group's smallest id is i0
            if (__ballot(xm[u] > fx || (xm[u] == fx && (uint32_t)i0 <= fid))) {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const float xj = xc[u][j];
                    const uint32_t id = (uint32_t)(i0 + j);
                    const bool ok = (i0 + j < hi) && (xj > fx || (xj == fx && id <= fid));  // false for NaN
                    top.offer_xid(xj, id, ok);
                }
                if (top.thr > pub) {  // publish this wave's K-th key
                    pub = top.thr;
                    if (lane == 0) atomicMax(&s_key, (unsigned long long)pub);
                }
            }
        }
        {
            // entering needs a key above the best published K-th key
            const uint64_t sk = *(volatile unsigned long long*)&s_key;
            if (sk) {
                const float tx = cand_value(sk);
                const uint32_t tid1 = cand_id(sk);
                if (tx > fx || (tx == fx && tid1 <= fid)) {
                    fx = tx;
                    fid = tid1 - 1;  // wraps for id 0 to "any id": looser, and offer re-checks the key
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
    const float wm = wave_max(m);
    double contrib = (m == -INFINITY) ? 0.0 : sum * exp((double)m - (double)wm);
    const double ws = STATS ? wave_sum(contrib) : 0.0;
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
            if (STATS) {
                pm[o] = M;
                ps[o] = tot;
            }
            pf[o] = anybad;
        }
        if (lane < K) pk[((size_t)row * S + s) * K + lane] = top.v;
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
// node score below tau (-inf if none; meaningful without overflow).
__device__ int plan_count(const PlanShared& sh, int Dp, int K, double tau, int cap, double* buf, double& m_out) {
    const int lane = lane_id();
    int total = 0;
    int plo = 0, phi = 0;  // parents of the current level in buf; level 0: the root
    double m = -INFINITY;
    for (int k = 0; k < Dp; ++k) {
        const int kk = sh.kfin[k];
        const float lpv = lane < kk ? sh.lp[k * K + lane] : -INFINITY;
        const int np = k == 0 ? 1 : phi - plo;
        const int nstart = total;
        for (int base = 0; base < np; base += kWave) {
            const int i = base + lane;
            const bool valid = i < np;
            const double s = (valid && k > 0) ? buf[plo + i] : 0.0;
            int c = 0;
            bool done = !valid;
            for (int j = 0; j < kk; ++j) {
                const double cs = s + (double)lane_f32(lpv, j);
                const bool ok = valid && cs >= tau;
                if (!done && !ok) {
                    m = fmax(m, cs);  // the parent's best child below tau
                    done = true;
                }
                if (!__ballot(ok)) break;
                c += ok ? 1 : 0;
            }
            int tot;
            const int off = wave_excl_scan<6>(c, tot);
            if (total + tot > cap) {
                m_out = -INFINITY;
                return cap + 1;
            }
            for (int j = 0; __ballot(j < c); ++j) {
                const float lj = lane_f32(lpv, j);
                if (j < c) buf[total + off + j] = s + (double)lj;
            }
            total += tot;
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
                                                          int32_t* __restrict__ req_status) {
    __shared__ PlanShared sh;
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

    // ---- threshold search (uniform control flow across the workgroup)
    const int cap = 2 * (B + 1);
    const int ns = min(kPlanWaves, kPlanBuf / cap);
    double hi_m = (Dp > 0 && sh.kfin[0] > 0) ? (double)sh.lp[0] : -INFINITY;  // the best node's score
    int hi_cnt = 0;
    double lo = -INFINITY;
    int mode = 3;  // 1: t* = hi_m; 2: t* selected in a wave's buffer; 3: every node is chosen
    int src = -1;
    // every round raises count(hi) by at least one (at most B + 1 rounds); the
    // guard only bounds the loop
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
    int n = 1, plo = 0, phi = 1;
    for (int k = 0; k < Dp && plo < phi; ++k) {
        const int kk = sh.kfin[k];
        const float lpv = lane < kk ? sh.lp[k * K + lane] : -INFINITY;
        for (int base = plo; base < phi; base += kWave) {
            const int i = base + lane;
            const bool valid = i < phi;
            const double s = valid ? sh.u.t.score[i] : 0.0;
            int cg = 0, ce = 0;
            for (int j = 0; j < kk; ++j) {
                const double cs = s + (double)lane_f32(lpv, j);
                const bool gt = valid && cs > tstar;
                const bool eq = valid && cs == tstar;
                if (!__ballot(gt || eq)) break;
                cg += gt ? 1 : 0;
                ce += eq ? 1 : 0;
            }
            int etot;
            const int eoff = wave_excl_scan<6>(ce, etot);
            const int adm = max(0, min(ce, quota - eoff));
            if (etot > 0 && quota > 0) tie_admitted = true;
            quota -= min(etot, quota);
            const int c = cg + adm;
            int tot;
            const int off = wave_excl_scan<6>(c, tot);
            for (int j = 0; __ballot(j < c); ++j) {
                const float lj = lane_f32(lpv, j);
                if (j < c && n + off + j <= B) {  // always true: the admitted nodes number at most B
                    const int x = n + off + j;
                    const double cs = s + (double)lj;
                    sh.u.t.score[x] = cs;
                    sh.u.t.par[x] = i;
                    sh.u.t.rank[x] = j;
                    sh.u.t.depth[x] = k + 1;
                    minsc = fmin(minsc, cs);
                }
            }
            if (valid) {
                sh.u.t.nch[i] = c;
                sh.u.t.fc[i] = c ? n + off : -1;
            }
            n = min(n + tot, B + 1);
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
                // the W-th largest score of the layer (with multiplicity)
                WaveTopList tl;
                tl.init(W);
                for (int base = lb; base < le; base += kWave) {
                    const int i = base + lane;
                    tl.offer(i < le ? ordered_bits64(sh.score[i]) : 0ull, i < le);
                }
                const uint64_t tk = lane_u64(tl.v, W - 1);
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
hipError_t launch_plan(const tsb_config& c, float invT, const void* draft, double* draft_lse, int32_t* topk_tok,
                       float* topk_lp, const tsb_tree& tree, int32_t* req_status, char* ws, hipStream_t st,
                       int frontier) {
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
            draft_partials<TSB_BF16, true, true><<<grid1, kBlock, 0, st>>>(draft, c.V, c.D, g.seg1, g.S1, invT, c.K, pm, ps,
                                                                     pk, pf, req_status);
        else
            draft_partials<TSB_BF16, false, true><<<grid1, kBlock, 0, st>>>(draft, c.V, c.D, g.seg1, g.S1, invT, c.K, pm, ps,
                                                                      pk, pf, req_status);
    } else {
        if (vec)
            draft_partials<TSB_F32, true, true><<<grid1, kBlock, 0, st>>>(draft, c.V, c.D, g.seg1, g.S1, invT, c.K, pm, ps,
                                                                    pk, pf, req_status);
        else
            draft_partials<TSB_F32, false, true><<<grid1, kBlock, 0, st>>>(draft, c.V, c.D, g.seg1, g.S1, invT, c.K, pm, ps,
                                                                     pk, pf, req_status);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((e = hook_after(TSB_KERNEL_DRAFT_PARTIALS, st)) != hipSuccess) return e;
    if ((e = hook_before(TSB_KERNEL_PLAN_TREE, st)) != hipSuccess) return e;
    if (frontier > 0)
        plan_ep<<<c.R, kPlanThreads, 0, st>>>(c.D, g.S1, c.K, c.B, frontier, invT, pm, ps, pk, pf, draft_lse,
                                              topk_tok, topk_lp, tree, req_status);
    else
        plan_tree<<<c.R, kPlanThreads, 0, st>>>(c.D, g.S1, c.K, c.B, invT, pm, ps, pk, pf, draft_lse, topk_tok,
                                                topk_lp, tree, req_status);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return hook_after(TSB_KERNEL_PLAN_TREE, st);
}

hipError_t launch_pool_partials(const tsb_config& c, int P, float invT, const void* draft, uint64_t* pk, int* pf,
                                int32_t* req_status, hipStream_t st) {
    const Geometry g = geometry(c);
    const dim3 grid1(g.S1, c.R * c.D);
    hipError_t e = hook_before(TSB_KERNEL_POOL_PARTIALS, st);
    if (e != hipSuccess) return e;
    const bool vec = (c.dtype == TSB_BF16) ? (c.V % 8 == 0 && ((uintptr_t)draft & 15) == 0)
                                           : (c.V % 4 == 0 && ((uintptr_t)draft & 15) == 0);
    if (c.dtype == TSB_BF16) {
        if (vec)
            draft_partials<TSB_BF16, true, false><<<grid1, kBlock, 0, st>>>(draft, c.V, c.D, g.seg1, g.S1, invT, P,
                                                                            nullptr, nullptr, pk, pf, req_status);
        else
            draft_partials<TSB_BF16, false, false><<<grid1, kBlock, 0, st>>>(draft, c.V, c.D, g.seg1, g.S1, invT, P,
                                                                             nullptr, nullptr, pk, pf, req_status);
    } else {
        if (vec)
            draft_partials<TSB_F32, true, false><<<grid1, kBlock, 0, st>>>(draft, c.V, c.D, g.seg1, g.S1, invT, P,
                                                                           nullptr, nullptr, pk, pf, req_status);
        else
            draft_partials<TSB_F32, false, false><<<grid1, kBlock, 0, st>>>(draft, c.V, c.D, g.seg1, g.S1, invT, P,
                                                                            nullptr, nullptr, pk, pf, req_status);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
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
