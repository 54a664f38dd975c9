// Verification of the replayed tree on gfx950 (Section 2.3, eq. (1);
// Appendix A: recursive rejection sampling without replacement; Section 3.3:
// the probabilities are those of the replayed candidates).
//
//   target_partials  grid (segment, request x node): one streaming read of
//                    every target row of the tree; online max and sum of
//                    exp per segment (binary32 terms, binary64 per lane).
//   verify_walk      cooperative grid (G workgroups per request). All G
//                    workgroups of a request replay the same scalar walk;
//                    every vocabulary-wide reduction of the walk (residual
//                    mass after a rejection, the bonus draw) is split over
//                    them and exchanged through a per-request barrier.
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

#include "tsb_device.hpp"
#include "tsb_kernels.hpp"

namespace tsb {

// ------------------------------------------------------------------ K4
template <int DT, bool VEC>
__global__ __launch_bounds__(kBlock) void target_partials(const void* __restrict__ target, int V, int B, int seg,
                                                          int S, float invT, const int32_t* __restrict__ n_nodes,
                                                          float* __restrict__ tm, double* __restrict__ ts,
                                                          int* __restrict__ tf, uint32_t* __restrict__ counters) {
    const int s = blockIdx.x;
    const int row = blockIdx.y;
    const int r = row / (B + 1);
    const int node = row % (B + 1);
    const int tid = threadIdx.x;
    if (s == 0 && node == 0 && tid == 0) counters[r] = 0u;
    if (node >= n_nodes[r]) return;

    const size_t rowbase = (size_t)row * (size_t)V;
    const int lo = s * seg;
    const int hi = min(V, lo + seg);
    float m = -INFINITY;
    double sum = 0.0;
    int bad = 0;
    for (int i0 = lo + tid * 8; i0 < hi; i0 += kBlock * 8) {
        float x[8];
        if (VEC && i0 + 8 <= hi) {
            if (DT == TSB_BF16) {
                const uint4 raw = *(const uint4*)((const uint16_t*)target + rowbase + i0);
                const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    x[2 * j] = __uint_as_float(w[j] << 16);
                    x[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
                }
            } else {
                const float4 a = *(const float4*)((const float*)target + rowbase + i0);
                const float4 b = *(const float4*)((const float*)target + rowbase + i0 + 4);
                x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
                x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
            }
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) x[j] = (i0 + j < hi) ? load_logit<DT>(target, rowbase + i0 + j) : -INFINITY;
        }
        float a[8];
        float cm = -INFINITY;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            a[j] = x[j] * invT;
            if (isnan(a[j]) || a[j] == INFINITY) {
                bad = 1;
                a[j] = -INFINITY;
            }
            cm = fmaxf(cm, a[j]);
        }
        if (cm > m) {
            sum = (m == -INFINITY) ? 0.0 : sum * (double)__expf(m - cm);
            m = cm;
        }
        if (m > -INFINITY) {
            float cs = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) cs += __expf(a[j] - m);
            sum += (double)cs;
        }
    }
    __shared__ float s_m[kBlock / kWave];
    __shared__ double s_s[kBlock / kWave];
    __shared__ int s_bad[kBlock / kWave];
    const int wave = tid / kWave, lane = tid % kWave;
    const float wm = wave_max(m);
    const double contrib = (m == -INFINITY) ? 0.0 : sum * exp((double)m - (double)wm);
    const double wsum = wave_sum(contrib);
    const int wb = wave_or(bad);
    if (lane == 0) {
        s_m[wave] = wm;
        s_s[wave] = wsum;
        s_bad[wave] = wb;
    }
    __syncthreads();
    if (tid == 0) {
        float M = s_m[0];
        for (int w = 1; w < kBlock / kWave; ++w) M = fmaxf(M, s_m[w]);
        double tot = 0.0;
        int anybad = 0;
        for (int w = 0; w < kBlock / kWave; ++w) {
            if (s_m[w] != -INFINITY) tot += s_s[w] * exp((double)s_m[w] - (double)M);
            anybad |= s_bad[w];
        }
        const size_t o = (size_t)row * S + s;
        tm[o] = M;
        ts[o] = tot;
        tf[o] = anybad;
    }
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
    uint32_t* counters;
    double* zpart;
    float* bkey;
    int* bidx;
    int V, D, B, S4, r0;
    float invT;
    uint32_t k0, k1, step;
};

// binary64 log-sum-exp of target row (r, node) from its segment partials
__device__ double target_lse(const WalkArgs& A, int r, int node, int* bad) {
    const size_t o = ((size_t)r * (A.B + 1) + node) * A.S4;
    float M = -INFINITY;
    int b = 0;
    for (int s = 0; s < A.S4; ++s) {
        M = fmaxf(M, A.tm[o + s]);
        b |= A.tf[o + s];
    }
    double tot = 0.0;
    for (int s = 0; s < A.S4; ++s)
        if (A.tm[o + s] != -INFINITY) tot += A.ts[o + s] * exp((double)A.tm[o + s] - (double)M);
    *bad = b || M == -INFINITY;
    return (double)M + log(tot);
}

// Per-request barrier over the G workgroups of a request: monotone counter,
// bounded spin (a wait that exceeds the limit sets *timeout and proceeds).
__device__ void request_barrier(uint32_t* counter, uint32_t target, int* timeout) {
    __syncthreads();
    if (threadIdx.x == 0) {
        __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        uint32_t spins = 0;
        while (__hip_atomic_load(counter, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < target) {
            __builtin_amdgcn_s_sleep(2);
            if (++spins > (1u << 22)) {
                *timeout = 1;
                break;
            }
        }
    }
    __syncthreads();
}

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

// sum_v exp(a_v - L0) over this slice of target row `trow`, binary64 terms.
template <int DT>
__device__ double mass_slice(const WalkArgs& A, bool vec, size_t trow, double L0, int v0, int v1) {
    double acc = 0.0;
    for (int g = v0 / 4 + (int)threadIdx.x; g * 4 < v1; g += kBlock) {
        const int e0 = g * 4;
        const int valid = min(4, v1 - e0);
        float xt[4];
        load4<DT>(A.target, trow + e0, valid, vec, xt);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float a = xt[e] * A.invT;
            if (e < valid && a > -INFINITY) acc += exp((double)a - L0);
        }
    }
    return block_sum(acc);
}

// Residual mass sum_v max(p_v - C q_v, 0) over this slice, binary64 terms
// (the difference cancels when the target is close to the draft).
template <int DT>
__device__ double residual_slice(const WalkArgs& A, bool vec, size_t trow, size_t drow, double Lt, double Ld,
                                 double C, int v0, int v1) {
    double acc = 0.0;
    for (int g = v0 / 4 + (int)threadIdx.x; g * 4 < v1; g += kBlock) {
        const int e0 = g * 4;
        const int valid = min(4, v1 - e0);
        float xt[4], xd[4];
        load4<DT>(A.target, trow + e0, valid, vec, xt);
        load4<DT>(A.draft, drow + e0, valid, vec, xd);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (e >= valid) continue;
            const double p = exp((double)(xt[e] * A.invT) - Lt);
            const double q = exp((double)(xd[e] * A.invT) - Ld);
            const double rr = p - C * q;
            acc += rr > 0.0 ? rr : 0.0;
        }
    }
    return block_sum(acc);
}

// Bonus keys ln max(p_v - C q_v, 0) + G_v over this slice; returns the best
// (key, token) and the slice's residual mass.
template <int DT>
__device__ void bonus_slice(const WalkArgs& A, bool vec, const RngKey& key, uint32_t node, size_t trow, size_t drow,
                            bool use_q, double Lt, double Ld, double C, int v0, int v1, float* bk, int* bi,
                            double* mass) {
    float best = -INFINITY;
    int bidx = 0x7FFFFFFF;
    double acc = 0.0;
    const SplitF Ls = split(Lt);
    for (int g = v0 / 4 + (int)threadIdx.x; g * 4 < v1; g += kBlock) {
        const int e0 = g * 4;
        const int valid = min(4, v1 - e0);
        float xt[4], xd[4];
        load4<DT>(A.target, trow + e0, valid, vec, xt);
        if (use_q) load4<DT>(A.draft, drow + e0, valid, vec, xd);
        const uint4 w = rng_block(key, node, kStreamBonus, (uint32_t)g);
        const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (e >= valid) continue;
            float lr;
            if (use_q) {
                const double p = exp((double)(xt[e] * A.invT) - Lt);
                const double q = exp((double)(xd[e] * A.invT) - Ld);
                const double rr = p - C * q;
                acc += rr > 0.0 ? rr : 0.0;
                lr = rr > 0.0 ? (float)log(rr) : -INFINITY;
            } else {
                lr = (xt[e] * A.invT - Ls.hi) - Ls.lo;  // ln p_v up to a constant
                acc += 1.0;
            }
            if (lr > -INFINITY) {
                const float kv = lr + gumbel_f32(ws[e]);
                const int v = e0 + e;
                if (kv > best || (kv == best && v < bidx)) {
                    best = kv;
                    bidx = v;
                }
            }
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const float ok = __shfl_xor(best, off, kWave);
        const int oi = __shfl_xor(bidx, off, kWave);
        if (ok > best || (ok == best && oi < bidx)) {
            best = ok;
            bidx = oi;
        }
    }
    __shared__ float rk[kBlock / kWave];
    __shared__ int ri[kBlock / kWave];
    __shared__ double rm[kBlock / kWave];
    const double wm = wave_sum(acc);
    if ((threadIdx.x % kWave) == 0) {
        rk[threadIdx.x / kWave] = best;
        ri[threadIdx.x / kWave] = bidx;
        rm[threadIdx.x / kWave] = wm;
    }
    __syncthreads();
    float fb = rk[0];
    int fi = ri[0];
    double fm = 0.0;
    for (int i = 0; i < kBlock / kWave; ++i) {
        if (rk[i] > fb || (rk[i] == fb && ri[i] < fi)) {
            fb = rk[i];
            fi = ri[i];
        }
        fm += rm[i];
    }
    __syncthreads();
    *bk = fb;
    *bi = fi;
    *mass = fm;
}

template <int DT, bool VEC>
__global__ __launch_bounds__(kBlock) void verify_walk(WalkArgs A) {
    const int g = blockIdx.x;
    const int G = gridDim.x;
    const int r = A.r0 + blockIdx.y;
    const int tid = threadIdx.x;
    const int B1 = A.B + 1;
    const size_t tb = (size_t)r * B1;
    const bool vec = VEC;
    int* status_p = A.out.req_status + r;
    const int n = A.tree.n_nodes[r];

    const bool lead = (g == 0 && tid == 0);
    int n_acc_out = -1, bonus_out = -1, add_status = 0;

    // vocabulary slice of this workgroup (multiple of 4)
    // (an empty slice is [0, 0): its start must stay a multiple of 4)
    const int span = ((A.V + G - 1) / G + 3) & ~3;
    const bool has_slice = (long long)g * span < A.V;
    const int v0 = has_slice ? g * span : 0;
    const int v1 = has_slice ? min(A.V, v0 + span) : 0;

    // target rows of every tree node must be finite
    __shared__ int s_bad;
    if (tid == 0) s_bad = 0;
    __syncthreads();
    const bool draft_bad = (*status_p & TSB_REQ_NONFINITE) != 0;
    if (!draft_bad) {
        for (int i = tid; i < n; i += kBlock) {
            int b;
            const double l = target_lse(A, r, i, &b);
            if (b) atomicOr(&s_bad, 1);
            if (A.out.target_lse && (i % G) == g) A.out.target_lse[tb + i] = b ? (double)NAN : l;
        }
    }
    __syncthreads();
    if (A.out.target_lse && (draft_bad || s_bad))
        for (int i = tid; i < B1; i += kBlock)
            if ((i % G) == g) A.out.target_lse[tb + i] = (double)NAN;
    if (A.out.target_lse && !draft_bad && !s_bad)
        for (int i = n + tid; i < B1; i += kBlock)
            if ((i % G) == g) A.out.target_lse[tb + i] = (double)NAN;

    int tcount = 0;
    auto trace_put = [&](int child, double U, double ratio, double z) {
        if (lead && A.out.trace && tcount < TSB_TRACE_MAX) {
            double* t = A.out.trace + ((size_t)r * TSB_TRACE_MAX + tcount) * 4;
            t[0] = child;
            t[1] = U;
            t[2] = ratio;
            t[3] = z;
        }
        ++tcount;
    };
    auto trace_set_z = [&](double z) {
        if (lead && A.out.trace && tcount >= 1 && tcount <= TSB_TRACE_MAX)
            A.out.trace[((size_t)r * TSB_TRACE_MAX + tcount - 1) * 4 + 3] = z;
    };

    if (!draft_bad && !s_bad) {
        RngKey key;
        key.k0 = A.k0;
        key.k1 = A.k1;
        key.request = (uint32_t)r;
        key.step = A.step;
        uint32_t nb = 0;  // barriers passed
        int timeout = 0;
        int u = 0;
        int nacc = 0;
        while (true) {
            const int m = A.tree.n_children[tb + u];
            const int d = A.tree.depth[tb + u];
            int tbad;
            const double Lt0 = target_lse(A, r, u, &tbad);
            const size_t trow = ((size_t)r * B1 + u) * (size_t)A.V;
            const size_t drow = ((size_t)r * A.D + (d < A.D ? d : 0)) * (size_t)A.V;
            const double Ld = (m > 0) ? A.draft_lse[(size_t)r * A.D + d] : 0.0;
            double Lt = Lt0;
            if (m > 0) {
                // binary64 normaliser of p_u (the streamed estimate has binary32 terms)
                const double part = mass_slice<DT>(A, vec, trow, Lt0, v0, v1);
                const int slot = (r * 2 + (nb & 1)) * kWalkGroupsMax + g;
                if (tid == 0) A.zpart[slot] = part;
                ++nb;
                request_barrier(&A.counters[r], nb * (uint32_t)G, &timeout);
                double S0 = 0.0;
                for (int h = 0; h < G; ++h)
                    S0 += __hip_atomic_load(&A.zpart[(r * 2 + ((nb - 1) & 1)) * kWalkGroupsMax + h], __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
                Lt = Lt0 + log(S0);
            }
            double C = 0.0, S = 1.0, Z = 1.0;
            bool accepted = false, degenerate = false;
            for (int j = 0; j < m; ++j) {
                const int c = A.tree.first_child[tb + u] + j;
                const int y = A.node_tok[tb + c];
                const double qy = exp((double)(load_logit<DT>(A.draft, drow + y) * A.invT) - Ld);
                const double py = exp((double)(load_logit<DT>(A.target, trow + y) * A.invT) - Lt);
                const double W = Z / S;
                const double num = py - C * qy;
                const double ratio = (num > 0.0 ? num : 0.0) / (W * qy);
                const double U = u24d(rng_word(key, (uint32_t)c, kStreamAccept, 0u));
                trace_put(c, U, ratio, -1.0);
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
                S = S - qy;
                if (j + 1 == m) break;
                // residual mass at the new C, summed over the G slices
                const double part = residual_slice<DT>(A, vec, trow, drow, Lt, Ld, C, v0, v1);
                const int slot = (r * 2 + (nb & 1)) * kWalkGroupsMax + g;
                if (tid == 0) A.zpart[slot] = part;
                ++nb;
                request_barrier(&A.counters[r], nb * (uint32_t)G, &timeout);
                Z = 0.0;
                for (int h = 0; h < G; ++h)
                    Z += __hip_atomic_load(&A.zpart[(r * 2 + ((nb - 1) & 1)) * kWalkGroupsMax + h], __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
                trace_set_z(Z);
                if (Z <= 0.0 || S <= 0.0) {
                    degenerate = true;
                    break;
                }
            }
            if (accepted) continue;
            // bonus token at the terminal node u
            bool use_q = !degenerate && C > 0.0;
            for (int attempt = 0; attempt < 2; ++attempt) {
                float bk;
                int bi;
                double mass;
                bonus_slice<DT>(A, vec, key, (uint32_t)u, trow, drow, use_q, Lt, Ld, C, v0, v1, &bk, &bi, &mass);
                const int slot = (r * 2 + (nb & 1)) * kWalkGroupsMax + g;
                if (tid == 0) {
                    A.bkey[slot] = bk;
                    A.bidx[slot] = bi;
                    A.zpart[slot] = mass;
                }
                ++nb;
                request_barrier(&A.counters[r], nb * (uint32_t)G, &timeout);
                float fb = -INFINITY;
                int fi = 0x7FFFFFFF;
                double fm = 0.0;
                for (int h = 0; h < G; ++h) {
                    const int sl = (r * 2 + ((nb - 1) & 1)) * kWalkGroupsMax + h;
                    const float kb = __hip_atomic_load(&A.bkey[sl], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    const int ib = __hip_atomic_load(&A.bidx[sl], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    fm += __hip_atomic_load(&A.zpart[sl], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (kb > fb || (kb == fb && ib < fi)) {
                        fb = kb;
                        fi = ib;
                    }
                }
                if (use_q) trace_set_z(fm);
                if (use_q && (fm <= 0.0 || fb == -INFINITY)) {
                    degenerate = true;
                    use_q = false;
                    continue;
                }
                bonus_out = fi;
                break;
            }
            if (degenerate) add_status |= TSB_REQ_DEGENERATE_RESIDUAL;
            if (timeout) add_status |= TSB_REQ_WALK_TIMEOUT;
            n_acc_out = nacc;
            break;
        }
        if (lead)
            for (int i = nacc; i < A.D; ++i) {
                A.out.acc_node[(size_t)r * A.D + i] = -1;
                A.out.acc_tok[(size_t)r * A.D + i] = -1;
            }
    } else {
        add_status |= TSB_REQ_NONFINITE;
        if (lead)
            for (int i = 0; i < A.D; ++i) {
                A.out.acc_node[(size_t)r * A.D + i] = -1;
                A.out.acc_tok[(size_t)r * A.D + i] = -1;
            }
    }
    if (lead) {
        A.out.n_acc[r] = n_acc_out;
        A.out.bonus[r] = bonus_out;
        *status_p |= add_status;
        if (A.out.trace)
            for (int i = tcount; i < TSB_TRACE_MAX; ++i)
                for (int f = 0; f < 4; ++f) A.out.trace[((size_t)r * TSB_TRACE_MAX + i) * 4 + f] = -1.0;
    }
}

// ------------------------------------------------------------------ launch
hipError_t launch_verify(const tsb_config& c, float invT, const void* draft, const double* draft_lse,
                         const void* target, const tsb_tree& tree, const int32_t* node_tok, uint32_t step,
                         const tsb_verdict& out, char* ws, hipStream_t st) {
    const Geometry g = geometry(c);
    const VerifyWs w = verify_ws(c);
    float* tm = (float*)(ws + w.tm);
    double* ts = (double*)(ws + w.ts);
    int* tf = (int*)(ws + w.tf);
    uint32_t* counters = (uint32_t*)(ws + w.counter);
    const bool vec8 = (c.dtype == TSB_BF16) ? (c.V % 8 == 0 && ((uintptr_t)target & 15) == 0)
                                            : (c.V % 4 == 0 && ((uintptr_t)target & 15) == 0);
    const dim3 grid4(g.S4, c.R * (c.B + 1));
    hipError_t e = hook_before(TSB_KERNEL_TARGET_PARTIALS, st);
    if (e != hipSuccess) return e;
    if (c.dtype == TSB_BF16) {
        if (vec8)
            target_partials<TSB_BF16, true><<<grid4, kBlock, 0, st>>>(target, c.V, c.B, g.seg4, g.S4, invT,
                                                                      tree.n_nodes, tm, ts, tf, counters);
        else
            target_partials<TSB_BF16, false><<<grid4, kBlock, 0, st>>>(target, c.V, c.B, g.seg4, g.S4, invT,
                                                                       tree.n_nodes, tm, ts, tf, counters);
    } else {
        if (vec8)
            target_partials<TSB_F32, true><<<grid4, kBlock, 0, st>>>(target, c.V, c.B, g.seg4, g.S4, invT,
                                                                     tree.n_nodes, tm, ts, tf, counters);
        else
            target_partials<TSB_F32, false><<<grid4, kBlock, 0, st>>>(target, c.V, c.B, g.seg4, g.S4, invT,
                                                                      tree.n_nodes, tm, ts, tf, counters);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((e = hook_after(TSB_KERNEL_TARGET_PARTIALS, st)) != hipSuccess) return e;

    WalkArgs A;
    A.draft = draft;
    A.draft_lse = draft_lse;
    A.target = target;
    A.tree = tree;
    A.node_tok = node_tok;
    A.out = out;
    A.tm = tm;
    A.ts = ts;
    A.tf = tf;
    A.counters = counters;
    A.zpart = (double*)(ws + w.zpart);
    A.bkey = (float*)(ws + w.bkey);
    A.bidx = (int*)(ws + w.bidx);
    A.V = c.V;
    A.D = c.D;
    A.B = c.B;
    A.S4 = g.S4;
    A.invT = invT;
    A.k0 = (uint32_t)c.seed;
    A.k1 = (uint32_t)(c.seed >> 32);
    A.step = step;

    const bool vec4 = c.V % 4 == 0 && ((uintptr_t)target & 15) == 0 && ((uintptr_t)draft & 15) == 0;
    const void* fn = nullptr;
    if (c.dtype == TSB_BF16)
        fn = vec4 ? (const void*)verify_walk<TSB_BF16, true> : (const void*)verify_walk<TSB_BF16, false>;
    else
        fn = vec4 ? (const void*)verify_walk<TSB_F32, true> : (const void*)verify_walk<TSB_F32, false>;

    int dev = 0, cus = 0, per_cu = 0;
    e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock, 0);
    if (e != hipSuccess) return e;
    const int cap = per_cu * cus;
    if (cap < 1) return hipErrorCooperativeLaunchTooLarge;
    int G = g.G;
    if (G * c.R > cap) G = cap / c.R > 0 ? cap / c.R : 1;
    const int chunk = cap / G;
    if ((e = hook_before(TSB_KERNEL_VERIFY_WALK, st)) != hipSuccess) return e;
    for (int r0 = 0; r0 < c.R; r0 += chunk) {
        A.r0 = r0;
        const int rc = min(chunk, c.R - r0);
        void* args[] = {&A};
        e = hipLaunchCooperativeKernel(fn, dim3(G, rc), dim3(kBlock), args, 0, st);
        if (e != hipSuccess) return e;
    }
    return hook_after(TSB_KERNEL_VERIFY_WALK, st);
}

}  // namespace tsb
