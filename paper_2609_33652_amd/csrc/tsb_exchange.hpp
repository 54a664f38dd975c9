// Exchange among the G workgroups that share one request in verification,
// through tagged slots that the workgroups poll (no counter barrier).
//
// Layout (the workspace's persistent region): seqs [R] and slots
// [R][2][kWalkGroupsMax][kSlotWords] 64-bit words; round e of request r uses
// the slot pair of parity e & 1. A publisher (thread 0 of a workgroup)
// writes each word with one relaxed agent-scope store; every word carries
// the round's 8-bit tag in its low bits, so a reader knows it holds all
// words of the current round without any ordering between the stores:
//   tag(seq, e) = (seq & 1) << 7 | (e & 1) << 6 | ((e >> 1) % 63 + 1)
// never 0, different for rounds e and e - 2 of one slot, and different for
// the previous call of the request (seq - 1).
//
// Invariant between calls: every word of every slot of a request is zero
// or belongs to the previous call's last round (a publish writes all words
// of its slot). A call that ran rounds keeps it with xfinish(): each
// workgroup zeroes its slot of the round before the last (all workgroups
// have read it), the request's first workgroup zeroes the slots of
// workgroups g >= G, and the sequence number advances. A wait that was
// abandoned (TSB_REQ_WALK_TIMEOUT) voids the invariant for that request until
// the caller zero-fills the workspace again.
#pragma once

#include "tsb_device.hpp"

namespace tsb {

constexpr int kSlotWords = 8;  // one 64-byte slot per (request, parity, workgroup)
constexpr uint64_t kTagMask = 0xFFull;
constexpr uint32_t kPollLimit = 1u << 20;  // ~1 s of polling before a wait is abandoned

struct XRegion {
    uint32_t* seqs;
    uint64_t* slots;
};

__device__ __forceinline__ uint64_t xtag(uint32_t seq, uint32_t e) {
    return ((uint64_t)(seq & 1u) << 7) | ((uint64_t)(e & 1u) << 6) | (uint64_t)((e >> 1) % 63u + 1u);
}

__device__ __forceinline__ uint64_t* xslot(const XRegion& X, int r, uint32_t e, int g) {
    return X.slots + (((size_t)r * 2 + (e & 1u)) * kWalkGroupsMax + g) * kSlotWords;
}

// Payload packing: a binary64 value keeps all but its 8 lowest mantissa bits
// (relative resolution 2^-44); 32-bit payloads sit in the high half.
__device__ __forceinline__ uint64_t xpack_f64(double x) { return (uint64_t)__double_as_longlong(x) & ~kTagMask; }
__device__ __forceinline__ double xunpack_f64(uint64_t w) { return __longlong_as_double((long long)(w & ~kTagMask)); }
__device__ __forceinline__ uint64_t xpack_u32(uint32_t x) { return (uint64_t)x << 32; }
__device__ __forceinline__ uint32_t xunpack_u32(uint64_t w) { return (uint32_t)(w >> 32); }

// Thread 0 publishes NW payload words of round e. The slot's other words get
// the bare tag: every word of a slot then belongs to the round last written,
// whatever the width of the exchanges before it (a word left from an older
// round could otherwise carry a tag that matches again two calls later).
template <int NW>
__device__ __forceinline__ void xpublish(const XRegion& X, int r, int g, uint32_t seq, uint32_t e,
                                         const uint64_t (&w)[NW]) {
    static_assert(NW <= kSlotWords, "slot width");
    if (threadIdx.x != 0) return;
    const uint64_t t = xtag(seq, e);
    uint64_t* s = xslot(X, r, e, g);
#pragma unroll
    for (int i = 0; i < kSlotWords; ++i)
        __hip_atomic_store(&s[i], i < NW ? ((w[i] & ~kTagMask) | t) : t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Polls the NW words of workgroup h's slot of round e until all carry the
// round's tag (lanes of wave 0 call this for their own slots). Returns false
// if the wait was abandoned.
template <int NW>
__device__ __forceinline__ bool xpoll(const XRegion& X, int r, int h, uint32_t seq, uint32_t e, uint64_t (&w)[NW]) {
    const uint64_t t = xtag(seq, e);
    const uint64_t* s = xslot(X, r, e, h);
    for (uint32_t spins = 0;; ++spins) {
        bool ok = true;
#pragma unroll
        for (int i = 0; i < NW; ++i) {
            w[i] = __hip_atomic_load(&s[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            ok = ok && (w[i] & kTagMask) == t;
        }
        if (ok) return true;
        if (spins >= kPollLimit) return false;
        __builtin_amdgcn_s_sleep(1);
    }
}

// End of a call that ran `rounds` rounds (> 0) for request r: see the
// invariant above. All threads of every workgroup of the request call it.
__device__ __forceinline__ void xfinish(const XRegion& X, int r, int g, int G, uint32_t seq, uint32_t rounds) {
    if (threadIdx.x < kSlotWords) {
        uint64_t* s = xslot(X, r, rounds, g);  // parity of round rounds - 2, i.e. the one before the last
        __hip_atomic_store(&s[threadIdx.x], 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (g == 0) {
        for (int i = threadIdx.x; i < 2 * (kWalkGroupsMax - G) * kSlotWords; i += blockDim.x) {
            const int q = i / kSlotWords;
            const int gg = G + q / 2;
            uint64_t* s = xslot(X, r, (uint32_t)(q & 1), gg);
            __hip_atomic_store(&s[i % kSlotWords], 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (threadIdx.x == 0) X.seqs[r] = seq + 1u;
    }
}

}  // namespace tsb
