// Exchange among the G workgroups that share one request in verification,
// through tagged slots that the workgroups poll (no counter barrier).
//
// Layout (a workspace region): slots [R][2][kWalkGroupsMax][kSlotWords]
// 64-bit words; round e of request r uses the slot pair of parity e & 1. A
// publisher (thread 0 of a workgroup) writes each word with one relaxed
// agent-scope store; every word carries the round's 8-bit tag in its low
// bits, so a reader knows it holds all words of the current round without
// any ordering between the stores:
//   tag(e) = (e & 1) << 7 | ((e >> 1) % 127 + 1)
// never 0, and different for rounds e and e - 2, the only earlier round a
// slot can still hold (a workgroup publishes round e only after reading
// round e - 1 from every workgroup, each of which had read round e - 2).
//
// Nothing persists between calls: a kernel enqueued before each walk in the
// same call (the target stream, or the naive walk's clearing kernel) clears
// the slots of every request of the call and the ticket counter (xclear),
// and stream order makes the zeros visible before the walk starts. Whatever the workspace
// held before the call (another entry point's scratch, an abandoned wait of
// an earlier call, uninitialised memory) can therefore never be taken for a
// current word.
#pragma once

#include "tsb_device.hpp"

namespace tsb {

constexpr int kSlotWords = 8;  // one 64-byte slot per (request, parity, workgroup)
constexpr uint64_t kTagMask = 0xFFull;
constexpr uint32_t kPollLimit = 1u << 20;  // ~1 s of polling before a wait is abandoned

struct XRegion {
    uint64_t* slots;
};

__device__ __forceinline__ uint64_t xtag(uint32_t e) {
    return ((uint64_t)(e & 1u) << 7) | (uint64_t)((e >> 1) % 127u + 1u);
}

__device__ __forceinline__ uint64_t* xslot(const XRegion& X, int r, uint32_t e, int g) {
    return X.slots + (((size_t)r * 2 + (e & 1u)) * kWalkGroupsMax + g) * kSlotWords;
}

// Words of the slots of R requests; one more 64-byte line after them holds
// the walk's ticket counter.
constexpr int kTicketWords = 8;
__host__ __device__ inline size_t xslot_words(int R) { return (size_t)R * 2 * kWalkGroupsMax * kSlotWords; }
// Words of the exchange region of R requests (slots and ticket counter).
__host__ __device__ inline size_t xwords(int R) { return xslot_words(R) + kTicketWords; }

// Tickets. A walk is one launch of R * G workgroups; each workgroup, once it
// runs, takes the next ticket t from a counter cleared before the launch and
// serves request t / G, slice t % G. Tickets go only to running workgroups,
// in order, so every request below the highest ticket taken has all its
// workgroups running or done, and its exchanges complete; as they finish,
// waiting workgroups start and take the next tickets. The launch therefore
// needs only G workgroups to fit on the device at once, whatever else runs
// there and however the hardware orders the dispatch of the grid.
__device__ __forceinline__ int xticket(const XRegion& X, int R) {
    __shared__ int s_ticket;
    if (threadIdx.x == 0)
        s_ticket = (int)__hip_atomic_fetch_add((uint32_t*)(X.slots + xslot_words(R)), 1u, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    return s_ticket;
}

// Zeroes the exchange slots of R requests and the ticket counter; thread `i`
// of `n` threads
// (grid-stride) takes every n-th word.
__device__ __forceinline__ void xclear(const XRegion& X, int R, size_t i, size_t n) {
    const size_t nw = xwords(R);
    for (; i < nw; i += n) __hip_atomic_store(&X.slots[i], 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Payload packing: a binary64 value keeps all but its 8 lowest mantissa bits
// (relative resolution 2^-44); 32-bit payloads sit in the high half.
__device__ __forceinline__ uint64_t xpack_f64(double x) { return (uint64_t)__double_as_longlong(x) & ~kTagMask; }
__device__ __forceinline__ double xunpack_f64(uint64_t w) { return __longlong_as_double((long long)(w & ~kTagMask)); }
__device__ __forceinline__ uint64_t xpack_u32(uint32_t x) { return (uint64_t)x << 32; }
__device__ __forceinline__ uint32_t xunpack_u32(uint64_t w) { return (uint32_t)(w >> 32); }

// Thread 0 publishes NW payload words of round e. The slot's other words get
// the bare tag: every word of a slot then belongs to the round last written,
// whatever the width of the exchanges before it.
template <int NW>
__device__ __forceinline__ void xpublish(const XRegion& X, int r, int g, uint32_t e, const uint64_t (&w)[NW]) {
    static_assert(NW <= kSlotWords, "slot width");
    if (threadIdx.x != 0) return;
    const uint64_t t = xtag(e);
    uint64_t* s = xslot(X, r, e, g);
#pragma unroll
    for (int i = 0; i < kSlotWords; ++i)
        __hip_atomic_store(&s[i], i < NW ? ((w[i] & ~kTagMask) | t) : t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Polls the NW words of workgroup h's slot of round e until all carry the
// round's tag (lanes of wave 0 call this for their own slots). Returns false
// if the wait was abandoned.
template <int NW>
__device__ __forceinline__ bool xpoll(const XRegion& X, int r, int h, uint32_t e, uint64_t (&w)[NW]) {
    const uint64_t t = xtag(e);
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

}  // namespace tsb
