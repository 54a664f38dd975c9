// Internal definitions shared by the host layer and the kernels of the
// tree-replay library: launch geometry and workspace layout.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/tsubame.h"

namespace tsb {

// RNG stream tags (word 1 of the Philox counter, above the node index).
enum : uint32_t { kStreamReplay = 0, kStreamAccept = 1, kStreamBonus = 2 };

constexpr int kBlock = 256;          // threads per workgroup of the streaming kernels
constexpr int kReplayTile = 4096;    // vocabulary tile of the replay scan
constexpr int kWalkGroupsMax = 128;  // workgroups per request in verification
constexpr int kWalkTokensPerGroup = 9728;  // tokens whose binary64 (p, q) one walk workgroup holds in LDS
constexpr int kTargetWorkgroups = 2048;  // target stream: 8 resident workgroups on each of 256 CUs
constexpr int kClearWorkgroups = 64;      // a target job without rows: workgroups that clear the exchange slots
// A walk that reads the target rows it enters takes the rows of nodes 0 and
// 1 of every request (the root and, in BFS order, its first child: rows that
// do not depend on the topology) from a stream beside the planner, in
// kChainPieces equal pieces per row.
constexpr int kChainRows = 2;
constexpr int kChainPieces = 8;
// Targets of up to this many bytes are streamed whole before the walk (one
// pass beside the replay scan costs less than a row read and an exchange at
// every node the walk enters); larger ones are read row by row as the walk
// enters nodes.
constexpr long long kStreamRowsBytes = 128ll << 20;
constexpr int kTargetMinChunk = 32768;   // shortest target chunk (logits), unless the whole target is shorter
constexpr int kDraftWorkgroups = 512;    // row statistics: two 512-thread workgroups on each of 256 CUs
constexpr int kDraftMinSeg = 16384;      // shortest draft segment (elements), unless the row is shorter

struct Geometry {
    int S1;          // workgroups per draft row (row statistics)
    int seg1;        // elements per draft segment (multiple of 8)
    int S4;          // partial slots per target row
    int G4;          // chunks of the target stream (one per workgroup of its own grid)
    long long chunk4;  // logits per chunk (multiple of 8)
    int T;           // replay tiles per row
    int G;           // workgroups per request in verification (upper bound)
};

inline int ceil_div(long long a, long long b) { return (int)((a + b - 1) / b); }

// Whether the RRS walk reads each target row when it enters the node (true)
// or takes the row normalisers from a stream of every row before it.
inline bool walk_reads_rows(const tsb_config& c) {
    if (c.flags & TSB_FLAG_READ_ROWS) return true;
    if (c.flags & TSB_FLAG_STREAM_ROWS) return false;
    const long long b = c.dtype == TSB_BF16 ? 2 : 4;
    return (long long)c.R * (c.B + 1) * c.V * b > kStreamRowsBytes;
}

inline Geometry geometry(const tsb_config& c) {
    Geometry g;
    const long long drows = (long long)c.R * c.D;
    int s1 = ceil_div(kDraftWorkgroups, drows);
    int s1max = ceil_div(c.V, kDraftMinSeg);
    g.S1 = s1 < 1 ? 1 : (s1 > s1max ? s1max : s1);
    g.seg1 = ceil_div(ceil_div(c.V, g.S1), 8) * 8;
    g.S1 = ceil_div(c.V, g.seg1);
    // target stream: equal chunks of the flat [R (B+1) V] array, one per
    // resident workgroup; a row meets at most (V - 1) / chunk + 2 chunks
    const long long n4 = (long long)c.R * (c.B + 1) * c.V;
    long long g4 = (n4 + kTargetMinChunk - 1) / kTargetMinChunk;
    if (g4 > kTargetWorkgroups) g4 = kTargetWorkgroups;
    if (g4 < 1) g4 = 1;
    g.chunk4 = ((n4 + g4 - 1) / g4 + 7) / 8 * 8;
    g.G4 = (int)((n4 + g.chunk4 - 1) / g.chunk4);
    g.S4 = (int)((c.V - 1) / g.chunk4) + 2;
    g.T = ceil_div(c.V, kReplayTile);
    // walk: about one workgroup per compute unit over the batch, and enough
    // per request that a slice fits the LDS cache
    int gw = 256 / (c.R > 0 ? c.R : 1);
    const int gmin = ceil_div(c.V, kWalkTokensPerGroup);
    if (gw < gmin) gw = gmin;
    g.G = gw < 1 ? 1 : (gw > kWalkGroupsMax ? kWalkGroupsMax : gw);
    return g;
}

// Workspace carving: every region starts on a 256-byte boundary.
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct PlanWs {  // row statistics partials
    size_t pm, ps, pk, pf, total;
};
struct ReplayWs {  // per (parent, tile) best keys, flat parent list, per-parent records
    size_t cand, cnt, plist, ptotal, thr, total;
};
// 32-bit words of the walk's node record: eight of header, four per child.
constexpr int kRecWords = 8 + 4 * TSB_MAX_K;

struct VerifyWs {  // target partials, node records of the walk
    size_t tm, ts, tf, nrec, total;
};

// The exchange slots of the walks come first: [R][2][kWalkGroupsMax][8]
// 64-bit words that the workgroups of a request poll (cleared by a kernel
// enqueued before each walk in the same call; nothing is kept between
// calls), then the partials of every request's rows 0 and 1 for a walk that
// reads the other rows itself. Every stage's scratch starts after them.
struct XchgWs {
    size_t slots, cm, cs, cf, total;
};

inline XchgWs xchg_ws(const tsb_config& c) {
    XchgWs w;
    size_t o = 0;
    // slots [R][2][kWalkGroupsMax][8] words, then one line for the ticket counter
    w.slots = o; o = align256(o + ((size_t)c.R * 2 * kWalkGroupsMax * 8 + 8) * sizeof(uint64_t));
    // partials of rows 0 and 1 of every request ([R][2][kChainPieces]), written
    // beside the planner and read by the walk (no stage's scratch overlaps them)
    const size_t nc = (size_t)c.R * kChainRows * kChainPieces;
    w.cm = o; o = align256(o + nc * sizeof(float));
    w.cs = o; o = align256(o + nc * sizeof(double));
    w.cf = o; o = align256(o + nc * sizeof(int32_t));
    w.total = o;
    return w;
}

inline PlanWs plan_ws(const tsb_config& c) {
    const Geometry g = geometry(c);
    const size_t n = (size_t)c.R * c.D * g.S1;
    PlanWs w;
    size_t o = xchg_ws(c).total;
    w.pm = o; o = align256(o + n * sizeof(float));
    w.ps = o; o = align256(o + n * sizeof(double));
    w.pk = o; o = align256(o + n * (size_t)c.K * sizeof(uint64_t));
    w.pf = o; o = align256(o + n * sizeof(int32_t));
    w.total = o;
    return w;
}

inline ReplayWs replay_ws(const tsb_config& c) {
    const Geometry g = geometry(c);
    const size_t slots = (size_t)c.R * (c.B + 1) * g.T;
    ReplayWs w;
    size_t o = xchg_ws(c).total;
    w.cand = o; o = align256(o + slots * TSB_MAX_K * sizeof(uint64_t));
    w.cnt = o; o = align256(o + slots * sizeof(int32_t));
    w.plist = o; o = align256(o + (size_t)c.R * (c.B + 1) * sizeof(int32_t));
    w.ptotal = o; o = align256(o + sizeof(int32_t));
    w.thr = o; o = align256(o + (size_t)c.R * (c.B + 1) * 4 * sizeof(float));  // per node (c_d, thr, d, m)
    w.total = o;
    return w;
}

inline VerifyWs verify_ws_at(const tsb_config& c, size_t base) {
    const Geometry g = geometry(c);
    const size_t n = (size_t)c.R * (c.B + 1) * g.S4;
    VerifyWs w;
    size_t o = base;
    w.tm = o; o = align256(o + n * sizeof(float));
    w.ts = o; o = align256(o + n * sizeof(double));
    w.tf = o; o = align256(o + n * sizeof(int32_t));
    w.nrec = o; o = align256(o + (size_t)c.R * (c.B + 1) * kRecWords * sizeof(uint32_t));
    w.total = o;
    return w;
}

// The target partials sit after the replay's region: a round streams the
// target in the replay scan's grid (after the planner, whose region they may
// reuse).
inline VerifyWs verify_ws(const tsb_config& c) { return verify_ws_at(c, replay_ws(c).total); }

// Whole workspace of the vocabulary-wide entry points.
inline size_t ws_bytes(const tsb_config& c) {
    const size_t a = plan_ws(c).total, v = verify_ws(c).total;
    return a > v ? a : v;
}

// Pools of P tokens per draft position: segment candidate lists of the pool
// selection, then the candidate lists of every (position, parent slot):
// list 0 is the root's, list 1 + (d - 1) P + i that of a node at depth d >= 1
// whose token holds slot i of pool d - 1; entries pack (lp bits << 32 | slot).
constexpr int kPoolMax = 64;
// LDS bitmap of the pool tokens in a walk workgroup's vocabulary slice
// (slices up to 262144 tokens).
constexpr size_t kPoolBitmapBytes = 32768;

inline int pool_lists_per_request(const tsb_config& c, int P) { return 1 + (c.D - 1) * P; }

struct PoolWs {
    size_t pk, pf, lists, nfin, total;
};

inline PoolWs pool_ws(const tsb_config& c, int P) {
    const Geometry g = geometry(c);
    const size_t n = (size_t)c.R * c.D * g.S1;
    const size_t nl = (size_t)c.R * pool_lists_per_request(c, P);
    PoolWs w;
    size_t o = xchg_ws(c).total;
    w.pk = o; o = align256(o + n * (size_t)P * sizeof(uint64_t));
    w.pf = o; o = align256(o + n * sizeof(int32_t));
    w.lists = o; o = align256(o + nl * (size_t)c.K * sizeof(uint64_t));
    w.nfin = o; o = align256(o + nl * sizeof(int32_t));
    w.total = o;
    return w;
}

// The target partials of a pool round follow the pool replay (which keeps
// nothing in the workspace) and may reuse the pool selection's region.
inline VerifyWs pool_verify_ws(const tsb_config& c) { return verify_ws_at(c, xchg_ws(c).total); }

inline size_t pool_ws_bytes(const tsb_config& c, int P) {
    const size_t a = pool_ws(c, P).total, v = pool_verify_ws(c).total;
    return a > v ? a : v;
}

}  // namespace tsb
