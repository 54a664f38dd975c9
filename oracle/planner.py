"""First pass: plan and freeze the tree topology (oracle side).

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

Section 3.1 and Appendix B.3: the first pass allocates the node budget by
cumulative draft path probability; node-wise max-heap expansion over the
parallel per-position distributions maximises the summed draft path
probability under the budget. Only the topology (parent-child relations and
child order) is kept (Section 3.1, Figure 1).

A node is a rank path rho = (j_1, ..., j_k), k <= D, j_i < K: the child of
rank j_i at depth i is the j_i-th planning candidate of draft position i-1.
Its score is sum_i lp[i-1, j_i], accumulated in binary64 from the root.

Lazy best-first (max-heap) expansion: the frontier starts with the root's
rank-0 child; each pop commits the best frontier node and pushes its rank-0
child (if depth < D) and its next younger sibling (if rank + 1 < K). A
candidate with lp = -inf is never pushed. B pops (or an empty frontier) end
the pass.

Order of the frontier (the paper gives no tie rule; this is the reading both
sides implement): higher score first, then smaller depth, then the
lexicographically smaller rank path. It is a static total order on rank
paths in which a parent and an older sibling always precede a node (lp <= 0
and lp is non-increasing in rank), so B pops commit exactly the first B rank
paths of that order. The root is committed first (pop index 0).

Output is in BFS order (depth, then parent's BFS index, then rank), node 0 =
root, so parent[i] < i and children are contiguous in rank order.
plan_margin = score(last committed) - score(best uncommitted) (inf if the
frontier is empty).
"""
import heapq

import numpy as np


def plan(lp, B):
    """lp: float32 array [D, K] of planning log-probabilities (sorted desc per row).

    Returns a dict with BFS-ordered arrays (length n_nodes <= B + 1): parent,
    depth, rank, n_children, first_child, score (float64), plus n_nodes,
    plan_margin and bfs_of_pop (BFS index of the i-th committed node).
    """
    lp = np.asarray(lp, dtype=np.float32)
    D, K = lp.shape
    lp64 = lp.astype(np.float64)

    # committed nodes in pop order: (parent_pop, rank, depth, score)
    c_parent = [-1]
    c_rank = [-1]
    c_depth = [0]
    c_score = [0.0]
    pop_of_path = {(): 0}

    # heap entries: (-score, depth, rank path); tuples compare lexicographically
    heap = []
    if D > 0 and K > 0 and np.isfinite(lp64[0, 0]):
        heapq.heappush(heap, (-(0.0 + lp64[0, 0]), 1, (0,)))
    while len(c_parent) - 1 < B and heap:
        neg_s, dep, path = heapq.heappop(heap)
        s = -neg_s
        rk = path[-1]
        ppop = pop_of_path[path[:-1]]
        pop_idx = len(c_parent)
        pop_of_path[path] = pop_idx
        c_parent.append(ppop)
        c_rank.append(rk)
        c_depth.append(dep)
        c_score.append(s)
        if dep < D and np.isfinite(lp64[dep, 0]):
            heapq.heappush(heap, (-(s + lp64[dep, 0]), dep + 1, path + (0,)))
        if rk + 1 < K and np.isfinite(lp64[dep - 1, rk + 1]):
            heapq.heappush(heap, (-(c_score[ppop] + lp64[dep - 1, rk + 1]), dep, path[:-1] + (rk + 1,)))

    n = len(c_parent)
    if heap:
        margin = c_score[-1] - (-heap[0][0]) if n > 1 else np.inf
    else:
        margin = np.inf

    # BFS canonical order: children of each committed node sorted by rank.
    kids = [[] for _ in range(n)]
    for p in range(1, n):
        kids[c_parent[p]].append(p)
    for k in kids:
        k.sort(key=lambda p: c_rank[p])
    bfs_of_pop = np.full(n, -1, dtype=np.int64)
    order = [0]
    bfs_of_pop[0] = 0
    head = 0
    while head < len(order):
        p = order[head]
        head += 1
        for ch in kids[p]:
            bfs_of_pop[ch] = len(order)
            order.append(ch)

    parent = np.full(n, -1, dtype=np.int64)
    depth = np.zeros(n, dtype=np.int64)
    rank = np.full(n, -1, dtype=np.int64)
    n_children = np.zeros(n, dtype=np.int64)
    first_child = np.full(n, -1, dtype=np.int64)
    score = np.zeros(n, dtype=np.float64)
    for i, p in enumerate(order):
        parent[i] = bfs_of_pop[c_parent[p]] if c_parent[p] >= 0 else -1
        depth[i] = c_depth[p]
        rank[i] = c_rank[p]
        score[i] = c_score[p]
        n_children[i] = len(kids[p])
        first_child[i] = bfs_of_pop[kids[p][0]] if kids[p] else -1
    return dict(parent=parent, depth=depth, rank=rank, n_children=n_children,
                first_child=first_child, score=score, n_nodes=n,
                plan_margin=float(margin), bfs_of_pop=bfs_of_pop.copy())


def max_nodes(D, K):
    """Number of rank paths of depth 1..D (the budget can never exceed it)."""
    return sum(K ** d for d in range(1, D + 1))
