"""First pass by expand-then-prune (oracle side).

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

Section 3.1 and Appendix B.3: for drafters that need a correction step per
new prefix, the first pass uses EAGLE-2-style expand-then-prune, which
batches the corrections of a whole frontier per depth; the paper keeps
EAGLE-2's frontier width of 10. Like max-heap expansion it allocates nodes by
cumulative draft path probability, and with a wide enough frontier it
recovers the max-heap topology.

Reading of the procedure (the paper names it, EAGLE-2 defines it):
  * layer 1 is the root's children: the K planning candidates of position 0;
  * the frontier of layer d is its w best nodes; layer d + 1 holds every
    child of every frontier node (the K candidates of position d);
  * the tree is the first B of all generated nodes.
"Best" is the static order of the max-heap planner: score desc, then depth
asc, then rank path lexicographically asc (within a layer the depth is
equal). Scores are binary64 sums of lp from the root; candidates with
lp = -inf are never generated. Because lp <= 0 and is non-increasing in
rank, the first B generated nodes are closed under parents and older
siblings, so they form a tree whose chosen children are a rank prefix.

Output: the same BFS-ordered dict as planner.plan (parent, depth, rank,
n_children, first_child, score, n_nodes, plan_margin); plan_margin is the
score of the last chosen node minus that of the first generated node left
out (inf if none is left out).
"""
import numpy as np


def plan_expand_prune(lp, B, w):
    """lp: float32 [D, K] planning log-probabilities (sorted desc per row); w >= 1 frontier width."""
    lp = np.asarray(lp, dtype=np.float32)
    D, K = lp.shape
    lp64 = lp.astype(np.float64)
    if w < 1:
        raise ValueError("frontier width must be >= 1")

    def children(path, score, d):
        return [(path + (j,), score + lp64[d, j]) for j in range(K) if np.isfinite(lp64[d, j])]

    generated = []
    layer = children((), 0.0, 0) if D > 0 else []
    generated += layer
    for d in range(1, D):
        frontier = sorted(layer, key=lambda t: (-t[1], t[0]))[:w]
        layer = [c for (p, s) in frontier for c in children(p, s, d)]
        generated += layer

    order = sorted(generated, key=lambda t: (-t[1], len(t[0]), t[0]))
    chosen = order[:B]
    margin = (chosen[-1][1] - order[B][1]) if (B < len(order) and chosen) else np.inf
    return _bfs_tree(chosen, margin)


def _bfs_tree(chosen, margin):
    """BFS-ordered arrays of a prefix-closed set of (rank path, score)."""
    score_of = {(): 0.0}
    for p, s in chosen:
        score_of[p] = s
    kids = {p: [] for p in score_of}
    for p in score_of:
        if p:
            if p[:-1] not in kids:
                raise AssertionError("chosen set is not closed under parents")
            kids[p[:-1]].append(p)
    for k in kids.values():
        k.sort()
    order = [()]
    head = 0
    while head < len(order):
        order += kids[order[head]]
        head += 1
    index = {p: i for i, p in enumerate(order)}
    n = len(order)
    parent = np.full(n, -1, dtype=np.int64)
    depth = np.zeros(n, dtype=np.int64)
    rank = np.full(n, -1, dtype=np.int64)
    n_children = np.zeros(n, dtype=np.int64)
    first_child = np.full(n, -1, dtype=np.int64)
    score = np.zeros(n, dtype=np.float64)
    for i, p in enumerate(order):
        if p:
            parent[i] = index[p[:-1]]
            rank[i] = p[-1]
        depth[i] = len(p)
        score[i] = score_of[p]
        n_children[i] = len(kids[p])
        first_child[i] = index[kids[p][0]] if kids[p] else -1
    return dict(parent=parent, depth=depth, rank=rank, n_children=n_children,
                first_child=first_child, score=score, n_nodes=n, plan_margin=float(margin))
