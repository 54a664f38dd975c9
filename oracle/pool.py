"""Sparse candidate pools with context-dependent draft distributions (oracle
side): first pass, replay and verification of one round.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

Section 3.1: because branching multiplies the prefixes that need a
conditional draft distribution, the drafter's vocabulary is restricted at
every position to a pool of the backbone's top-scoring tokens; the
drafter's corrections are computed only inside the pool and the corrected
logits are normalised over the pool. DFlash2 obtains its conditional
distributions by looking up precomputed transition scores between
candidates and is planned by node-wise max-heap expansion. Section 3.2,
eq. (2): replay recomputes q_u = q(. | x, y_path(u)) under the replayed
prefix, with the same pools. Section 3.3: verification uses the
probabilities of the replayed candidates, normalised within the pool (zero
outside it). Appendix B.1 (draft candidate pools): the pools restrict only
the draft proposals, not the target distribution, which stays
vocabulary-wide. Pool sizes in the paper: 16 (DFlash2), 64 (Domino).

This project's drafter correction is such a transition-score lookup: a table
c[d-1] of shape [P, P] per draft position d >= 1 scores pool slot j of
position d given that the parent's token holds pool slot i of position d-1.
Readings (the paper fixes no formula for the correction):
  pool_d       the first P tokens of draft row d by (logit desc, id asc)
  a_{d,j}      fl32(x_{d, pool_d[j]} * invT)
  z_u(j)       fl32(a_{d,j} + fl32(c[d-1][s_u, j] * invT)), a binary32 sum,
               for a node u at depth d >= 1 whose token holds slot s_u of
               pool_{d-1}; z_root(j) = a_{0,j}. Being binary32 like the
               logits, fl32(L_u) >= max z_u, so lp_u <= 0 and path scores never
               grow along a path.
  q_u(j)       exp(z_u(j) - L_u), L_u = binary64 log-sum-exp of z_u over the pool
  lp_u(j)      fl32(z_u(j) - fl32(L_u)), the planning log-probabilities
  candidates   the pool slots of u by (lp_u desc, slot asc), the first K with
               lp_u > -inf; the child of rank k of u is the k-th candidate
First pass: max-heap expansion (as planner.plan) in which every node has its
own candidate list: the tree is the first B rank paths under the static order
(score desc, depth asc, rank path lexicographic asc), score = binary64 sum of
lp along the path. Replay: the m children of u receive, in rank order, the
pool tokens with the m largest keys z_u(j) + G(seed, step, request, u, v),
v = pool_d[j] (binary64; equal keys to the smaller token id), G from the
REPLAY stream with the token id as draw index, as in the vocabulary-wide
replay. Verification: WoR-RRS of verify.verify with q_u over the vocabulary
(zero outside the pool).
"""
import heapq

import numpy as np

from . import philox, verify as verify_mod
from .planner_ep import _bfs_tree
from .rowstats import (STATUS_BUDGET_SHORT, STATUS_NONFINITE, inv_temperature, lse64, probs, row_ok,
                       scaled, topk)


def pools(draft, P):
    """pool_d for every draft row: int64 [D, P] (logit desc, id asc)."""
    draft = np.asarray(draft)
    return np.stack([topk(draft[d], P) for d in range(draft.shape[0])]) if draft.shape[0] else \
        np.zeros((0, P), np.int64)


def pool_logits(draft, invT, pool):
    """a_{d,j} = fl32(x_{d, pool_d[j]} * invT) as float64, [D, P]."""
    out = np.zeros(pool.shape, np.float64)
    for d in range(pool.shape[0]):
        out[d] = scaled(np.asarray(draft[d], np.float32)[pool[d]], invT)
    return out


def scaled_corrections(trans, invT):
    """fl32(c * invT) as float64, same shape as trans ([D-1, P, P])."""
    return scaled(np.asarray(trans, np.float32), invT)


def corrected(a_pool, cs, d, s):
    """z_u over the pool of position d for a node at depth d whose token holds slot s (ignored at d = 0)."""
    z = a_pool[d].copy()
    if d > 0:
        z = (z.astype(np.float32) + cs[d - 1][s].astype(np.float32)).astype(np.float64)
    return z


def pool_q(z):
    """(q, L, lp32): pool-normalised probabilities, their binary64 normaliser, planning lp."""
    L = lse64(z)
    q = np.exp(z - L)
    lp = (z.astype(np.float64) - np.float64(np.float32(L))).astype(np.float32)
    return q, L, lp


def candidates(z, K):
    """(slots, lp) of the first K candidates by (lp desc, slot asc), lp > -inf only."""
    _, _, lp = pool_q(z)
    lp64 = lp.astype(np.float64)
    order = np.lexsort((np.arange(lp.shape[0]), -lp64))
    order = [int(j) for j in order if np.isfinite(lp64[j])][:K]
    return order, [float(lp64[j]) for j in order]


def plan_ctx(a_pool, cs, K, B):
    """First pass over context-dependent candidate lists.

    Best-first search that pushes every candidate child of a committed node;
    because a child never precedes its parent in the static order, the pops
    come in that order and the first B pops are the first B rank paths.
    Returns the BFS tree dict of planner.plan plus plan_slot (pool slot of
    each node's planning token, -1 at the root).
    """
    D = a_pool.shape[0]
    heap = []
    slot_of = {(): -1}
    score_of = {(): 0.0}

    def push_children(path, score):
        d = len(path)
        if d >= D:
            return
        slots, lps = candidates(corrected(a_pool, cs, d, slot_of[path]), K)
        for k, (j, lp) in enumerate(zip(slots, lps)):
            child = path + (k,)
            slot_of[child] = j
            heapq.heappush(heap, (-(score + lp), d + 1, child))

    push_children((), 0.0)
    chosen = []
    while len(chosen) < B and heap:
        neg, _, path = heapq.heappop(heap)
        score_of[path] = -neg
        chosen.append((path, -neg))
        push_children(path, -neg)
    margin = (chosen[-1][1] - (-heap[0][0])) if (chosen and heap) else np.inf
    tree = _bfs_tree(chosen, margin)
    tree["plan_slot"] = _slots_in_bfs(tree, chosen, slot_of)
    return tree


def _slots_in_bfs(tree, chosen, slot_of):
    """Pool slot of every node of a BFS tree built from rank paths."""
    n = tree["n_nodes"]
    path = [()] * n
    for i in range(1, n):
        path[i] = path[int(tree["parent"][i])] + (int(tree["rank"][i]),)
    return np.array([slot_of[p] for p in path], dtype=np.int64)


def plan_tokens(tree, pool, slots):
    """Token of every node from its pool slot (-1 at the root)."""
    tok = np.full(tree["n_nodes"], -1, np.int64)
    for i in range(1, tree["n_nodes"]):
        tok[i] = pool[int(tree["depth"][i]) - 1][int(slots[i])]
    return tok


def replay_pool(a_pool, cs, pool, tree, seed, step, request):
    """Refill every non-root node. Returns (node_tok, node_slot, per-parent margins)."""
    n = tree["n_nodes"]
    node_tok = np.full(n, -1, np.int64)
    node_slot = np.full(n, -1, np.int64)
    margins = {}
    for u in range(n):  # BFS order: a parent is filled before its children
        m = int(tree["n_children"][u])
        if m == 0:
            continue
        d = int(tree["depth"][u])
        z = corrected(a_pool, cs, d, int(node_slot[u]))
        toks = pool[d]
        g = philox.gumbel(philox.uniforms(seed, step, request, u, philox.STREAM_REPLAY,
                                          toks.astype(np.uint64)))
        keys = z + g
        order = np.lexsort((toks, -keys))
        top = keys[order[:m + 1]]
        gaps = top[:-1] - top[1:]
        margins[u] = float(gaps.min()) if gaps.size else np.inf
        fc = int(tree["first_child"][u])
        node_slot[fc:fc + m] = order[:m]
        node_tok[fc:fc + m] = toks[order[:m]]
    return node_tok, node_slot, margins


def q_full(a_pool, cs, pool, d, s, V):
    """q_u over the whole vocabulary (zero outside pool_d)."""
    q, _, _ = pool_q(corrected(a_pool, cs, d, s))
    out = np.zeros(V, np.float64)
    out[pool[d]] = q
    return out


def step_pool_request(draft, target, trans, T, K, P, B, seed, step, request, target_fn=None):
    """Full round for one request with pools of P tokens and transition table trans [D-1, P, P].

    target: array [B+1, V] (slot-keyed rows), or None with target_fn(tree,
    node_tok) -> array [n_nodes, V]. Returns a dict of stage outputs and the
    margin log (plan, replay, accept and bonus decisions).
    """
    invT = inv_temperature(T)
    draft = np.asarray(draft)
    D, V = draft.shape
    ok = all(row_ok(scaled(draft[d], invT)) for d in range(D)) and bool(np.isfinite(np.asarray(trans)).all())
    status = 0
    pool = pools(draft, P)
    a_pool = pool_logits(draft, invT, pool)
    cs = scaled_corrections(trans, invT)
    if not ok:
        tree = _bfs_tree([], np.inf)
        tree["plan_slot"] = np.full(1, -1, np.int64)
        return dict(tree=tree, pool=pool, node_tok=np.full(1, -1, np.int64), node_slot=np.full(1, -1, np.int64),
                    n_acc=-1, acc_node=[], acc_tok=[], bonus=-1, status=STATUS_NONFINITE,
                    margins=[("plan", -1, np.inf)], verify=None)
    tree = plan_ctx(a_pool, cs, K, B)
    if tree["n_nodes"] < B + 1:
        status |= STATUS_BUDGET_SHORT
    margins = [("plan", -1, tree["plan_margin"])]
    node_tok, node_slot, rmg = replay_pool(a_pool, cs, pool, tree, seed, step, request)
    margins += [("replay", u, m) for u, m in rmg.items()]
    if target is None:
        target = target_fn(tree, node_tok)
    n = tree["n_nodes"]
    a_t = [scaled(target[u], invT) for u in range(n)]
    if not all(row_ok(a) for a in a_t):
        return dict(tree=tree, pool=pool, node_tok=node_tok, node_slot=node_slot, n_acc=-1, acc_node=[],
                    acc_tok=[], bonus=-1, status=status | STATUS_NONFINITE, margins=margins, verify=None)
    lse_t = np.array([lse64(a) for a in a_t])
    depth = tree["depth"]
    vr = verify_mod.verify(lambda u: probs(a_t[u], lse_t[u]), None, tree, node_tok, seed, step, request,
                           q_node=lambda u: q_full(a_pool, cs, pool, int(depth[u]), int(node_slot[u]), V))
    vr["lse_t"] = lse_t
    margins += vr["margins"]
    return dict(tree=tree, pool=pool, node_tok=node_tok, node_slot=node_slot, n_acc=vr["n_acc"],
                acc_node=vr["acc_node"], acc_tok=vr["acc_tok"], bonus=vr["bonus"],
                status=status | vr["status"], margins=margins, verify=vr)
