"""Traversal verification of a replayed tree (oracle side): sequence-level
recursive rejection sampling over a tree whose siblings were drawn without
replacement.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

Appendix A: Traversal Verification (Weng et al., 2025) extends the
sequence-level verification of Block Verification (Sun et al., 2025) from
chains to trees, as sequence-level RRS with WoR candidates; Table 2 lists it
as the sequence-level verifier paired with WoR sampling, and Section 4.2
compares it with layer-wise RRS on replayed trees. The paper states the
method by reference only; this module restates it from its published
definition (the reading is listed in the design notes and pinned by the
tests: exact losslessness, reduction to WoR-RRS on one layer, and the
Block-Verification optimum on a chain).

Each node u carries three quantities, set when the traversal first reaches
it and updated whenever one of its children is rejected:
  Mb_u   the distribution a bonus at u is drawn from (initially p_u, the
         target's next-token distribution at u),
  Ms_u   the distribution u's remaining children were drawn from (initially
         q_u; the rejected child's token is removed and Ms_u renormalised:
         the without-replacement update),
  alpha_u  the probability of accepting the path root..u when u is tested:
         alpha_root = 1 and, for a child c of u with token y,
         alpha_c = min(1, alpha_u * Mb_u(y) / Ms_u(y)) with u's quantities
         at the time c is reached (a running capped product of
         target-to-draft ratios along the path).
The traversal is post-order, siblings in slot order: starting from the root
it follows the first remaining child down to a node with no remaining
children and tests it with U ~ uniform (ACCEPT stream of that node):
  * U < alpha_c: the path root..c is accepted; the bonus token is a sample
    of Mb_c (Gumbel-max, BONUS stream of c).
  * otherwise c is removed from the tree and its parent u updates, with the
    quantities from which c was drawn:
        T      = sum_v max(alpha_u Mb_u(v) - Ms_u(v), 0)
        Mb_u  <- max(alpha_u Mb_u - Ms_u, 0) / T
        alpha_u <- T / (T + 1 - alpha_u)
        Ms_u(y) <- 0, Ms_u <- Ms_u / sum Ms_u
    and the traversal continues from u (its next child, or u itself once
    it has none left).
The root keeps alpha = 1 (T / (T + 0)), so once every child of the root is
rejected the root is accepted and the bonus is a sample of its residual:
on a tree of one layer this is exactly WoR-RRS. On a chain Mb and alpha
follow Block Verification's residual distributions and acceptance
probabilities.

Readings where the method is silent (measure-zero events in exact
arithmetic, handled deterministically):
  * T <= 0 at a node with alpha_u < 1: alpha_u <- 0 (the formula's value),
    Mb_u <- 0; u and its remaining children can no longer be accepted.
  * T <= 0 at a node with alpha_u = 1, or Ms_u exhausted (sum <= 0) while
    u has children left: the walk stops at u, the bonus is drawn from p_u and
    DEGENERATE_RESIDUAL is set (as for RRS).
The root is accepted without a uniform (alpha_root = 1).

closed_form_state() restates the node update in the closed form the GPU
walk uses (derived here, not printed anywhere): a node's Mb is
max(A p - C q, 0) / Z and its Ms is q / S over the unremoved tokens, with
A = 1, C = 0, Z = 1, S = 1 when the node is first reached; a rejection of the
child with token y maps (alpha, A, C, Z, S) to
  A' = alpha A / Z,  C' = alpha C / Z + 1 / S,  Z' = T = sum_v max(A' p - C' q, 0),
  alpha' = T / (T + 1 - alpha),  S' = S - q(y).
(Removed tokens contribute nothing: their A' p - C' q is <= 0.)
"""
import numpy as np

from . import philox
from .rowstats import STATUS_DEGENERATE_RESIDUAL


def child_alpha(alpha_u, Mb_u, Ms_u, y):
    """Acceptance probability of the path to the child of u holding token y."""
    b, s = float(Mb_u[y]), float(Ms_u[y])
    if s <= 0.0:
        return 1.0 if (b > 0.0 and alpha_u > 0.0) else 0.0
    return min(1.0, alpha_u * b / s)


def reject_child(alpha_u, Mb_u, Ms_u, y):
    """Update of node u after its child holding token y was rejected.

    Returns (alpha', Mb', Ms', T, S) with T the residual mass and S the draft
    mass left before renormalising Ms.
    """
    R = np.maximum(alpha_u * Mb_u - Ms_u, 0.0)
    T = float(R.sum())
    if T > 0.0:
        Mb_n = R / T
        alpha_n = T / (T + (1.0 - alpha_u))
    else:
        Mb_n = np.zeros_like(Mb_u)
        alpha_n = 0.0 if alpha_u < 1.0 else float("nan")
    Ms_n = Ms_u.copy()
    Ms_n[y] = 0.0
    S = float(Ms_n.sum())
    if S > 0.0:
        Ms_n = Ms_n / S
    return alpha_n, Mb_n, Ms_n, T, S


def bonus_sample(P, seed, step, request, node):
    """Gumbel-max sample of distribution P (zero entries excluded). Returns (token, margin)."""
    V = P.shape[0]
    with np.errstate(divide="ignore"):
        keys = np.log(P) + philox.gumbels(seed, step, request, node, philox.STREAM_BONUS, V)
    order = np.lexsort((np.arange(V), -keys))
    margin = float(keys[order[0]] - keys[order[1]]) if V > 1 else np.inf
    return int(order[0]), margin


def verify_traversal(p_rows, q_rows, tree, node_tok, seed, step, request, q_node=None):
    """Traverse the replayed tree.

    p_rows(u) -> float64 target distribution at node u (length V)
    q_rows(d) -> float64 draft distribution of position d (the children of
                 a node at depth d were drawn from it)
    q_node(u) -> draft distribution of u's children, replacing q_rows when
                 given (drafters whose q_u depends on the replayed prefix)
    Returns dict: n_acc, acc_node, acc_tok, bonus, terminal, status, tests
    (list of (node, U, alpha, accepted) in traversal order), residual_T
    (list of T per rejection), margins (list of (kind, id, margin)).
    """
    n_children = tree["n_children"]
    first_child = tree["first_child"]
    depth = tree["depth"]

    def q_of(u):
        return q_node(u) if q_node is not None else q_rows(int(depth[u]))

    Mb = {0: p_rows(0)}
    Ms = {0: q_of(0) if int(n_children[0]) > 0 else None}
    alpha = {0: 1.0}
    left = {0: 0}
    path = [0]
    tests, res_T, margins = [], [], []
    status = 0

    def finish(u, P):
        bonus, mg = bonus_sample(P, seed, step, request, u)
        margins.append(("bonus", u, mg))
        acc = [c for c in path[1:]]
        return dict(n_acc=len(acc), acc_node=acc, acc_tok=[int(node_tok[c]) for c in acc], bonus=bonus,
                    terminal=u, status=status, tests=tests, residual_T=res_T, margins=margins)

    while True:
        u = path[-1]
        if left[u] < int(n_children[u]):       # descend to the next remaining child
            c = int(first_child[u]) + left[u]
            alpha[c] = child_alpha(alpha[u], Mb[u], Ms[u], int(node_tok[c]))
            Mb[c] = p_rows(c)
            Ms[c] = q_of(c) if int(n_children[c]) > 0 else None
            left[c] = 0
            path.append(c)
            continue
        if u == 0:                             # every child of the root rejected
            return finish(0, Mb[0])
        U = float(philox.uniforms(seed, step, request, u, philox.STREAM_ACCEPT, 0))
        ok = U < alpha[u]
        tests.append((u, U, alpha[u], ok))
        margins.append(("accept", u, abs(U - alpha[u])))
        if ok:
            return finish(u, Mb[u])
        path.pop()
        w = path[-1]
        a_new, Mb_new, Ms_new, T, S = reject_child(alpha[w], Mb[w], Ms[w], int(node_tok[u]))
        res_T.append(T)
        left[w] += 1
        if (T <= 0.0 and alpha[w] >= 1.0) or (S <= 0.0 and left[w] < int(n_children[w])):
            status |= STATUS_DEGENERATE_RESIDUAL
            return finish(w, p_rows(w))
        alpha[w], Mb[w], Ms[w] = a_new, Mb_new, Ms_new


def closed_form_state(p, q, alpha0, ys):
    """Closed form of a node's state along successive child rejections (tokens ys), from its first visit
    with alpha0. Returns the list of (alpha, A, C, Z, S) after each rejection."""
    alpha, A, C, Z, S = alpha0, 1.0, 0.0, 1.0, 1.0
    out = []
    for y in ys:
        A, C = alpha * A / Z, alpha * C / Z + 1.0 / S
        T = float(np.maximum(A * p - C * q, 0.0).sum())
        alpha = T / (T + (1.0 - alpha)) if T > 0.0 else 0.0
        Z = T if T > 0.0 else 1.0
        if T <= 0.0:
            A, C = 0.0, 0.0
        S = S - float(q[y])
        out.append((alpha, A, C, Z, S))
    return out


def closed_form_mb(p, q, A, C, Z):
    """Mb of the closed form: max(A p - C q, 0) / Z."""
    return np.maximum(A * p - C * q, 0.0) / Z
