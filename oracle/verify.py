"""Verification of the replayed tree: recursive rejection sampling without
replacement, plus the bonus token (oracle side).

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

Section 2.3, eq. (1): a proposed token v ~ q is accepted with probability
min{1, p(v)/q(v)}; on rejection the output is corrected by sampling the
normalised residual max(p - q, 0). Appendix A: candidates drawn without
replacement are verified with the WoR variant of recursive rejection
sampling (RRS) across siblings; Table 2 lists RRS as the step-wise tree
verifier paired with WoR sampling. Section 3.3: the probabilities used are
those of the replayed candidates, q_u of eq. (2).

Literal procedure (the form this module follows), per request, starting at
the root u:
  P <- p_u, Q <- q_{depth(u)}
  for each child c of u in slot order, token y:
      U ~ uniform (ACCEPT stream, node c)
      accept iff U < P(y) / Q(y)        (min{1, .} is implied since U < 1)
      -> emit y, move to c and start over with P <- p_c, Q <- q_{depth(c)}
      otherwise  P <- max(P - Q, 0) / sum max(P - Q, 0)
                 Q(y) <- 0, Q <- Q / sum Q
  when no child is accepted (or u is a leaf) the bonus token is a sample of
  P, taken as argmax_v ln P(v) + G_v (Gumbel-max, BONUS stream, node u).
An empty residual or an exhausted Q (measure zero in exact arithmetic) sets
the DEGENERATE_RESIDUAL status bit and the bonus is drawn from p_u.

closed_form_node() restates the same recursion in closed form (derived, not
printed in the paper): after i rejections P is proportional to
max(p - C_i q, 0) and Q to q over the unremoved tokens / S_i, with C_0 = 0,
S_0 = 1, Z_0 = 1, W_i = Z_i / S_i, C_{i+1} = C_i + W_i, S_{i+1} = S_i - q(y),
Z_{i+1} = sum_v max(p_v - C_{i+1} q_v, 0), ratio_i = max(p(y) - C_i q(y), 0)
/ (W_i q(y)). The tests hold it to the literal form to 1e-12.
"""
import numpy as np

from . import philox
from .rowstats import STATUS_DEGENERATE_RESIDUAL


def accept_ratio(P, Q, y):
    """P(y) / Q(y) of the current (normalised) residual pair."""
    qy = Q[y]
    if qy <= 0.0:
        return np.inf if P[y] > 0.0 else 0.0
    return float(P[y] / qy)


def reject(P, Q, y):
    """Literal WoR-RRS update after rejecting token y: returns (P', Q', Z, S)."""
    R = np.maximum(P - Q, 0.0)
    Z = float(R.sum())
    Qn = Q.copy()
    Qn[y] = 0.0
    S = float(Qn.sum())
    Pn = R / Z if Z > 0.0 else R
    Qn = Qn / S if S > 0.0 else Qn
    return Pn, Qn, Z, S


def bonus_sample(P, seed, step, request, node):
    """Gumbel-max sample of distribution P (zero entries excluded). Returns (token, margin)."""
    V = P.shape[0]
    with np.errstate(divide="ignore"):
        keys = np.log(P) + philox.gumbels(seed, step, request, node, philox.STREAM_BONUS, V)
    order = np.lexsort((np.arange(V), -keys))
    margin = float(keys[order[0]] - keys[order[1]]) if V > 1 else np.inf
    return int(order[0]), margin


def verify(p_rows, q_rows, tree, node_tok, seed, step, request, q_node=None):
    """Walk the replayed tree.

    p_rows(u) -> float64 target distribution at node u (length V)
    q_rows(d) -> float64 draft distribution of position d
    q_node(u) -> float64 draft distribution q_u of the children of node u;
                 when given it replaces q_rows (drafters whose q_u depends on
                 the replayed prefix, eq. (2))
    Returns dict: n_acc, acc_node, acc_tok, bonus, status, tests (list of
    (child, U, ratio, accepted)), residual_Z (list), margins (list of
    (kind, id, margin)).
    """
    n_children = tree["n_children"]
    first_child = tree["first_child"]
    depth = tree["depth"]
    u = 0
    acc_node, acc_tok, tests, zs, margins = [], [], [], [], []
    status = 0
    while True:
        m = int(n_children[u])
        P = p_rows(u)
        if m == 0:
            Q = None
        elif q_node is not None:
            Q = q_node(u)
        else:
            Q = q_rows(int(depth[u]))
        accepted = False
        degenerate = False
        for j in range(m):
            c = int(first_child[u]) + j
            y = int(node_tok[c])
            U = float(philox.uniforms(seed, step, request, c, philox.STREAM_ACCEPT, 0))
            ratio = accept_ratio(P, Q, y)
            ok = U < ratio
            tests.append((c, U, ratio, ok))
            margins.append(("accept", c, abs(U - ratio)))
            if ok:
                acc_node.append(c)
                acc_tok.append(y)
                u = c
                accepted = True
                break
            P, Q, Z, S = reject(P, Q, y)
            zs.append(Z)
            if Z <= 0.0 or (j + 1 < m and S <= 0.0):
                degenerate = True
                break
        if accepted:
            continue
        if degenerate:
            status |= STATUS_DEGENERATE_RESIDUAL
            P = p_rows(u)
        bonus, mg = bonus_sample(P, seed, step, request, u)
        margins.append(("bonus", u, mg))
        return dict(n_acc=len(acc_node), acc_node=acc_node, acc_tok=acc_tok,
                    bonus=bonus, terminal=u, status=status, tests=tests,
                    residual_Z=zs, margins=margins)


def closed_form_node(p, q, ys, Us):
    """Closed-form WoR-RRS at one node for children tokens ys and uniforms Us.

    Returns (index of the accepted child or -1, ratios, Zs, C at exit).
    """
    C, S, Z = 0.0, 1.0, 1.0
    ratios, zs = [], []
    for j, (y, U) in enumerate(zip(ys, Us)):
        W = Z / S
        qy = q[y]
        ratio = max(p[y] - C * qy, 0.0) / (W * qy)
        ratios.append(ratio)
        if U < ratio:
            return j, ratios, zs, C
        C = C + W
        S = S - qy
        Z = float(np.maximum(p - C * q, 0.0).sum())
        zs.append(Z)
    return -1, ratios, zs, C
