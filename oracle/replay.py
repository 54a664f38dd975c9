"""Second pass: tree replay by Gumbel-top-k sampling (oracle side).

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

Section 3.2, eq. (2): the frozen topology is refilled layer by layer; every
parent u draws fresh tokens for its fixed child slots from
q_u = q(. | x, y_path(u)), without replacement (Appendix A: each draw excludes
the previously drawn tokens and renormalises q). This project's drafter is a
parallel block predictor, so q_u depends only on the depth of u:
q_u = softmax(a_{depth(u)}) over the whole vocabulary.

Sampling without replacement is realised with the Gumbel-top-k construction
(Kool, van Hoof and Welling, ICML 2019): with independent standard Gumbel
noise G_v, the tokens ordered by decreasing a_v + G_v are an ordered sample
without replacement from softmax(a) (Plackett-Luce law). Child slot j (rank
order) receives the j-th largest key; equal keys go to the smaller token id.
G_v comes from the REPLAY stream of the counter-based generator, keyed by
(seed, step, request, parent u, token v).
"""
import numpy as np

from . import philox


def replay_node(a_row, m, seed, step, request, node):
    """Top-m tokens of a_v + G_v for one parent. Returns (tokens, margin).

    margin is the smallest gap between consecutive keys among the m + 1
    largest (the decision that fixes which token lands in which slot).
    """
    a = np.asarray(a_row, dtype=np.float64)
    V = a.shape[0]
    keys = a + philox.gumbels(seed, step, request, node, philox.STREAM_REPLAY, V)
    order = np.lexsort((np.arange(V), -keys))
    top = keys[order[:m + 1]]
    gaps = top[:-1] - top[1:]
    margin = float(gaps.min()) if gaps.size else np.inf
    return order[:m].astype(np.int64), margin


def replay(a_draft, tree, seed, step, request):
    """Fill every non-root node. a_draft: float64 [D, V] scaled draft logits.

    Returns (node_tok [n_nodes] with -1 at the root, per-parent margins dict).
    """
    n = tree["n_nodes"]
    node_tok = np.full(n, -1, dtype=np.int64)
    margins = {}
    for u in range(n):
        m = int(tree["n_children"][u])
        if m == 0:
            continue
        d = int(tree["depth"][u])
        toks, mg = replay_node(a_draft[d], m, seed, step, request, u)
        fc = int(tree["first_child"][u])
        node_tok[fc:fc + m] = toks
        margins[u] = mg
    return node_tok, margins
