"""The first-pass tree with its planning tokens (First) and target-sample
matching verification (Naive), oracle side.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

Section 3.1: the first pass yields a deterministic, context-aware tree; kept
with its planning tokens and verified directly it is the deterministic
baseline First (the TopK candidate selection of Tables 3 and 4). A node of
depth d and rank j carries the j-th planning candidate of draft position
d - 1.

Table 2 (Naive) and Section 2.3: target-sample matching. At node u a token y
is drawn from the target distribution p_u; if y is the token of a child of u
that child is accepted and the walk goes on from it, otherwise y is emitted
as the bonus token and the round ends. Every emitted token is then a target
sample given its prefix, so the rule is lossless for any tree and any node
tokens (Replay + Naive as well as First + Naive).

The draw at node u is the Gumbel-max sample argmax_v a_v + G_v with
a = fl32(t_u invT) and G from the BONUS stream (node u): the same draw the
RRS verifier makes for a bonus from p_u (a common shift by the normaliser
does not change the argmax).
"""
import numpy as np

from . import philox
from .rowstats import STATUS_NONFINITE, inv_temperature, row_ok, scaled


def first_tokens(tree, topk_tok):
    """Planning tokens of the first-pass tree: node of depth d, rank j -> topk_tok[d - 1, j]; root -1."""
    n = int(tree["n_nodes"])
    tok = np.full(n, -1, dtype=np.int64)
    for i in range(1, n):
        tok[i] = int(topk_tok[int(tree["depth"][i]) - 1, int(tree["rank"][i])])
    return tok


def target_sample(a, seed, step, request, node):
    """Gumbel-max draw from softmax(a): (token, margin between the two best keys)."""
    V = a.shape[0]
    keys = a.astype(np.float64) + philox.gumbels(seed, step, request, node, philox.STREAM_BONUS, V)
    order = np.lexsort((np.arange(V), -keys))
    margin = float(keys[order[0]] - keys[order[1]]) if V > 1 else np.inf
    return int(order[0]), margin


def verify_naive(target, tree, node_tok, T, seed, step, request):
    """Target-sample matching over a tree.

    target: raw target logits [n_nodes (or more), V], row u for node u.
    Returns dict: n_acc, acc_node, acc_tok, bonus, terminal, status, margins
    (list of (node, margin)). A visited row with NaN or +inf (after scaling)
    or with no finite entry ends the round with NONFINITE (n_acc = bonus = -1).
    """
    invT = inv_temperature(T)
    n_children = tree["n_children"]
    first_child = tree["first_child"]
    u = 0
    acc_node, acc_tok, margins = [], [], []
    while True:
        a = scaled(target[u], invT)
        if not row_ok(a):
            return dict(n_acc=-1, acc_node=[], acc_tok=[], bonus=-1, terminal=u, status=STATUS_NONFINITE,
                        margins=margins)
        y, mg = target_sample(a, seed, step, request, u)
        margins.append((u, mg))
        m = int(n_children[u])
        fc = int(first_child[u])
        match = -1
        for j in range(m):
            if int(node_tok[fc + j]) == y:
                match = fc + j
                break
        if match < 0:
            return dict(n_acc=len(acc_node), acc_node=acc_node, acc_tok=acc_tok, bonus=y, terminal=u, status=0,
                        margins=margins)
        acc_node.append(match)
        acc_tok.append(y)
        u = match



def first_naive_request(draft, target, T, K, B, seed, step, request):
    """One First + Naive round for one request: plan, keep the planning tokens, verify by matching.

    draft: [D, V] logits; target: [B+1, V] logits, one row per tree node in BFS order.
    """
    from .step import plan_request

    pl = plan_request(draft, T, K, B)
    tree = pl["tree"]
    if pl["status"] & STATUS_NONFINITE:
        return dict(plan=pl, tree=tree, node_tok=np.full(tree["n_nodes"], -1, np.int64), n_acc=-1,
                    acc_node=[], acc_tok=[], bonus=-1, terminal=-1, status=pl["status"], margins=[])
    node_tok = first_tokens(tree, pl["topk_tok"])
    vr = verify_naive(target, tree, node_tok, T, seed, step, request)
    out = dict(vr)
    out.update(plan=pl, tree=tree, node_tok=node_tok, status=pl["status"] | vr["status"])
    return out
