"""One decoding round of tree replay for a batch of independent requests
(oracle side): plan -> replay -> verify.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

Section 3 (Figure 1): the first pass plans and freezes the topology from the
draft path scores, the second pass replays it with fresh samples, and the
replayed tree is verified against the target (Section 3.3, Proposition 1:
lossless when the topology is fixed before replay and the verifier is
lossless for any fixed topology).

Inputs per request: draft logits x[D, V] (one row per block position) and
target logits t[B+1, V] (one row per tree node in BFS order, root first).
Row d of the draft is the distribution of the tokens at depth d + 1.
"""
import numpy as np

from . import planner, replay as replay_mod, traversal as traversal_mod, verify as verify_mod
from .rowstats import (STATUS_BUDGET_SHORT, STATUS_NONFINITE, draft_rowstats,
                       inv_temperature, lse64, probs, row_ok, scaled)

NEAR_TIE = 1e-5


def plan_request(draft, T, K, B):
    """Row statistics + first pass for one request (draft: [D, V])."""
    invT = inv_temperature(T)
    D = draft.shape[0]
    ok_all = True
    l64 = np.zeros(D)
    l32 = np.zeros(D, np.float32)
    ids = np.zeros((D, K), np.int64)
    lp = np.zeros((D, K), np.float32)
    for d in range(D):
        ok, a, b, c, e = draft_rowstats(draft[d], invT, K)
        ok_all &= ok
        l64[d], l32[d], ids[d], lp[d] = a, b, c, e
    status = 0
    if not ok_all:
        tree = planner.plan(np.zeros((0, K), np.float32), B)
        status |= STATUS_NONFINITE
    else:
        tree = planner.plan(lp, B)
        if tree["n_nodes"] < B + 1:
            status |= STATUS_BUDGET_SHORT
    return dict(invT=invT, lse64=l64, lse32=l32, topk_tok=ids, topk_lp=lp,
                tree=tree, status=status)


VERIFIERS = ("rrs", "traversal")


class _RowNotFinite(Exception):
    """A target row the walk visits holds a NaN or +inf, or no finite entry."""


def verify_request(draft, target, tree, node_tok, lse_draft64, T, seed, step, request, verifier="rrs"):
    """Target normalisers + the verification walk for one request: WoR-RRS (eq. (1); Appendix A) or
    traversal verification (Appendix A; Table 2), both with the replayed candidates' probabilities.

    Unusable target rows (a NaN, a +inf, or no finite entry; the paper has no such rows) end the round
    with NONFINITE. WoR-RRS reads a row only when its walk enters the node, so only the rows of the
    nodes it enters count, as in target-sample matching; traversal verification counts every row of the
    tree. lse_t holds each row's normaliser (NaN for an unusable row) whatever the status.
    """
    invT = inv_temperature(T)
    n = tree["n_nodes"]
    a_t = [scaled(target[u], invT) for u in range(n)]
    ok = [row_ok(a) for a in a_t]
    lse_t = np.array([lse64(a) if ok[u] else np.nan for u, a in enumerate(a_t)])
    unusable = dict(n_acc=-1, acc_node=[], acc_tok=[], bonus=-1, terminal=-1,
                    status=STATUS_NONFINITE, tests=[], residual_Z=[], margins=[], lse_t=lse_t)
    if verifier != "rrs" and not all(ok):
        return unusable

    def p_rows(u):
        if not ok[u]:
            raise _RowNotFinite(u)
        return probs(a_t[u], lse_t[u])

    a_d = scaled(draft, invT)
    walk = verify_mod.verify if verifier == "rrs" else traversal_mod.verify_traversal
    try:
        res = walk(p_rows, lambda d: probs(a_d[d], lse_draft64[d]), tree, node_tok, seed, step, request)
    except _RowNotFinite:
        return unusable
    res["lse_t"] = lse_t
    return res


def step_request(draft, target, T, K, B, seed, step, request, target_fn=None, verifier="rrs"):
    """Full round for one request.

    target: array [B+1, V] (slot-keyed rows), or None with target_fn(tree,
    node_tok) -> array [n_nodes, V] built after replay (prefix-keyed tests).
    Returns a dict of all stage outputs and the margin log.
    """
    pl = plan_request(draft, T, K, B)
    tree = pl["tree"]
    out = dict(plan=pl, tree=tree)
    margins = [("plan", -1, pl["tree"]["plan_margin"])]
    if pl["status"] & STATUS_NONFINITE:
        out.update(node_tok=np.full(tree["n_nodes"], -1, np.int64), n_acc=-1, acc_node=[],
                   acc_tok=[], bonus=-1, status=pl["status"], margins=margins, verify=None)
        return out
    a_d = scaled(draft, pl["invT"])
    node_tok, rmg = replay_mod.replay(a_d, tree, seed, step, request)
    margins += [("replay", u, m) for u, m in rmg.items()]
    if target is None:
        target = target_fn(tree, node_tok)
    vr = verify_request(draft, target, tree, node_tok, pl["lse64"], T, seed, step, request, verifier)
    margins += vr["margins"]
    out.update(node_tok=node_tok, n_acc=vr["n_acc"], acc_node=vr["acc_node"],
               acc_tok=vr["acc_tok"], bonus=vr["bonus"], status=pl["status"] | vr["status"],
               margins=margins, verify=vr)
    return out


def near_ties(margins, thr=NEAR_TIE):
    """Decisions whose margin is positive but below the near-tie threshold."""
    return [m for m in margins if 0.0 < m[2] < thr]
