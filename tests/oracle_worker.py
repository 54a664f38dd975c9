"""Oracle side of the GPU parity tests, run in worker processes (or in
process for small cases).

TEST INFRASTRUCTURE: calls the CPU oracle; imports numpy and the oracle only
(no torch, no HIP), so worker processes start fast and never touch the GPU.

A task is one request of one round: the CPU oracle plans it from the very
draft bytes the HIP path read, then replays and verifies it on the topology
and node tokens the HIP path produced (so each stage is compared on the same
inputs, and a flagged near-tie in one stage does not hide the next). Inputs
arrive as memory-mapped files written by the test process: bf16 logits as
raw 16-bit patterns, binary32 logits as is.
"""
import numpy as np

from oracle import naive as onaive, pool as opool, replay as oreplay, step as ostep, verify as overify
from oracle.rowstats import STATUS_BUDGET_SHORT, STATUS_NONFINITE, inv_temperature, lse64, probs, row_ok, scaled

_MAPS = {}


def _rows(spec, r):
    """Row block r of a shared logit array spec = (path, shape, dtype) as float32."""
    path, shape, dtype = spec
    m = _MAPS.get(path)
    if m is None:
        if len(_MAPS) > 4:
            _MAPS.clear()
        m = np.memmap(path, dtype=np.uint16 if dtype == "bf16" else np.float32, mode="r", shape=tuple(shape))
        _MAPS[path] = m
    x = np.array(m[r])
    if dtype == "bf16":
        x = (x.astype(np.uint32) << 16).view(np.float32)
    return x


def request_step(d, t, T, K, B, seed, step, r, gtree, gtok):
    """Oracle outputs of one request-step.

    d: draft rows [D, V]; t: target rows [B+1, V] (or None for plan only);
    gtree: the HIP path's topology of this request (oracle tree format) and
    gtok its node tokens, or None to skip replay and verification.
    """
    pl = ostep.plan_request(d, T, K, B)
    out = dict(plan=pl, replay=None, verify=None)
    if gtree is None or pl["status"] & STATUS_NONFINITE:
        return out
    a_d = scaled(d, inv_temperature(T))
    tok, mg = oreplay.replay(a_d, gtree, seed, step, r)
    out["replay"] = (tok, mg)
    if t is not None:
        vr = ostep.verify_request(d, t, gtree, gtok, pl["lse64"], T, seed, step, r)
        out["verify"] = vr
    return out


def request_step_traversal(d, t, T, K, B, seed, step, r, gtree, gtok):
    """As request_step with traversal verification on the HIP path's topology and tokens."""
    pl = ostep.plan_request(d, T, K, B)
    out = dict(plan=pl, replay=None, verify=None)
    if gtree is None or pl["status"] & STATUS_NONFINITE:
        return out
    tok, mg = oreplay.replay(scaled(d, inv_temperature(T)), gtree, seed, step, r)
    out["replay"] = (tok, mg)
    if t is not None:
        out["verify"] = ostep.verify_request(d, t, gtree, gtok, pl["lse64"], T, seed, step, r, verifier="traversal")
    return out


def request_step_naive(d, t, T, K, B, seed, step, r, gtree, gtok):
    """First + Naive oracle outputs of one request-step: the plan and First tokens from the draft, and
    target-sample matching on the HIP path's topology and node tokens."""
    pl = ostep.plan_request(d, T, K, B)
    out = dict(plan=pl, first_tok=None, naive=None)
    if pl["status"] & STATUS_NONFINITE:
        return out
    out["first_tok"] = onaive.first_tokens(pl["tree"], pl["topk_tok"])
    if gtree is not None and t is not None:
        out["naive"] = onaive.verify_naive(t, gtree, gtok, T, seed, step, r)
    return out


def request_step_pool(d, t, T, K, B, seed, step, r, gtree, gtok, trans, P):
    """Sparse-pool oracle outputs of one request-step: pools and the first pass over per-node candidate lists
    from the draft and transition scores; replay and verification on the HIP path's topology and tokens."""
    invT = inv_temperature(T)
    D, V = d.shape
    pool = opool.pools(d, P)
    out = dict(pool=pool, tree=None, status=0, plan_tok=None, replay=None, verify=None)
    if not (all(row_ok(scaled(d[j], invT)) for j in range(D)) and bool(np.isfinite(trans).all())):
        out["status"] = STATUS_NONFINITE
        return out
    a_pool = opool.pool_logits(d, invT, pool)
    cs = opool.scaled_corrections(trans, invT)
    tree = opool.plan_ctx(a_pool, cs, K, B)
    out["tree"] = tree
    out["status"] = STATUS_BUDGET_SHORT if tree["n_nodes"] < B + 1 else 0
    out["plan_tok"] = opool.plan_tokens(tree, pool, tree["plan_slot"])
    if gtree is None:
        return out
    tok, _, mg = opool.replay_pool(a_pool, cs, pool, gtree, seed, step, r)
    out["replay"] = (tok, mg)
    if t is None or gtok is None:
        return out
    n = gtree["n_nodes"]
    a_t = [scaled(t[u], invT) for u in range(n)]
    if not all(row_ok(a) for a in a_t):
        out["verify"] = dict(n_acc=-1, status=STATUS_NONFINITE)
        return out
    lse_t = np.array([lse64(a) for a in a_t])
    depth = gtree["depth"]
    # pool slot of every node's token in its position's pool (the context of its children)
    slot = np.full(n, -1, np.int64)
    for u in range(1, n):
        hit = np.nonzero(pool[int(depth[u]) - 1] == int(gtok[u]))[0]
        slot[u] = int(hit[0]) if hit.size else 0
    vr = overify.verify(lambda u: probs(a_t[u], lse_t[u]), None, gtree, gtok, seed, step, r,
                        q_node=lambda u: opool.q_full(a_pool, cs, pool, int(depth[u]), int(slot[u]), V))
    vr["lse_t"] = lse_t
    out["verify"] = vr
    return out


KINDS = {"rrs": request_step, "naive": request_step_naive, "pool": request_step_pool,
         "traversal": request_step_traversal}


def run(task):
    """Pool entry: task = (kind, draft spec, target spec, T, K, B, seed, step, r, gtree, gtok[, trans spec, P])."""
    kind, dspec, tspec, T, K, B, seed, step, r, gtree, gtok = task[:11]
    d = _rows(dspec, r)
    t = _rows(tspec, r) if tspec is not None else None
    if kind == "pool":
        return r, step, request_step_pool(d, t, T, K, B, seed, step, r, gtree, gtok, _rows(task[11], r), task[12])
    return r, step, KINDS[kind](d, t, T, K, B, seed, step, r, gtree, gtok)
