"""GPU parity of the expand-then-prune first pass (Section 3.1; Appendix B.3)
against the oracle (oracle/planner_ep.py), through the C ABI.

The row statistics and candidates are those of tsb_plan (compared as in the
main parity tests); the topology, scores and margin must match the oracle
bit for bit, except plan near-ties, which are reported. Cases: every
workload at the paper's frontier width (10) and at widths 1 and 4; a
frontier at least as wide as the budget must reproduce tsb_plan's tree;
exact-tie inputs; zero budget, non-finite rows and budgets larger than the
generated set; and a full round (plan_ep, replay, verify) against the
oracle.
"""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import planner_ep, replay as oreplay, step as ostep
from oracle.rowstats import STATUS_BUDGET_SHORT, STATUS_NONFINITE, inv_temperature, scaled
import paper_2609_33652_amd as tsb
from parity_util import compare_plan, compare_request, make_round, to_np, tree_dict_np
from tally import Tally

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tsb.load()


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def plan_request_ep(draft, T, K, B, w):
    pl = ostep.plan_request(draft, T, K, B)
    if pl["status"] & STATUS_NONFINITE:
        return pl
    pl["tree"] = planner_ep.plan_expand_prune(pl["topk_lp"], B, w)
    pl["status"] = STATUS_BUDGET_SHORT if pl["tree"]["n_nodes"] < B + 1 else 0
    return pl


def run_ep(cfg, w, steps=1, requests=None, gen_device="cpu", name=""):
    R, D, B, K, T = cfg["R"], cfg["D"], cfg["B"], cfg["K"], cfg["T"]
    requests = list(range(R)) if requests is None else list(requests)
    rnd = make_round(cfg, 3, trace=False)
    tally = Tally("plan_ep %s w=%d" % (name, w))
    for s in range(steps):
        say("plan_ep %s w=%d step %d (%s)" % (name, w, s, W.describe(cfg)))
        base, _ = W.base_rows(cfg, set_idx=s, device=gen_device)
        draft = W.draft_from_base(cfg, base)
        d_host = to_np(draft[requests].cpu())
        rnd.plan_ep(draft.cuda().contiguous(), w)
        h = rnd.host()
        for i, r in enumerate(requests):
            pl = plan_request_ep(d_host[i], T, K, B, w)
            compare_plan(h, r, pl, tally, "%s w=%d step %d req %d" % (name, w, s, r))
            if not pl["status"] & STATUS_NONFINITE:
                assert bool(int(h["req_status"][r]) & tsb.REQ_BUDGET_SHORT) == bool(pl["status"] & STATUS_BUDGET_SHORT)
    say(tally.line())
    assert tally.flagged <= 1, tally.notes
    return tally


@pytest.mark.parametrize("cfg_id,steps,w", [(1, 40, 10), (1, 20, 1), (2, 20, 10), (2, 10, 4), (3, 10, 10)])
def test_plan_ep_small_workloads(cfg_id, steps, w):
    t = run_ep(W.config(cfg_id), w, steps=steps, name=W.config(cfg_id)["name"])
    assert t.exact["plan"] + t.flagged_by["plan"] == steps


def test_plan_ep_batched_and_large_budget():
    t = run_ep(W.config(4), 10, steps=4, gen_device="cuda", name="batched")
    assert t.exact["plan"] + t.flagged_by["plan"] == 64
    t = run_ep(W.config(5), 10, steps=2, gen_device="cuda", name="large_budget")
    assert t.exact["plan"] + t.flagged_by["plan"] == 128


def test_wide_frontier_reproduces_max_heap_tree():
    cfg = W.config(2, R=3, V=20000, D=6, B=40, K=6, name="wide")
    base, _ = W.base_rows(cfg, 0)
    draft = W.draft_from_base(cfg, base).cuda()
    a = make_round(cfg, 1, trace=False)
    b = make_round(cfg, 1, trace=False)
    a.plan(draft)
    b.plan_ep(draft, 64)
    ha, hb = a.host(), b.host()
    for k in ("parent", "depth", "rank", "n_children", "first_child", "score", "n_nodes", "topk_tok", "draft_lse"):
        assert torch.equal(ha[k], hb[k]), k


@pytest.mark.parametrize("B,K,D,w", [(1, 4, 6, 2), (7, 4, 6, 3), (50, 6, 8, 10), (200, 8, 10, 10), (1023, 16, 20, 16)])
def test_plan_ep_exact_ties(B, K, D, w):
    V = 96
    rng = np.random.default_rng(B * 5 + K)
    d = np.zeros((5, D, V), dtype=np.float32)
    d[1] = rng.integers(0, 4, size=(D, V)).astype(np.float32)
    d[2] = rng.standard_normal((D, V)).astype(np.float32)
    d[2, :, :3] = 5.0
    d[3] = (rng.standard_normal((D, V)) * 3).astype(np.float32)
    d[4] = np.round(rng.standard_normal((D, V)) * 4) / 4
    cfg = dict(name="ep-ties", R=5, V=V, D=D, B=B, K=K, T=1.0, dtype="f32", steps=1)
    rnd = make_round(cfg, 11, trace=False)
    rnd.plan_ep(torch.from_numpy(d).cuda(), w)
    h = rnd.host()
    tally = Tally("plan_ep ties B=%d K=%d D=%d w=%d" % (B, K, D, w), register=False)
    for r in range(5):
        compare_plan(h, r, plan_request_ep(d[r], 1.0, K, B, w), tally, "ties req %d" % r)
    say(tally.line())
    assert tally.exact["plan"] >= 4 and tally.flagged <= 1


def test_plan_ep_edges():
    rng = np.random.default_rng(9)
    cfg = dict(name="ep-edge", R=3, V=300, D=3, B=0, K=3, T=1.0, dtype="f32", steps=1)
    d = (rng.standard_normal((3, 3, 300)) * 2).astype(np.float32)
    rnd = make_round(cfg, 1, trace=False)
    rnd.plan_ep(torch.from_numpy(d).cuda(), 2)
    h = rnd.host()
    assert (h["n_nodes"] == 1).all() and (h["n_children"][:, 0] == 0).all()
    assert np.isinf(h["plan_margin"].numpy()).all()
    # non-finite row: root-only tree and the flag; budget above the generated set
    cfg = dict(name="ep-edge", R=3, V=300, D=3, B=200, K=3, T=1.0, dtype="f32", steps=1)
    d[1, 2, 7] = np.nan
    rnd = make_round(cfg, 1, trace=False)
    rnd.plan_ep(torch.from_numpy(d).cuda(), 2)
    h = rnd.host()
    st = h["req_status"].numpy()
    assert st[1] & tsb.REQ_NONFINITE and int(h["n_nodes"][1]) == 1
    tally = Tally("plan_ep edges", register=False)
    for r in (0, 2):
        pl = plan_request_ep(d[r], 1.0, 3, 200, 2)
        assert pl["tree"]["n_nodes"] == 1 + 3 + 2 * 3 + 2 * 3
        assert st[r] & tsb.REQ_BUDGET_SHORT
        compare_plan(h, r, pl, tally, "edge req %d" % r)
    assert tally.exact["plan"] == 2


def test_round_on_expand_then_prune_tree():
    """plan_ep -> replay -> verify: the plan against the expand-then-prune oracle, then replay and verification
    on the HIP path's tree against the oracle, stage by stage."""
    import oracle_worker
    cfg = W.config(2, R=2, V=32000, D=8, B=48, K=6, name="ep-round")
    seed = 77
    rnd = make_round(cfg, seed)
    tally = Tally("plan_ep full rounds")
    for s in range(6):
        base, sigma = W.base_rows(cfg, s)
        draft = W.draft_from_base(cfg, base)
        d_host = to_np(draft)
        rnd.plan_ep(draft.cuda(), 10)
        h = rnd.host()
        dep = h["depth"].long().clamp(min=0)
        target = W.target_from_base(cfg, base, sigma, dep, set_idx=s)
        rnd.replay(draft.cuda(), s)
        rnd.verify(draft.cuda(), target.cuda(), s)
        h = rnd.host()
        t_host = to_np(target)
        for r in range(2):
            where = "round step %d req %d" % (s, r)
            n = int(h["n_nodes"][r])
            res = oracle_worker.request_step(d_host[r], t_host[r], cfg["T"], cfg["K"], cfg["B"], seed, s, r,
                                             tree_dict_np(h, r), h["node_tok"][r, :n].numpy().astype(np.int64))
            res["plan"] = plan_request_ep(d_host[r], cfg["T"], cfg["K"], cfg["B"], 10)
            compare_request(h, r, res, tally, cfg["D"], where)
    say(tally.line())
    assert tally.exact["verify"] + tally.flagged_by["verify"] == 12 and tally.flagged <= 1
