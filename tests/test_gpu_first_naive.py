"""GPU parity of the First + Naive baseline (Section 3.1; Table 2, Naive)
against the CPU oracle, through the C ABI.

Stage by stage on the same seeded bytes: the plan (as in the main parity
tests), the First node tokens (bit-exact), then target-sample matching on
that tree (accepted path and bonus bit-exact, except a draw whose oracle
margin is below the near-tie threshold, which is reported). tsb_step_first
must equal the staged calls bit for bit. Full-size workloads check sampled
requests. Edge cases: root-only budget, a non-finite row that is visited
(flags the request) or never visited (does not), masked tokens, a minimal
vocabulary, a non-finite draft (plan flag carried through), and matching on
replayed tokens.
"""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import naive as onaive, replay as oreplay, step as ostep
from oracle.rowstats import STATUS_NONFINITE, inv_temperature, scaled
import paper_2609_33652_amd as tsb
from parity_util import NEAR_TIE, Tally, compare_plan, make_round, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tsb.load()


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def compare_naive(h, r, vr, tally, D, where=""):
    n_acc = int(h["n_acc"][r])
    got = (n_acc, [int(x) for x in h["acc_node"][r, :max(n_acc, 0)]], [int(x) for x in h["acc_tok"][r, :max(n_acc, 0)]],
           int(h["bonus"][r]))
    exp = (vr["n_acc"], [int(x) for x in vr["acc_node"]], [int(x) for x in vr["acc_tok"]], int(vr["bonus"]))
    if got == exp:
        assert [int(x) for x in h["acc_node"][r, max(n_acc, 0):]] == [-1] * (D - max(n_acc, 0)), where
        if vr["n_acc"] < 0:
            assert int(h["req_status"][r]) & tsb.REQ_NONFINITE, where
        else:
            assert not int(h["req_status"][r]) & (tsb.REQ_NONFINITE | tsb.REQ_WALK_TIMEOUT), where
        tally.exact += 1
        return True
    if any(0 < m < NEAR_TIE for _, m in vr["margins"]):
        tally.flag("naive near-tie " + where)
        return False
    raise AssertionError("naive verification differs %s: gpu %s oracle %s" % (where, got, exp))


def _depths(pls, h, R, B):
    dep = torch.zeros(R, B + 1, dtype=torch.int64)
    for r in range(R):
        if pls[r] is not None:
            t = pls[r]["tree"]
            dep[r, : t["n_nodes"]] = torch.from_numpy(t["depth"])
        else:
            n = int(h["n_nodes"][r])
            dep[r, :n] = h["depth"][r, :n].long()
    return dep


def run_first(cfg, seed, steps, sets=4, requests=None, gen_device="cpu", check_step=True, name=""):
    R, D, B, K, T = cfg["R"], cfg["D"], cfg["B"], cfg["K"], cfg["T"]
    requests = list(range(R)) if requests is None else list(requests)
    rnd = make_round(cfg, seed, trace=False)
    rnd2 = make_round(cfg, seed, trace=False) if check_step else None
    tally, ptally = Tally(), Tally()
    for s in range(steps):
        say("first+naive %s step %d (%s)" % (name, s, W.describe(cfg)))
        base, sigma = W.base_rows(cfg, set_idx=s % sets, device=gen_device)
        draft = W.draft_from_base(cfg, base)
        d_host = to_np(draft[requests].cpu())
        pls = [None] * R
        for i, r in enumerate(requests):
            pls[r] = ostep.plan_request(d_host[i], T, K, B)
        draft_g = draft.cuda().contiguous()
        rnd.plan(draft_g)
        rnd.first_tokens()
        h = rnd.host()
        target = W.target_from_base(cfg, base, sigma, _depths(pls, h, R, B).to(base.device), set_idx=s % sets)
        t_host = to_np(target[requests].cpu())
        target_g = target.cuda().contiguous()
        ok = {}
        for i, r in enumerate(requests):
            where = "%s step %d req %d" % (name, s, r)
            ok[r] = compare_plan(h, r, pls[r], ptally, where)
            if ok[r]:
                n = pls[r]["tree"]["n_nodes"]
                o_tok = onaive.first_tokens(pls[r]["tree"], pls[r]["topk_tok"])
                assert np.array_equal(h["node_tok"][r, :n].numpy().astype(np.int64), o_tok), where
                assert (h["node_tok"][r, n:] == -1).all(), where
        rnd.verify_naive(target_g, s)
        h = rnd.host()
        for i, r in enumerate(requests):
            if not ok[r]:
                continue
            tree = pls[r]["tree"]
            vr = onaive.verify_naive(t_host[i], tree, onaive.first_tokens(tree, pls[r]["topk_tok"]), T, seed, s, r)
            compare_naive(h, r, vr, tally, D, "%s step %d req %d" % (name, s, r))
        if check_step:
            rnd2.step_first(draft_g, target_g, s)
            h2 = rnd2.host()
            for k in ("draft_lse", "topk_tok", "topk_lp", "parent", "depth", "rank", "n_children", "first_child",
                      "score", "n_nodes", "node_tok", "n_acc", "acc_node", "acc_tok", "bonus", "req_status"):
                assert torch.equal(h[k], h2[k]), k
    say("first+naive %s: plans exact %d flagged %d; walks exact %d flagged %d %s"
        % (name, ptally.exact, ptally.flagged, tally.exact, tally.flagged, (ptally.notes + tally.notes)[:5]))
    return tally


def test_first_naive_tiny_fp32():
    cfg = W.config(1)
    t = run_first(cfg, W.replay_seed(1), steps=24, name="tiny")
    assert t.exact >= 22 and t.flagged <= 2


def test_first_naive_ragged_scalar_path():
    cfg = W.config(2, R=3, V=9001, D=5, B=20, K=6, T=1.3, name="ragged")
    t = run_first(cfg, 12345, steps=6, name="ragged")
    assert t.exact >= 16 and t.flagged <= 2


def test_first_naive_small_bf16():
    cfg = W.config(2)
    t = run_first(cfg, W.replay_seed(2), steps=6, name="small")
    assert t.exact >= 5 and t.flagged <= 1


def test_first_naive_qwen_vocab():
    cfg = W.config(3)
    t = run_first(cfg, W.replay_seed(3), steps=3, name="qwen_vocab")
    assert t.exact >= 2 and t.flagged <= 1


def test_first_naive_batched_full_size():
    cfg = W.config(4)
    t = run_first(cfg, W.replay_seed(4), steps=1, sets=1, requests=list(range(16)), gen_device="cuda",
                  name="batched")
    assert t.exact >= 15


def test_first_naive_large_budget_sampled():
    cfg = W.config(5)
    t = run_first(cfg, W.replay_seed(5), steps=1, sets=1, requests=[0, 17, 40, 63], gen_device="cuda",
                  check_step=False, name="large_budget")
    assert t.exact >= 3


def _edge(cfg, d, t, seed=5, step=0, replayed=False):
    """One round through the C ABI, compared request by request with the oracle."""
    rnd = make_round(cfg, seed, trace=False)
    draft = torch.from_numpy(d).cuda()
    target = torch.from_numpy(t).cuda()
    rnd.plan(draft)
    if replayed:
        rnd.replay(draft, step)
    else:
        rnd.first_tokens()
    rnd.verify_naive(target, step)
    h = rnd.host()
    tally, ptally = Tally(), Tally()
    for r in range(cfg["R"]):
        pl = ostep.plan_request(d[r], cfg["T"], cfg["K"], cfg["B"])
        plan_ok = compare_plan(h, r, pl, ptally, "edge req %d" % r)
        if pl["status"] & STATUS_NONFINITE:
            assert int(h["n_acc"][r]) == -1 and int(h["bonus"][r]) == -1
            continue
        if not plan_ok:
            continue
        tree = pl["tree"]
        if replayed:
            tok, _ = oreplay.replay(scaled(d[r], inv_temperature(cfg["T"])), tree, seed, step, r)
            n = tree["n_nodes"]
            if not np.array_equal(h["node_tok"][r, :n].numpy().astype(np.int64), tok):
                tally.flag("replay differs %d" % r)
                continue
        else:
            tok = onaive.first_tokens(tree, pl["topk_tok"])
        vr = onaive.verify_naive(t[r], tree, tok, cfg["T"], seed, step, r)
        compare_naive(h, r, vr, tally, cfg["D"], "edge req %d" % r)
    return h, tally


def _edge_cfg(**kw):
    c = dict(name="edge", R=3, V=600, D=3, B=6, K=3, T=1.0, dtype="f32", steps=1)
    c.update(kw)
    return c


def test_naive_edge_root_only_budget():
    cfg = _edge_cfg(B=0)
    rng = np.random.default_rng(11)
    d = (rng.standard_normal((3, 3, 600)) * 2).astype(np.float32)
    t = (rng.standard_normal((3, 1, 600)) * 2).astype(np.float32)
    for s in range(4):
        h, tally = _edge(cfg, d, t, step=s)
        assert (h["n_nodes"] == 1).all() and (h["n_acc"] == 0).all() and tally.exact == 3


def test_naive_edge_nonfinite_visited_or_not():
    cfg = _edge_cfg(B=6, R=4)
    rng = np.random.default_rng(12)
    d = (rng.standard_normal((4, 3, 600)) * 2).astype(np.float32)
    t = (rng.standard_normal((4, 7, 600)) * 2).astype(np.float32)
    t[0, 0, 5] = np.nan          # root row: always visited -> flagged
    t[1, 6, 9] = np.inf          # last node, visited only if the walk reaches it
    t[2, 0, :] = -np.inf         # root row with no finite logit -> flagged
    d[3, 1, 3] = np.nan          # non-finite draft: root-only tree, flag carried from the plan
    h, tally = _edge(cfg, d, t)
    st = h["req_status"].numpy()
    assert st[0] & tsb.REQ_NONFINITE and int(h["n_acc"][0]) == -1 and int(h["bonus"][0]) == -1
    assert st[2] & tsb.REQ_NONFINITE and int(h["n_acc"][2]) == -1
    assert st[3] & tsb.REQ_NONFINITE and int(h["n_acc"][3]) == -1
    assert tally.exact == 3


def test_naive_edge_masked_tokens_and_minimal_vocabulary():
    cfg = _edge_cfg(R=2, V=4, D=4, B=4, K=1)
    rng = np.random.default_rng(13)
    d = rng.standard_normal((2, 4, 4)).astype(np.float32)
    t = rng.standard_normal((2, 5, 4)).astype(np.float32)
    t[1, :, 2] = -np.inf
    for s in range(20):
        h, tally = _edge(cfg, d, t, step=s)
        assert tally.exact == 2
        assert int(h["bonus"][1]) != 2


def test_naive_on_replayed_tokens():
    cfg = _edge_cfg(R=3, V=3000, D=4, B=12, K=4)
    rng = np.random.default_rng(14)
    d = (rng.standard_normal((3, 4, 3000)) * 3).astype(np.float32)
    t = np.repeat(d[:, :1], 13, axis=1).copy()
    t += rng.standard_normal(t.shape).astype(np.float32) * 0.3
    for s in range(6):
        h, tally = _edge(cfg, d, t, step=s, replayed=True)
        assert tally.exact + tally.flagged == 3


def test_naive_deterministic_repeat():
    cfg = W.config(2, R=4, V=20000, D=8, B=30, K=5, name="repeat")
    base, sigma = W.base_rows(cfg, 0)
    draft = W.draft_from_base(cfg, base).cuda()
    target = W.target_from_base(cfg, base, sigma, torch.ones(4, 31, dtype=torch.int64)).cuda()
    outs = []
    for _ in range(2):
        rnd = make_round(cfg, 7, trace=False)
        rnd.step_first(draft, target, 3)
        outs.append(rnd.host())
    for k in ("node_tok", "n_acc", "acc_tok", "bonus", "req_status"):
        assert torch.equal(outs[0][k], outs[1][k]), k


def test_exchange_state_across_calls():
    """Verification keeps exchange state in the workspace between calls: alternating RRS and naive
    rounds on one workspace must give the same results as a fresh workspace for every call."""
    cfg = W.config(2, R=4, V=20000, D=6, B=24, K=4, name="xstate")
    base, sigma = W.base_rows(cfg, 0)
    draft = W.draft_from_base(cfg, base).cuda()
    target = W.target_from_base(cfg, base, sigma, torch.ones(4, 25, dtype=torch.int64)).cuda()
    reused = make_round(cfg, 21, trace=False)
    for i in range(12):
        fresh = make_round(cfg, 21, trace=False)
        kind = "step" if i % 3 != 2 else "step_first"
        getattr(reused, kind)(draft, target, i)
        getattr(fresh, kind)(draft, target, i)
        a, b = reused.host(), fresh.host()
        for k in ("node_tok", "n_acc", "acc_node", "acc_tok", "bonus", "req_status"):
            assert torch.equal(a[k], b[k]), (i, kind, k)


def test_exchange_state_many_calls_full_size():
    """Hundreds of rounds on one workspace (mixed exchange widths in the walk) against a workspace
    zero-filled before every call: identical results and no abandoned wait. A stale slot word
    accepted as current makes the workgroups of a request diverge, which shows up here."""
    cfg = W.config(4)
    base, sigma = W.base_rows(cfg, 0, device="cuda")
    draft = W.draft_from_base(cfg, base)
    a = make_round(cfg, W.replay_seed(4), trace=False)
    b = make_round(cfg, W.replay_seed(4), trace=False)
    a.plan(draft)
    target = W.target_from_base(cfg, base, sigma, a.tree["depth"].long().clamp(min=0))
    del base
    flags = 0
    for s in range(240):
        kind = "step" if s % 5 else "step_first"
        getattr(a, kind)(draft, target, s)
        b.ws.zero_()
        getattr(b, kind)(draft, target, s)
        if s % 40 == 39:
            say("exchange state: %d calls" % (s + 1))
        flags |= int((a.req_status & tsb.REQ_WALK_TIMEOUT).any())
        for k in ("n_acc", "acc_tok", "bonus", "req_status"):
            assert torch.equal(getattr(a, k), getattr(b, k)), (s, kind, k)
    assert flags == 0
