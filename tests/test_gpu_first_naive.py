"""GPU parity of the First + Naive baseline (Section 3.1; Table 2, Naive)
against the CPU oracle, through the C ABI.

Stage by stage on the same seeded bytes, every request of every round run:
the plan (as in the main parity tests), the First node tokens (bit-exact),
then target-sample matching on the HIP path's tree and tokens (path and
bonus bit-exact; the first differing draw is excused only at its own oracle
near-tie, see tests/parity_util.py). tsb_step_first must equal the staged
calls bit for bit. Edge cases: root-only budget, a non-finite row that is
visited (flags the request) or never visited (does not), masked tokens, a
minimal vocabulary, a non-finite draft (plan flag carried through), and
matching on replayed tokens.
"""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import naive as onaive, replay as oreplay, step as ostep
from oracle.rowstats import STATUS_NONFINITE, inv_temperature, scaled
import paper_2609_33652_amd as tsb
from parity_util import check_tally, compare_naive, compare_plan, make_round, run_rounds
from tally import Tally

pytestmark = pytest.mark.gpu

KEYS = ("draft_lse", "topk_tok", "topk_lp", "parent", "depth", "rank", "n_children", "first_child", "score",
        "n_nodes", "node_tok", "n_acc", "acc_node", "acc_tok", "bonus", "req_status")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tsb.load()


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_first(pool, cfg, seed, steps, step0=0, sets=4, gen_device="cpu", check_step=True, name=""):
    rnd2 = make_round(cfg, seed, trace=False) if check_step else None

    def gpu_round(rnd, draft_g, target_g, s):
        rnd.first_tokens()
        rnd.verify_naive(target_g, s)

    def check(h, draft_g, target_g, s):
        rnd2.step_first(draft_g, target_g, s)
        h2 = rnd2.host()
        for k in KEYS:
            assert torch.equal(h[k], h2[k]), (name, s, k)

    return run_rounds(pool, cfg, seed, steps, "naive", gpu_round, step0=step0, sets=sets, gen_device=gen_device,
                      name=name, check=check if check_step else None, trace=False)


def test_first_naive_tiny_all_steps(opool):
    cfg = W.config(1)
    check_tally(run_first(opool, cfg, W.replay_seed(1), steps=cfg["steps"], name="tiny"), cfg["steps"], 1)


def test_first_naive_ragged_scalar_path(opool):
    cfg = W.config(2, R=3, V=9001, D=5, B=20, K=6, T=1.3, name="ragged")
    check_tally(run_first(opool, cfg, 12345, steps=30, name="ragged"), 30, 3)


def test_first_naive_small_all_steps(opool):
    cfg = W.config(2)
    check_tally(run_first(opool, cfg, W.replay_seed(2), steps=cfg["steps"], name="small"), cfg["steps"], 1)


def test_first_naive_qwen_vocab_100_steps(opool):
    cfg = W.config(3)
    check_tally(run_first(opool, cfg, W.replay_seed(3), steps=100, name="qwen_vocab"), 100, 1)


def test_first_naive_batched_every_request_16_steps(opool):
    cfg = W.config(4)
    check_tally(run_first(opool, cfg, W.replay_seed(4), steps=16, gen_device="cuda", name="batched"), 16, 16)


def test_first_naive_large_budget_every_request_4_steps(opool):
    cfg = W.config(5)
    check_tally(run_first(opool, cfg, W.replay_seed(5), steps=4, sets=2, gen_device="cuda", name="large_budget"),
                4, 64)


def _edge(cfg, d, t, seed=5, step=0, replayed=False):
    """One round through the C ABI, compared request by request with the oracle (on the HIP path's tree)."""
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
    tally = Tally("naive edge %s step %d" % (W.describe(cfg), step), register=False)
    for r in range(cfg["R"]):
        pl = ostep.plan_request(d[r], cfg["T"], cfg["K"], cfg["B"])
        compare_plan(h, r, pl, tally, "edge req %d" % r)
        if pl["status"] & STATUS_NONFINITE:
            assert int(h["n_acc"][r]) == -1 and int(h["bonus"][r]) == -1
            continue
        tree = pl["tree"]
        n = tree["n_nodes"]
        if replayed:
            tok, mg = oreplay.replay(scaled(d[r], inv_temperature(cfg["T"])), tree, seed, step, r)
            g = h["node_tok"][r, :n].numpy().astype(np.int64)
            for u in range(n):
                m, fc = int(tree["n_children"][u]), int(tree["first_child"][u])
                if m and not np.array_equal(g[fc:fc + m], tok[fc:fc + m]):
                    assert 0 < mg[u] < 1e-5, ("replay differs", r, u)
        tok = h["node_tok"][r, :n].numpy().astype(np.int64)
        if not replayed:
            assert np.array_equal(tok, onaive.first_tokens(tree, pl["topk_tok"])), r
        vr = onaive.verify_naive(t[r], tree, tok, cfg["T"], seed, step, r)
        compare_naive(h, r, vr, tally, cfg["D"], "edge req %d" % r)
    assert tally.flagged <= 1, tally.notes
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
        assert (h["n_nodes"] == 1).all() and (h["n_acc"] == 0).all() and tally.exact["verify"] == 3


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
    assert tally.exact["verify"] == 3


def test_naive_edge_masked_tokens_and_minimal_vocabulary():
    cfg = _edge_cfg(R=2, V=4, D=4, B=4, K=1)
    rng = np.random.default_rng(13)
    d = rng.standard_normal((2, 4, 4)).astype(np.float32)
    t = rng.standard_normal((2, 5, 4)).astype(np.float32)
    t[1, :, 2] = -np.inf
    for s in range(20):
        h, tally = _edge(cfg, d, t, step=s)
        assert tally.exact["verify"] == 2
        assert int(h["bonus"][1]) != 2


def test_naive_on_replayed_tokens():
    cfg = _edge_cfg(R=3, V=3000, D=4, B=12, K=4)
    rng = np.random.default_rng(14)
    d = (rng.standard_normal((3, 4, 3000)) * 3).astype(np.float32)
    t = np.repeat(d[:, :1], 13, axis=1).copy()
    t += rng.standard_normal(t.shape).astype(np.float32) * 0.3
    for s in range(6):
        h, tally = _edge(cfg, d, t, step=s, replayed=True)
        assert tally.exact["verify"] + tally.flagged_by["verify"] == 3


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
    """Alternating RRS and naive rounds on one workspace (never cleared by the caller) give the same results
    as a fresh workspace for every call: nothing a walk leaves in the workspace is read by the next."""
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
    accepted as current would make the workgroups of a request diverge, which would show up here."""
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
