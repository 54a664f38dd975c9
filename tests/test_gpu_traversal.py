"""GPU parity of traversal verification (Appendix A; Table 2) against the CPU
oracle (oracle/traversal.py), through the C ABI.

Stage by stage on the same seeded bytes, every request of every round run:
the plan and the replay as in the RRS parity tests, then the traversal on
the HIP path's tree and tokens, test by test (tested node and uniform
exact; alpha and the residual mass T to 1e-5 relative; the first differing
decision excused only at its own oracle margin; path and bonus exact unless
the bonus key gap is a near-tie). tsb_step_traversal must equal the staged
calls bit for bit. Edge cases: root-only budget, chains (one candidate per
position) on a tiny vocabulary, masked tokens, non-finite rows, and a
workspace left with garbage by other entry points.
"""
import numpy as np
import pytest
import torch

import oracle_worker
import workloads as W
import paper_2609_33652_amd as tsb
from oracle.rowstats import STATUS_NONFINITE
from parity_util import check_tally, compare_request_traversal, make_round, run_rounds, tree_dict_np
from tally import Tally

pytestmark = pytest.mark.gpu

KEYS = ("draft_lse", "topk_tok", "topk_lp", "parent", "depth", "rank", "n_children", "first_child", "score",
        "n_nodes", "node_tok", "n_acc", "acc_node", "acc_tok", "bonus", "req_status", "target_lse", "trace")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tsb.load()


def _same(a, b):
    return torch.equal(a, b) or (a.dtype.is_floating_point and torch.equal(a.nan_to_num(7.0), b.nan_to_num(7.0)))


def run_traversal(pool, cfg, seed, steps, step0=0, sets=4, gen_device="cpu", check_step=True, name=""):
    rnd2 = make_round(cfg, seed) if check_step else None

    def gpu_round(rnd, draft_g, target_g, s):
        rnd.replay(draft_g, s)
        rnd.verify_traversal(draft_g, target_g, s)

    def check(h, draft_g, target_g, s):
        rnd2.step_traversal(draft_g, target_g, s)
        h2 = rnd2.host()
        for k in KEYS:
            assert _same(h[k], h2[k]), (name, s, k)

    return run_rounds(pool, cfg, seed, steps, "traversal", gpu_round, step0=step0, sets=sets,
                      gen_device=gen_device, name=name, check=check if check_step else None)


def test_traversal_tiny_all_steps(opool):
    cfg = W.config(1)
    check_tally(run_traversal(opool, cfg, W.replay_seed(1), steps=cfg["steps"], name="tiny"), cfg["steps"], 1)


def test_traversal_small_200_steps(opool):
    cfg = W.config(2)
    check_tally(run_traversal(opool, cfg, W.replay_seed(2), steps=200, name="small"), 200, 1)


def test_traversal_qwen_vocab_60_steps(opool):
    cfg = W.config(3)
    check_tally(run_traversal(opool, cfg, W.replay_seed(3), steps=60, name="qwen_vocab"), 60, 1)


def test_traversal_batched_every_request_8_steps(opool):
    cfg = W.config(4)
    check_tally(run_traversal(opool, cfg, W.replay_seed(4), steps=8, gen_device="cuda", name="batched"), 8, 16)


def test_traversal_large_budget_every_request_2_steps(opool):
    cfg = W.config(5)
    check_tally(run_traversal(opool, cfg, W.replay_seed(5), steps=2, sets=2, gen_device="cuda", check_step=False,
                              name="large_budget"), 2, 64)


def test_traversal_ragged_scalar_path(opool):
    # V not a multiple of 4 (scalar loads), T != 1
    cfg = W.config(2, R=3, V=9001, D=5, B=20, K=6, T=1.3, name="ragged")
    check_tally(run_traversal(opool, cfg, 12345, steps=30, name="ragged"), 30, 3)


def test_traversal_slices_beyond_the_lds_cache(opool):
    # V = 300001 with two requests: slices longer than the LDS cache (recomputed chunk by chunk)
    cfg = W.config(2, R=2, V=300001, D=4, B=24, K=6, T=1.0, name="wide")
    check_tally(run_traversal(opool, cfg, 31337, steps=6, name="wide"), 6, 2)


def _edge(cfg, d, t, seed=5, step=0):
    rnd = make_round(cfg, seed)
    draft = torch.from_numpy(d).cuda()
    target = torch.from_numpy(t).cuda()
    rnd.step_traversal(draft, target, step)
    h = rnd.host()
    tally = Tally("traversal edge %s step %d" % (W.describe(cfg), step), register=False)
    for r in range(cfg["R"]):
        res = oracle_worker.request_step_traversal(d[r], t[r], cfg["T"], cfg["K"], cfg["B"], seed, step, r,
                                                   tree_dict_np(h, r),
                                                   h["node_tok"][r, :int(h["n_nodes"][r])].numpy().astype(np.int64))
        if res["plan"]["status"] & STATUS_NONFINITE:
            assert int(h["req_status"][r]) & tsb.REQ_NONFINITE and int(h["n_acc"][r]) == -1
            continue
        compare_request_traversal(h, r, res, tally, cfg["D"], "edge req %d" % r)
    assert tally.flagged <= 1, tally.notes
    return h, tally


def _edge_cfg(**kw):
    c = dict(name="edge", R=3, V=600, D=3, B=6, K=3, T=1.0, dtype="f32", steps=1)
    c.update(kw)
    return c


def test_traversal_edge_root_only_budget():
    cfg = _edge_cfg(B=0)
    rng = np.random.default_rng(21)
    d = (rng.standard_normal((3, 3, 600)) * 2).astype(np.float32)
    t = (rng.standard_normal((3, 1, 600)) * 2).astype(np.float32)
    h, tally = _edge(cfg, d, t)
    assert (h["n_nodes"] == 1).all() and (h["n_acc"] == 0).all() and tally.exact["verify"] == 3


def test_traversal_edge_chains_and_minimal_vocabulary():
    # K = 1: every tree is a chain (Block Verification); V = 4
    cfg = _edge_cfg(R=2, V=4, D=4, B=4, K=1)
    rng = np.random.default_rng(22)
    d = rng.standard_normal((2, 4, 4)).astype(np.float32)
    t = rng.standard_normal((2, 5, 4)).astype(np.float32)
    for s in range(30):
        h, tally = _edge(cfg, d, t, step=s)
        assert tally.exact["verify"] == 2


def test_traversal_edge_masked_tokens_and_budget_short():
    cfg = _edge_cfg(D=2, K=2, B=10)
    rng = np.random.default_rng(23)
    d = (rng.standard_normal((3, 2, 600)) * 2).astype(np.float32)
    d[1, 1, 1:] = -np.inf  # request 1, position 1: a single finite token
    t = (rng.standard_normal((3, 11, 600)) * 2).astype(np.float32)
    t[2, :, 5:300] = -np.inf
    for s in range(6):
        h, tally = _edge(cfg, d, t, step=s)
        assert int(h["req_status"][0]) & tsb.REQ_BUDGET_SHORT
        assert tally.exact["verify"] + tally.flagged_by["verify"] == 3


def test_traversal_edge_nonfinite_rows_flag_only_their_request():
    cfg = _edge_cfg(B=6)
    rng = np.random.default_rng(24)
    d = (rng.standard_normal((3, 3, 600)) * 2).astype(np.float32)
    t = (rng.standard_normal((3, 7, 600)) * 2).astype(np.float32)
    d[0, 2, 17] = np.nan
    t[2, 3, 5] = np.inf
    h, tally = _edge(cfg, d, t)
    st = h["req_status"].numpy()
    assert st[0] & tsb.REQ_NONFINITE and int(h["n_acc"][0]) == -1
    assert not st[1] & tsb.REQ_NONFINITE and int(h["n_acc"][1]) >= 0
    assert st[2] & tsb.REQ_NONFINITE and int(h["n_acc"][2]) == -1


def test_traversal_after_other_walks_on_one_workspace():
    cfg = W.config(2, R=3, V=12000, D=5, B=20, K=4, name="shared")
    base, sigma = W.base_rows(cfg, 0)
    draft = W.draft_from_base(cfg, base).cuda()
    target = W.target_from_base(cfg, base, sigma, torch.ones(3, 21, dtype=torch.int64)).cuda()
    shared = make_round(cfg, 9)
    shared.ws.fill_(0x3C)
    for s, kind in enumerate(["step", "step_traversal", "step_first", "step_traversal", "step_traversal"]):
        fresh = make_round(cfg, 9)
        fresh.ws.zero_()
        getattr(shared, kind)(draft, target, s)
        getattr(fresh, kind)(draft, target, s)
        a, b = shared.host(), fresh.host()
        for k in ("n_acc", "acc_node", "acc_tok", "bonus", "req_status", "node_tok"):
            assert _same(a[k], b[k]), (kind, s, k)
