"""GPU parity of the round over sparse candidate pools with context-dependent
q_u (Section 3.1 pools and transition-score lookups; Section 3.2, eq. (2);
Section 3.3) against the CPU oracle, through the C ABI.

Stage by stage on the same seeded bytes, every request of every round run:
pools (bit-exact), the first pass over per-node candidate lists (topology,
scores, plan margin and planning tokens bit-exact unless the oracle's plan
margin is a near-tie), the replay on the HIP path's topology (parent by
parent), and the walk on its topology and tokens (test by test: uniforms
exact, ratios and residual masses to 1e-5 relative; the first differing
decision excused only at its own near-tie; see tests/parity_util.py).
tsb_pool_step must equal the staged calls bit for bit. Workloads: the tiny
and small workloads with pools of 4, 13 and 16 tokens, the Qwen-vocabulary
workload with 64, the batched workload at full size with 16 and 64, and the
large-budget workload (whose candidate lists exceed the planner's LDS).
Edge cases: root-only budget, non-finite transition score or draft row,
pools holding -inf logits, a pool as wide as the vocabulary, a node token
outside its pool, and a workspace shared with the vocabulary-wide walk.
"""
import sys

import numpy as np
import pytest
import torch

import oracle_worker
import workloads as W
from oracle.rowstats import STATUS_NONFINITE
import paper_2609_33652_amd as tsb
from parity_util import check_tally, compare_request_pool, run_rounds, tree_dict_np
from tally import Tally

pytestmark = pytest.mark.gpu

KEYS = ("pool_tok", "parent", "depth", "rank", "n_children", "first_child", "score", "n_nodes", "node_tok", "n_acc",
        "acc_node", "acc_tok", "bonus", "req_status", "target_lse", "trace")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tsb.load()


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def pool_round(cfg, seed, P, trace=True):
    c = tsb.make_config(cfg["R"], cfg["D"], cfg["V"], cfg["B"], cfg["K"], cfg["T"], cfg["dtype"], seed)
    return tsb.Round(c, "cuda", target_lse=True, trace=trace, pool=P)


def run_pool(opool, cfg, P, seed, steps, step0=0, sets=4, gen_device="cpu", check_step=True, name=""):
    rnd2 = pool_round(cfg, seed, P) if check_step else None

    def gpu_round(rnd, draft_g, target_g, s, trans_g):
        rnd.pool_replay(draft_g, trans_g, s)
        rnd.pool_verify(draft_g, trans_g, target_g, s)

    def check(h, draft_g, target_g, s, trans_g):
        rnd2.pool_step(draft_g, trans_g, target_g, s)
        h2 = rnd2.host()
        for k in KEYS:
            assert torch.equal(h[k].nan_to_num(7.0), h2[k].nan_to_num(7.0)) if h[k].dtype.is_floating_point \
                else torch.equal(h[k], h2[k]), (name, s, k)

    return run_rounds(opool, cfg, seed, steps, "pool", gpu_round, step0=step0, sets=sets, gen_device=gen_device,
                      name=name, check=check if check_step else None, P=P)


@pytest.mark.parametrize("P", [4, 16])
def test_pool_tiny_fp32(opool, P):
    cfg = W.config(1)
    check_tally(run_pool(opool, cfg, P, W.replay_seed(1), steps=100, name="tiny"), 100, 1)


def test_pool_ragged_scalar_path(opool):
    cfg = W.config(2, R=3, V=9001, D=5, B=20, K=6, T=1.3, name="ragged")
    check_tally(run_pool(opool, cfg, 13, 12345, steps=20, name="ragged"), 20, 3)


def test_pool_small_bf16(opool):
    cfg = W.config(2)
    check_tally(run_pool(opool, cfg, 16, W.replay_seed(2), steps=100, name="small"), 100, 1)


def test_pool_qwen_vocab_p64(opool):
    cfg = W.config(3)
    check_tally(run_pool(opool, cfg, 64, W.replay_seed(3), steps=50, name="qwen_vocab"), 50, 1)


@pytest.mark.parametrize("P", [16, 64])
def test_pool_batched_every_request(opool, P):
    cfg = W.config(4)
    check_tally(run_pool(opool, cfg, P, W.replay_seed(4), steps=4, gen_device="cuda", name="batched"), 4, 16)


def test_pool_full_budget_many_internal_nodes(opool):
    # B = 1023 with K = 2: a 1024-node tree with several hundred internal
    # nodes, beyond those whose Gumbel draws the replay computes ahead
    cfg = W.config(2, R=2, V=4096, D=12, B=1023, K=2, T=1.0, name="deep")
    t = run_pool(opool, cfg, 8, 4242, steps=4, name="deep")
    check_tally(t, 4, 2)
    assert t.exact["replay"] + t.flagged_by["replay"] > 400


def test_pool_large_budget_every_request(opool):
    cfg = W.config(5)
    check_tally(run_pool(opool, cfg, 64, W.replay_seed(5), steps=2, sets=2, gen_device="cuda", check_step=False,
                         name="large_budget"), 2, 64)


# ------------------------------------------------------------------ edges
def _edge_cfg(**kw):
    c = dict(name="edge", R=3, V=600, D=3, B=6, K=3, T=1.0, dtype="f32", steps=1)
    c.update(kw)
    return c


def _edge(cfg, P, d, tr, t, seed=5, step=0):
    rnd = pool_round(cfg, seed, P)
    draft, trans, target = (torch.from_numpy(x).cuda() for x in (d, tr, t))
    rnd.pool_plan(draft, trans)
    rnd.pool_replay(draft, trans, step)
    rnd.pool_verify(draft, trans, target, step)
    h = rnd.host()
    tally = Tally("pool edge %s P=%d" % (W.describe(cfg), P), register=False)
    outs = []
    for r in range(cfg["R"]):
        n = int(h["n_nodes"][r])
        o = oracle_worker.request_step_pool(d[r], t[r], cfg["T"], cfg["K"], cfg["B"], seed, step, r,
                                            tree_dict_np(h, r), h["node_tok"][r, :n].numpy().astype(np.int64),
                                            tr[r], P)
        outs.append(o)
        compare_request_pool(h, r, o, tally, cfg["D"], "edge req %d" % r)
    assert tally.flagged <= 1, tally.notes
    return h, tally, outs


def _edge_inputs(cfg, P, rng):
    R, D, V, B = cfg["R"], cfg["D"], cfg["V"], cfg["B"]
    d = (rng.standard_normal((R, D, V)) * 2).astype(np.float32)
    tr = (rng.standard_normal((R, max(D - 1, 0), P, P)) * 1.5).astype(np.float32)
    t = (rng.standard_normal((R, B + 1, V)) * 2).astype(np.float32)
    return d, tr, t


def test_pool_edge_root_only_budget():
    cfg = _edge_cfg(B=0)
    d, tr, t = _edge_inputs(cfg, 8, np.random.default_rng(1))
    h, tally, _ = _edge(cfg, 8, d, tr, t)
    assert (h["n_nodes"] == 1).all() and (h["n_acc"] == 0).all() and tally.exact["verify"] == 3


def test_pool_edge_nonfinite_transition_and_draft():
    cfg = _edge_cfg()
    d, tr, t = _edge_inputs(cfg, 8, np.random.default_rng(2))
    tr[0, 1, 3, 5] = np.nan
    tr[1, 0, 7, 0] = np.inf
    d[2, 2, 17] = np.nan
    h, _, outs = _edge(cfg, 8, d, tr, t)
    for r in range(3):
        assert outs[r]["status"] & STATUS_NONFINITE
        assert int(h["req_status"][r]) & tsb.REQ_NONFINITE and int(h["n_acc"][r]) == -1


def test_pool_edge_masked_pool_entries():
    # rows with only 5 finite logits: pools of 8 hold three -inf entries
    cfg = _edge_cfg(V=64, K=4, B=12)
    rng = np.random.default_rng(3)
    d, tr, t = _edge_inputs(cfg, 8, rng)
    mask = np.ones_like(d, dtype=bool)
    for r in range(cfg["R"]):
        for dd in range(cfg["D"]):
            mask[r, dd, rng.choice(cfg["V"], 5, replace=False)] = False
    d[mask] = -np.inf
    h, tally, outs = _edge(cfg, 8, d, tr, t)
    assert tally.exact["verify"] + tally.flagged_by["verify"] == 3
    for r in range(3):
        n = int(h["n_nodes"][r])
        assert (h["n_children"][r, :n] <= 4).all()


def test_pool_edge_pool_as_wide_as_vocabulary():
    cfg = _edge_cfg(V=48, K=4, B=10, R=2)
    d, tr, t = _edge_inputs(cfg, 48, np.random.default_rng(4))
    h, tally, _ = _edge(cfg, 48, d, tr, t)
    assert tally.exact["verify"] + tally.flagged_by["verify"] == 2


def test_pool_bad_token_is_flagged():
    cfg = _edge_cfg(R=1, V=300, K=3, B=6)
    d, tr, t = _edge_inputs(cfg, 8, np.random.default_rng(5))
    # a target that accepts everything likely: copy the draft into the target rows
    rnd = pool_round(cfg, 9, 8)
    draft, trans, target = (torch.from_numpy(x).cuda() for x in (d, tr, t))
    rnd.pool_plan(draft, trans)
    rnd.pool_replay(draft, trans, 0)
    h = rnd.host()
    pool0 = set(h["pool_tok"][0, 0].tolist())
    outside = next(v for v in range(cfg["V"]) if v not in pool0)
    fc = int(h["first_child"][0, 0])
    rnd.node_tok[0, fc] = outside  # the root's first child now holds a token outside pool 0
    t2 = t.copy()
    t2[0, 0, :] = -30.0
    t2[0, 0, outside] = 30.0  # the target puts all its mass on it
    rnd.pool_verify(draft, trans, torch.from_numpy(t2).cuda(), 0)
    h = rnd.host()
    assert int(h["req_status"][0]) & tsb.REQ_BAD_TOKEN
    assert int(h["n_acc"][0]) >= 1 and int(h["acc_tok"][0, 0]) == outside


def test_pool_and_vocabulary_walks_share_a_workspace():
    cfg = W.config(2, R=2, V=20000, D=6, B=24, K=6, T=1.0, name="shared")
    P, seed = 16, 77
    c = tsb.make_config(cfg["R"], cfg["D"], cfg["V"], cfg["B"], cfg["K"], cfg["T"], cfg["dtype"], seed)
    rnd = tsb.Round(c, "cuda", target_lse=True, trace=False, pool=P)
    ref_pool = pool_round(cfg, seed, P, trace=False)
    ref_vocab = tsb.Round(c, "cuda", target_lse=True, trace=False)
    for s in range(12):
        base, sigma = W.base_rows(cfg, set_idx=s % 3)
        draft = W.draft_from_base(cfg, base).cuda().contiguous()
        trans = W.transitions(cfg, P, set_idx=s % 3).cuda().contiguous()
        dep = torch.zeros(cfg["R"], cfg["B"] + 1, dtype=torch.int64)
        target = W.target_from_base(cfg, base, sigma, dep, set_idx=s % 3).cuda().contiguous()
        for other, call in ((ref_pool, "pool"), (ref_vocab, "vocab")) if s % 2 else \
                ((ref_vocab, "vocab"), (ref_pool, "pool")):
            if call == "pool":
                rnd.pool_step(draft, trans, target, s)
                other.pool_step(draft, trans, target, s)
            else:
                rnd.step(draft, target, s)
                other.step(draft, target, s)
            h, ho = rnd.host(), other.host()
            for k in ("n_acc", "acc_node", "acc_tok", "bonus", "req_status"):
                assert torch.equal(h[k], ho[k]), (s, call, k)
            assert not (h["req_status"] & tsb.REQ_WALK_TIMEOUT).any()
