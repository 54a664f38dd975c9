"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Every case feeds the same seeded bytes to both sides and compares stage by
stage (plan; replay on the HIP path's topology; verification on its topology
and node tokens), decision by decision, with the rules of
tests/parity_util.py. The workloads are checked on every request of every
step run: all steps of the tiny and small workloads, 160 steps of the
Qwen-vocabulary one, 16 steps of the batched one and 4 of the large-budget
one (the oracle runs in a process pool over the host's cores). tsb_step must
equal the staged calls bit for bit, with the normaliser output requested
and without it; the other way of reading the target rows (each row as the
walk enters its node, or every row streamed first) must take the same
decisions. Each case allows at most one flagged near-tie; the tallies are
printed at the end of the run.
"""
import sys

import numpy as np
import pytest
import torch

import oracle_worker
import workloads as W
from oracle import replay as oreplay, step as ostep
from oracle.rowstats import STATUS_NONFINITE, inv_temperature, scaled
import paper_2609_33652_amd as tsb
from parity_util import (check_tally, compare_plan, compare_request, make_round, run_rounds,
                         tree_dict_np)
from tally import Tally

pytestmark = pytest.mark.gpu

STEP_KEYS = ("draft_lse", "topk_tok", "topk_lp", "parent", "depth", "rank", "n_children", "first_child", "score",
             "n_nodes", "node_tok", "n_acc", "acc_node", "acc_tok", "bonus", "req_status", "target_lse", "trace")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tsb.load()


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _same(a, b):
    return torch.equal(a, b) or (a.dtype.is_floating_point and torch.equal(a.nan_to_num(7.0), b.nan_to_num(7.0)))


def run_case(pool, cfg, seed, steps, step0=0, sets=4, gen_device="cpu", check_step=True, name=""):
    """Stage-wise parity of every request of rounds step0 .. step0 + steps - 1 (plan, replay, verify), with
    tsb_step on two more workspaces (with and without the normaliser output) compared with the staged calls
    bit for bit."""
    rnd2 = make_round(cfg, seed) if check_step else None
    rnd3 = make_round(cfg, seed, target_lse=False) if check_step else None
    other = tsb.FLAG_STREAM_ROWS if tsb.walk_reads_rows(rnd2.cfg) else tsb.FLAG_READ_ROWS
    rnd4 = make_round(cfg, seed, flags=other) if check_step else None

    def gpu_round(rnd, draft_g, target_g, s):
        rnd.replay(draft_g, s)
        rnd.verify(draft_g, target_g, s)

    def check(h, draft_g, target_g, s):
        rnd2.step(draft_g, target_g, s)
        h2 = rnd2.host()
        for k in STEP_KEYS:
            assert _same(h[k], h2[k]), (name, s, k)
        rnd3.step(draft_g, target_g, s)
        h3 = rnd3.host()
        assert h3["target_lse"] is None
        for k in STEP_KEYS:
            if k != "target_lse":
                assert _same(h[k], h3[k]), (name, s, k, "no normaliser output")
        rnd4.step(draft_g, target_g, s)
        h4 = rnd4.host()
        for k in STEP_KEYS:
            if k == "trace":
                # a test taken clear of the band with the streamed normaliser records its ratio to ~1e-6
                assert torch.allclose(h[k], h4[k], rtol=1e-5, atol=0.0, equal_nan=True), (name, s, k, other)
            else:
                assert _same(h[k], h4[k]), (name, s, k, other)

    return run_rounds(pool, cfg, seed, steps, "rrs", gpu_round, step0=step0, sets=sets, gen_device=gen_device,
                      name=name, check=check if check_step else None)


_check = check_tally


def test_tiny_all_steps(opool):
    cfg = W.config(1)
    _check(run_case(opool, cfg, W.replay_seed(1), steps=cfg["steps"], name="tiny"), cfg["steps"], 1)


def test_small_all_steps(opool):
    cfg = W.config(2)
    _check(run_case(opool, cfg, W.replay_seed(2), steps=cfg["steps"], name="small"), cfg["steps"], 1)


@pytest.mark.parametrize("step0", [0, 80])
def test_qwen_vocab_160_steps(opool, step0):
    cfg = W.config(3)
    _check(run_case(opool, cfg, W.replay_seed(3), steps=80, step0=step0, name="qwen_vocab"), 80, 1)


@pytest.mark.parametrize("step0", [0, 8])
def test_batched_every_request_16_steps(opool, step0):
    cfg = W.config(4)
    _check(run_case(opool, cfg, W.replay_seed(4), steps=8, step0=step0, gen_device="cuda", name="batched"), 8, 16)


@pytest.mark.parametrize("step0", [0, 2])
def test_large_budget_every_request_4_steps(opool, step0):
    cfg = W.config(5)
    _check(run_case(opool, cfg, W.replay_seed(5), steps=2, step0=step0, sets=2, gen_device="cuda",
                    name="large_budget"), 2, 64)


def test_ragged_multi_tile_scalar_path(opool):
    # V not a multiple of 8 or 4 (scalar loads), 3 replay tiles with a ragged tail, T != 1
    cfg = W.config(2, R=3, V=9001, D=5, B=20, K=6, T=1.3, name="ragged")
    _check(run_case(opool, cfg, 12345, steps=40, name="ragged"), 40, 3)


def test_vocab_beyond_64_replay_tiles(opool):
    # V = 300001: 74 replay tiles of 4096 (more than one per lane in the merge,
    # which then inserts key by key) with a ragged last tile, scalar loads
    cfg = W.config(2, R=2, V=300001, D=4, B=24, K=6, T=1.0, name="wide")
    _check(run_case(opool, cfg, 31337, steps=8, name="wide"), 8, 2)


def test_pruning_does_not_change_replay():
    cfg = W.config(2, R=2, V=32000, D=6, B=40, K=8, name="prune")
    seed = 99
    base, sigma = W.base_rows(cfg, 0)
    draft = W.draft_from_base(cfg, base).cuda()
    a = make_round(cfg, seed, 0)
    b = make_round(cfg, seed, tsb.FLAG_NO_PRUNE)
    for s in range(4):
        a.plan(draft)
        a.replay(draft, s)
        b.plan(draft)
        b.replay(draft, s)
        assert torch.equal(a.node_tok, b.node_tok)


def test_deterministic_repeat():
    cfg = W.config(2, R=4, V=20000, D=8, B=30, K=5, name="repeat")
    base, sigma = W.base_rows(cfg, 0)
    draft = W.draft_from_base(cfg, base).cuda()
    target = W.target_from_base(cfg, base, sigma, torch.ones(4, 31, dtype=torch.int64)).cuda()
    outs = []
    for _ in range(2):
        rnd = make_round(cfg, 7)
        rnd.step(draft, target, 3)
        outs.append(rnd.host())
    for k in ("topk_tok", "node_tok", "n_acc", "acc_tok", "bonus", "trace"):
        assert torch.equal(outs[0][k], outs[1][k]), k


def _edge_cfg(**kw):
    c = dict(name="edge", R=3, V=600, D=3, B=6, K=3, T=1.0, dtype="f32", steps=1)
    c.update(kw)
    return c


def _run_edge(cfg, draft_np, target_np, seed=5, step=0, name="edge", flags=0):
    rnd = make_round(cfg, seed, flags=flags)
    draft = torch.from_numpy(draft_np).cuda()
    target = torch.from_numpy(target_np).cuda()
    rnd.step(draft, target, step)
    h = rnd.host()
    tally = Tally("%s %s step %d" % (name, W.describe(cfg), step), register=False)
    for r in range(cfg["R"]):
        res = oracle_worker.request_step(draft_np[r], target_np[r], cfg["T"], cfg["K"], cfg["B"], seed, step, r,
                                         tree_dict_np(h, r),
                                         h["node_tok"][r, :int(h["n_nodes"][r])].numpy().astype(np.int64))
        if res["plan"]["status"] & STATUS_NONFINITE:
            assert int(h["req_status"][r]) & tsb.REQ_NONFINITE and int(h["n_acc"][r]) == -1
            assert int(h["bonus"][r]) == -1
            tally.ok("plan")
            continue
        compare_request(h, r, res, tally, cfg["D"], "%s req %d" % (name, r))
    assert tally.flagged <= 1, tally.notes
    return h, tally


@pytest.mark.parametrize("flags", [0, tsb.FLAG_READ_ROWS])
def test_edge_root_only_budget(flags):
    cfg = _edge_cfg(B=0)
    rng = np.random.default_rng(1)
    d = (rng.standard_normal((3, 3, 600)) * 2).astype(np.float32)
    t = (rng.standard_normal((3, 1, 600)) * 2).astype(np.float32)
    h, tally = _run_edge(cfg, d, t, flags=flags)
    assert (h["n_nodes"] == 1).all() and (h["n_acc"] == 0).all()


def test_edge_budget_short_and_masked_tokens():
    cfg = _edge_cfg(D=2, K=2, B=10)
    rng = np.random.default_rng(2)
    d = (rng.standard_normal((3, 2, 600)) * 2).astype(np.float32)
    d[1, 1, 1:] = -np.inf  # request 1, position 1: a single finite token
    t = (rng.standard_normal((3, 11, 600)) * 2).astype(np.float32)
    h, tally = _run_edge(cfg, d, t)
    assert int(h["n_nodes"][0]) == 7 and int(h["req_status"][0]) & tsb.REQ_BUDGET_SHORT
    assert tally.exact["plan"] >= 2 and tally.exact["verify"] >= 2


@pytest.mark.parametrize("flags", [0, tsb.FLAG_READ_ROWS])
def test_edge_nonfinite_rows_flag_only_their_request(flags):
    cfg = _edge_cfg(B=6)
    rng = np.random.default_rng(3)
    d = (rng.standard_normal((3, 3, 600)) * 2).astype(np.float32)
    t = (rng.standard_normal((3, 7, 600)) * 2).astype(np.float32)
    d[0, 2, 17] = np.nan
    t[2, 0, 5] = np.inf
    h, tally = _run_edge(cfg, d, t, flags=flags)
    st = h["req_status"].numpy()
    assert st[0] & tsb.REQ_NONFINITE and int(h["n_nodes"][0]) == 1 and int(h["n_acc"][0]) == -1
    assert not st[1] & tsb.REQ_NONFINITE and int(h["n_acc"][1]) >= 0
    assert st[2] & tsb.REQ_NONFINITE and int(h["n_acc"][2]) == -1


@pytest.mark.parametrize("flags", [0, tsb.FLAG_READ_ROWS])
def test_edge_nonfinite_rows_off_the_walk(flags):
    """A NaN or +inf in a target row counts only when the walk enters its node: the rows of the last tree
    node (never entered at this acceptance level) get one, the requests keep their results, and the
    normaliser output marks just that row; in the root row it ends the request."""
    cfg = _edge_cfg(R=4, B=6)
    rng = np.random.default_rng(31)
    d = (rng.standard_normal((4, 3, 600)) * 2).astype(np.float32)
    t = (rng.standard_normal((4, 7, 600)) * 2).astype(np.float32)
    ref, _ = _run_edge(cfg, d, t, name="edge clean", flags=flags)
    t2 = t.copy()
    for r in range(3):
        entered = {0} | {int(x) for x in ref["acc_node"][r, :max(0, int(ref["n_acc"][r]))]}
        spare = [u for u in range(int(ref["n_nodes"][r])) if u not in entered]
        t2[r, spare[-1], 11 + r] = np.nan if r % 2 else np.inf
    t2[3, 0, 7] = np.nan
    h, tally = _run_edge(cfg, d, t2, name="edge off-walk rows", flags=flags)
    for r in range(3):
        assert not int(h["req_status"][r]) & tsb.REQ_NONFINITE
        for k in ("n_acc", "acc_node", "acc_tok", "bonus"):
            assert torch.equal(h[k][r], ref[k][r]), (r, k)
        assert int(torch.isnan(h["target_lse"][r, :int(h["n_nodes"][r])]).sum()) == 1
    assert int(h["req_status"][3]) & tsb.REQ_NONFINITE and int(h["n_acc"][3]) == -1
    rnd = make_round(cfg, 5, flags=flags, target_lse=False)
    rnd.step(torch.from_numpy(d).cuda(), torch.from_numpy(t2).cuda(), 0)
    h3 = rnd.host()
    for k in ("n_acc", "acc_node", "acc_tok", "bonus", "req_status", "trace"):
        assert _same(h[k], h3[k]), k


@pytest.mark.parametrize("flags", [0, tsb.FLAG_READ_ROWS])
def test_edge_chain_and_minimal_vocabulary(flags):
    cfg = _edge_cfg(R=2, V=4, D=4, B=4, K=1)
    rng = np.random.default_rng(4)
    d = rng.standard_normal((2, 4, 4)).astype(np.float32)
    t = rng.standard_normal((2, 5, 4)).astype(np.float32)
    for s in range(20):
        h, tally = _run_edge(cfg, d, t, step=s, flags=flags)
        assert tally.exact["verify"] == 2


def _plan_only(cfg, draft_np):
    rnd = make_round(cfg, 11)
    rnd.plan(torch.from_numpy(draft_np).cuda())
    h = rnd.host()
    tally = Tally("plan-only %s" % W.describe(cfg), register=False)
    for r in range(cfg["R"]):
        pl = ostep.plan_request(draft_np[r], cfg["T"], cfg["K"], cfg["B"])
        compare_plan(h, r, pl, tally, "plan req %d" % r)  # raises on a mismatch that is not a near-tie
    say(tally.line())
    assert tally.flagged <= 1, tally.notes
    return h, tally


@pytest.mark.parametrize("B,K,D", [(1, 4, 6), (7, 4, 6), (50, 6, 8), (200, 8, 10), (1023, 32, 64)])
def test_planner_exact_ties(B, K, D):
    """Exact score ties (identical logits, few distinct values) at small and maximal budgets: the
    topology is decided by depth and rank path, so it must match bit for bit."""
    V = 96
    rng = np.random.default_rng(B * 7 + K)
    d = np.zeros((5, D, V), dtype=np.float32)
    d[0] = 0.0                                                   # every candidate ties
    d[1] = rng.integers(0, 4, size=(D, V)).astype(np.float32)    # four distinct values
    d[2] = rng.standard_normal((D, V)).astype(np.float32)
    d[2, :, :3] = 5.0                                            # three tied peaks per row
    d[3] = (rng.standard_normal((D, V)) * 3).astype(np.float32)  # no designed ties
    d[4] = np.round(rng.standard_normal((D, V)) * 4) / 4         # quarter steps
    cfg = dict(name="ties", R=5, V=V, D=D, B=B, K=K, T=1.0, dtype="f32", steps=1)
    h, tally = _plan_only(cfg, d)
    assert tally.exact["plan"] >= 4
    nmax = sum(K ** i for i in range(1, D + 1))
    assert (h["n_nodes"] == min(B, nmax) + 1).all()


def _special_rows(rng, R, D, V):
    """bf16-exact draft rows [R, D, V] with values outside the exponential table planted: exact zeros,
    values below its smallest binade (+-2^-20 and bf16 subnormals), values at or beyond 64 (some the
    row maximum), masked -inf entries, one row whose every value lies outside the table, and rows
    rising along the vocabulary (every late group passes the first candidate filter)."""
    d = (rng.standard_normal((R, D, V)) * 2.5).astype(np.float32)
    d[:, :, rng.integers(0, V, 16)] += 6.0
    for r in range(R):
        for j in range(D):
            kind = (r * D + j) % 6
            pos = rng.choice(V, 4000, replace=False)
            if kind == 0:
                d[r, j, pos] = 0.0
            elif kind == 1:
                d[r, j, pos[:2000]] = 2.0 ** -20
                d[r, j, pos[2000:]] = -(2.0 ** -20)
            elif kind == 2:
                d[r, j, pos[:50]] = np.float32(np.ldexp(1.0, -130))  # a bf16 subnormal
                d[r, j, pos[50:60]] = 64.0
                d[r, j, pos[60:63]] = 100.0
                d[r, j, pos[63:80]] = -100.0
            elif kind == 3:
                d[r, j, pos] = -np.inf
            elif kind == 4:
                d[r, j, pos[:20]] = 70.0
                d[r, j, pos[20:40]] = -70.0
    d[1, 4] = 64.0 + (rng.random(V).astype(np.float32) * 30.0)  # every value outside the table
    # rising along the vocabulary: every group after the first chunk passes
    # the first filter (the per-lane lists of candidate groups run full),
    # with long runs of equal bf16 values
    d[0, 5] = np.linspace(-5.0, 15.0, V, dtype=np.float32)
    d[1, 9] = np.linspace(20.0, -5.0, V, dtype=np.float32)[::-1].copy()
    return torch.from_numpy(d).to(torch.bfloat16).float().numpy()


@pytest.mark.parametrize("T", [1.0, 0.05])
def test_draft_table_path_special_values(T):
    """Row statistics on full-vocabulary bf16 rows whose segments are long enough for the exponential
    table (T = 1; at T = 0.05 the scaled logits leave the table's range and every logit is evaluated):
    zeros, tiny, subnormal, large and masked logits must give the oracle's binary64 normaliser to 1e-12,
    its canonical binary32 rounding, the same candidates and the same topology; NaN and +inf rows flag
    only their own request."""
    R, D, V = 4, 32, 151936  # 128 draft rows: four segments of 37984 logits each
    rng = np.random.default_rng(31 if T == 1.0 else 32)
    d = _special_rows(rng, R, D, V)
    d[2, 7, 12345] = np.nan
    d[3, 30, 777] = np.inf
    cfg = dict(name="special", R=R, V=V, D=D, B=20, K=8, T=T, dtype="bf16", steps=1)
    rnd = make_round(cfg, 11)
    rnd.plan(torch.from_numpy(d).to(torch.bfloat16).cuda())
    h = rnd.host()
    st = h["req_status"].numpy()
    tally = Tally("special rows T=%g" % T)
    for r in range(R):
        pl = ostep.plan_request(d[r], T, cfg["K"], cfg["B"])
        if r >= 2:
            assert pl["status"] & STATUS_NONFINITE and st[r] & tsb.REQ_NONFINITE, r
            continue
        assert not st[r] & tsb.REQ_NONFINITE, r
        compare_plan(h, r, pl, tally, "special T=%g req %d" % (T, r))
    say(tally.line())
    assert tally.exact["plan"] >= 1 and tally.flagged <= 1
