"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Every case feeds the same seeded bytes to both sides and compares stage by
stage (plan, then replay on the same tree, then verify on the same tree and
tokens), with the rules of tests/parity_util.py. Full-size workloads are
checked on sampled requests and parents. tsb_step must equal the staged
calls bit for bit.
"""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import replay as oreplay, step as ostep
from oracle.rowstats import STATUS_NONFINITE, inv_temperature, scaled
import paper_2609_33652_amd as tsb
from parity_util import (Tally, compare_plan, compare_replay, compare_verify, make_round, to_np, tree_dict_np)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tsb.load()


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _depths(pls, R, B):
    dep = torch.zeros(R, B + 1, dtype=torch.int64)
    for r, pl in enumerate(pls):
        if pl is not None:
            t = pl["tree"]
            dep[r, : t["n_nodes"]] = torch.from_numpy(t["depth"])
    return dep


def run_case(cfg, seed, steps, sets=4, requests=None, parents_per_req=None, gen_device="cpu", flags=0,
             check_step=True, name=""):
    """Stage-wise parity for `steps` rounds. requests: indices checked against the oracle."""
    R, D, B, K, T = cfg["R"], cfg["D"], cfg["B"], cfg["K"], cfg["T"]
    requests = list(range(R)) if requests is None else list(requests)
    rnd = make_round(cfg, seed, flags)
    rnd2 = make_round(cfg, seed, flags) if check_step else None
    invT = inv_temperature(T)
    tally = Tally()
    for s in range(steps):
        say("case %s step %d (%s)" % (name, s, W.describe(cfg)))
        base, sigma = W.base_rows(cfg, set_idx=s % sets, device=gen_device)
        draft = W.draft_from_base(cfg, base)
        d_host = to_np(draft[requests].cpu()) if gen_device != "cpu" else to_np(draft)[requests]
        pls = [None] * R
        for i, r in enumerate(requests):
            pls[r] = ostep.plan_request(d_host[i], T, K, B)
        draft_g = draft.cuda().contiguous()
        rnd.plan(draft_g)
        h = rnd.host()
        dep = _depths(pls, R, B)
        for r in range(R):
            if pls[r] is None:
                n = int(h["n_nodes"][r])
                dep[r, :n] = h["depth"][r, :n].long()
        target = W.target_from_base(cfg, base, sigma, dep.to(base.device), set_idx=s % sets)
        t_host = to_np(target[requests].cpu()) if gen_device != "cpu" else to_np(target)[requests]
        target_g = target.cuda().contiguous()
        plan_ok = {}
        for i, r in enumerate(requests):
            plan_ok[r] = compare_plan(h, r, pls[r], tally, "%s step %d req %d" % (name, s, r))
        rnd.replay(draft_g, s)
        h = rnd.host()
        tok_ok = {}
        for i, r in enumerate(requests):
            if not plan_ok[r]:
                continue
            tree = pls[r]["tree"]
            a_d = scaled(d_host[i], invT)
            n = tree["n_nodes"]
            g_tok = h["node_tok"][r, :n].numpy().astype(np.int64)
            if parents_per_req is None:
                o_tok, mg = oreplay.replay(a_d, tree, seed, s, r)
                tok_ok[r] = compare_replay(g_tok, o_tok, mg, tally, "%s step %d req %d" % (name, s, r))
            else:
                par = [u for u in range(n) if tree["n_children"][u] > 0]
                pick = par[:parents_per_req] + par[-1:]
                for u in pick:
                    m = int(tree["n_children"][u])
                    toks, mg = oreplay.replay_node(a_d[int(tree["depth"][u])], m, seed, s, r, u)
                    fc = int(tree["first_child"][u])
                    compare_replay(g_tok[fc:fc + m], toks, {u: mg}, tally, "%s step %d req %d parent %d"
                                   % (name, s, r, u))
                tok_ok[r] = False
        rnd.verify(draft_g, target_g, s)
        h = rnd.host()
        for i, r in enumerate(requests):
            if not tok_ok.get(r):
                continue
            tree = pls[r]["tree"]
            n = tree["n_nodes"]
            vr = ostep.verify_request(d_host[i], t_host[i], tree, h["node_tok"][r, :n].numpy(), pls[r]["lse64"], T,
                                      seed, s, r)
            compare_verify(h, r, vr, tally, D, "%s step %d req %d" % (name, s, r))
        if check_step:
            rnd2.step(draft_g, target_g, s)
            h2 = rnd2.host()
            for k in ("draft_lse", "topk_tok", "topk_lp", "parent", "depth", "rank", "n_children", "first_child",
                      "score", "n_nodes", "node_tok", "n_acc", "acc_node", "acc_tok", "bonus", "req_status",
                      "target_lse", "trace"):
                a, b = h[k], h2[k]
                assert torch.equal(a, b) or (a.dtype.is_floating_point and torch.equal(a.nan_to_num(7.0),
                                                                                     b.nan_to_num(7.0))), k
    say("case %s: exact %d flagged %d max|dlse_t| %.2e %s" % (name, tally.exact, tally.flagged,
                                                            getattr(tally, "max_lse_err", 0.0), tally.notes[:5]))
    return tally


def test_tiny_fp32_end_to_end():
    cfg = W.config(1)
    t = run_case(cfg, W.replay_seed(1), steps=24, name="tiny")
    assert t.exact > 0 and t.flagged <= 2


def test_ragged_multi_tile_scalar_path():
    # V not a multiple of 8 or 4 (scalar loads), 3 replay tiles with a ragged tail, T != 1
    cfg = W.config(2, R=3, V=9001, D=5, B=20, K=6, T=1.3, name="ragged")
    t = run_case(cfg, 12345, steps=8, name="ragged")
    assert t.exact > 0 and t.flagged <= 2


def test_small_bf16():
    cfg = W.config(2)
    t = run_case(cfg, W.replay_seed(2), steps=6, name="small")
    assert t.exact > 0 and t.flagged <= 2


def test_qwen_vocab_single_request():
    cfg = W.config(3)
    t = run_case(cfg, W.replay_seed(3), steps=3, name="qwen_vocab")
    assert t.exact > 0 and t.flagged <= 1


def test_batched_full_size_sampled():
    cfg = W.config(4)
    t = run_case(cfg, W.replay_seed(4), steps=1, sets=1, requests=[0, 5, 11, 15], gen_device="cuda",
                 check_step=True, name="batched")
    assert t.exact >= 8


def test_batched_full_size_parents_sampled():
    cfg = W.config(4)
    t = run_case(cfg, W.replay_seed(4), steps=1, sets=1, requests=list(range(16)), parents_per_req=2,
                 gen_device="cuda", check_step=False, name="batched-parents")
    assert t.exact >= 16


def test_large_budget_full_size_sampled():
    cfg = W.config(5)
    t = run_case(cfg, W.replay_seed(5), steps=1, sets=1, requests=[0, 63], gen_device="cuda", check_step=False,
                 name="large_budget")
    assert t.exact >= 4


def test_vocab_beyond_64_replay_tiles():
    # V = 300001: 74 replay tiles of 4096 (more than one per lane in the merge,
    # which then inserts key by key) with a ragged last tile, scalar loads
    cfg = W.config(2, R=2, V=300001, D=4, B=24, K=6, T=1.0, name="wide")
    t = run_case(cfg, 31337, steps=2, name="wide")
    assert t.exact >= 3 and t.flagged <= 1


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


def _run_edge(cfg, draft_np, target_np, seed=5, step=0):
    rnd = make_round(cfg, seed)
    draft = torch.from_numpy(draft_np).cuda()
    target = torch.from_numpy(target_np).cuda()
    rnd.step(draft, target, step)
    h = rnd.host()
    tally = Tally()
    for r in range(cfg["R"]):
        pl = ostep.plan_request(draft_np[r], cfg["T"], cfg["K"], cfg["B"])
        if not compare_plan(h, r, pl, tally, "edge req %d" % r):
            continue
        n = pl["tree"]["n_nodes"]
        o_tok, mg = oreplay.replay(scaled(draft_np[r], inv_temperature(cfg["T"])), pl["tree"], seed, step, r)
        if not compare_replay(h["node_tok"][r, :n].numpy().astype(np.int64), o_tok, mg, tally, "edge %d" % r):
            continue
        vr = ostep.verify_request(draft_np[r], target_np[r], pl["tree"], o_tok, pl["lse64"], cfg["T"], seed, step, r)
        st = int(h["req_status"][r])
        if vr["n_acc"] < 0:
            assert st & tsb.REQ_NONFINITE and int(h["n_acc"][r]) == -1 and int(h["bonus"][r]) == -1
            continue
        compare_verify(h, r, vr, tally, cfg["D"], "edge %d" % r)
    return h, tally


def test_edge_root_only_budget():
    cfg = _edge_cfg(B=0)
    rng = np.random.default_rng(1)
    d = (rng.standard_normal((3, 3, 600)) * 2).astype(np.float32)
    t = (rng.standard_normal((3, 1, 600)) * 2).astype(np.float32)
    h, tally = _run_edge(cfg, d, t)
    assert (h["n_nodes"] == 1).all() and (h["n_acc"] == 0).all()


def test_edge_budget_short_and_masked_tokens():
    cfg = _edge_cfg(D=2, K=2, B=10)
    rng = np.random.default_rng(2)
    d = (rng.standard_normal((3, 2, 600)) * 2).astype(np.float32)
    d[1, 1, 1:] = -np.inf  # request 1, position 1: a single finite token
    t = (rng.standard_normal((3, 11, 600)) * 2).astype(np.float32)
    h, tally = _run_edge(cfg, d, t)
    assert int(h["n_nodes"][0]) == 7 and int(h["req_status"][0]) & tsb.REQ_BUDGET_SHORT
    assert tally.exact >= 6


def test_edge_nonfinite_rows_flag_only_their_request():
    cfg = _edge_cfg(B=6)
    rng = np.random.default_rng(3)
    d = (rng.standard_normal((3, 3, 600)) * 2).astype(np.float32)
    t = (rng.standard_normal((3, 7, 600)) * 2).astype(np.float32)
    d[0, 2, 17] = np.nan
    t[2, 0, 5] = np.inf
    h, tally = _run_edge(cfg, d, t)
    st = h["req_status"].numpy()
    assert st[0] & tsb.REQ_NONFINITE and int(h["n_nodes"][0]) == 1 and int(h["n_acc"][0]) == -1
    assert not st[1] & tsb.REQ_NONFINITE and int(h["n_acc"][1]) >= 0
    assert st[2] & tsb.REQ_NONFINITE and int(h["n_acc"][2]) == -1


def test_edge_chain_and_minimal_vocabulary():
    cfg = _edge_cfg(R=2, V=4, D=4, B=4, K=1)
    rng = np.random.default_rng(4)
    d = rng.standard_normal((2, 4, 4)).astype(np.float32)
    t = rng.standard_normal((2, 5, 4)).astype(np.float32)
    for s in range(20):
        h, tally = _run_edge(cfg, d, t, step=s)
        assert tally.exact >= 4


def _plan_only(cfg, draft_np):
    rnd = make_round(cfg, 11)
    rnd.plan(torch.from_numpy(draft_np).cuda())
    h = rnd.host()
    tally = Tally()
    for r in range(cfg["R"]):
        pl = ostep.plan_request(draft_np[r], cfg["T"], cfg["K"], cfg["B"])
        compare_plan(h, r, pl, tally, "plan req %d" % r)  # raises on a mismatch that is not a near-tie
    say("plan-only %s: exact %d flagged %d %s" % (W.describe(cfg), tally.exact, tally.flagged, tally.notes[:3]))
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
    assert tally.exact >= 4
    nmax = sum(K ** i for i in range(1, D + 1))
    assert (h["n_nodes"] == min(B, nmax) + 1).all()


def _special_rows(rng, R, D, V):
    """bf16-exact draft rows [R, D, V] with values outside the exponential table planted: exact zeros,
    values below its smallest binade (+-2^-20 and bf16 subnormals), values at or beyond 64 (some the
    row maximum), masked -inf entries, and one row whose every value lies outside the table."""
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
    tally = Tally()
    for r in range(R):
        pl = ostep.plan_request(d[r], T, cfg["K"], cfg["B"])
        if r >= 2:
            assert pl["status"] & STATUS_NONFINITE and st[r] & tsb.REQ_NONFINITE, r
            continue
        assert not st[r] & tsb.REQ_NONFINITE, r
        compare_plan(h, r, pl, tally, "special T=%g req %d" % (T, r))
    say("special rows T=%g: exact %d flagged %d %s" % (T, tally.exact, tally.flagged, tally.notes[:3]))
    assert tally.exact >= 1
