"""GPU parity of the round over sparse candidate pools with context-dependent
q_u (Section 3.1 pools and transition-score lookups; Section 3.2, eq. (2);
Section 3.3) against the CPU oracle, through the C ABI.

Stage by stage on the same seeded bytes: pools (bit-exact), the first pass
over per-node candidate lists (topology, scores, plan margin and planning
tokens bit-exact unless the oracle's plan margin is a near-tie), the replay
(node tokens bit-exact unless a replay key gap is a near-tie) and the walk
(accepted path and bonus bit-exact unless an acceptance or bonus margin is a
near-tie; acceptance ratios to 1e-5 relative; streamed target normalisers
to 2e-6). tsb_pool_step must equal the staged calls bit for bit.
Workloads: the tiny and small workloads with pools of 4, 13 and 16 tokens,
the Qwen-vocabulary workload with 64, the batched workload at full size with
16 and 64, and sampled requests of the large-budget workload (whose
candidate lists exceed the planner's LDS). Edge cases: root-only budget,
non-finite transition score or draft row, pools holding -inf logits, a pool
as wide as the vocabulary, a node token outside its pool, and a workspace
shared with the vocabulary-wide walk.
"""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import pool as opool
from oracle.rowstats import STATUS_BUDGET_SHORT, STATUS_NONFINITE, inv_temperature
import paper_2609_33652_amd as tsb
from parity_util import LSE_T_ATOL, NEAR_TIE, Tally, make_round, to_np, tree_dict_np

pytestmark = pytest.mark.gpu


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


def oracle_plan(d_host, tr_host, T, K, P, B):
    invT = inv_temperature(T)
    pl = opool.pools(d_host, P)
    a_pool = opool.pool_logits(d_host, invT, pl)
    cs = opool.scaled_corrections(tr_host, invT)
    return pl, opool.plan_ctx(a_pool, cs, K, B)


def compare_pool_plan(h, r, pl, tree, status, tally, where):
    """Returns True if the GPU plan of request r equals the oracle's."""
    if status & STATUS_NONFINITE:
        assert int(h["req_status"][r]) & tsb.REQ_NONFINITE, where
        assert int(h["n_nodes"][r]) == 1, where
        return False
    assert not int(h["req_status"][r]) & tsb.REQ_NONFINITE, where
    assert np.array_equal(h["pool_tok"][r].numpy().astype(np.int64), pl), where
    g = tree_dict_np(h, r)
    margin = tree["plan_margin"]
    same = g["n_nodes"] == tree["n_nodes"] and all(
        np.array_equal(g[k], tree[k]) for k in ("parent", "depth", "rank", "n_children", "first_child"))
    if not same:
        if 0 < margin < NEAR_TIE:
            tally.flag("plan near-tie %g %s" % (margin, where))
            return False
        raise AssertionError("topology differs %s (margin %g): gpu n=%d oracle n=%d"
                             % (where, margin, g["n_nodes"], tree["n_nodes"]))
    assert np.array_equal(g["score"], tree["score"]), where
    if np.isfinite(margin):
        assert g["plan_margin"] == margin, where
    else:
        assert not np.isfinite(g["plan_margin"]), where
    n = tree["n_nodes"]
    assert np.array_equal(h["plan_tok"][r, :n].numpy().astype(np.int64),
                          opool.plan_tokens(tree, pl, tree["plan_slot"])), where
    assert (h["plan_tok"][r, n:] == -1).all(), where
    assert bool(int(h["req_status"][r]) & tsb.REQ_BUDGET_SHORT) == bool(status & STATUS_BUDGET_SHORT), where
    tally.exact += 1
    return True


def compare_pool_verify(h, r, o, tally, D, where):
    n_acc = int(h["n_acc"][r])
    got = (n_acc, [int(x) for x in h["acc_node"][r, :max(n_acc, 0)]],
           [int(x) for x in h["acc_tok"][r, :max(n_acc, 0)]], int(h["bonus"][r]))
    exp = (o["n_acc"], [int(x) for x in o["acc_node"]], [int(x) for x in o["acc_tok"]], int(o["bonus"]))
    vr = o["verify"]
    if vr is not None:
        tr = h["trace"][r].numpy()
        for i, (c, U, ratio, _) in enumerate(vr["tests"][: tr.shape[0]]):
            if int(tr[i, 0]) != c:
                break
            assert tr[i, 1] == U, where
            if np.isfinite(ratio):
                assert abs(tr[i, 2] - ratio) <= 1e-5 * abs(ratio) + 1e-7, (where, i, tr[i, 2], ratio)
        lt = h["target_lse"][r].numpy()[: len(vr["lse_t"])]
        np.testing.assert_allclose(lt, vr["lse_t"], rtol=0, atol=LSE_T_ATOL, err_msg=where)
    if got == exp:
        assert [int(x) for x in h["acc_node"][r, max(n_acc, 0):]] == [-1] * (D - max(n_acc, 0)), where
        assert not int(h["req_status"][r]) & (tsb.REQ_WALK_TIMEOUT | tsb.REQ_BAD_TOKEN), where
        tally.exact += 1
        return True
    if any(0 < m[2] < NEAR_TIE for m in o["margins"] if m[0] in ("accept", "bonus")):
        tally.flag("verify near-tie " + where)
        return False
    raise AssertionError("pool verification differs %s: gpu %s oracle %s" % (where, got, exp))


def _depths(trees, h, R, B):
    dep = torch.zeros(R, B + 1, dtype=torch.int64)
    for r in range(R):
        if trees[r] is not None:
            dep[r, : trees[r]["n_nodes"]] = torch.from_numpy(trees[r]["depth"])
        else:
            n = int(h["n_nodes"][r])
            dep[r, :n] = h["depth"][r, :n].long()
    return dep


def run_pool(cfg, P, seed, steps, sets=4, requests=None, gen_device="cpu", check_step=True, name=""):
    R, D, B, K, T = cfg["R"], cfg["D"], cfg["B"], cfg["K"], cfg["T"]
    requests = list(range(R)) if requests is None else list(requests)
    rnd = pool_round(cfg, seed, P)
    rnd2 = pool_round(cfg, seed, P) if check_step else None
    ptally, rtally, vtally = Tally(), Tally(), Tally()
    for s in range(steps):
        say("pool %s P=%d step %d (%s)" % (name, P, s, W.describe(cfg)))
        base, sigma = W.base_rows(cfg, set_idx=s % sets, device=gen_device)
        draft = W.draft_from_base(cfg, base)
        trans = W.transitions(cfg, P, set_idx=s % sets, device=gen_device)
        d_host = to_np(draft[requests].cpu())
        tr_host = trans[requests].cpu().numpy()
        draft_g, trans_g = draft.cuda().contiguous(), trans.cuda().contiguous()
        rnd.pool_plan(draft_g, trans_g)
        h = rnd.host()
        trees = [None] * R
        pls = {}
        for i, r in enumerate(requests):
            pls[r], trees[r] = oracle_plan(d_host[i], tr_host[i], T, K, P, B)
        target = W.target_from_base(cfg, base, sigma, _depths(trees, h, R, B).to(base.device), set_idx=s % sets)
        t_host = to_np(target[requests].cpu())
        target_g = target.cuda().contiguous()
        rnd.pool_replay(draft_g, trans_g, s)
        rnd.pool_verify(draft_g, trans_g, target_g, s)
        h = rnd.host()
        for i, r in enumerate(requests):
            where = "%s P=%d step %d req %d" % (name, P, s, r)
            o = opool.step_pool_request(d_host[i], t_host[i], tr_host[i], T, K, P, B, seed, s, r)
            if not compare_pool_plan(h, r, pls[r], o["tree"], o["status"], ptally, where):
                continue
            n = o["tree"]["n_nodes"]
            gtok = h["node_tok"][r, :n].numpy().astype(np.int64)
            if not np.array_equal(gtok, o["node_tok"]):
                if any(0 < m[2] < NEAR_TIE for m in o["margins"] if m[0] == "replay"):
                    rtally.flag("replay near-tie " + where)
                    continue
                diff = np.nonzero(gtok != o["node_tok"])[0]
                raise AssertionError("node tokens differ %s at %s: gpu %s oracle %s"
                                     % (where, diff[:8], gtok[diff[:8]], o["node_tok"][diff[:8]]))
            assert (h["node_tok"][r, n:] == -1).all(), where
            rtally.exact += 1
            compare_pool_verify(h, r, o, vtally, D, where)
        if check_step:
            rnd2.pool_step(draft_g, trans_g, target_g, s)
            h2 = rnd2.host()
            for k in ("pool_tok", "parent", "depth", "rank", "n_children", "first_child", "score", "n_nodes",
                      "node_tok", "n_acc", "acc_node", "acc_tok", "bonus", "req_status", "target_lse", "trace"):
                assert torch.equal(h[k], h2[k]), k
    say("pool %s P=%d: plans exact %d flagged %d; replays exact %d flagged %d; walks exact %d flagged %d %s"
        % (name, P, ptally.exact, ptally.flagged, rtally.exact, rtally.flagged, vtally.exact, vtally.flagged,
           (ptally.notes + rtally.notes + vtally.notes)[:5]))
    return ptally, rtally, vtally


@pytest.mark.parametrize("P", [4, 16])
def test_pool_tiny_fp32(P):
    cfg = W.config(1)
    p, rp, v = run_pool(cfg, P, W.replay_seed(1), steps=16, name="tiny")
    assert v.exact >= 14 and p.flagged + rp.flagged + v.flagged <= 2


def test_pool_ragged_scalar_path():
    cfg = W.config(2, R=3, V=9001, D=5, B=20, K=6, T=1.3, name="ragged")
    p, rp, v = run_pool(cfg, 13, 12345, steps=5, name="ragged")
    assert v.exact >= 13


def test_pool_small_bf16():
    cfg = W.config(2)
    p, rp, v = run_pool(cfg, 16, W.replay_seed(2), steps=5, name="small")
    assert v.exact >= 4


def test_pool_qwen_vocab_p64():
    cfg = W.config(3)
    p, rp, v = run_pool(cfg, 64, W.replay_seed(3), steps=3, name="qwen_vocab")
    assert v.exact >= 2


@pytest.mark.parametrize("P", [16, 64])
def test_pool_batched_full_size(P):
    cfg = W.config(4)
    p, rp, v = run_pool(cfg, P, W.replay_seed(4), steps=1, sets=1, gen_device="cuda", name="batched")
    assert v.exact >= 15


def test_pool_full_budget_many_internal_nodes():
    # B = 1023 with K = 2: a 1024-node tree with several hundred internal
    # nodes, beyond those whose Gumbel draws the replay computes ahead
    cfg = W.config(2, R=2, V=4096, D=12, B=1023, K=2, T=1.0, name="deep")
    p, rp, v = run_pool(cfg, 8, 4242, steps=2, name="deep")
    assert rp.exact + rp.flagged == 4 and rp.exact >= 3


def test_pool_large_budget_sampled():
    cfg = W.config(5)
    p, rp, v = run_pool(cfg, 64, W.replay_seed(5), steps=1, sets=1, requests=[0, 21, 63], gen_device="cuda",
                        check_step=False, name="large_budget")
    assert v.exact >= 2


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
    tally = Tally()
    outs = []
    for r in range(cfg["R"]):
        o = opool.step_pool_request(d[r], t[r], tr[r], cfg["T"], cfg["K"], P, cfg["B"], seed, step, r)
        outs.append(o)
        pl, _ = oracle_plan(d[r], tr[r], cfg["T"], cfg["K"], P, cfg["B"])
        if not compare_pool_plan(h, r, pl, o["tree"], o["status"], Tally(), "edge req %d" % r):
            if o["status"] & STATUS_NONFINITE:
                assert int(h["n_acc"][r]) == -1 and int(h["bonus"][r]) == -1
            continue
        n = o["tree"]["n_nodes"]
        assert np.array_equal(h["node_tok"][r, :n].numpy().astype(np.int64), o["node_tok"]), r
        compare_pool_verify(h, r, o, tally, cfg["D"], "edge req %d" % r)
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
    assert (h["n_nodes"] == 1).all() and (h["n_acc"] == 0).all() and tally.exact == 3


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
    assert tally.exact + tally.flagged == 3
    for r in range(3):
        n = int(h["n_nodes"][r])
        assert (h["n_children"][r, :n] <= 4).all()


def test_pool_edge_pool_as_wide_as_vocabulary():
    cfg = _edge_cfg(V=48, K=4, B=10, R=2)
    d, tr, t = _edge_inputs(cfg, 48, np.random.default_rng(4))
    h, tally, _ = _edge(cfg, 48, d, tr, t)
    assert tally.exact + tally.flagged == 2


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
