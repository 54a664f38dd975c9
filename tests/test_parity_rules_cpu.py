"""The GPU-parity comparison rules, checked on the CPU: outputs shaped like
the HIP path's but built from the oracle itself must compare exact, and a
planted difference must fail unless it sits at a decision whose own oracle
margin is a near-tie (an earlier or later near-tie elsewhere in the request
must not excuse it)."""
import copy

import numpy as np
import pytest
import torch

import oracle_worker
from oracle import replay as oreplay
from oracle.rowstats import STATUS_NONFINITE, inv_temperature, scaled
from parity_util import NEAR_TIE, compare_request, near_f32_boundary
from tally import REGISTRY, Tally

R, D, V, B, K, T = 3, 4, 600, 14, 3, 1.0
SEED, STEP = 21, 5
TRACE_MAX = 256


def _closed_z(vr, parent):
    """Closed-form residual mass after each rejection: product of the literal (normalised) masses at a node."""
    out, zi, prod, cur = [], 0, 1.0, None
    for c, U, ratio, ok in vr["tests"]:
        u = int(parent[c])
        if u != cur:
            cur, prod = u, 1.0
        if ok:
            out.append(-1.0)
        else:
            prod *= vr["residual_Z"][zi]
            zi += 1
            out.append(prod)
    return out


def _fake_gpu(seed=0):
    """Oracle results for R requests plus outputs in the HIP path's layout built from them."""
    rng = np.random.default_rng(seed)
    d = (rng.standard_normal((R, D, V)) * 2.5).astype(np.float32)
    t = (rng.standard_normal((R, B + 1, V)) * 2.5).astype(np.float32)
    res = []
    h = dict(draft_lse=torch.zeros(R, D, dtype=torch.float64), topk_tok=torch.zeros(R, D, K, dtype=torch.int32),
             topk_lp=torch.zeros(R, D, K, dtype=torch.float32),
             node_tok=torch.full((R, B + 1), -1, dtype=torch.int32), n_acc=torch.zeros(R, dtype=torch.int32),
             acc_node=torch.full((R, D), -1, dtype=torch.int32), acc_tok=torch.full((R, D), -1, dtype=torch.int32),
             bonus=torch.zeros(R, dtype=torch.int32), req_status=torch.zeros(R, dtype=torch.int32),
             target_lse=torch.full((R, B + 1), float("nan"), dtype=torch.float64),
             trace=torch.full((R, TRACE_MAX, 4), -1.0, dtype=torch.float64),
             n_nodes=torch.zeros(R, dtype=torch.int32), plan_margin=torch.zeros(R, dtype=torch.float64),
             score=torch.zeros(R, B + 1, dtype=torch.float64))
    for k in ("parent", "depth", "rank", "n_children", "first_child"):
        h[k] = torch.full((R, B + 1), -1, dtype=torch.int32)
    for r in range(R):
        pl = oracle_worker.request_step(d[r], None, T, K, B, SEED, STEP, r, None, None)["plan"]
        tree = pl["tree"]
        n = tree["n_nodes"]
        tok, _ = oreplay.replay(scaled(d[r], inv_temperature(T)), tree, SEED, STEP, r)
        full = oracle_worker.request_step(d[r], t[r], T, K, B, SEED, STEP, r, tree, tok)
        vr = full["verify"]
        res.append(full)
        h["draft_lse"][r] = torch.from_numpy(pl["lse64"])
        h["topk_tok"][r] = torch.from_numpy(pl["topk_tok"].astype(np.int32))
        h["topk_lp"][r] = torch.from_numpy(pl["topk_lp"])
        for k in ("parent", "depth", "rank", "n_children", "first_child"):
            h[k][r, :n] = torch.from_numpy(tree[k].astype(np.int32))
        h["score"][r, :n] = torch.from_numpy(tree["score"])
        h["n_nodes"][r] = n
        h["plan_margin"][r] = tree["plan_margin"]
        h["node_tok"][r, :n] = torch.from_numpy(tok.astype(np.int32))
        h["n_acc"][r] = vr["n_acc"]
        h["acc_node"][r, :vr["n_acc"]] = torch.tensor(vr["acc_node"], dtype=torch.int32)
        h["acc_tok"][r, :vr["n_acc"]] = torch.tensor(vr["acc_tok"], dtype=torch.int32)
        h["bonus"][r] = vr["bonus"]
        h["target_lse"][r, :n] = torch.from_numpy(vr["lse_t"])
        zc = _closed_z(vr, tree["parent"])
        for i, (c, U, ratio, ok) in enumerate(vr["tests"]):
            h["trace"][r, i] = torch.tensor([c, U, ratio, zc[i]], dtype=torch.float64)
    return h, res


@pytest.fixture(scope="module")
def fake():
    return _fake_gpu()


def _run(h, res):
    t = Tally("rules")
    REGISTRY.remove(t)
    for r in range(R):
        compare_request(h, r, res[r], t, D, "req %d" % r)
    return t


def test_identical_outputs_compare_exact(fake):
    h, res = fake
    t = _run(h, res)
    assert t.flagged == 0 and t.exact["plan"] == R and t.exact["verify"] == R
    assert t.exact["replay"] == sum(int((res[r]["plan"]["tree"]["n_children"] > 0).sum()) for r in range(R))
    assert any(not ok for r in range(R) for (_, _, _, ok) in res[r]["verify"]["tests"])  # rejections are covered


def _parents(res, r):
    tree = res[r]["plan"]["tree"]
    return [u for u in range(tree["n_nodes"]) if tree["n_children"][u] > 0]


def test_replay_mismatch_fails_even_if_another_parent_is_a_near_tie(fake):
    h, res = fake
    h = copy.deepcopy(h)
    res = copy.deepcopy(res)
    par = _parents(res, 0)
    assert len(par) >= 2
    tok, mg = res[0]["replay"]
    mg[par[0]] = NEAR_TIE / 3          # a near-tie at one parent ...
    fc = int(res[0]["plan"]["tree"]["first_child"][par[1]])
    h["node_tok"][0, fc] = (int(h["node_tok"][0, fc]) + 1) % V  # ... cannot excuse a mismatch at another
    mg[par[1]] = max(mg[par[1]], 1e-3)
    with pytest.raises(AssertionError):
        _run(h, res)
    mg[par[1]] = NEAR_TIE / 2          # at its own near-tie it is flagged
    t = _run(h, res)
    assert t.flagged_by["replay"] == 1


def test_bonus_mismatch_fails_away_from_its_own_margin(fake):
    h, res = fake
    h = copy.deepcopy(h)
    res = copy.deepcopy(res)
    vr = res[1]["verify"]
    h["bonus"][1] = (vr["bonus"] + 1) % V
    for i, m in enumerate(vr["margins"]):
        if m[0] == "accept":
            vr["margins"][i] = ("accept", m[1], NEAR_TIE / 4)   # near-ties elsewhere in the walk excuse nothing
    with pytest.raises(AssertionError):
        _run(h, res)


def test_residual_mass_is_compared(fake):
    h, res = fake
    h = copy.deepcopy(h)
    r, i = next((r, i) for r in range(R) for i, (_, _, _, ok) in enumerate(res[r]["verify"]["tests"]) if not ok)
    h["trace"][r, i, 3] *= 1.0 + 1e-3
    with pytest.raises(AssertionError):
        _run(h, res)


def test_acceptance_flip_is_excused_only_at_its_own_near_tie(fake):
    h, res = fake
    h = copy.deepcopy(h)
    res = copy.deepcopy(res)
    r = 0
    c, U, ratio, ok = res[r]["verify"]["tests"][0]
    # the HIP ratio moves across U by less than the probability tolerance
    gr = U + (-1 if ok else 1) * 1e-9
    h["trace"][r, 0, 2] = gr
    res[r]["verify"]["tests"][0] = (c, U, U - (-1 if ok else 1) * 2e-9, ok)  # oracle margin 2e-9: a near-tie
    t = _run(h, res)
    assert t.flagged_by["verify"] == 1
    res[r]["verify"]["tests"][0] = (c, U, ratio, ok)
    if abs(U - ratio) >= NEAR_TIE:
        with pytest.raises(AssertionError):
            _run(h, res)


def test_lse32_rounding_boundary_rule():
    rng = np.random.default_rng(3)
    for _ in range(200):
        f = np.float32(rng.uniform(-30, 30))
        nb = np.nextafter(f, np.float32(np.inf))
        mid = (float(f) + float(nb)) / 2.0
        assert near_f32_boundary(mid + 1e-14 * abs(mid)) and near_f32_boundary(mid - 1e-14 * abs(mid))
        assert not near_f32_boundary(float(f))            # a binary32 value is half an ulp from any boundary
        assert not near_f32_boundary(mid + 1e-9 * abs(mid))


def test_plan_normaliser_beyond_its_tolerance_fails(fake):
    h, res = fake
    h = copy.deepcopy(h)
    h["draft_lse"][2, 1] = float(h["draft_lse"][2, 1]) * (1 + 1e-11)
    with pytest.raises(AssertionError):
        _run(h, res)


def test_nonfinite_request_needs_the_flag(fake):
    h, res = fake
    h = copy.deepcopy(h)
    res = copy.deepcopy(res)
    res[0]["plan"]["status"] |= STATUS_NONFINITE
    with pytest.raises(AssertionError):
        _run(h, res)
    h["req_status"][0] = 1
    h["n_acc"][0] = -1
    h["bonus"][0] = -1
    res[0]["replay"] = None
    t = _run(h, res)
    assert t.exact["plan"] == R
