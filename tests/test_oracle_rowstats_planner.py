"""Pins of the oracle's row statistics (oracle/rowstats.py) and first-pass
planner (oracle/planner.py).

Row statistics: scipy's logsumexp (a different routine) and closed forms for
uniform and two-level rows; candidates against a plain Python sort.
Planner (Section 3.1, Appendix B.3): brute force over every rank path sorted
by the static order (score desc, depth asc, path lex asc); the chosen set
maximises the summed draft path probability over all prefix-closed node sets
of the same size; tree invariants; budget-short and masked-token cases.
"""
import itertools

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st
from scipy.special import logsumexp

from oracle import planner, rowstats


# ---------------------------------------------------------------- row stats

def test_lse_against_scipy_and_closed_forms():
    rng = np.random.default_rng(3)
    for scale in (0.1, 1.0, 5.0, 30.0):
        a = rng.standard_normal(5000) * scale
        assert rowstats.lse64(a) == pytest.approx(float(logsumexp(a)), rel=1e-13, abs=1e-12)
    # uniform row: ln(V) + a
    assert rowstats.lse64(np.full(1024, 2.5)) == pytest.approx(2.5 + np.log(1024), abs=1e-13)
    # two levels: n1 at x, n2 at y
    a = np.r_[np.full(3, 1.0), np.full(5, -2.0)]
    assert rowstats.lse64(a) == pytest.approx(np.log(3 * np.e + 5 * np.exp(-2.0)), abs=1e-14)
    # -inf entries drop out
    assert rowstats.lse64(np.r_[0.0, -np.inf, 0.0]) == pytest.approx(np.log(2.0), abs=1e-15)


def test_scaling_and_canonical_lp():
    invT = rowstats.inv_temperature(0.8)
    assert invT == np.float32(1.25)
    x = np.array([1.5, -3.0, 0.1], dtype=np.float32)
    assert np.array_equal(rowstats.scaled(x, invT), (x * np.float32(1.25)).astype(np.float64))
    ok, l64, l32, ids, lp = rowstats.draft_rowstats(np.array([0.0, 0.0, 0.0, 0.0], np.float32), invT, 2)
    assert ok and l32 == np.float32(np.log(4.0)) and list(ids) == [0, 1]
    assert np.all(lp == np.float32(np.float32(0.0) - np.float32(np.log(4.0))))
    with pytest.raises(ValueError):
        rowstats.inv_temperature(0.0)


def test_topk_order_matches_plain_sort():
    rng = np.random.default_rng(5)
    for _ in range(50):
        x = rng.integers(-4, 5, size=40).astype(np.float64)  # many exact ties
        K = int(rng.integers(1, 12))
        ref = sorted(range(40), key=lambda i: (-x[i], i))[:K]
        assert list(rowstats.topk(x, K)) == ref


def test_nonfinite_rows():
    assert not rowstats.row_ok(np.array([0.0, np.nan]))
    assert not rowstats.row_ok(np.array([0.0, np.inf]))
    assert not rowstats.row_ok(np.array([-np.inf, -np.inf]))
    assert rowstats.row_ok(np.array([-np.inf, 0.0]))


# ---------------------------------------------------------------- planner

def _all_paths(D, K):
    for d in range(1, D + 1):
        yield from itertools.product(range(K), repeat=d)


def _score(lp64, path):
    s = 0.0
    for i, j in enumerate(path):
        s = s + lp64[i, j]
    return s


def _brute_force_plan(lp, B):
    lp64 = np.asarray(lp, np.float32).astype(np.float64)
    D, K = lp64.shape
    paths = [p for p in _all_paths(D, K) if np.isfinite(_score(lp64, p))]
    paths.sort(key=lambda p: (-_score(lp64, p), len(p), p))
    return paths[:B]


def _paths_of(tree):
    n = tree["n_nodes"]
    paths = [()] * n
    for i in range(1, n):
        paths[i] = paths[tree["parent"][i]] + (int(tree["rank"][i]),)
    return paths


def _check_invariants(tree, lp, B):
    n = tree["n_nodes"]
    par, dep, rk = tree["parent"], tree["depth"], tree["rank"]
    nc, fc, sc = tree["n_children"], tree["first_child"], tree["score"]
    assert par[0] == -1 and dep[0] == 0 and sc[0] == 0.0
    for i in range(1, n):
        assert 0 <= par[i] < i
        assert dep[i] == dep[par[i]] + 1
        assert sc[i] <= sc[par[i]]                       # monotone along paths
        assert sc[i] == sc[par[i]] + np.float64(np.float32(lp[dep[i] - 1, rk[i]]))
    assert np.all(np.diff(dep) >= 0)                     # BFS: depth non-decreasing
    for u in range(n):
        kids = [i for i in range(1, n) if par[i] == u]
        assert nc[u] == len(kids)
        if kids:
            assert kids == list(range(fc[u], fc[u] + nc[u]))   # contiguous
            assert [rk[i] for i in kids] == list(range(nc[u]))  # ranks 0..m-1
    assert n <= B + 1


def _random_lp(rng, D, K, ties=False):
    if ties:
        x = rng.integers(-6, 1, size=(D, K)).astype(np.float64) * 0.5
    else:
        x = rng.standard_normal((D, K)) * 2
    x = -np.sort(-x, axis=1)
    lp = (x - np.log(np.exp(x).sum(axis=1, keepdims=True) + 1.0)).astype(np.float32)
    return lp


@pytest.mark.parametrize("ties", [False, True])
def test_planner_equals_brute_force(ties):
    rng = np.random.default_rng(7 + ties)
    for _ in range(60):
        D, K = int(rng.integers(1, 4)), int(rng.integers(1, 5))
        lp = _random_lp(rng, D, K, ties)
        total = planner.max_nodes(D, K)
        for B in sorted({0, 1, 2, total // 2, total, total + 3}):
            tree = planner.plan(lp, B)
            ref = _brute_force_plan(lp, B)
            got = _paths_of(tree)[1:]
            assert sorted(got) == sorted(ref)
            assert tree["n_nodes"] == len(ref) + 1
            _check_invariants(tree, lp, B)
            # BFS order = (depth, lexicographic path)
            assert got == sorted(got, key=lambda p: (len(p), p))


def _prefix_closed_sets(D, K, B):
    paths = list(_all_paths(D, K))
    for combo in itertools.combinations(paths, B):
        s = set(combo)
        if all(p[:-1] in s or len(p) == 1 for p in s):
            yield s


def test_planner_maximises_summed_path_probability():
    # Appendix B.3: max-heap expansion maximises the summed draft path
    # probability under a node budget.
    rng = np.random.default_rng(13)
    for _ in range(25):
        D, K, B = 3, 2, int(rng.integers(1, 6))
        lp = _random_lp(rng, D, K)
        lp64 = lp.astype(np.float64)
        tree = planner.plan(lp, B)
        chosen = sum(np.exp(s) for s in tree["score"][1:])
        best = max(sum(np.exp(_score(lp64, p)) for p in s) for s in _prefix_closed_sets(D, K, B))
        assert chosen == pytest.approx(best, rel=1e-12)


def test_budget_short_and_masked_candidates():
    lp = np.array([[-0.1, -2.0], [-0.5, -np.inf]], np.float32)
    tree = planner.plan(lp, 10)
    # reachable rank paths: (0), (1), (0,0), (1,0)
    assert tree["n_nodes"] == 5 and tree["plan_margin"] == np.inf
    assert sorted(_paths_of(tree)[1:]) == [(0,), (0, 0), (1,), (1, 0)]


def test_plan_margin():
    lp = np.array([[-0.1, -2.0]], np.float32)
    tree = planner.plan(lp, 1)
    assert tree["plan_margin"] == pytest.approx(np.float64(np.float32(-0.1)) - np.float64(np.float32(-2.0)))


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 4), st.integers(1, 4), st.integers(0, 40), st.integers(0, 2 ** 31 - 1))
def test_planner_invariants_hypothesis(D, K, B, seed):
    rng = np.random.default_rng(seed)
    lp = _random_lp(rng, D, K, ties=bool(seed & 1))
    tree = planner.plan(lp, B)
    _check_invariants(tree, lp, B)
    assert tree["n_nodes"] == min(B, planner.max_nodes(D, K)) + 1
