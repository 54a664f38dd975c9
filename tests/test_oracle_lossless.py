"""Losslessness of the oracle's round (Section 3.3, Proposition 1).

Exact enumeration (no random numbers) at V=4, D=3, B<=6 on the paper's
Figure 1 topology and on planner-produced topologies: the law of the emitted
sequence, continued by target sampling to D+1 tokens, equals the target's own
law prod_i p(s_i | s_<i) to 1e-12. The target is prefix-keyed, built per
token path as a target model would. A planted mistake in the residual update
must break the equality. A chi^2 check at V=64 runs the Philox-driven oracle.
"""
import os

import numpy as np
import pytest
from scipy import stats

from oracle import exact, planner, replay, step, verify

HERE = os.path.dirname(os.path.abspath(__file__))


def _softmax(a):
    e = np.exp(a - a.max())
    return e / e.sum()


def _figure1_tree():
    rows = []
    with open(os.path.join(HERE, "golden", "figure1_topology.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            rows.append([int(w) for w in line.split()])
    rows = np.array(rows)
    n = rows.shape[0]
    parent, depth, rank = rows[:, 1], rows[:, 2], rows[:, 3]
    nc = np.array([(parent == u).sum() for u in range(n)])
    fc = np.array([int(np.argmax(parent == u)) if nc[u] else -1 for u in range(n)])
    return dict(n_nodes=n, parent=parent, depth=depth, rank=rank, n_children=nc, first_child=fc,
                score=np.zeros(n))


def _prefix_target(rng, V, D, scale=1.5):
    tab = {}

    def p_of(s):
        s = tuple(s)
        if s not in tab:
            tab[s] = _softmax(rng.standard_normal(V) * scale)
        return tab[s]
    # materialise every prefix up to length D so the table is fixed
    import itertools
    for L in range(D + 1):
        for s in itertools.product(range(V), repeat=L):
            p_of(s)
    return p_of


def _check_lossless(tree, q, p_of, V, D):
    law = exact.emitted_law(tree, q, p_of)
    assert sum(law.values()) == pytest.approx(1.0, abs=1e-12)
    ext = exact.extend_law(law, p_of, D + 1)
    ref = exact.target_law(p_of, V, D + 1)
    for k in ref:
        assert ext.get(k, 0.0) == pytest.approx(ref[k], abs=1e-12)
    return law


def test_figure1_topology_is_lossless():
    rng = np.random.default_rng(100)
    V, D = 4, 3
    tree = _figure1_tree()
    assert tree["n_nodes"] == 7 and list(tree["n_children"]) == [2, 2, 1, 1, 0, 0, 0]
    for _ in range(3):
        q = np.stack([_softmax(rng.standard_normal(V) * 1.5) for _ in range(D)])
        _check_lossless(tree, q, _prefix_target(rng, V, D), V, D)


def test_planner_topologies_are_lossless():
    rng = np.random.default_rng(101)
    V, D = 4, 3
    for B in range(0, 7):
        q = np.stack([_softmax(rng.standard_normal(V) * 1.5) for _ in range(D)])
        lp = np.log(np.sort(q, axis=1)[:, ::-1]).astype(np.float32)
        tree = planner.plan(lp, B)
        _check_lossless(tree, q, _prefix_target(rng, V, D), V, D)


def test_planted_residual_mistake_breaks_losslessness(monkeypatch):
    # Plant a plausible slip (residual max(P - Q, 0) replaced by max(P - Q/2, 0))
    # in the oracle and check that the enumeration catches it.
    rng = np.random.default_rng(102)
    V, D = 4, 3
    tree = _figure1_tree()
    q = np.stack([_softmax(rng.standard_normal(V) * 1.5) for _ in range(D)])
    p_of = _prefix_target(rng, V, D)
    good = verify.reject

    def bad(P, Q, y):
        return good(P, Q * 0.5, y)

    monkeypatch.setattr(verify, "reject", bad)
    with pytest.raises(AssertionError):
        _check_lossless(tree, q, p_of, V, D)


def test_chi2_first_tokens_v64():
    rng = np.random.default_rng(103)
    V, D, B, K = 64, 3, 6, 3
    draft = (rng.standard_normal((D, V)) * 1.5).astype(np.float32)
    tab = {}

    def p_of(s):
        s = tuple(s)
        if s not in tab:
            tab[s] = (rng.standard_normal(V) * 1.5).astype(np.float32)
        return tab[s]

    def target_fn(tree, node_tok):
        rows = []
        for u in range(tree["n_nodes"]):
            path, w = [], u
            while w > 0:
                path.append(int(node_tok[w]))
                w = int(tree["parent"][w])
            rows.append(p_of(tuple(reversed(path))))
        return np.stack(rows)

    n = 6000
    first = np.zeros(V)
    pairs = {}
    for s in range(n):
        out = step.step_request(draft, None, 1.0, K, B, seed=0xABC, step=s, request=0, target_fn=target_fn)
        seq = list(out["acc_tok"]) + [out["bonus"]]
        first[seq[0]] += 1
    p0 = _softmax(p_of(()).astype(np.float64))
    big = p0 * n >= 5
    obs = np.r_[first[big], first[~big].sum()]
    exp_ = np.r_[p0[big] * n, p0[~big].sum() * n]
    assert stats.chisquare(obs, exp_).pvalue > 1e-3
