"""Pins of the traversal-verification oracle (oracle/traversal.py; Appendix A:
sequence-level RRS over WoR trees; Table 2).

* Losslessness (Section 3.3, Proposition 1: the round is lossless when the
  verifier is lossless for every fixed topology): exact enumeration of the
  replay draws of every parent and every accept/reject branch, on the
  Figure 1 topology and on planner topologies at V=4, D=3, B<=6, with a
  prefix-keyed target and with a draft conditioned on the replayed prefix;
  extended by target sampling to D+1 tokens, the law equals the target's to
  1e-12.
* On a chain the method is Block Verification, which attains the largest
  expected number of accepted tokens of any lossless verifier: checked
  against that optimum computed independently by linear programming over
  every valid verifier of the chain (V=3, chains of 1 and 2 tokens).
* On a tree of one layer the method is WoR recursive rejection sampling:
  every test and output equals the RRS oracle's on the same uniforms.
* The closed form of the node update (the GPU's) equals the literal update.
* Plausible mistakes (the parent's alpha update without its - alpha term,
  no without-replacement removal, no residual, the path's alpha product
  dropped) must break the exact law.
* The Philox-driven sampling oracle follows the enumerated law (chi^2).
"""
import itertools
import os

import numpy as np
import pytest
from scipy import stats
from scipy.optimize import linprog

from oracle import exact, planner, step, traversal as trav, verify

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


def _chain(G):
    n = G + 1
    return dict(n_nodes=n, parent=np.arange(-1, G), depth=np.arange(n), rank=np.r_[-1, np.zeros(G, np.int64)],
                n_children=np.r_[np.ones(G, np.int64), 0], first_child=np.r_[np.arange(1, n), -1],
                score=np.zeros(n))


def _star(m):
    n = m + 1
    return dict(n_nodes=n, parent=np.r_[-1, np.zeros(m, np.int64)], depth=np.r_[0, np.ones(m, np.int64)],
                rank=np.r_[-1, np.arange(m)], n_children=np.r_[m, np.zeros(m, np.int64)],
                first_child=np.r_[1, -np.ones(m, np.int64)], score=np.zeros(n))


def _table(rng, V, L, scale=1.5):
    tab = {}
    for k in range(L + 1):
        for s in itertools.product(range(V), repeat=k):
            tab[s] = _softmax(rng.standard_normal(V) * scale)
    return lambda s: tab[tuple(s)]


def _check_lossless(tree, q, p_of, V, D):
    law = exact.traversal_law(tree, q, p_of)
    assert sum(law.values()) == pytest.approx(1.0, abs=1e-12)
    ext = exact.extend_law(law, p_of, D + 1)
    ref = exact.target_law(p_of, V, D + 1)
    for k in ref:
        assert ext.get(k, 0.0) == pytest.approx(ref[k], abs=1e-12)
    return law


def _expected_length(law):
    return sum(w * len(k) for k, w in law.items())


# ------------------------------------------------------------ losslessness
def test_figure1_topology_is_lossless():
    rng = np.random.default_rng(300)
    V, D = 4, 3
    tree = _figure1_tree()
    for _ in range(3):
        q = np.stack([_softmax(rng.standard_normal(V) * 1.5) for _ in range(D)])
        _check_lossless(tree, q, _table(rng, V, D + 1), V, D)


def test_planner_topologies_are_lossless():
    rng = np.random.default_rng(301)
    V, D = 4, 3
    for B in range(0, 7):
        q = np.stack([_softmax(rng.standard_normal(V) * 1.5) for _ in range(D)])
        lp = np.log(np.sort(q, axis=1)[:, ::-1]).astype(np.float32)
        tree = planner.plan(lp, B)
        law = _check_lossless(tree, q, _table(rng, V, D + 1), V, D)
        assert max(len(k) for k in law) <= D + 1


def test_context_dependent_draft_is_lossless():
    # q of a node's children depends on the node's whole replayed prefix (eq. (2))
    rng = np.random.default_rng(302)
    V, D = 4, 3
    tree = _figure1_tree()
    _check_lossless(tree, _table(rng, V, D, scale=2.0), _table(rng, V, D + 1), V, D)


def test_peaked_and_masked_distributions_are_lossless():
    # draft and target with zero-probability tokens and near-deterministic rows
    rng = np.random.default_rng(303)
    V, D = 4, 3
    tree = _figure1_tree()
    q = np.stack([_softmax(rng.standard_normal(V) * 5.0) for _ in range(D)])
    q[1, 3] = 0.0
    q[1] /= q[1].sum()
    tab = {}
    for k in range(D + 2):
        for s in itertools.product(range(V), repeat=k):
            row = _softmax(rng.standard_normal(V) * 4.0)
            if k == 1:
                row[2] = 0.0
                row /= row.sum()
            tab[s] = row
    _check_lossless(tree, q, lambda s: tab[tuple(s)], V, D)


# ---------------------------------------------------- chain: Block Verification optimum
def _lp_optimum(P, Q, V, G):
    """Largest expected number of accepted draft tokens over every lossless verifier of a G-token chain.

    Variables pi(x, tau, y) >= 0: draft chain x (drawn from Q), the verifier keeps its first tau tokens and
    emits y. Constraints: sum over (tau, y) of pi(x, .) = Q(x); the output, continued by target sampling to
    G + 1 tokens, has the target's law."""
    xs = list(itertools.product(range(V), repeat=G))
    var = [(x, t, y) for x in xs for t in range(G + 1) for y in range(V)]
    idx = {v: i for i, v in enumerate(var)}
    A, b = [], []

    def seq_prob(tab, s):
        w = 1.0
        for i in range(len(s)):
            w *= tab(s[:i])[s[i]]
        return w

    for x in xs:
        row = np.zeros(len(var))
        for t in range(G + 1):
            for y in range(V):
                row[idx[(x, t, y)]] = 1.0
        A.append(row)
        b.append(seq_prob(Q, x))
    for s in itertools.product(range(V), repeat=G + 1):
        row = np.zeros(len(var))
        for (x, t, y), i in idx.items():
            if x[:t] + (y,) == s[:t + 1]:
                w = 1.0
                for j in range(t + 1, G + 1):
                    w *= P(s[:j])[s[j]]
                row[i] += w
        A.append(row)
        b.append(seq_prob(P, s))
    r = linprog(-np.array([t for (x, t, y) in var], float), A_eq=np.array(A), b_eq=np.array(b),
                bounds=(0, None), method="highs")
    assert r.status == 0, r.message
    return -r.fun


@pytest.mark.parametrize("G", [1, 2])
def test_chain_attains_the_optimal_expected_accepted_length(G):
    rng = np.random.default_rng(310 + G)
    V = 3
    for _ in range(3):
        P = _table(rng, V, G + 1, scale=1.2)
        Q = _table(rng, V, G, scale=1.2)
        law = exact.traversal_law(_chain(G), Q, P)
        accepted = _expected_length(law) - 1.0
        assert accepted == pytest.approx(_lp_optimum(P, Q, V, G), abs=1e-9)
        # token-wise rejection sampling on the same chain accepts no more
        assert _expected_length(exact.emitted_law(_chain(G), Q, P)) - 1.0 <= accepted + 1e-12


# ---------------------------------------------------- one layer: WoR-RRS
def test_one_layer_is_wor_rrs():
    rng = np.random.default_rng(320)
    V = 40
    for trial in range(60):
        m = int(rng.integers(1, 6))
        tree = _star(m)
        p_root = _softmax(rng.standard_normal(V) * rng.uniform(0.5, 3.0))
        q0 = _softmax(rng.standard_normal(V) * rng.uniform(0.5, 3.0))
        leaf = {u: _softmax(rng.standard_normal(V)) for u in range(1, m + 1)}
        toks = np.r_[-1, rng.choice(V, m, replace=False, p=q0)]
        p_rows = lambda u: p_root if u == 0 else leaf[u]  # noqa: E731
        a = trav.verify_traversal(p_rows, lambda d: q0, tree, toks, 77, trial, 3)
        b = verify.verify(p_rows, lambda d: q0, tree, toks, 77, trial, 3)
        assert (a["n_acc"], a["acc_node"], a["acc_tok"], a["bonus"]) == \
            (b["n_acc"], b["acc_node"], b["acc_tok"], b["bonus"])
        assert len(a["tests"]) == len(b["tests"])
        for (c1, U1, al, ok1), (c2, U2, ratio, ok2) in zip(a["tests"], b["tests"]):
            assert c1 == c2 and U1 == U2 and ok1 == ok2
            assert al == pytest.approx(min(1.0, ratio), rel=1e-12, abs=1e-15)


# ---------------------------------------------------- closed form
def test_closed_form_equals_literal_update():
    rng = np.random.default_rng(330)
    V = 50
    checked = 0
    for _ in range(200):
        p = _softmax(rng.standard_normal(V) * rng.uniform(0.5, 3))
        q = _softmax(rng.standard_normal(V) * rng.uniform(0.5, 3))
        alpha0 = float(rng.choice([1.0, rng.uniform(0.05, 1.0)]))
        Mb, Ms, alpha = p.copy(), q.copy(), alpha0
        ys = []
        lit = []
        for _ in range(int(rng.integers(1, 6))):
            # a child is rejected only if its path's alpha is below 1: alpha Mb(y) < Ms(y)
            cand = [y for y in range(V) if Ms[y] > 0 and alpha * Mb[y] < Ms[y] and y not in ys]
            if not cand or alpha <= 0.0:
                break
            y = int(rng.choice(cand))
            alpha, Mb, Ms, T, S = trav.reject_child(alpha, Mb, Ms, y)
            ys.append(y)
            lit.append((alpha, Mb.copy(), Ms.copy(), T))
        for (a_l, Mb_l, Ms_l, T_l), (a_c, A, C, Z, S) in zip(lit, trav.closed_form_state(p, q, alpha0, ys)):
            assert a_c == pytest.approx(a_l, rel=1e-12, abs=1e-300)
            if T_l > 0:
                assert Z == pytest.approx(T_l, rel=1e-12)
                np.testing.assert_allclose(trav.closed_form_mb(p, q, A, C, Z), Mb_l, rtol=1e-10, atol=1e-15)
            ms = q.copy()
            ms[ys[:len(lit)]] = 0.0
            checked += 1
        if ys:
            ms = q.copy()
            ms[ys] = 0.0
            assert S == pytest.approx(ms.sum(), rel=1e-12)
            np.testing.assert_allclose(ms / S, lit[-1][2], rtol=1e-12)
    assert checked > 300


def test_alpha_never_increases_on_rejection():
    rng = np.random.default_rng(331)
    V = 30
    for _ in range(300):
        Mb = _softmax(rng.standard_normal(V) * 2)
        Ms = _softmax(rng.standard_normal(V) * 2)
        alpha = float(rng.uniform(0, 1))
        y = int(rng.integers(V))
        a2, _, _, T, _ = trav.reject_child(alpha, Mb, Ms, y)
        assert 0.0 <= T <= alpha + 1e-15 and 0.0 <= a2 <= alpha + 1e-15


# ---------------------------------------------------- planted mistakes
def _tiny_case(seed):
    rng = np.random.default_rng(seed)
    V, D = 4, 3
    q = np.stack([_softmax(rng.standard_normal(V) * 1.5) for _ in range(D)])
    return _figure1_tree(), q, _table(rng, V, D + 1), V, D


@pytest.mark.parametrize("slip", ["alpha_update", "no_removal", "no_residual", "local_ratio"])
def test_planted_mistakes_break_losslessness(monkeypatch, slip):
    tree, q, p_of, V, D = _tiny_case(340)
    _check_lossless(tree, q, p_of, V, D)
    real_reject, real_alpha = trav.reject_child, trav.child_alpha

    if slip == "alpha_update":      # alpha' = T / (T + 1): the parent's own alpha left out
        def bad(alpha, Mb, Ms, y):
            a, Mb2, Ms2, T, S = real_reject(alpha, Mb, Ms, y)
            return (T / (T + 1.0) if T > 0 else 0.0), Mb2, Ms2, T, S
        monkeypatch.setattr(trav, "reject_child", bad)
    elif slip == "no_removal":      # the rejected token stays in the draft distribution
        def bad(alpha, Mb, Ms, y):
            a, Mb2, _, T, S = real_reject(alpha, Mb, Ms, y)
            return a, Mb2, Ms.copy(), T, S
        monkeypatch.setattr(trav, "reject_child", bad)
    elif slip == "no_residual":     # the bonus distribution is never corrected
        def bad(alpha, Mb, Ms, y):
            a, _, Ms2, T, S = real_reject(alpha, Mb, Ms, y)
            return a, Mb.copy(), Ms2, T, S
        monkeypatch.setattr(trav, "reject_child", bad)
    else:                           # the path's product dropped: token-level ratios in traversal order
        def bad(alpha, Mb, Ms, y):
            return real_alpha(1.0, Mb, Ms, y)
        monkeypatch.setattr(trav, "child_alpha", bad)
    with pytest.raises(AssertionError):
        _check_lossless(tree, q, p_of, V, D)


# ---------------------------------------------------- sampling oracle
def test_sampling_round_follows_the_exact_law():
    """plan -> replay (Philox Gumbel-top-k) -> traversal (Philox uniforms and bonus draws) through
    step_request against the enumerated law of the same round."""
    rng = np.random.default_rng(350)
    V, D, B, K = 5, 3, 6, 3
    draft = (rng.standard_normal((D, V)) * 1.2).astype(np.float32)
    tab = {}

    def table(s):
        s = tuple(s)
        if s not in tab:
            tab[s] = (rng.standard_normal(V) * 1.5).astype(np.float32)
        return tab[s]

    for k in range(D + 1):
        for s in itertools.product(range(V), repeat=k):
            table(s)

    def target_fn(tree, node_tok):
        rows = []
        for u in range(tree["n_nodes"]):
            path, w = [], u
            while w > 0:
                path.append(int(node_tok[w]))
                w = int(tree["parent"][w])
            rows.append(table(tuple(reversed(path))))
        return np.stack(rows)

    pl = step.plan_request(draft, 1.0, K, B)
    qd = np.stack([np.exp(draft[d].astype(np.float64) - pl["lse64"][d]) for d in range(D)])
    law = exact.traversal_law(pl["tree"], qd, lambda s: _softmax(table(s).astype(np.float64)))
    n = 4000
    counts = {}
    for s in range(n):
        out = step.step_request(draft, None, 1.0, K, B, seed=0x7A5, step=s, request=1, target_fn=target_fn,
                                verifier="traversal")
        seq = tuple(out["acc_tok"]) + (out["bonus"],)
        counts[seq] = counts.get(seq, 0) + 1
    assert set(counts) <= set(law)
    keys = sorted(law, key=lambda k: -law[k])
    big = [k for k in keys if law[k] * n >= 5]
    small = [k for k in keys if law[k] * n < 5]
    obs = [counts.get(k, 0) for k in big] + [sum(counts.get(k, 0) for k in small)]
    exp_ = [law[k] * n for k in big] + [sum(law[k] for k in small) * n]
    assert stats.chisquare(obs, exp_).pvalue > 1e-3
