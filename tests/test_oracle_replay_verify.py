"""Pins of the oracle's replay (oracle/replay.py) and verifier (oracle/verify.py).

Replay (Section 3.2, Appendix A): the ordered Gumbel-top-k draws follow the
Plackett-Luce law of sampling without replacement from softmax(a): chi^2 on
ordered pairs and on single draws, with Philox draws keyed by distinct steps.
Verifier (eq. (1), Appendix A): the closed form equals the literal recursion;
a single child is accepted with probability sum_v min{p, q}; a chain accepts
its first j tokens with probability prod alpha_i when p and q depend only on
the depth; p = q always accepts; the sampling verifier's empirical law equals
the exact enumerated law.
"""
import numpy as np
import pytest
from scipy import stats

from oracle import exact, philox, planner, replay, verify


def _softmax(a):
    e = np.exp(a - a.max())
    return e / e.sum()


def test_replay_plackett_luce_law():
    rng = np.random.default_rng(2)
    V = 6
    a = rng.standard_normal(V) * 1.2
    q = _softmax(a)
    n = 30000
    counts = np.zeros((V, V))
    for s in range(n):
        toks, _ = replay.replay_node(a, 2, seed=77, step=s, request=0, node=0)
        counts[toks[0], toks[1]] += 1
    exp_ = np.array([[q[i] * q[j] / (1 - q[i]) if i != j else 0.0 for j in range(V)] for i in range(V)]) * n
    mask = exp_ > 0
    assert counts[~mask].sum() == 0
    assert stats.chisquare(counts[mask], exp_[mask]).pvalue > 1e-3


def test_replay_single_draw_is_softmax_and_slots_distinct():
    rng = np.random.default_rng(4)
    V = 10
    a = rng.standard_normal(V)
    q = _softmax(a)
    n = 20000
    c = np.zeros(V)
    for s in range(n):
        toks, _ = replay.replay_node(a, 3, seed=5, step=s, request=1, node=2)
        assert len(set(toks.tolist())) == 3
        c[toks[0]] += 1
    assert stats.chisquare(c, q * n).pvalue > 1e-3


def test_replay_key_formula():
    a = np.array([0.5, -1.0, 2.0, 0.0])
    toks, margin = replay.replay_node(a, 2, seed=9, step=3, request=4, node=5)
    g = -np.log(-np.log(philox.u24(philox.draw_words(9, 3, 4, 5, philox.STREAM_REPLAY, np.arange(4)))))
    keys = a + g
    order = sorted(range(4), key=lambda v: (-keys[v], v))
    assert list(toks) == order[:2]
    assert margin == pytest.approx(min(keys[order[0]] - keys[order[1]], keys[order[1]] - keys[order[2]]))


def _literal_node(p, q, ys, Us):
    P, Q = p.copy(), q.copy()
    ratios, zs = [], []
    for j, (y, U) in enumerate(zip(ys, Us)):
        r = verify.accept_ratio(P, Q, y)
        ratios.append(r)
        if U < r:
            return j, ratios, zs
        P, Q, Z, S = verify.reject(P, Q, y)
        zs.append(Z)
    return -1, ratios, zs


def test_closed_form_equals_literal():
    rng = np.random.default_rng(8)
    for _ in range(300):
        V = int(rng.integers(2, 40))
        p = _softmax(rng.standard_normal(V) * 2)
        q = _softmax(rng.standard_normal(V) * 2)
        m = int(rng.integers(1, min(V, 8) + 1))
        ys = rng.choice(V, size=m, replace=False, p=q)
        Us = rng.random(m)
        j1, r1, z1 = _literal_node(p, q, ys, Us)
        j2, r2, z2, _ = verify.closed_form_node(p, q, ys, Us)
        assert j1 == j2
        np.testing.assert_allclose(r2, r1, rtol=1e-12, atol=1e-15)
        # literal Z is the normaliser of the residual of an already normalised P;
        # closed-form Z is unnormalised: Z_lit_i = Z_cf_i / Z_cf_{i-1}
        zc = [1.0] + z2
        np.testing.assert_allclose([zc[i + 1] / zc[i] for i in range(len(z2))], z1, rtol=1e-11, atol=1e-15)


def _chain_tree(D):
    n = D + 1
    return dict(n_nodes=n, parent=np.arange(-1, D), depth=np.arange(n),
                rank=np.r_[-1, np.zeros(D, int)], n_children=np.r_[np.ones(D, int), 0],
                first_child=np.r_[np.arange(1, n), -1], score=np.zeros(n))


def test_single_child_accepts_with_rs_overlap():
    # eq. (1): alpha_RS(p, q) = sum_v min{p(v), q(v)}
    rng = np.random.default_rng(12)
    for _ in range(20):
        V = int(rng.integers(2, 7))
        p = _softmax(rng.standard_normal(V) * 1.5)
        q = _softmax(rng.standard_normal(V) * 1.5)
        tree = _chain_tree(1)
        law = exact.emitted_law(tree, q[None, :], lambda s: p if len(s) == 0 else np.ones(V) / V)
        acc = sum(w for seq, w in law.items() if len(seq) == 2)
        assert acc == pytest.approx(np.minimum(p, q).sum(), abs=1e-14)


def test_chain_acceptance_is_product_of_overlaps():
    rng = np.random.default_rng(21)
    V, D = 4, 3
    q = np.stack([_softmax(rng.standard_normal(V)) for _ in range(D)])
    p = np.stack([_softmax(rng.standard_normal(V)) for _ in range(D + 1)])
    law = exact.emitted_law(_chain_tree(D), q, lambda s: p[len(s)])
    alpha = np.minimum(p[:D], q).sum(axis=1)
    for j in range(1, D + 1):
        got = sum(w for seq, w in law.items() if len(seq) - 1 >= j)
        assert got == pytest.approx(np.prod(alpha[:j]), abs=1e-13)


def test_equal_distributions_always_accept_first_child():
    rng = np.random.default_rng(1)
    V = 5
    q = np.stack([_softmax(rng.standard_normal(V)) for _ in range(2)])
    lp = np.log(np.sort(q, axis=1)[:, ::-1]).astype(np.float32)
    tree = planner.plan(lp, 5)
    law = exact.emitted_law(tree, q, lambda s: q[min(len(s), 1)])
    # every emitted sequence goes through the first child at depth 1
    assert sum(w for seq, w in law.items() if len(seq) >= 2) == pytest.approx(1.0, abs=1e-13)


def test_sampling_verifier_matches_exact_law():
    # the oracle's Philox-driven replay + verify reproduces the enumerated law
    rng = np.random.default_rng(31)
    V, D = 3, 2
    q = np.stack([_softmax(rng.standard_normal(V) * 1.3) for _ in range(D)])
    ptab = {}

    def p_of(s):
        if s not in ptab:
            ptab[s] = _softmax(rng.standard_normal(V) * 1.3)
        return ptab[s]

    lp = np.log(np.sort(q, axis=1)[:, ::-1]).astype(np.float32)
    tree = planner.plan(lp, 4)
    law = exact.emitted_law(tree, q, p_of)
    n = 20000
    counts = {}
    for s in range(n):
        a = np.log(q)
        node_tok, _ = replay.replay(a, tree, seed=123, step=s, request=0)

        def prow(u, node_tok=node_tok):
            path = []
            while u > 0:
                path.append(int(node_tok[u]))
                u = int(tree["parent"][u])
            return p_of(tuple(reversed(path)))

        res = verify.verify(prow, lambda d: q[d], tree, node_tok, 123, s, 0)
        seq = tuple(res["acc_tok"]) + (res["bonus"],)
        counts[seq] = counts.get(seq, 0) + 1
    keys = sorted(set(law) | set(counts))
    obs = np.array([counts.get(k, 0) for k in keys], float)
    exp_ = np.array([law.get(k, 0.0) for k in keys]) * n
    assert obs[exp_ == 0].sum() == 0
    big = exp_ >= 5
    obs2 = np.r_[obs[big], obs[~big].sum()]
    exp2 = np.r_[exp_[big], exp_[~big].sum()]
    if exp2[-1] == 0:
        obs2, exp2 = obs2[:-1], exp2[:-1]
    assert stats.chisquare(obs2, exp2).pvalue > 1e-3


def test_rrs_reads_only_the_target_rows_its_walk_enters():
    """An unusable target row (here a NaN) ends a WoR-RRS round only when the walk enters its node: in a
    row the walk never reads it changes no output but that row's normaliser; in the root row it ends the
    round with NONFINITE. Traversal verification rejects it anywhere in the tree."""
    from oracle import step
    rng = np.random.default_rng(311)
    V, D, B, K = 12, 3, 8, 3
    draft = (rng.standard_normal((D, V)) * 1.5).astype(np.float32)
    target = (rng.standard_normal((B + 1, V)) * 1.5).astype(np.float32)
    for s in range(6):
        ref = step.step_request(draft, target, 1.0, K, B, seed=0x7A, step=s, request=1)
        entered = {0} | {int(c) for c in ref["acc_node"]}
        spare = [u for u in range(ref["tree"]["n_nodes"]) if u not in entered]
        assert spare and ref["n_acc"] >= 0
        t = target.copy()
        t[spare[-1], 3] = np.nan
        out = step.step_request(draft, t, 1.0, K, B, seed=0x7A, step=s, request=1)
        assert (out["n_acc"], out["acc_node"], out["acc_tok"], out["bonus"]) == \
            (ref["n_acc"], ref["acc_node"], ref["acc_tok"], ref["bonus"])
        assert not out["status"] & 1
        lse_a, lse_b = ref["verify"]["lse_t"], out["verify"]["lse_t"]
        assert np.isnan(lse_b[spare[-1]])
        keep = np.arange(len(lse_a)) != spare[-1]
        assert np.array_equal(lse_a[keep], lse_b[keep])
        trav = step.step_request(draft, t, 1.0, K, B, seed=0x7A, step=s, request=1, verifier="traversal")
        assert trav["status"] & 1 and trav["n_acc"] == -1
        t = target.copy()
        t[0, 5] = np.inf
        out = step.step_request(draft, t, 1.0, K, B, seed=0x7A, step=s, request=1)
        assert out["status"] & 1 and out["n_acc"] == -1 and out["bonus"] == -1
