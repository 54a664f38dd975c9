"""Pins of the pool oracle (oracle/pool.py; Section 3.1 sparse candidate
pools, Section 3.2 eq. (2) with the replayed prefix, Section 3.3).

* Pool selection: every pool token precedes every other token under
  (logit desc, id asc), checked pair by pair on tie-heavy rows.
* A pool holding the whole vocabulary with a zero transition table is the
  vocabulary-wide round: tree, node tokens, accepted path and bonus equal
  oracle.step's (itself pinned by enumeration and closed forms).
* First pass: equal to brute-force enumeration of every rank path of the
  context-dependent candidate tree, sorted by the static order; invariants.
* Losslessness with context-dependent, pool-restricted q_u: the exact law of
  the emitted sequence (enumeration) equals the target's, with P < V so the
  residuals carry mass outside the pool.
* The Philox-driven oracle round (Gumbel-top-k over the pool, per-node q_u in
  verification) follows that exact law (chi^2); planting a replay that
  ignores the context, or a verifier that ignores it, breaks a pin.
"""
import itertools

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st
from scipy import stats

from oracle import exact, planner_ep, pool, step
from oracle.rowstats import STATUS_BUDGET_SHORT, STATUS_NONFINITE


def _softmax(a):
    e = np.exp(a - a.max())
    return e / e.sum()


def test_pool_is_the_first_p_tokens_by_logit_then_id():
    rng = np.random.default_rng(200)
    for _ in range(30):
        V, P = int(rng.integers(4, 40)), int(rng.integers(1, 4))
        row = rng.integers(0, 5, size=V).astype(np.float32)  # many ties
        ids = pool.pools(row[None, :], P)[0]
        assert len(set(ids.tolist())) == P
        inside = set(ids.tolist())
        for i in inside:
            for o in set(range(V)) - inside:
                assert row[i] > row[o] or (row[i] == row[o] and i < o)
        for a, b in zip(ids[:-1], ids[1:]):
            assert row[a] > row[b] or (row[a] == row[b] and a < b)


def _prefix_rows(rng, V, scale=1.5):
    tab = {}

    def p_of(s):
        s = tuple(s)
        if s not in tab:
            tab[s] = (rng.standard_normal(V) * scale).astype(np.float32)
        return tab[s]
    return p_of


def _target_fn(p_of):
    def fn(tree, node_tok):
        rows = []
        for u in range(tree["n_nodes"]):
            path, w = [], u
            while w > 0:
                path.append(int(node_tok[w]))
                w = int(tree["parent"][w])
            rows.append(p_of(tuple(reversed(path))))
        return np.stack(rows)
    return fn


def test_whole_vocabulary_pool_without_corrections_is_the_vocabulary_wide_round():
    rng = np.random.default_rng(201)
    V, D, K, B = 48, 3, 4, 10
    checked = 0
    for trial in range(12):
        draft = (rng.standard_normal((D, V)) * 2).astype(np.float32)
        trans = np.zeros((D - 1, V, V), np.float32)
        p_of = _prefix_rows(rng, V)
        for s in range(4):
            a = pool.step_pool_request(draft, None, trans, 1.0, K, V, B, 7, s, trial, target_fn=_target_fn(p_of))
            b = step.step_request(draft, None, 1.0, K, B, 7, s, trial, target_fn=_target_fn(p_of))
            ta, tb = a["tree"], b["tree"]
            for k in ("parent", "depth", "rank", "n_children", "first_child", "score"):
                assert np.array_equal(ta[k], tb[k]), k
            assert np.array_equal(a["node_tok"], b["node_tok"])
            if not step.near_ties(a["margins"]) and not step.near_ties(b["margins"]):
                assert a["n_acc"] == b["n_acc"] and a["acc_tok"] == b["acc_tok"] and a["bonus"] == b["bonus"]
                checked += 1
    assert checked >= 40


def _brute_force_tree(a_pool, cs, K, B):
    """Every rank path of the candidate tree, sorted by the static order, first B."""
    D = a_pool.shape[0]
    nodes = []

    def grow(path, slot, score):
        d = len(path)
        if d >= D:
            return
        slots, lps = pool.candidates(pool.corrected(a_pool, cs, d, slot), K)
        for k, (j, lp) in enumerate(zip(slots, lps)):
            nodes.append((path + (k,), score + lp))
            grow(path + (k,), j, score + lp)

    grow((), -1, 0.0)
    order = sorted(nodes, key=lambda t: (-t[1], len(t[0]), t[0]))
    chosen = order[:B]
    margin = (chosen[-1][1] - order[B][1]) if (chosen and B < len(order)) else np.inf
    return planner_ep._bfs_tree(chosen, margin), len(nodes)


def _tiny_pool_case(rng, D, V, P, ties=False):
    if ties:
        draft = rng.integers(0, 4, size=(D, V)).astype(np.float32)
        trans = rng.integers(-2, 3, size=(max(D - 1, 0), P, P)).astype(np.float32)
    else:
        draft = (rng.standard_normal((D, V)) * 2).astype(np.float32)
        trans = (rng.standard_normal((max(D - 1, 0), P, P)) * 1.5).astype(np.float32)
    pl = pool.pools(draft, P)
    return draft, trans, pl, pool.pool_logits(draft, np.float32(1.0), pl), pool.scaled_corrections(trans, 1.0)


@pytest.mark.parametrize("ties", [False, True])
def test_first_pass_equals_brute_force_enumeration(ties):
    rng = np.random.default_rng(202 + ties)
    for _ in range(40):
        D, P = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        K = int(rng.integers(1, P + 1))
        _, _, _, a_pool, cs = _tiny_pool_case(rng, D, 6, P, ties)
        B = int(rng.integers(0, 20))
        got = pool.plan_ctx(a_pool, cs, K, B)
        ref, total = _brute_force_tree(a_pool, cs, K, B)
        assert got["n_nodes"] == min(B, total) + 1
        for k in ("parent", "depth", "rank", "n_children", "first_child", "score"):
            assert np.array_equal(got[k], ref[k]), k
        assert got["plan_margin"] == ref["plan_margin"] or (np.isinf(got["plan_margin"]) and np.isinf(ref["plan_margin"]))


@settings(max_examples=60, deadline=None)
@given(D=st.integers(1, 5), P=st.integers(1, 6), B=st.integers(0, 40), seed=st.integers(0, 10**6))
def test_first_pass_invariants(D, P, B, seed):
    rng = np.random.default_rng(seed)
    K = 1 + seed % P
    _, _, pl, a_pool, cs = _tiny_pool_case(rng, D, 8, P, ties=bool(seed % 2))
    t = pool.plan_ctx(a_pool, cs, K, B)
    n = t["n_nodes"]
    assert 1 <= n <= B + 1
    for i in range(1, n):
        p = t["parent"][i]
        assert 0 <= p < i and t["depth"][i] == t["depth"][p] + 1 <= D
        assert t["score"][i] <= t["score"][p]
        assert 0 <= t["plan_slot"][i] < P
    for u in range(n):
        c, f = t["n_children"][u], t["first_child"][u]
        if c:
            assert list(t["rank"][f:f + c]) == list(range(c))
            # the children's planning slots are the parent's candidates in order
            slots, _ = pool.candidates(pool.corrected(a_pool, cs, int(t["depth"][u]), int(t["plan_slot"][u])), K)
            assert list(t["plan_slot"][f:f + c]) == slots[:c]
    assert all(np.diff(t["depth"]) >= 0) and all(np.diff(t["parent"][1:]) >= 0)


def test_context_changes_the_candidates():
    # slot 2 after slot 0 and slot 1 after slot 1 get a large transition score
    draft = np.array([[3.0, 2.0, 1.0, 0.0], [3.0, 2.0, 1.0, 0.0]], np.float32)
    trans = np.zeros((1, 3, 3), np.float32)
    trans[0, 0, 2] = 10.0
    trans[0, 1, 1] = 10.0
    pl = pool.pools(draft, 3)
    t = pool.plan_ctx(pool.pool_logits(draft, np.float32(1.0), pl), pool.scaled_corrections(trans, 1.0), 2, 4)
    # root children: slots 0, 1; the best child of each follows its own row of the table
    f = t["first_child"]
    assert list(t["plan_slot"][1:3]) == [0, 1]
    assert t["plan_slot"][f[1]] == 2 and t["plan_slot"][f[2]] == 1
    assert list(pool.plan_tokens(t, pl, t["plan_slot"])[f[1]:f[1] + 1]) == [2]


def _q_of_prefix(a_pool, cs, pl, V):
    def q(prefix):
        d = len(prefix)
        s = -1 if d == 0 else int(np.nonzero(pl[d - 1] == prefix[-1])[0][0])
        return pool.q_full(a_pool, cs, pl, d, s, V)
    return q


def _prefix_target(rng, V, D, scale=1.5):
    tab = {}
    for L in range(D + 1):
        for s in itertools.product(range(V), repeat=L):
            tab[s] = _softmax(rng.standard_normal(V) * scale)
    return lambda s: tab[tuple(s)]


def _check_lossless(tree, q, p_of, V, D):
    law = exact.emitted_law(tree, q, p_of)
    assert sum(law.values()) == pytest.approx(1.0, abs=1e-12)
    ext = exact.extend_law(law, p_of, D + 1)
    ref = exact.target_law(p_of, V, D + 1)
    for k in ref:
        assert ext.get(k, 0.0) == pytest.approx(ref[k], abs=1e-12)


def test_context_dependent_pool_round_is_lossless():
    rng = np.random.default_rng(204)
    V, D, P, K = 5, 3, 3, 2
    for B in (1, 3, 6):
        _, _, pl, a_pool, cs = _tiny_pool_case(rng, D, V, P)
        tree = pool.plan_ctx(a_pool, cs, K, B)
        _check_lossless(tree, _q_of_prefix(a_pool, cs, pl, V), _prefix_target(rng, V, D), V, D)


def test_verifier_ignoring_the_context_breaks_losslessness(monkeypatch):
    # replay draws from the corrected q_u, the planted verifier uses the
    # uncorrected pool distribution of the depth: the enumeration must catch it
    rng = np.random.default_rng(205)
    V, D, P, K = 5, 3, 3, 2
    _, _, pl, a_pool, cs = _tiny_pool_case(rng, D, V, P)
    tree = pool.plan_ctx(a_pool, cs, K, 6)
    q_true = _q_of_prefix(a_pool, cs, pl, V)
    q_flat = _q_of_prefix(a_pool, np.zeros_like(cs), pl, V)
    p_of = _prefix_target(rng, V, D)
    _check_lossless(tree, q_true, p_of, V, D)
    current = {}
    real_wor = exact._wor_orders

    def q_verified(prefix):
        current["prefix"] = prefix
        return q_flat(prefix)

    def drawn_with_context(qd, m):
        # called right after q_verified at the same node: draw from q_true
        return list(real_wor(q_true(current["prefix"]), m))

    monkeypatch.setattr(exact, "_wor_orders", drawn_with_context)
    with pytest.raises(AssertionError):
        _check_lossless(tree, q_verified, p_of, V, D)


def _round_law_case(trans_scale=1.5):
    rng = np.random.default_rng(206)
    V, D, P, K, B = 6, 2, 4, 2, 4
    draft = (rng.standard_normal((D, V)) * 2).astype(np.float32)
    trans = (rng.standard_normal((D - 1, P, P)) * trans_scale).astype(np.float32)
    pl = pool.pools(draft, P)
    a_pool, cs = pool.pool_logits(draft, np.float32(1.0), pl), pool.scaled_corrections(trans, 1.0)
    tab = {}
    for L in range(D + 1):
        for s in itertools.product(range(V), repeat=L):
            tab[s] = (rng.standard_normal(V) * 1.5).astype(np.float32)
    tree = pool.plan_ctx(a_pool, cs, K, B)
    law = exact.emitted_law(tree, _q_of_prefix(a_pool, cs, pl, V),
                            lambda s: _softmax(tab[tuple(s)].astype(np.float64)))
    return draft, trans, K, P, B, (lambda s: tab[tuple(s)]), law


def _empirical(draft, trans, K, P, B, p_of_rows, n):
    counts = {}
    for s in range(n):
        out = pool.step_pool_request(draft, None, trans, 1.0, K, P, B, 0x5EED, s, 3,
                                     target_fn=_target_fn(p_of_rows))
        seq = tuple(out["acc_tok"]) + (out["bonus"],)
        counts[seq] = counts.get(seq, 0) + 1
    return counts


def _chi2_pvalue(counts, law, n):
    keys = sorted(law, key=lambda k: -law[k])
    big = [k for k in keys if law[k] * n >= 5]
    small = [k for k in keys if law[k] * n < 5]
    assert set(counts) <= set(law), "an emitted sequence the exact law gives probability zero"
    obs = [counts.get(k, 0) for k in big] + [sum(counts.get(k, 0) for k in small)]
    exp_ = [law[k] * n for k in big] + [sum(law[k] for k in small) * n]
    return stats.chisquare(obs, exp_).pvalue


def test_sampling_round_follows_the_exact_law():
    draft, trans, K, P, B, p_of_rows, law = _round_law_case()
    n = 3000
    assert _chi2_pvalue(_empirical(draft, trans, K, P, B, p_of_rows, n), law, n) > 1e-3


def test_replay_ignoring_the_context_breaks_the_law(monkeypatch):
    draft, trans, K, P, B, p_of_rows, law = _round_law_case(trans_scale=4.0)
    real = pool.replay_pool

    def context_free(a_pool, cs, pl, tree, seed, step_, request):
        return real(a_pool, np.zeros_like(cs), pl, tree, seed, step_, request)

    monkeypatch.setattr(pool, "replay_pool", context_free)
    n = 3000
    assert _chi2_pvalue(_empirical(draft, trans, K, P, B, p_of_rows, n), law, n) < 1e-3


def test_replayed_tokens_are_distinct_pool_members():
    rng = np.random.default_rng(207)
    for _ in range(20):
        D, V, P = 3, 20, 6
        draft, trans, pl, a_pool, cs = _tiny_pool_case(rng, D, V, P)
        tree = pool.plan_ctx(a_pool, cs, 4, 15)
        tok, slot, _ = pool.replay_pool(a_pool, cs, pl, tree, 11, int(rng.integers(1 << 30)), 0)
        for u in range(tree["n_nodes"]):
            c, f = tree["n_children"][u], tree["first_child"][u]
            if c:
                kids = tok[f:f + c]
                assert len(set(kids.tolist())) == c
                d = tree["depth"][u]
                assert all(pl[d][slot[f:f + c]] == kids)


def test_status_bits():
    rng = np.random.default_rng(208)
    D, V, P = 2, 16, 4
    draft, trans, _, _, _ = _tiny_pool_case(rng, D, V, P)
    target = (rng.standard_normal((4, V))).astype(np.float32)
    bad = trans.copy()
    bad[0, 1, 2] = np.nan
    out = pool.step_pool_request(draft, target, bad, 1.0, 2, P, 3, 1, 0, 0)
    assert out["status"] & STATUS_NONFINITE and out["n_acc"] == -1 and out["tree"]["n_nodes"] == 1
    out = pool.step_pool_request(draft, np.zeros((40, V), np.float32), trans, 1.0, 2, P, 30, 1, 0, 0)
    assert out["status"] & STATUS_BUDGET_SHORT and out["tree"]["n_nodes"] == 1 + 2 + 4


def test_target_row_slip_below_the_root_breaks_the_law(monkeypatch):
    """A node other than the root verified against its parent's target row (a row-selection mistake below the
    root) must be caught by the sampled law of the whole emitted sequence."""
    draft, trans, K, P, B, p_of_rows, law = _round_law_case()
    real = pool.verify_mod.verify

    def slipped(p_rows, q_rows, tree, node_tok, seed, step_, request, q_node=None):
        par = tree["parent"]
        return real(lambda u: p_rows(int(par[u]) if u > 0 else 0), q_rows, tree, node_tok, seed, step_, request,
                    q_node)

    monkeypatch.setattr(pool.verify_mod, "verify", slipped)
    n = 3000
    counts = _empirical(draft, trans, K, P, B, p_of_rows, n)
    impossible = not set(counts) <= set(law)
    assert impossible or _chi2_pvalue(counts, law, n) < 1e-3
