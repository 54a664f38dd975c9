"""Pins of the First + Naive oracle (Section 3.1; Table 2, Naive).

* first_tokens: each node carries the planning candidate of its depth and
  rank; siblings take the top-m candidates of their position in rank order,
  checked against a brute-force enumeration of the best rank paths.
* Exact losslessness of target-sample matching: the law of the emitted
  sequence (enumerated, no random numbers), continued by target sampling to
  D + 1 tokens, equals the target's own law to 1e-12, on the Figure 1
  topology with arbitrary sibling tokens and on First trees.
* The sampling oracle against that law: chi^2 of the emitted sequences over
  many Philox steps; a planted greedy draw must fail it.
* Special cases: B = 0 reduces to one target sample, the same draw as the
  RRS bonus at a leaf; near-zero temperature with draft = target accepts the
  whole rank-0 chain and emits the target argmax as bonus.
"""
import itertools

import numpy as np
import pytest
from scipy import stats

from oracle import exact, naive, philox, planner, step, verify
from oracle.rowstats import inv_temperature, lse64, probs, scaled

from test_oracle_lossless import _figure1_tree, _prefix_target, _softmax


def _check_naive_lossless(tree, node_tok, p_of, V, D):
    law = exact.naive_law(tree, node_tok, p_of)
    assert sum(law.values()) == pytest.approx(1.0, abs=1e-12)
    ext = exact.extend_law(law, p_of, D + 1)
    ref = exact.target_law(p_of, V, D + 1)
    for k in ref:
        assert ext.get(k, 0.0) == pytest.approx(ref[k], abs=1e-12)
    return law


def _random_sibling_tokens(tree, V, rng):
    tok = np.full(tree["n_nodes"], -1, np.int64)
    for u in range(tree["n_nodes"]):
        m = int(tree["n_children"][u])
        if m:
            fc = int(tree["first_child"][u])
            tok[fc:fc + m] = rng.choice(V, size=m, replace=False)
    return tok


def test_first_tokens_follow_best_rank_paths():
    rng = np.random.default_rng(200)
    V, D, K = 40, 3, 3
    draft = (rng.standard_normal((D, V)) * 2.0).astype(np.float32)
    for B in (1, 4, 9, 20, 39):
        pl = step.plan_request(draft, 1.0, K, B)
        tree = pl["tree"]
        tok = naive.first_tokens(tree, pl["topk_tok"])
        # brute force: all rank paths, best B by (score desc, depth asc, ranks lex asc)
        lp = pl["topk_lp"].astype(np.float64)
        paths = []
        for L in range(1, D + 1):
            for r in itertools.product(range(K), repeat=L):
                paths.append((-sum(float(lp[d, r[d]]) for d in range(L)), L, r))
        paths.sort()
        want = {tuple(int(pl["topk_tok"][d, r[d]]) for d in range(L)) for _, L, r in paths[:B]}
        got = set()
        for u in range(1, tree["n_nodes"]):
            path, w = [], u
            while w > 0:
                path.append(int(tok[w]))
                w = int(tree["parent"][w])
            got.add(tuple(reversed(path)))
        assert got == want
        assert tok[0] == -1
        for u in range(tree["n_nodes"]):
            m = int(tree["n_children"][u])
            fc = int(tree["first_child"][u])
            if m:
                d = int(tree["depth"][u])
                assert list(tok[fc:fc + m]) == list(pl["topk_tok"][d, :m])


def test_naive_figure1_lossless_any_sibling_tokens():
    rng = np.random.default_rng(201)
    V, D = 4, 3
    tree = _figure1_tree()
    for _ in range(4):
        tok = _random_sibling_tokens(tree, V, rng)
        _check_naive_lossless(tree, tok, _prefix_target(rng, V, D), V, D)


def test_naive_first_trees_lossless():
    rng = np.random.default_rng(202)
    V, D, K = 4, 3, 3
    for B in range(0, 10):
        draft = (rng.standard_normal((D, V)) * 1.5).astype(np.float32)
        pl = step.plan_request(draft, 1.0, K, B)
        tok = naive.first_tokens(pl["tree"], pl["topk_tok"])
        _check_naive_lossless(pl["tree"], tok, _prefix_target(rng, V, D), V, D)


def test_planted_matching_mistake_breaks_exact_law(monkeypatch):
    # Plant a plausible slip in the enumeration (the walk continues at the
    # first child whatever token was drawn) and check that the law breaks.
    rng = np.random.default_rng(203)
    V, D = 4, 3
    tree = _figure1_tree()
    tok = _random_sibling_tokens(tree, V, rng)
    p_of = _prefix_target(rng, V, D)
    bad_tok = tok.copy()
    for u in range(tree["n_nodes"]):
        m = int(tree["n_children"][u])
        if m > 1:
            fc = int(tree["first_child"][u])
            bad_tok[fc + 1] = bad_tok[fc]      # a duplicated sibling token: second child unreachable
    law_bad = exact.naive_law(tree, bad_tok, p_of)
    law_ok = exact.naive_law(tree, tok, p_of)
    # still a distribution and still lossless (matching is lossless for any tokens) ...
    _check_naive_lossless(tree, bad_tok, p_of, V, D)
    # ... but a different emitted law; the planted slip below is the one that must fail
    assert any(abs(law_bad.get(k, 0.0) - law_ok.get(k, 0.0)) > 1e-6 for k in set(law_ok) | set(law_bad))

    def greedy_walk(u, prefix, w, law, p_of=p_of):
        p = np.asarray(p_of(prefix))
        y = int(np.argmax(p))
        m = int(tree["n_children"][u])
        fc = int(tree["first_child"][u])
        for j in range(m):
            if int(tok[fc + j]) == y:
                return greedy_walk(fc + j, prefix + (y,), w, law)
        law[prefix + (y,)] = law.get(prefix + (y,), 0.0) + w

    law_greedy = {}
    greedy_walk(0, (), 1.0, law_greedy)
    monkeypatch.setattr(exact, "naive_law", lambda t, n, p: law_greedy)
    with pytest.raises(AssertionError):
        _check_naive_lossless(tree, tok, p_of, V, D)


def _sample_law(tree, tok, target_rows, n, seed, request=0):
    counts = {}
    for s in range(n):
        r = naive.verify_naive(target_rows, tree, tok, 1.0, seed, s, request)
        seq = tuple(r["acc_tok"]) + (r["bonus"],)
        counts[seq] = counts.get(seq, 0) + 1
    return counts


def _chi2_p(counts, law, n):
    keys = sorted(law, key=lambda k: -law[k])
    big = [k for k in keys if law[k] * n >= 5]
    small = [k for k in keys if law[k] * n < 5]
    obs = [counts.get(k, 0) for k in big] + [sum(counts.get(k, 0) for k in small)]
    exp_ = [law[k] * n for k in big] + [sum(law[k] for k in small) * n]
    assert sum(counts.values()) == n
    assert all(k in law for k in counts)
    if exp_[-1] == 0:
        obs, exp_ = obs[:-1], exp_[:-1]
    return stats.chisquare(obs, exp_).pvalue


def _tree_target_rows(tree, tok, p_logits):
    rows = []
    for u in range(tree["n_nodes"]):
        path, w = [], u
        while w > 0:
            path.append(int(tok[w]))
            w = int(tree["parent"][w])
        rows.append(p_logits(tuple(reversed(path))))
    return np.stack(rows).astype(np.float32)


def _logit_table(rng, V):
    tab = {}

    def x_of(s):
        if s not in tab:
            tab[s] = (rng.standard_normal(V) * 1.5).astype(np.float32)
        return tab[s]
    return x_of


def test_sampling_oracle_matches_exact_law():
    rng = np.random.default_rng(204)
    V, D = 4, 3
    tree = _figure1_tree()
    tok = _random_sibling_tokens(tree, V, rng)
    x_of = _logit_table(rng, V)
    rows = _tree_target_rows(tree, tok, x_of)
    invT = inv_temperature(1.0)

    def p_of(s):
        a = scaled(x_of(tuple(s)), invT)
        return probs(a, lse64(a))
    law = exact.naive_law(tree, tok, p_of)
    n = 6000
    assert _chi2_p(_sample_law(tree, tok, rows, n, 0x5EED), law, n) > 1e-3


def test_planted_greedy_draw_fails_chi2(monkeypatch):
    rng = np.random.default_rng(205)
    V, D = 4, 3
    tree = _figure1_tree()
    tok = _random_sibling_tokens(tree, V, rng)
    x_of = _logit_table(rng, V)
    rows = _tree_target_rows(tree, tok, x_of)
    invT = inv_temperature(1.0)

    def p_of(s):
        a = scaled(x_of(tuple(s)), invT)
        return probs(a, lse64(a))
    law = exact.naive_law(tree, tok, p_of)
    monkeypatch.setattr(naive, "target_sample", lambda a, *k: (int(np.argmax(a)), 1.0))
    n = 2000
    with pytest.raises(AssertionError):
        assert _chi2_p(_sample_law(tree, tok, rows, n, 0x5EED), law, n) > 1e-3


def test_root_only_budget_is_one_target_sample():
    rng = np.random.default_rng(206)
    V = 50
    tree = planner.plan(np.zeros((0, 2), np.float32), 0)
    for s in range(20):
        x = (rng.standard_normal((1, V)) * 2).astype(np.float32)
        r = naive.verify_naive(x, tree, np.array([-1]), 0.8, 7, s, 3)
        invT = inv_temperature(0.8)
        a = scaled(x[0], invT)
        y, _ = verify.bonus_sample(probs(a, lse64(a)), 7, s, 3, 0)
        assert r["n_acc"] == 0 and r["bonus"] == y and r["terminal"] == 0


def test_near_zero_temperature_accepts_rank0_chain():
    rng = np.random.default_rng(207)
    V, D, K, B = 64, 4, 3, 12
    T = 1e-6
    for s in range(4):
        draft = (rng.standard_normal((D, V)) * 2).astype(np.float32)
        pl = step.plan_request(draft, T, K, B)
        tree = pl["tree"]
        tok = naive.first_tokens(tree, pl["topk_tok"])
        # target at a node of depth d < D is the draft row d; at depth D a fresh row
        leaf_row = (rng.standard_normal(V) * 2).astype(np.float32)
        rows = np.stack([draft[int(tree["depth"][u])] if int(tree["depth"][u]) < D else leaf_row
                         for u in range(tree["n_nodes"])])
        r = naive.verify_naive(rows, tree, tok, T, 11, s, 0)
        assert r["n_acc"] == D
        assert r["acc_tok"] == [int(np.argmax(draft[d])) for d in range(D)]
        assert r["bonus"] == int(np.argmax(leaf_row))


def test_nonfinite_visited_row_sets_status():
    V = 16
    tree = planner.plan(np.log(np.full((2, 2), 0.5, np.float32)), 3)
    tok = naive.first_tokens(tree, np.array([[0, 1], [2, 3]]))
    rows = np.zeros((tree["n_nodes"], V), np.float32)
    rows[0, 5] = np.nan
    r = naive.verify_naive(rows, tree, tok, 1.0, 1, 0, 0)
    assert r["status"] == 1 and r["n_acc"] == -1 and r["bonus"] == -1


def test_first_naive_round_first_token_chi2_v64():
    rng = np.random.default_rng(208)
    V, D, B, K = 64, 3, 6, 3
    draft = (rng.standard_normal((D, V)) * 1.5).astype(np.float32)
    target = (rng.standard_normal((B + 1, V)) * 1.5).astype(np.float32)
    n = 4000
    first = np.zeros(V)
    for s in range(n):
        out = naive.first_naive_request(draft, target, 1.0, K, B, seed=0xF1, step=s, request=0)
        seq = list(out["acc_tok"]) + [out["bonus"]]
        first[seq[0]] += 1
    p0 = _softmax(target[0].astype(np.float64))
    big = p0 * n >= 5
    obs = np.r_[first[big], first[~big].sum()]
    exp_ = np.r_[p0[big] * n, p0[~big].sum() * n]
    assert stats.chisquare(obs, exp_).pvalue > 1e-3
