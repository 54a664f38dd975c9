"""Losslessness of the oracle's round (Section 3.3, Proposition 1).

Exact enumeration (no random numbers) at V=4, D=3, B<=6 on the paper's
Figure 1 topology and on planner-produced topologies: the law of the emitted
sequence, continued by target sampling to D+1 tokens, equals the target's own
law prod_i p(s_i | s_<i) to 1e-12. The target is prefix-keyed, built per
token path as a target model would. A planted mistake in the residual update
must break the equality. Sampling checks run the Philox-driven oracle through
step.step_request: the whole emitted sequence against the enumerated law of
the same round (V=5), and the first two emitted tokens against p(a) p(b | a)
of the prefix-keyed target (V=64); a node verified against its parent's
target row, or against the wrong draft row, must fail them.
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


def _path_target(table):
    """Target rows built after replay from each node's token path (prefix-keyed), as a target model would."""
    def target_fn(tree, node_tok):
        rows = []
        for u in range(tree["n_nodes"]):
            path, w = [], u
            while w > 0:
                path.append(int(node_tok[w]))
                w = int(tree["parent"][w])
            rows.append(table(tuple(reversed(path))))
        return np.stack(rows)
    return target_fn


def _logit_table(rng, V, scale=1.5):
    tab = {}

    def p_of(s):
        s = tuple(s)
        if s not in tab:
            tab[s] = (rng.standard_normal(V) * scale).astype(np.float32)
        return tab[s]
    return p_of


@pytest.fixture
def parent_row_slip(monkeypatch):
    """A plausible mistake below the root: a node other than the root is verified against its parent's
    target row (the root's own row is untouched, so every first emitted token keeps its law)."""
    real = step.verify_request

    def slipped(draft, target, tree, node_tok, lse, T, seed, step_, request, verifier="rrs"):
        t = np.array(target, copy=True)
        for u in range(1, tree["n_nodes"]):
            t[u] = target[int(tree["parent"][u])]
        return real(draft, t, tree, node_tok, lse, T, seed, step_, request, verifier)
    monkeypatch.setattr(step, "verify_request", slipped)


@pytest.fixture
def draft_row_slip(monkeypatch):
    """A mistake in the draft row a node's children are verified with: always row 0 instead of depth(u)."""
    real = verify.verify

    def slipped(p_rows, q_rows, tree, node_tok, seed, step_, request, q_node=None):
        return real(p_rows, lambda d: q_rows(0), tree, node_tok, seed, step_, request, q_node)
    monkeypatch.setattr(verify, "verify", slipped)


def _small_round_case():
    rng = np.random.default_rng(104)
    V, D, B, K = 5, 3, 6, 3
    draft = (rng.standard_normal((D, V)) * 1.2).astype(np.float32)
    table = _logit_table(rng, V)
    pl = step.plan_request(draft, 1.0, K, B)
    q = np.stack([np.exp(draft[d].astype(np.float64) - pl["lse64"][d]) for d in range(D)])
    law = exact.emitted_law(pl["tree"], q, lambda s: _softmax(table(s).astype(np.float64)))
    return draft, table, K, B, law


def _round_pvalue(draft, table, K, B, law, n=4000):
    counts = {}
    for s in range(n):
        out = step.step_request(draft, None, 1.0, K, B, seed=0x51CE, step=s, request=2,
                                target_fn=_path_target(table))
        seq = tuple(out["acc_tok"]) + (out["bonus"],)
        counts[seq] = counts.get(seq, 0) + 1
    if not set(counts) <= set(law):
        return 0.0  # an emitted sequence the exact law gives probability zero
    keys = sorted(law, key=lambda k: -law[k])
    big = [k for k in keys if law[k] * n >= 5]
    small = [k for k in keys if law[k] * n < 5]
    obs = [counts.get(k, 0) for k in big] + [sum(counts.get(k, 0) for k in small)]
    exp_ = [law[k] * n for k in big] + [sum(law[k] for k in small) * n]
    return stats.chisquare(obs, exp_).pvalue


def test_sampling_round_follows_the_exact_law():
    """The whole emitted sequence of step_request (plan, replay with Philox draws, the walk with its row
    selection at every visited node, the bonus) against the enumerated law of the same round."""
    draft, table, K, B, law = _small_round_case()
    assert max(len(k) for k in law) >= 3          # accepted paths reach depth 2: rows below the root are used
    assert _round_pvalue(draft, table, K, B, law) > 1e-3


def test_round_law_catches_a_target_row_slip_below_the_root(parent_row_slip):
    draft, table, K, B, law = _small_round_case()
    assert _round_pvalue(draft, table, K, B, law) < 1e-3


def test_round_law_catches_a_draft_row_slip(draft_row_slip):
    draft, table, K, B, law = _small_round_case()
    assert _round_pvalue(draft, table, K, B, law) < 1e-3


def _first_two(n, seed=103):
    """First two tokens of n sampled rounds at V = 64 through step_request (a one-token output is continued by
    one target draw, as decoding would), with the prefix-keyed target table."""
    rng = np.random.default_rng(seed)
    V, D, B, K = 64, 3, 6, 3
    draft = (rng.standard_normal((D, V)) * 1.5).astype(np.float32)
    table = _logit_table(rng, V)
    ext = np.random.default_rng(seed + 1)
    pairs = np.zeros((V, V))
    for s in range(n):
        out = step.step_request(draft, None, 1.0, K, B, seed=0xABC, step=s, request=0,
                                target_fn=_path_target(table))
        seq = list(out["acc_tok"]) + [out["bonus"]]
        if len(seq) == 1:
            seq.append(int(ext.choice(V, p=_softmax(table((seq[0],)).astype(np.float64)))))
        pairs[seq[0], seq[1]] += 1
    p0 = _softmax(table(()).astype(np.float64))
    joint = p0[:, None] * np.stack([_softmax(table((a,)).astype(np.float64)) for a in range(V)])
    return pairs, p0, joint


def _binned_pvalue(obs, exp_):
    obs, exp_ = obs.ravel(), exp_.ravel()
    big = exp_ >= 5
    return stats.chisquare(np.r_[obs[big], obs[~big].sum()], np.r_[exp_[big], exp_[~big].sum()]).pvalue


def test_chi2_first_two_tokens_v64():
    """Law of the first emitted token against p(.) and of the first two against p(a) p(b | a) of the
    prefix-keyed target (Section 3.3, Proposition 1), through step_request."""
    n = 6000
    pairs, p0, joint = _first_two(n)
    assert _binned_pvalue(pairs.sum(axis=1), p0 * n) > 1e-3
    assert _binned_pvalue(pairs, joint * n) > 1e-3


def test_chi2_first_two_tokens_catches_a_row_slip_below_the_root(parent_row_slip):
    n = 6000
    pairs, p0, joint = _first_two(n)
    assert _binned_pvalue(pairs.sum(axis=1), p0 * n) > 1e-3     # the root is untouched
    assert _binned_pvalue(pairs, joint * n) < 1e-3              # the second token is not
