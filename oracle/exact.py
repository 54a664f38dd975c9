"""Exact law of one replay-and-verify round, by enumeration (oracle side).

TEST INFRASTRUCTURE ONLY: used by the tests to check the losslessness claim
(Section 3.3, Proposition 1) with no random numbers at all.

For a fixed topology, a draft table q[d] (or a draft distribution keyed by
the replayed prefix) and a prefix-keyed target p(. | s), every random choice
of the round is enumerated:
  * replay draws at each parent u: ordered samples without replacement from
    q[depth(u)] with Plackett-Luce weight prod_j q(y_j) / (1 - sum_{i<j} q(y_i))
    (Appendix A, sampling without replacement);
  * each acceptance test: accept child j with probability min{1, ratio_j},
    ratios and residual updates taken from oracle.verify (the same code the
    sampling oracle runs);
  * the bonus token: the normalised final residual (or p at a leaf).
Subtrees that the walk never enters are marginalised out, which is exact
because the draws of different parents are independent.

naive_law() enumerates target-sample matching (Table 2, Naive) over a tree
whose node tokens are fixed (the First tree of Section 3.1): at each visited
node every token of p_u either matches a child and continues there, or ends
the round as the bonus.

traversal_law() enumerates a round verified by traversal (Appendix A; Table
2): the traversal starts below the root and can visit every node, so the
replay draws of every parent are enumerated (Plackett-Luce weights as
above), and for each complete assignment every accept/reject branch of the
traversal, with the updates taken from oracle.traversal.
"""
import itertools

import numpy as np

from . import traversal as trav_mod
from . import verify as verify_mod


def _wor_orders(q, m):
    """All ordered m-samples without replacement from q with their probabilities."""
    V = q.shape[0]
    for seq in itertools.permutations(range(V), m):
        w = 1.0
        used = 0.0
        for y in seq:
            rem = 1.0 - used
            if rem <= 0.0 or q[y] <= 0.0:
                w = 0.0
                break
            w *= q[y] / rem
            used += q[y]
        if w > 0.0:
            yield seq, w


def emitted_law(tree, q, p_of_prefix):
    """Exact distribution of the emitted sequence (accepted tokens + bonus).

    tree: BFS topology dict (n_children, first_child, depth).
    q: array [D, V] of draft distributions per depth, or a callable
       q(prefix) -> draft distribution of the children of the node reached
       by that token prefix (a drafter conditioned on the replayed prefix,
       eq. (2)).
    p_of_prefix(tuple) -> target distribution after that token prefix.
    Returns dict {tuple(sequence): probability}.
    """
    law = {}

    def add(seq, w):
        law[seq] = law.get(seq, 0.0) + w

    def at_node(u, prefix, weight):
        m = int(tree["n_children"][u])
        p_u = np.asarray(p_of_prefix(prefix), dtype=np.float64)
        if m == 0:
            for v in range(p_u.shape[0]):
                if p_u[v] > 0:
                    add(prefix + (v,), weight * p_u[v])
            return
        qd = np.asarray(q(prefix) if callable(q) else q[int(tree["depth"][u])], dtype=np.float64)
        fc = int(tree["first_child"][u])
        for seq, w_draw in _wor_orders(qd, m):
            P, Q = p_u.copy(), qd.copy()
            reach = weight * w_draw
            degenerate = False
            for j, y in enumerate(seq):
                ratio = verify_mod.accept_ratio(P, Q, y)
                pa = min(1.0, ratio)
                if pa > 0.0:
                    at_node(fc + j, prefix + (y,), reach * pa)
                reach *= (1.0 - pa)
                if reach == 0.0:
                    break
                P, Q, Z, S = verify_mod.reject(P, Q, y)
                if Z <= 0.0 or (j + 1 < m and S <= 0.0):
                    degenerate = True
                    break
            if reach == 0.0:
                continue
            final = p_u if degenerate else P
            tot = final.sum()
            for v in range(final.shape[0]):
                if final[v] > 0:
                    add(prefix + (v,), reach * final[v] / tot)

    at_node(0, (), 1.0)
    return law


def extend_law(law, p_of_prefix, length):
    """Continue every emitted sequence by sampling the target up to `length` tokens."""
    out = {}
    stack = list(law.items())
    while stack:
        seq, w = stack.pop()
        if len(seq) >= length:
            key = seq[:length]
            out[key] = out.get(key, 0.0) + w
            continue
        p = np.asarray(p_of_prefix(seq), dtype=np.float64)
        for v in range(p.shape[0]):
            if p[v] > 0:
                stack.append((seq + (v,), w * p[v]))
    return out


def target_law(p_of_prefix, V, length):
    """Law of `length` tokens sampled autoregressively from the target."""
    out = {}
    for seq in itertools.product(range(V), repeat=length):
        w = 1.0
        for i in range(length):
            w *= p_of_prefix(seq[:i])[seq[i]]
        out[seq] = w
    return out


def naive_law(tree, node_tok, p_of_prefix):
    """Exact law of the emitted sequence under target-sample matching on fixed node tokens."""
    law = {}

    def walk(u, prefix, w):
        p = np.asarray(p_of_prefix(prefix), dtype=np.float64)
        m = int(tree["n_children"][u])
        fc = int(tree["first_child"][u])
        child_of = {}
        for j in range(m):
            child_of.setdefault(int(node_tok[fc + j]), fc + j)
        for y in range(p.shape[0]):
            if p[y] <= 0.0:
                continue
            if y in child_of:
                walk(child_of[y], prefix + (y,), w * p[y])
            else:
                seq = prefix + (y,)
                law[seq] = law.get(seq, 0.0) + w * p[y]

    walk(0, (), 1.0)
    return law


def traversal_law(tree, q, p_of_prefix):
    """Exact distribution of the emitted sequence of a round verified by traversal.

    tree, q, p_of_prefix as in emitted_law (q: [D, V] per depth or a callable
    of the replayed prefix). Returns dict {tuple(sequence): probability}.
    """
    n = int(tree["n_nodes"])
    n_children, first_child, parent, depth = (tree["n_children"], tree["first_child"], tree["parent"],
                                             tree["depth"])
    internal = [u for u in range(n) if int(n_children[u]) > 0]
    law = {}

    def add(seq, w):
        law[seq] = law.get(seq, 0.0) + w

    def prefix_of(u, tok):
        path = []
        while u > 0:
            path.append(int(tok[u]))
            u = int(parent[u])
        return tuple(reversed(path))

    def q_at(u, tok):
        return np.asarray(q(prefix_of(u, tok)) if callable(q) else q[int(depth[u])], dtype=np.float64)

    def p_at(u, tok):
        return np.asarray(p_of_prefix(prefix_of(u, tok)), dtype=np.float64)

    def emit(u, P, tok, w):
        pre = prefix_of(u, tok)
        tot = P.sum()
        for v in range(P.shape[0]):
            if P[v] > 0:
                add(pre + (v,), w * P[v] / tot)

    def branch(tok, Mb, Ms, alpha, left, path, w):
        """Continue the traversal from the current state with probability weight w."""
        while True:
            u = path[-1]
            if left[u] < int(n_children[u]):
                c = int(first_child[u]) + left[u]
                alpha[c] = trav_mod.child_alpha(alpha[u], Mb[u], Ms[u], int(tok[c]))
                Mb[c] = p_at(c, tok)
                Ms[c] = q_at(c, tok) if int(n_children[c]) > 0 else None
                left[c] = 0
                path.append(c)
                continue
            if u == 0:
                emit(0, Mb[0], tok, w)
                return
            a = alpha[u]
            if a > 0.0:
                emit(u, Mb[u], tok, w * a)
            if a >= 1.0:
                return
            w *= 1.0 - a
            path.pop()
            v = path[-1]
            a_new, Mb_new, Ms_new, T, S = trav_mod.reject_child(alpha[v], Mb[v], Ms[v], int(tok[u]))
            left[v] += 1
            if (T <= 0.0 and alpha[v] >= 1.0) or (S <= 0.0 and left[v] < int(n_children[v])):
                emit(v, p_at(v, tok), tok, w)
                return
            alpha[v], Mb[v], Ms[v] = a_new, Mb_new, Ms_new

    def assign(i, tok, w):
        if i == len(internal):
            root_q = q_at(0, tok) if int(n_children[0]) > 0 else None
            branch(tok, {0: p_at(0, tok)}, {0: root_q}, {0: 1.0}, {0: 0}, [0], w)
            return
        u = internal[i]
        m = int(n_children[u])
        fc = int(first_child[u])
        for seq, w_draw in _wor_orders(q_at(u, tok), m):
            t2 = tok.copy()
            t2[fc:fc + m] = seq
            assign(i + 1, t2, w * w_draw)

    assign(0, np.full(n, -1, np.int64), 1.0)
    return law
