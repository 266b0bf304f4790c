"""Pins of oracle.expand (Algorithm 2, ExpandLayer):

* top-k against rank counting on small rows with ties and signed zeros:
  rank(t) = #{u : x_u > x_t in float32 order, or x_u == x_t and u < t};
  the children are the tokens of rank < k in rank order;
* the children's draft probabilities against scipy's softmax, and the
  probabilities of all V children of a row summing to one;
* a depth-3 tree grown layer by layer from a path-dependent draft table:
  parents precede children, and its root-to-leaf token paths are exactly
  the k^d paths a brute-force recursion over top-k choices gives;
* argument checks (k outside [1, V], too few node slots)."""

import itertools

import numpy as np
import pytest
from scipy.special import softmax

from oracle.expand import expand_layer, full_tree_layout, top_k_tokens


def _rank_topk(row, k):
    r32 = np.asarray(row, dtype=np.float32)
    V = len(r32)

    def greater(u, t):   # float32 order with -0 below +0
        a, b = float(r32[u]), float(r32[t])
        if a != b:
            return a > b
        if a == 0.0 and b == 0.0:
            return (not np.signbit(r32[u])) and np.signbit(r32[t])
        return False

    rank = [sum(1 for u in range(V) if greater(u, t) or (r32[u] == r32[t] and np.signbit(r32[u]) ==
                                                           np.signbit(r32[t]) and u < t)) for t in range(V)]
    return [t for _, t in sorted((rank[t], t) for t in range(V) if rank[t] < k)]


def test_top_k_matches_rank_counting():
    rng = np.random.default_rng(0)
    for _ in range(300):
        V = int(rng.integers(1, 9))
        row = rng.choice([-1.5, -0.0, 0.0, 0.25, 2.0, 3.0], size=V).astype(np.float32)
        for k in range(1, V + 1):
            assert top_k_tokens(row, k).tolist() == _rank_topk(row, k), (row, k)


def test_signed_zero_and_ties():
    row = np.array([0.0, -0.0, 1.0, 1.0], dtype=np.float32)
    row[1] = -0.0
    assert top_k_tokens(row, 4).tolist() == [2, 3, 0, 1]


def test_child_probabilities():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal((2, 3, 50)) * 3).astype(np.float32)
    tok, par, q = expand_layer(x, 50, frontier0=4, first_child=0, N=150)
    for b in range(2):
        for f in range(3):
            sl = slice(f * 50, (f + 1) * 50)
            assert abs(q[b, sl].sum() - 1.0) < 1e-12
            assert np.allclose(q[b, sl], softmax(x[b, f].astype(np.float64))[tok[b, sl]], rtol=1e-12)
            assert np.all(par[b, sl] == 4 + f)


def test_layer_by_layer_tree_equals_brute_force_paths():
    k, depth, V = 2, 3, 6
    rng = np.random.default_rng(2)
    table = {}

    def draft(path):   # the draft's logits after a token path (a fixed random table)
        if path not in table:
            table[path] = rng.standard_normal(V).astype(np.float32)
        return table[path]

    layers, N = full_tree_layout(k, depth)
    assert [l[:2] for l in layers] == [(-1, 0), (0, 2), (2, 6)] and N == 14
    tok = par = q = None
    path_of = {-1: ()}
    for frontier0, first, F in layers:
        nodes = [-1] if frontier0 < 0 else list(range(frontier0, frontier0 + F))
        logits = np.stack([draft(path_of[n]) for n in nodes])[None]
        tok, par, q = expand_layer(logits, k, frontier0, first, N, tok, par, q)
        for n in range(first, first + F * k):
            path_of[n] = path_of[int(par[0, n])] + (int(tok[0, n]),)
    assert all(par[0, n] < n for n in range(N))
    leaves = {path_of[n] for n in range(N - k ** depth, N)}

    def brute(path, d):
        if d == 0:
            return [path]
        out = []
        for t in top_k_tokens(draft(path), k):
            out += brute(path + (int(t),), d - 1)
        return out

    assert leaves == set(brute((), depth)) and len(leaves) == k ** depth


def test_argument_checks():
    x = np.zeros((1, 1, 4), dtype=np.float32)
    with pytest.raises(ValueError):
        expand_layer(x, 5, -1, 0, 8)
    with pytest.raises(ValueError):
        expand_layer(x, 0, -1, 0, 8)
    with pytest.raises(ValueError):
        expand_layer(x, 3, -1, 6, 8)
