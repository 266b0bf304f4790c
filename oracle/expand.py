"""Draft-side tree expansion (Algorithm 2, ExpandLayer), float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The draft model grows its proposal tree one layer at a time: every node of
the current frontier gets as children the top-k tokens of the draft's
next-token distribution q_t at that node, and the draft probability of each
child is kept with the tree (the correction step needs q_t).  Readings (the
paper states none of them): "top-k" ranks by the logit as a float32 value
(order keys, -0 below +0), equal logits by increasing token id; the children
of frontier node f are numbered first_child + f*k + j in rank order j, so a
tree built layer by layer lists parents before children; q(child) =
exp(logit - logsumexp(row)) of the row's float32 logits widened to float64.
"""

from __future__ import annotations

import numpy as np

from .warp import order_keys


def top_k_tokens(row32, k: int) -> np.ndarray:
    """The k highest-ranked token ids of one row, best first."""
    keys = order_keys(np.asarray(row32, dtype=np.float32)).astype(np.int64)
    ids = np.arange(keys.shape[0])
    order = np.lexsort((ids, -keys))          # key descending, then id ascending
    return order[:k]


def expand_layer(draft_logits, k: int, frontier0: int, first_child: int, N: int, tokens=None, parent=None,
                 q_child=None):
    """One ExpandLayer over B requests with F frontier nodes each.

    draft_logits [B][F][V] float32: row (b, f) is the draft's logits at
    frontier node frontier0 + f (frontier0 = -1: the frontier is the root).
    Writes entries first_child .. first_child + F*k - 1 of tokens, parent and
    q_child ([B][N] arrays, created filled with -1 / -1 / 0 when not given)
    and returns the three arrays.
    """
    x = np.asarray(draft_logits, dtype=np.float32)
    B, F, V = x.shape
    if not 1 <= k <= V or first_child + F * k > N:
        raise ValueError("need 1 <= k <= V and room for F*k children")
    if tokens is None:
        tokens = np.full((B, N), -1, dtype=np.int32)
        parent = np.full((B, N), -1, dtype=np.int32)
        q_child = np.zeros((B, N), dtype=np.float64)
    for b in range(B):
        for f in range(F):
            row = x[b, f].astype(np.float64)
            m = row.max()
            lse = m + np.log(np.exp(row - m).sum())
            best = top_k_tokens(x[b, f], k)
            for j, t in enumerate(best):
                n = first_child + f * k + j
                tokens[b, n] = int(t)
                parent[b, n] = -1 if frontier0 < 0 else frontier0 + f
                q_child[b, n] = np.exp(row[t] - lse)
    return tokens, parent, q_child


def full_tree_layout(k: int, depth: int):
    """(frontier0, first_child, F) of each layer of a full k-ary tree of the
    given depth numbered layer by layer, and the node count."""
    layers = []
    first, frontier0, F = 0, -1, 1
    for _ in range(depth):
        layers.append((frontier0, first, F))
        frontier0, first, F = first, first + F * k, F * k
    return layers, first
