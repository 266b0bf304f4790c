"""Tree verification, float64: tree-masked attention and lossless acceptance
of a candidate tree.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Source: Algorithm 2 and the paragraphs after it.  The drafter expands a
proposal tree whose every node carries the top-k candidates for the next
token (ExpandLayer); the target scores every node's prefix in one forward
pass, each node attending to the verified prefix, the root (the last verified
token) and its own ancestors.  The paper then tests every root-to-leaf path on
its own and keeps the longest, which does not preserve the target
distribution (a reading recorded in the design notes: with two candidates the
emitted token can follow (0.7, 0.3) for p = (0.5, 0.5)).  This module
verifies the tree losslessly instead, treating the candidates of a node as
point-mass proposals in the Leviathan test the paper adopts (Sec. 2): at a
node with target distribution p,
  * its children c_1, c_2, ... are tested in increasing node index; child c_j
    passes iff u[c_j] < p(c_j) / (1 - sum of p over the children rejected
    before it) (a candidate token seen earlier among its siblings has mass 0);
  * the first child that passes is accepted and the walk continues at it;
  * if every child is rejected, the final token is drawn from p with the
    rejected candidates removed (renormalised), by inverse CDF with the final
    draw u[N]; at a node without children (a leaf, or the root of an empty
    tree) the final token is a bonus drawn from p itself.
Each emitted token is then distributed exactly as the target's next-token
distribution, so the sequence is.  The draft distributions q are not used:
the candidate set of a node is what the drafter chose.

Layout (N nodes, G = N + 1 positions): position 0 is the root, position i + 1
is node i; parent[i] in [-1, i) is the parent node (-1: the root); the rows of
p and the query positions follow the positions; tokens[i] is node i's token;
u[i] tests node i and u[N] drives the final sample.
"""

from __future__ import annotations

from typing import List, Tuple

import numpy as np

from .accept import FINAL_BAND, RATIO_BAND


def ancestor_masks(parent) -> np.ndarray:
    """[G] uint64: bit a of mask[g] is set iff position a is position g itself,
    the root or an ancestor of it."""
    parent = np.asarray(parent, dtype=np.int64)
    N = parent.shape[0]
    masks = np.zeros(N + 1, dtype=np.uint64)
    masks[0] = np.uint64(1)
    for i in range(N):
        pp = int(parent[i])
        if not -1 <= pp < i:
            raise ValueError("parents must precede their children")
        masks[i + 1] = masks[pp + 1] | (np.uint64(1) << np.uint64(i + 1))
    return masks


def tree_attention(q, k_pool, v_pool, kv_off, kv_len, n_kv_heads, parent, scale=None):
    """Attention of the G = N + 1 tree positions of each request.

    Same layout as oracle.attention.verify_attention (q [B][G][Hq][D]; the
    request's cache [Hkv][L][D] at kv_off, its last G entries being the root
    and the nodes in position order); parent [B][N].  Position g sees the
    prefix keys 0 .. L - G - 1 and the tail key L - G + a iff bit a of its
    ancestor mask is set.
    """
    q = np.asarray(q, dtype=np.float64)
    B, G, Hq, D = q.shape
    Hkv = n_kv_heads
    group = Hq // Hkv
    scale = 1.0 / np.sqrt(D) if scale is None else scale
    out = np.empty_like(q)
    k_pool = np.asarray(k_pool)
    v_pool = np.asarray(v_pool)
    for b in range(B):
        L = int(kv_len[b])
        off = int(kv_off[b])
        K = k_pool[off:off + Hkv * L * D].reshape(Hkv, L, D).astype(np.float64)
        V = v_pool[off:off + Hkv * L * D].reshape(Hkv, L, D).astype(np.float64)
        masks = ancestor_masks(parent[b])
        for g in range(G):
            vis = np.zeros(L, dtype=bool)
            vis[:L - G] = True
            for a in range(G):
                if (int(masks[g]) >> a) & 1:
                    vis[L - G + a] = True
            for h in range(Hq):
                kh = h // group
                s = (K[kh][vis] @ q[b, g, h]) * scale
                w = np.exp(s - s.max())
                out[b, g, h] = (w / w.sum()) @ V[kh][vis]
    return out


def accept_tree_request(p_rows, tokens, parent, u) -> Tuple[List[int], List[int], int, dict]:
    """Verify one request's tree.

    p_rows [G][V]: target distribution at each position (row 0: after the root);
    tokens [N], parent [N], u [G].  Returns (path, emitted, final_row, trace):
    the accepted nodes in order, the emitted tokens (their tokens, then the
    final one), the position whose row the final token was drawn from, and
    the values the decision band needs.
    """
    p_rows = np.asarray(p_rows, dtype=np.float64)
    G, V = p_rows.shape
    N = G - 1
    children = [[] for _ in range(G)]            # by position
    for i in range(N):
        children[int(parent[i]) + 1].append(i)
    pos = 0
    path: List[int] = []
    tests = []                                   # (u, threshold) of every test made
    while True:
        p = p_rows[pos]
        rejected_mass = 0.0
        rejected_tok: List[int] = []
        accepted = None
        for c in children[pos]:
            t = int(tokens[c])
            if t in rejected_tok or not 0 <= t < V:
                thr = 0.0
            else:
                rest = 1.0 - rejected_mass
                thr = p[t] / rest if rest > 0.0 else 0.0
            tests.append((float(u[c]), thr))
            if float(u[c]) < thr:
                accepted = c
                break
            if 0 <= t < V and t not in rejected_tok:
                rejected_mass += p[t]
                rejected_tok.append(t)
        if accepted is None:
            break
        path.append(accepted)
        pos = accepted + 1

    r = p_rows[pos].copy()
    if rejected_tok:
        r[rejected_tok] = 0.0
    c = np.cumsum(r)
    z = float(c[-1])
    source = "residual" if rejected_tok else "bonus"
    if not z > 0.0:
        r = p_rows[pos].copy()
        c = np.cumsum(r)
        z = float(c[-1])
        source += "+fallback"
    thr = float(u[N]) * z
    t = int(np.searchsorted(c, thr, side="right"))
    if t >= V:
        t = int(np.nonzero(r > 0.0)[0][-1])
    emitted = [int(tokens[i]) for i in path] + [t]
    trace = {"tests": tests, "z": z, "threshold": thr, "c_before": float(c[t - 1]) if t > 0 else 0.0,
             "c_at": float(c[t]), "source": source}
    return path, emitted, pos, trace


def accept_tree(logits_or_probs, row_lse, tokens, parent, u, kv_len=None):
    """Batched tree verification mirroring the library's call.

    logits_or_probs [B*G][V] (logits when row_lse is given: p = exp(logit - lse)
    in float64 after widening), tokens [B][N], parent [B][N], u [B][G].
    Returns accept_len [B], out_tok [B][G] and out_node [B][G] (-1 padded: the
    accepted nodes, then -1 for the final token), new_kv_len [B] (the cache
    keeps its prefix, the root and the accepted nodes: L - N + accept_len) or
    None, and per-request traces.
    """
    x = np.asarray(logits_or_probs)
    tokens = np.asarray(tokens)
    parent = np.asarray(parent)
    u = np.asarray(u)
    B, N = tokens.shape
    G = N + 1
    accept_len = np.zeros(B, dtype=np.int32)
    out_tok = np.full((B, G), -1, dtype=np.int32)
    out_node = np.full((B, G), -1, dtype=np.int32)
    traces = []
    for b in range(B):
        rows = x[b * G:(b + 1) * G].astype(np.float64)
        if row_lse is not None:
            lse = np.asarray(row_lse[b * G:(b + 1) * G], dtype=np.float64)
            rows = np.exp(rows - lse[:, None])
        path, emitted, _, tr = accept_tree_request(rows, tokens[b], parent[b], u[b])
        accept_len[b] = len(path)
        out_tok[b, :len(emitted)] = emitted
        out_node[b, :len(path)] = path
        traces.append(tr)
    new_kv_len = None
    if kv_len is not None:
        new_kv_len = (np.asarray(kv_len, dtype=np.int64) - N + accept_len).astype(np.int32)
    return {"accept_len": accept_len, "out_tok": out_tok, "out_node": out_node, "new_kv_len": new_kv_len,
            "traces": traces}


def tree_near_threshold(trace, band: float = RATIO_BAND, final_band: float = FINAL_BAND) -> bool:
    """A draw within ``band`` of a test threshold, or the final draw within
    final_band * Z of the chosen token's CDF interval ends (the bands of
    ``oracle.accept``)."""
    for ui, thr in trace["tests"]:
        if 0.0 < thr and abs(ui - thr) < band:
            return True
    z = trace["z"]
    return ((trace["threshold"] - trace["c_before"]) < final_band * z
            or (trace["c_at"] - trace["threshold"]) < final_band * z)


def tree_commit_kv(k_pool, v_pool, kv_off, kv_len, n_kv_heads, head_dim, out_node, accept_len, N):
    """Copies of the pools after moving each request's accepted nodes next to
    the root: for every KV head, tail position j + 1 receives the row of tail
    position out_node[b][j] + 1, for j < accept_len[b], in increasing j (the
    tail is the last N + 1 rows of the request's cache).  Rows are moved as
    raw values; nothing else changes."""
    k = np.array(k_pool, copy=True)
    v = np.array(v_pool, copy=True)
    G = N + 1
    D = head_dim
    for b in range(len(kv_len)):
        L = int(kv_len[b])
        off = int(kv_off[b])
        tail0 = L - G
        for g in range(n_kv_heads):
            base = off + g * L * D
            for j in range(int(accept_len[b])):
                src = base + (tail0 + int(out_node[b][j]) + 1) * D
                dst = base + (tail0 + j + 1) * D
                k[dst:dst + D] = k[src:src + D]
                v[dst:dst + D] = v[src:src + D]
    return k, v
