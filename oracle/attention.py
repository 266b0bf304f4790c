"""Causal multi-query verification attention, float64, by definition.

Source: Algorithm 2 of the paper (verification loop) runs the target model
along the prefixes y, y+[x_1], ..., y+[x_1..x_d] of a draft path and notes the
gamma + 1 evaluations may run in parallel; Sec. 2 ("Tree-based proposals")
describes scoring the candidates in one batched forward pass.  This module is
the attention part of that forward for one layer: softmax(Q K^T * scale) V,
restricted causally.

Conventions (the paper states none of them; each is a reading recorded in the
design notes):
* scale defaults to 1/sqrt(head_dim);
* grouped-query attention maps query head h to KV head floor(h / (Hq / Hkv));
* Q and K arrive already position-encoded (no rotary embedding here);
* ``kv_len[b]`` = L_b includes the G = gamma + 1 positions of this step at the
  tail of the cache, so query j (0 = root, j >= 1 = draft x_j) sits at absolute
  position L_b - G + j and sees keys 0 .. L_b - G + j.
"""

from __future__ import annotations

import numpy as np


def verify_attention(q, k_pool, v_pool, kv_off, kv_len, n_kv_heads, scale=None):
    """Return O[B][G][Hq][D] (float64).

    q        [B][G][Hq][D] float array
    k_pool   flat float array; request b's keys are the [Hkv][kv_len[b]][D]
             block starting at element kv_off[b]
    v_pool   same layout as k_pool
    """
    q = np.asarray(q)
    B, G, Hq, D = q.shape
    Hkv = int(n_kv_heads)
    if Hq % Hkv:
        raise ValueError("n_q_heads must be a multiple of n_kv_heads")
    group = Hq // Hkv
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    out = np.zeros((B, G, Hq, D), dtype=np.float64)
    for b in range(B):
        L = int(kv_len[b])
        off = int(kv_off[b])
        if L < G:
            raise ValueError("kv_len must include the gamma + 1 positions of the step")
        Kb = np.asarray(k_pool[off:off + Hkv * L * D], dtype=np.float64).reshape(Hkv, L, D)
        Vb = np.asarray(v_pool[off:off + Hkv * L * D], dtype=np.float64).reshape(Hkv, L, D)
        # visible[j, t] is True when key t is at or before query j's position.
        last = L - G + np.arange(G)
        visible = np.arange(L)[None, :] <= last[:, None]
        for h in range(Hq):
            g = h // group
            s = (q[b, :, h, :].astype(np.float64) @ Kb[g].T) * scale      # [G][L]
            s = np.where(visible, s, -np.inf)
            s = s - s.max(axis=1, keepdims=True)
            e = np.exp(s)
            wgt = e / e.sum(axis=1, keepdims=True)
            out[b, :, h, :] = wgt @ Vb[g]
    return out
