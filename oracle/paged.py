"""Paged KV caches, float64: the verification attention of requests whose
K and V rows live in pages of a shared pool.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Per-session (per-tag) KV state is what Algorithm 1 isolates; here a session's
cache is the list of its pages.  Pool layout [num_pages][Hkv][P][D]; request
b's key k of KV head g is row k % P of head g in page block_table[b][k // P].
The attention itself is the chain definition of oracle.attention applied to
the gathered rows.
"""

from __future__ import annotations

import numpy as np

from .attention import verify_attention


def gather_request(pool, table_row, L: int, page_size: int) -> np.ndarray:
    """[Hkv][L][D] rows of one request, key by key from its pages."""
    pool = np.asarray(pool)
    _, Hkv, P, D = pool.shape
    if P != page_size:
        raise ValueError("pool page size mismatch")
    out = np.empty((Hkv, L, D), dtype=pool.dtype)
    for k in range(L):
        page = int(table_row[k // page_size])
        out[:, k, :] = pool[page, :, k % page_size, :]
    return out


def paged_attention(q, k_pages, v_pages, block_table, kv_len, page_size: int, scale=None) -> np.ndarray:
    """verify_attention over the gathered caches (q [B][G][Hq][D])."""
    k_pages = np.asarray(k_pages)
    B = len(kv_len)
    Hkv = k_pages.shape[1]
    segs_k, segs_v, offs = [], [], []
    off = 0
    for b in range(B):
        L = int(kv_len[b])
        segs_k.append(gather_request(k_pages, block_table[b], L, page_size).ravel())
        segs_v.append(gather_request(v_pages, block_table[b], L, page_size).ravel())
        offs.append(off)
        off += segs_k[-1].size
    return verify_attention(q, np.concatenate(segs_k), np.concatenate(segs_v), np.array(offs), np.asarray(kv_len),
                            Hkv, scale)
