"""Pins of oracle.paged: pages written from contiguous per-request caches by
an independent scatter (the header's layout: request b's key k of head g is
row k % P of head g in page table[b][k // P]) gather back to those caches
exactly, and paged attention then equals the segment-layout attention of
oracle.attention bit for bit, for shuffled and interleaved page tables and
lengths that end inside, at and one past a page boundary."""

import numpy as np
import pytest

from oracle import gather_request, paged_attention, verify_attention


def _scatter(segs, Hkv, D, P, rng, spare=3):
    """Pool [num_pages][Hkv][P][D] holding each request's rows in shuffled
    pages (unused rows NaN), and the block table."""
    need = [(s.shape[1] + P - 1) // P for s in segs]
    num_pages = sum(need) + spare
    order = rng.permutation(num_pages)
    pool = np.full((num_pages, Hkv, P, D), np.nan)
    table = np.full((len(segs), max(need) + 1), -1, dtype=np.int32)
    nxt = 0
    for b, seg in enumerate(segs):
        for j in range(need[b]):
            table[b, j] = order[nxt]
            nxt += 1
        L = seg.shape[1]
        for g in range(Hkv):
            for k in range(L):
                pool[table[b, k // P], g, k % P] = seg[g, k]
    return pool, table


@pytest.mark.parametrize("P", [64, 128])
def test_gather_inverts_the_layout(P):
    rng = np.random.default_rng(P)
    Hkv, D = 2, 8
    lengths = [5, P, P + 1, 3 * P - 1, 2 * P]
    segs = [rng.standard_normal((Hkv, L, D)) for L in lengths]
    pool, table = _scatter(segs, Hkv, D, P, rng)
    for b, seg in enumerate(segs):
        got = gather_request(pool, table[b], seg.shape[1], P)
        assert np.array_equal(got, seg)
        assert not np.isnan(got).any()


def test_paged_attention_equals_segment_attention():
    rng = np.random.default_rng(7)
    B, G, Hq, Hkv, D, P = 4, 3, 4, 2, 16, 64
    lengths = [G, 64, 65, 200]
    kseg = [rng.standard_normal((Hkv, L, D)) for L in lengths]
    vseg = [rng.standard_normal((Hkv, L, D)) for L in lengths]
    q = rng.standard_normal((B, G, Hq, D))
    kp, table = _scatter(kseg, Hkv, D, P, np.random.default_rng(1))
    vp = np.full_like(kp, np.nan)
    for b, seg in enumerate(vseg):
        for g in range(Hkv):
            for k in range(seg.shape[1]):
                vp[table[b, k // P], g, k % P] = seg[g, k]
    got = paged_attention(q, kp, vp, table, lengths, P)
    offs = np.cumsum([0] + [s.size for s in kseg[:-1]])
    want = verify_attention(q, np.concatenate([s.ravel() for s in kseg]), np.concatenate([s.ravel() for s in vseg]),
                            offs, lengths, Hkv)
    assert np.array_equal(got, want)


def test_interleaved_tables_keep_requests_apart():
    # Two requests sharing one pool with alternating pages: swapping their
    # tables swaps their gathered caches.
    rng = np.random.default_rng(3)
    Hkv, D, P = 1, 4, 64
    a, b = rng.standard_normal((Hkv, 130, D)), rng.standard_normal((Hkv, 130, D))
    pool = np.zeros((6, Hkv, P, D))
    ta, tb = [0, 2, 4], [1, 3, 5]
    for k in range(130):
        pool[ta[k // P], 0, k % P] = a[0, k]
        pool[tb[k // P], 0, k % P] = b[0, k]
    assert np.array_equal(gather_request(pool, ta, 130, P), a)
    assert np.array_equal(gather_request(pool, tb, 130, P), b)
