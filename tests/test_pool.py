"""The library's host-side KV page allocator (sd_kv_pool_*), on the CPU:
per-tag page counts are ceil(length / P), no page is held by two tags, pages
are conserved, a failed reservation changes nothing, truncation keeps the
leading pages (the roll-back to the accepted prefix), freed pages are reused
first, and block tables list pages in key order.  The page ids a tag gets are
not unique to the method; the tests check what is (counts, disjointness,
order of a tag's pages) and that the rest is valid."""

import numpy as np
import pytest

import paper_2601_21622_amd as sd


def _held(pool, tags, max_pages=64):
    t = pool.block_table(tags, max_pages)
    return {tag: [int(p) for p in row if p >= 0] for tag, row in zip(tags, t)}


def test_reserve_truncate_release_invariants():
    rng = np.random.default_rng(5)
    P, N = 64, 200
    pool = sd.KVPool(N, P)
    lengths = {}
    for _ in range(400):
        tag = int(rng.integers(0, 12))
        op = rng.integers(0, 3)
        if op == 0:
            want = lengths.get(tag, 0) + int(rng.integers(0, 300))
            before = _held(pool, list(range(12)))
            free0 = pool.free_pages()
            try:
                pool.reserve(tag, want)
                lengths[tag] = max(lengths.get(tag, 0), want)
            except sd.SdError as e:
                assert e.status == sd.SD_ERR_CAPACITY
                assert _held(pool, list(range(12))) == before and pool.free_pages() == free0
        elif op == 1 and tag in lengths:
            keep = int(rng.integers(0, lengths[tag] + 1))
            lead = _held(pool, [tag])[tag][:(keep + P - 1) // P]
            pool.truncate(tag, keep)
            lengths[tag] = keep
            assert _held(pool, [tag])[tag] == lead
        elif op == 2:
            pool.release(tag)
            lengths.pop(tag, None)
        held = _held(pool, list(range(12)))
        for t in range(12):
            assert pool.tag_pages(t) == (lengths.get(t, 0) + P - 1) // P
            assert len(held[t]) == pool.tag_pages(t)
        every = [p for v in held.values() for p in v]
        assert len(every) == len(set(every))
        assert all(0 <= p < N for p in every)
        assert len(every) + pool.free_pages() == N


def test_fresh_pool_order_reuse_and_table_padding():
    pool = sd.KVPool(8, 128)
    pool.reserve(0, 300)                      # 3 pages
    pool.reserve(1, 1)                        # 1 page
    t = pool.block_table([0, 1, 5], 4)
    assert t[0].tolist() == [0, 1, 2, -1] and t[1].tolist() == [3, -1, -1, -1] and t[2].tolist() == [-1] * 4
    pool.truncate(0, 128)                     # frees pages 2 and 1 (last first)
    pool.reserve(2, 129)
    assert pool.block_table([2], 2)[0].tolist() == [1, 2]
    pool.release(0)
    assert pool.free_pages() == 8 - 1 - 2
    with pytest.raises(sd.SdError):
        pool.block_table([2], 1)             # holds 2 pages
    pool.reserve(1, 1)                        # no growth needed
    assert pool.tag_pages(1) == 1


def test_invalid_arguments():
    with pytest.raises(sd.SdError):
        sd.KVPool(0, 64)
    for bad in (32, 96, 8192):
        with pytest.raises(sd.SdError):
            sd.KVPool(4, bad)
    pool = sd.KVPool(4, 64)
    for call in (lambda: pool.reserve(-1, 4), lambda: pool.reserve(0, -4), lambda: pool.truncate(-2, 0),
                 lambda: pool.release(-1)):
        with pytest.raises(sd.SdError) as e:
            call()
        assert e.value.status == sd.SD_ERR_INVALID_ARGUMENT
    with pytest.raises(sd.SdError) as e:
        pool.reserve(0, 64 * 5)
    assert e.value.status == sd.SD_ERR_CAPACITY and pool.tag_pages(0) == 0 and pool.free_pages() == 4
