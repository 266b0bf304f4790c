"""Pins of the oracle's causal verification attention (oracle.attention).

The definition softmax(Q K^T / sqrt(D)) V with the causal offset is fixed by
special cases with closed-form answers, by invariances, and by an independent
library routine (torch's scaled_dot_product_attention on the CPU in float64,
with an explicit mask).  The convention that query j of a request with
kv_len = L sits at position L - G + j is pinned by the L = G case.
"""

import numpy as np
import pytest
import torch

from oracle.attention import verify_attention


def _make(rng, B, G, Hq, Hkv, D, lens):
    q = rng.normal(size=(B, G, Hq, D))
    lens = np.asarray(lens)
    seg = Hkv * lens * D
    off = np.concatenate([[0], np.cumsum(seg)[:-1]])
    k = rng.normal(size=int(seg.sum()))
    v = rng.normal(size=int(seg.sum()))
    return q, k, v, off, lens


def _kv(pool, off, L, Hkv, D):
    return pool[off:off + Hkv * L * D].reshape(Hkv, L, D)


def test_shortest_cache_query0_returns_first_value():
    rng = np.random.default_rng(0)
    G, Hq, D = 4, 2, 8
    q, k, v, off, lens = _make(rng, 1, G, Hq, Hq, D, [G])
    o = verify_attention(q, k, v, off, lens, Hq)
    V_ = _kv(v, 0, G, Hq, D)
    for h in range(Hq):
        assert np.array_equal(o[0, 0, h], V_[h, 0])      # sees exactly one key
        assert not np.allclose(o[0, 1, h], V_[h, 0])     # query 1 sees two


def test_identical_keys_average_visible_values():
    rng = np.random.default_rng(1)
    G, H, D, L = 3, 2, 16, 11
    q, k, v, off, lens = _make(rng, 1, G, H, H, D, [L])
    K = _kv(k, 0, L, H, D)
    K[:] = K[:, :1, :]
    o = verify_attention(q, k, v, off, lens, H)
    V_ = _kv(v, 0, L, H, D)
    for j in range(G):
        vis = L - G + j + 1
        for h in range(H):
            assert np.allclose(o[0, j, h], V_[h, :vis].mean(axis=0), atol=1e-13)


def test_dominant_key():
    rng = np.random.default_rng(2)
    G, H, D, L = 2, 1, 32, 20
    q, k, v, off, lens = _make(rng, 1, G, H, H, D, [L])
    K = _kv(k, 0, L, H, D)
    K[0, 7] = 50.0 * q[0, 0, 0] / np.linalg.norm(q[0, 0, 0])
    o = verify_attention(q, k, v, off, lens, H)
    assert np.allclose(o[0, 0, 0], _kv(v, 0, L, H, D)[0, 7], atol=1e-6)


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (8, 2), (6, 1)])
def test_matches_torch_sdpa_with_explicit_mask(Hq, Hkv):
    rng = np.random.default_rng(3)
    G, D = 5, 16
    lens = [5, 9, 37]
    q, k, v, off, lens = _make(rng, 3, G, Hq, Hkv, D, lens)
    o = verify_attention(q, k, v, off, lens, Hkv)
    for b in range(3):
        L = int(lens[b])
        K = torch.from_numpy(_kv(k, off[b], L, Hkv, D)).repeat_interleave(Hq // Hkv, dim=0)
        V_ = torch.from_numpy(_kv(v, off[b], L, Hkv, D)).repeat_interleave(Hq // Hkv, dim=0)
        Q = torch.from_numpy(q[b]).permute(1, 0, 2)  # [Hq][G][D]
        mask = torch.arange(L)[None, :] <= (L - G + torch.arange(G))[:, None]
        ref = torch.nn.functional.scaled_dot_product_attention(Q, K, V_, attn_mask=mask)
        assert np.allclose(o[b], ref.permute(1, 0, 2).numpy(), atol=1e-12, rtol=1e-12)


def test_causal_future_keys_do_not_matter():
    rng = np.random.default_rng(4)
    G, H, D, L = 4, 2, 8, 15
    q, k, v, off, lens = _make(rng, 1, G, H, H, D, [L])
    o1 = verify_attention(q, k, v, off, lens, H)
    k2, v2 = k.copy(), v.copy()
    _kv(k2, 0, L, H, D)[:, L - 1] += 3.0     # only the last query sees position L-1
    _kv(v2, 0, L, H, D)[:, L - 1] -= 2.0
    o2 = verify_attention(q, k2, v2, off, lens, H)
    assert np.array_equal(o1[:, :G - 1], o2[:, :G - 1])
    assert not np.allclose(o1[:, G - 1], o2[:, G - 1])


def test_scale_and_permutation_invariance():
    rng = np.random.default_rng(5)
    G, H, D, L = 3, 2, 8, 12
    q, k, v, off, lens = _make(rng, 1, G, H, H, D, [L])
    o = verify_attention(q, k, v, off, lens, H)
    o2 = verify_attention(q * 2.0, k, v, off, lens, H, scale=0.5 / np.sqrt(D))
    assert np.allclose(o, o2, atol=1e-13)
    # Permuting keys/values jointly among positions every query sees.
    perm = rng.permutation(L - G + 1)
    k3, v3 = k.copy(), v.copy()
    K3, V3 = _kv(k3, 0, L, H, D), _kv(v3, 0, L, H, D)
    K3[:, :L - G + 1] = _kv(k, 0, L, H, D)[:, perm]
    V3[:, :L - G + 1] = _kv(v, 0, L, H, D)[:, perm]
    assert np.allclose(verify_attention(q, k3, v3, off, lens, H), o, atol=1e-13)


def test_requests_are_isolated():
    rng = np.random.default_rng(6)
    G, H, D = 2, 2, 8
    q, k, v, off, lens = _make(rng, 2, G, H, H, D, [6, 9])
    o = verify_attention(q, k, v, off, lens, H)
    k2 = k.copy()
    k2[off[1]:] += rng.normal(size=k2[off[1]:].shape)
    o2 = verify_attention(q, k2, v, off, lens, H)
    assert np.array_equal(o[0], o2[0]) and not np.allclose(o[1], o2[1])
