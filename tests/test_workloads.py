"""The seeded input generator: determinism, layouts and value recipes."""

import numpy as np
import pytest
import torch

from workloads import CONFIGS, bf16_bits, get_config, make_inputs
from workloads.generate import bf16_bits_to_f32


def small(name, **kw):
    base = dict(batch=3, vocab=777, lengths=("uniform", 20, 90))
    base.update(kw)
    c = get_config(name)
    if c.hidden != c.n_q_heads * c.head_dim:
        raise AssertionError
    return c.replace(**base)


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.normal(size=10000).astype(np.float32),
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8, 0.0, -0.0], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bf16_bits(x), ref)
    assert np.array_equal(bf16_bits_to_f32(ref), torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy())


@pytest.mark.parametrize("name", ["tiny", "vicuna7b", "pooled", "llama3_8b"])
def test_deterministic_and_shaped(name):
    c = get_config(name) if name == "tiny" else small(name)
    a, b = make_inputs(c), make_inputs(c)
    for f in ("kv_len", "kv_off", "q", "k_pool", "v_pool", "hidden", "w", "q_draft", "draft", "u"):
        assert np.array_equal(getattr(a, f), getattr(b, f)), f
    B, G = c.batch, c.positions
    assert a.q.shape == (B, G, c.n_q_heads, c.head_dim)
    assert a.hidden.shape == (B * G, c.hidden)
    assert a.w.shape == (c.vocab, c.hidden)
    assert a.q_draft.shape == (B, c.gamma, c.vocab)
    assert a.draft.shape == (B, c.gamma) and a.u.shape == (B, G)
    assert a.k_pool.size == a.kv_elements == a.v_pool.size
    assert (a.kv_off[1:] == a.kv_off[:-1] + c.n_kv_heads * a.kv_len[:-1].astype(np.int64) * c.head_dim).all()
    assert np.all(a.kv_len >= G)
    want = np.uint16 if c.dtype == "bf16" else np.float32
    assert a.k_pool.dtype == want and a.w.dtype == want
    # draws are multiples of 2^-24 in [0, 1)
    assert np.all((a.u >= 0) & (a.u < 1))
    assert np.array_equal(a.u.astype(np.float64) * 2 ** 24, np.floor(a.u.astype(np.float64) * 2 ** 24))
    assert np.allclose(a.q_draft.sum(axis=-1), 1.0, atol=1e-5)
    assert np.all(a.q_draft[np.arange(B)[:, None], np.arange(c.gamma)[None, :], a.draft] > 0)


def test_seed_changes_values():
    c = small("vicuna7b")
    assert not np.array_equal(make_inputs(c).w, make_inputs(c, seed=5).w)


def test_value_distributions():
    c = small("vicuna7b", vocab=2000)
    a = make_inputs(c)
    w = a.f32("w")
    assert abs(w.std() * np.sqrt(c.hidden) - 1.0) < 0.02
    k = a.f32("k_pool")
    assert abs(k.mean()) < 0.01 and abs(k.std() - 1.0) < 0.01
    c4 = small("llama3_8b", vocab=3000)
    assert abs(make_inputs(c4).f32("w").std() * np.sqrt(c4.hidden) - 16.0) < 0.4


def test_length_recipes():
    a = make_inputs(get_config("vicuna7b"))
    assert a.kv_len.min() >= 512 and a.kv_len.max() <= 2048
    c = get_config("pooled").replace(vocab=100, batch=400, n_q_heads=1, n_kv_heads=1, head_dim=64, hidden=64)
    L = make_inputs(c).kv_len
    assert L.max() <= 8192 and L.min() >= c.positions
    assert 800 < np.median(L) < 1300
    assert get_config("llama70b_share").max_kv_len() == 32768
    e = small("vicuna7b", batch=2, lengths=("explicit", (6, 33)))
    assert list(make_inputs(e).kv_len) == [6, 33]


def test_draft_tokens_follow_q():
    c = get_config("tiny").replace(batch=400, gamma=1, vocab=5, lengths=("fixed", 2), hidden=256)
    a = make_inputs(c)
    counts = np.bincount(a.draft[:, 0], minlength=5)
    expected = a.q_draft[:, 0, :].sum(axis=0)
    chi2 = ((counts - expected) ** 2 / expected).sum()
    assert chi2 < 25.0  # 4 dof; p ~ 5e-5


def test_smoothed_onehot_and_independent_recipes():
    a = make_inputs(small("llama3_8b"))
    mx = a.q_draft.max(axis=-1)
    assert np.allclose(mx, 0.9, atol=1e-7)
    a5 = make_inputs(get_config("llama70b_share").replace(batch=2, vocab=300, hidden=512, n_q_heads=4,
                                                        n_kv_heads=2, lengths=("fixed", 40)))
    assert np.allclose(a5.q_draft.sum(-1), 1.0, atol=1e-5)
