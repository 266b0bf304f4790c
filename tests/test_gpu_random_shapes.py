"""GPU parity of the whole verification step on seeded random shapes.

Each case draws a shape inside the boundary's limits (batch up to 70, so some
cases take two launches of at most 64 requests; gamma up to 15; grouped
queries up to 128 rows per KV head; head dimension 64 or 128; vocabularies
that are not multiples of any tile; ragged cache lengths down to gamma + 1;
the packed or row-major LM head; bfloat16, and float32 where its limits
allow) and runs sd_verify_step.  Checks, as in the fixed-shape tests:
attention output and logits against the float64 oracle within the tolerance
rule, the row log-sum-exps against the logits' own, and accept lengths,
emitted tokens and new cache lengths bit-exact against the oracle re-run on
the GPU's logits (near-threshold requests excluded and bounded)."""

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

from oracle import accept_resample, verify_attention, verify_logits
from workloads import get_config, make_inputs

from gpu_util import RTOL, DeviceBatch, announce, assert_accept_parity, assert_close_rows, to_np

pytestmark = pytest.mark.gpu

NCASES = 16


def random_config(i: int):
    rng = np.random.default_rng(20260 + i)
    f32 = i % 5 == 4
    D = 64 if (f32 or rng.random() < 0.35) else 128
    hkv = int(rng.choice([1, 2, 4, 8]))
    gamma = int(rng.integers(1, 16))
    G = gamma + 1
    max_rows = 64 if f32 else 128
    groups = [g for g in (1, 2, 4, 8) if G * g <= max_rows]
    group = int(rng.choice(groups))
    hq = hkv * group
    batch = int(rng.integers(1, 71)) if not f32 else int(rng.integers(1, 9))
    if i % 4 == 1:
        batch = int(rng.integers(65, 71))        # two launches
    vocab = int(rng.integers(100, 70000)) if not f32 else int(rng.integers(50, 3000))
    hidden = hq * D
    lengths = tuple(int(x) for x in rng.integers(G, G + (400 if f32 else 3000), size=batch))
    if batch > 2:
        lengths = (G,) + lengths[1:]             # a request whose cache is just this step
    draft = [("noisy", 1.0), ("independent", 1.0), ("smoothed_onehot", 0.9), ("noisy", 0.2)][i % 4]
    base = get_config("tiny" if f32 else "vicuna7b")
    return base.replace(name=f"rand{i}", batch=batch, gamma=gamma, n_q_heads=hq, n_kv_heads=hkv, head_dim=D,
                        hidden=hidden, vocab=vocab, lengths=("explicit", lengths), draft=draft, seed=i)


@pytest.mark.parametrize("i", range(NCASES))
def test_random_shape_step_matches_oracle(i):
    cfg = random_config(i)
    packed = cfg.dtype == "bf16" and i % 2 == 0
    announce(f"random step case={i} B={cfg.batch} gamma={cfg.gamma} Hq/Hkv={cfg.n_q_heads}/{cfg.n_kv_heads} "
             f"D={cfg.head_dim} V={cfg.vocab} dtype={cfg.dtype} packed={packed}")
    x = make_inputs(cfg)
    db = DeviceBatch(x, packed_vocab=packed)
    db.ws.fill_(0xA5)
    db.step(use_hidden=True)
    torch.cuda.synchronize()
    rtol = RTOL[cfg.dtype]
    attn_ref = verify_attention(x.f32("q"), x.f32("k_pool"), x.f32("v_pool"), x.kv_off, x.kv_len, cfg.n_kv_heads)
    assert_close_rows(to_np(db.attn), attn_ref, rtol, f"random attention[{i}]")
    logits_ref, _ = verify_logits(x.f32("hidden"), x.f32("w"))
    g_logits, g_lse = to_np(db.logits), to_np(db.lse)
    assert_close_rows(g_logits, logits_ref, rtol, f"random logits[{i}]")
    assert np.max(np.abs(g_lse - logsumexp(g_logits.astype(np.float64), axis=1))) < 1e-4
    ref = accept_resample(g_logits, g_lse, x.q_draft, x.draft, x.u, kv_len=x.kv_len)
    near = assert_accept_parity(to_np(db.accept_len), to_np(db.out_tok), to_np(db.new_kv_len), ref)
    announce(f"random step case={i}: near-threshold {near}, mean accept {to_np(db.accept_len).mean():.2f}")


NSAMPLED = 6
# (temperature, top-k, top-p): greedy, plain, top-p, top-k + top-p, top-1,
# a hot top-k with a tight top-p.
SAMPLED_SETTINGS = [(0.0, 0, 1.0), (1.0, 0, 0.9), (0.8, 40, 0.9), (0.7, 1, 1.0), (1.3, 100, 0.5), (1.0, 8, 1.0)]


@pytest.mark.parametrize("i", range(NSAMPLED))
def test_random_shape_sampled_step_matches_oracle(i):
    """sd_verify_step_sampled on random shapes and warp settings: the cut
    against the oracle's warp of the GPU logits, acceptance bit-exact."""
    import paper_2601_21622_amd as sd
    from oracle import accept_resample_sampled
    from test_gpu_sampling import _check_cut, _gpu_cut

    cfg = random_config(100 + 5 * i + i % 4)  # an index that is never 4 mod 5: bfloat16
    T, k, p = SAMPLED_SETTINGS[i]
    announce(f"random sampled step case={i} B={cfg.batch} gamma={cfg.gamma} V={cfg.vocab} T={T} k={k} p={p}")
    x = make_inputs(cfg)
    db = DeviceBatch(x, packed_vocab=i % 2 == 0)
    db.ws.fill_(0x5A)
    mn = torch.empty_like(db.lse)
    sd.sd_verify_step_sampled(db.dims, sd.Sampling(T, k, p), db.q, db.k, db.v, x.kv_off, x.kv_len, db.scale,
                              db.hidden, db.w, db.q_draft, db.draft, db.u, db.attn, db.logits, db.lse, mn,
                              db.accept_len, db.out_tok, db.new_kv_len, db.ws)
    torch.cuda.synchronize()
    logits = to_np(db.logits)
    logits_ref, _ = verify_logits(x.f32("hidden"), x.f32("w"))
    assert_close_rows(logits, logits_ref, RTOL[cfg.dtype], f"random sampled logits[{i}]")
    g_lse, g_min = to_np(db.lse), to_np(mn)
    _check_cut(logits, T, k, p, g_lse, g_min)
    ref = accept_resample_sampled(logits, x.q_draft, x.draft, x.u, T, k, p, x.kv_len,
                                  cut=_gpu_cut(logits, T, g_lse, g_min))
    near = assert_accept_parity(to_np(db.accept_len), to_np(db.out_tok), to_np(db.new_kv_len), ref)
    announce(f"random sampled step case={i}: near-threshold {near}")


NTREE = 6


@pytest.mark.parametrize("i", range(NTREE))
def test_random_shape_tree_step_matches_oracle(i):
    """sd_verify_step_tree on random shapes and random candidate trees:
    attention against the tree oracle, the folded row log-sum-exps against
    the logits, and the walk and final draw bit-exact against the oracle on
    the GPU logits."""
    import paper_2601_21622_amd as sd
    from oracle import accept_tree, tree_attention
    from test_gpu_tree import _assert_tree_parity, random_parents
    from gpu_util import tensor

    cfg = random_config(400 + 5 * i + i % 4)  # bfloat16, as above
    rng = np.random.default_rng(600 + i)
    announce(f"random tree step case={i} B={cfg.batch} nodes={cfg.gamma} Hq/Hkv={cfg.n_q_heads}/{cfg.n_kv_heads} "
             f"V={cfg.vocab}")
    x = make_inputs(cfg)
    parent = random_parents(rng, cfg.batch, cfg.gamma)
    tokens = rng.integers(0, cfg.vocab, size=(cfg.batch, cfg.gamma)).astype(np.int32)
    db = DeviceBatch(x, packed_vocab=i % 2 == 1)
    db.ws.fill_(0xFF)
    node = torch.empty_like(db.out_tok)
    sd.sd_verify_step_tree(db.dims, db.q, db.k, db.v, x.kv_off, x.kv_len, tensor(parent), db.scale, db.hidden, db.w,
                           tensor(tokens), db.u, db.attn, db.logits, db.lse, db.accept_len, db.out_tok, node,
                           db.new_kv_len, db.ws)
    torch.cuda.synchronize()
    ref_attn = tree_attention(x.f32("q"), x.f32("k_pool"), x.f32("v_pool"), x.kv_off, x.kv_len, cfg.n_kv_heads, parent)
    assert_close_rows(to_np(db.attn), ref_attn, RTOL[cfg.dtype], f"random tree attention[{i}]")
    g_logits, g_lse = to_np(db.logits), to_np(db.lse)
    assert np.max(np.abs(g_lse - logsumexp(g_logits.astype(np.float64), axis=1))) < 1e-4
    ref = accept_tree(g_logits, g_lse, tokens, parent, x.u, kv_len=x.kv_len)
    near = _assert_tree_parity([to_np(db.accept_len), to_np(db.out_tok), to_np(node), to_np(db.new_kv_len)], ref)
    announce(f"random tree step case={i}: near-threshold {near}, mean depth {to_np(db.accept_len).mean():.2f}")
