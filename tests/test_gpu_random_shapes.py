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
