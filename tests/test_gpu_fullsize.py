"""GPU parity at the full sizes of the bf16 workloads, in the launch
configuration bench.py times (sd_verify_step with caller-supplied hidden).

Every output is compared with the oracle: the attention output of every
request and head, the logits and log-sum-exp of every row (each a full
float64 dot product over the whole vocabulary), and the acceptance of every
request re-run on the GPU's own logits and log-sum-exp (bit-exact outside the
decision bands).  Properties that hold at any size are checked too: finite
outputs, rows of p summing to one, accept lengths in range, emitted tokens
inside the vocabulary."""

import numpy as np
import pytest
import torch

from oracle import accept_resample, verify_attention, verify_logits
from workloads import get_config, make_inputs

from gpu_util import RTOL, DeviceBatch, announce, assert_accept_parity, assert_close_rows, to_np

pytestmark = pytest.mark.gpu


def _attention(x):
    c = x.cfg
    return verify_attention(x.f32("q"), x.f32("k_pool"), x.f32("v_pool"), x.kv_off, x.kv_len, c.n_kv_heads)


@pytest.mark.parametrize("name,packed", [("vicuna7b", True), ("vicuna7b", False), ("pooled", True),
                                         ("llama3_8b", True), ("llama70b_share", True)])
def test_full_size_step(name, packed):
    cfg = get_config(name)
    announce(f"full-size step case={name} packed_vocab={packed} B={cfg.batch} gamma={cfg.gamma} V={cfg.vocab} "
             f"hidden={cfg.hidden}")
    x = make_inputs(cfg)
    db = DeviceBatch(x, packed_vocab=packed)
    db.step(use_hidden=True)
    torch.cuda.synchronize()
    announce(f"full-size step case={name}: GPU step done")
    rtol = RTOL[cfg.dtype]
    B, G, V = cfg.batch, cfg.positions, cfg.vocab

    # Attention: every request and query head.
    err = assert_close_rows(to_np(db.attn), _attention(x), rtol, f"attention[{name}]")
    announce(f"full-size step case={name}: attention of all {B} requests, max rel err {err:.2e}")

    # Logits and log-sum-exp: every row.
    logits = to_np(db.logits)
    lse = to_np(db.lse)
    assert np.all(np.isfinite(logits)) and np.all(np.isfinite(lse))
    ref_logits, ref_lse = verify_logits(x.f32("hidden"), x.f32("w"))
    err = assert_close_rows(logits, ref_logits, rtol, f"logits[{name}]")
    assert np.all(np.abs(lse - ref_lse) <= rtol * np.maximum(np.abs(ref_lse), 1.0))
    announce(f"full-size step case={name}: logits of all {cfg.rows} rows, max rel err {err:.2e}")
    del ref_logits
    p_sum = np.exp(logits.astype(np.float64) - lse.astype(np.float64)[:, None]).sum(axis=1)
    assert np.allclose(p_sum, 1.0, atol=1e-4)

    # Acceptance on the GPU's own p, every request.
    acc, tok, new = to_np(db.accept_len), to_np(db.out_tok), to_np(db.new_kv_len)
    assert np.all((acc >= 0) & (acc <= cfg.gamma))
    assert np.all(tok[np.arange(B), acc] >= 0) and np.all(tok[np.arange(B), acc] < V)
    ref = accept_resample(logits, lse, x.q_draft, x.draft, x.u, kv_len=x.kv_len)
    near = assert_accept_parity(acc, tok, new, ref)
    announce(f"full-size step case={name}: mean accept {acc.mean():.2f}, near-threshold {near}")
