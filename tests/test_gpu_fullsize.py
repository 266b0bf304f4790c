"""GPU parity at the full sizes of the bf16 workloads, in the launch
configuration bench.py times (sd_verify_step with caller-supplied hidden).

The oracle cannot afford whole batches here, so it checks sampled outputs it
can compute one by one: the attention output of a few requests, the logits and
log-sum-exp of a few rows (each row a full float64 dot product over the whole
vocabulary), and the acceptance of every request re-run on the GPU's own
logits and log-sum-exp (bit-exact outside the 1e-6 band).  Properties that
hold at any size are checked on everything: finite outputs, rows of p summing
to one, accept lengths in range, emitted tokens inside the vocabulary."""

import numpy as np
import pytest
import torch

from oracle import accept_resample, verify_attention, verify_logits
from workloads import get_config, make_inputs

from gpu_util import RTOL, DeviceBatch, announce, assert_accept_parity, assert_close_rows, to_np

pytestmark = pytest.mark.gpu


def _sampled_attention(x, reqs):
    c = x.cfg
    return verify_attention(x.f32("q")[reqs], x.f32("k_pool"), x.f32("v_pool"), x.kv_off[reqs], x.kv_len[reqs],
                            c.n_kv_heads)


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

    # Attention: the shortest, the longest and one middle request.
    order = np.argsort(x.kv_len)
    reqs = np.unique([order[0], order[len(order) // 2], order[-1]])
    ref_attn = _sampled_attention(x, reqs)
    assert_close_rows(to_np(db.attn)[reqs], ref_attn, rtol, f"attention[{name}]")

    # Logits and log-sum-exp: first and last row, plus two inside.
    M = cfg.rows
    rows = np.unique([0, M // 3, (2 * M) // 3, M - 1])
    logits = to_np(db.logits)
    lse = to_np(db.lse)
    assert np.all(np.isfinite(logits)) and np.all(np.isfinite(lse))
    ref_logits, ref_lse = verify_logits(x.f32("hidden")[rows], x.f32("w"))
    assert_close_rows(logits[rows], ref_logits, rtol, f"logits[{name}]")
    assert np.all(np.abs(lse[rows] - ref_lse) <= rtol * np.maximum(np.abs(ref_lse), 1.0))
    p_sum = np.exp(logits.astype(np.float64) - lse.astype(np.float64)[:, None]).sum(axis=1)
    assert np.allclose(p_sum, 1.0, atol=1e-4)

    # Acceptance on the GPU's own p, every request.
    acc, tok, new = to_np(db.accept_len), to_np(db.out_tok), to_np(db.new_kv_len)
    assert np.all((acc >= 0) & (acc <= cfg.gamma))
    assert np.all(tok[np.arange(B), acc] >= 0) and np.all(tok[np.arange(B), acc] < V)
    ref = accept_resample(logits, lse, x.q_draft, x.draft, x.u, kv_len=x.kv_len)
    near = assert_accept_parity(acc, tok, new, ref)
    announce(f"full-size step case={name}: mean accept {acc.mean():.2f}, near-threshold {near}")
