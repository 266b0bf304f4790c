"""GPU parity of the whole verification step (sd_verify_step).

* attention output and logits against the independent float64 oracle
  (tolerance rule), and
* acceptance bit-exact against the oracle re-run on the GPU's own logits and
  row log-sum-exp (same p on both sides), near-threshold draws excluded;
* the agreement of emitted tokens with the fully independent oracle is
  reported as a rate (a 2e-2 logit tolerance moves p by far more than the
  1e-6 band, so it cannot be bit-exact)."""

import numpy as np
from scipy.special import logsumexp
import pytest
import torch

from oracle import accept_resample, verify_attention, verify_logits
from workloads import get_config, make_inputs

from gpu_util import RTOL, DeviceBatch, announce, assert_accept_parity, assert_close_rows, to_np

pytestmark = pytest.mark.gpu

CASES = {
    "tiny_f32": get_config("tiny"),
    "vicuna_small": get_config("vicuna7b").replace(batch=3, n_q_heads=4, n_kv_heads=4, hidden=512, vocab=3000,
                                                   lengths=("explicit", (6, 600, 1300))),
    "gqa_small": get_config("llama3_8b").replace(batch=2, n_q_heads=8, n_kv_heads=2, hidden=1024, vocab=2500,
                                                 lengths=("explicit", (7, 900))),
    # Degenerate vocabularies: one token (p = q = 1, every draft accepted)
    # on the deep projection, two tokens on the shallow one.
    "vocab1_deep": get_config("vicuna7b").replace(batch=20, gamma=4, n_q_heads=2, n_kv_heads=2, hidden=64, vocab=1,
                                                  lengths=("fixed", 40)),
    "vocab2": get_config("vicuna7b").replace(batch=3, n_q_heads=2, n_kv_heads=2, hidden=64, vocab=2,
                                             lengths=("explicit", (6, 70, 300))),
}


def _check(name, use_hidden):
    cfg = CASES[name]
    announce(f"step parity case={name} use_hidden={use_hidden}")
    x = make_inputs(cfg)
    db = DeviceBatch(x)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    db.step(use_hidden=use_hidden, kernel_events=ev)
    torch.cuda.synchronize()
    assert all(ev[2 * i].elapsed_time(ev[2 * i + 1]) > 0 for i in range(3))
    rtol = RTOL[cfg.dtype]
    attn_ref = verify_attention(x.f32("q"), x.f32("k_pool"), x.f32("v_pool"), x.kv_off, x.kv_len, cfg.n_kv_heads)
    assert_close_rows(to_np(db.attn), attn_ref, rtol, f"step attention[{name}]")
    if use_hidden:
        h = x.f32("hidden")
    else:
        # The GPU projects its own (rounded) attention output; so does this check.
        h = to_np(db.attn).reshape(cfg.rows, -1)
    logits_ref, lse_ref = verify_logits(h, x.f32("w"))
    assert_close_rows(to_np(db.logits), logits_ref, rtol, f"step logits[{name}]")
    g_logits, g_lse = to_np(db.logits), to_np(db.lse)
    # The acceptance folds the row log-sum-exps from the projection's tile
    # statistics; they must be those of the logits themselves.
    assert np.max(np.abs(g_lse - logsumexp(g_logits.astype(np.float64), axis=1))) < 1e-4
    ref = accept_resample(g_logits, g_lse, x.q_draft, x.draft, x.u, kv_len=x.kv_len)
    near = assert_accept_parity(to_np(db.accept_len), to_np(db.out_tok), to_np(db.new_kv_len), ref)
    indep = accept_resample(logits_ref, lse_ref, x.q_draft, x.draft, x.u, kv_len=x.kv_len)
    agree = float(np.mean(np.all(to_np(db.out_tok) == indep["out_tok"], axis=1)))
    announce(f"step case={name}: near-threshold {near}; token agreement with the independent oracle {agree:.3f}")


@pytest.mark.parametrize("name", sorted(CASES))
def test_step_with_hidden(name):
    _check(name, True)


@pytest.mark.parametrize("name", ["tiny_f32", "vicuna_small"])
def test_step_projects_attention_output(name):
    _check(name, False)


# 70 requests: two acceptance launches (at most 64 requests each), whose
# arrival counters are indexed by the global request number.
MANY = get_config("vicuna7b").replace(batch=70, n_q_heads=4, n_kv_heads=4, hidden=256, vocab=5000,
                                      lengths=("explicit", tuple(6 + 37 * i for i in range(70))))


@pytest.mark.parametrize("fill", [0x00, 0xFF])
def test_step_acceptance_on_a_stale_workspace(fill):
    """The step's acceptance runs as one launch whose per-request arrival
    counters live in the workspace; the step's projection launch clears them.
    A workspace full of stale bytes, and a second step over the first one's
    leftovers, give the same outputs as the two-launch sd_accept_resample on
    the step's own logits and log-sum-exps, and both match the oracle."""
    cfg = MANY
    announce(f"stale-workspace step case=vicuna_many fill={fill:#x} B={cfg.batch}")
    x = make_inputs(cfg)
    db = DeviceBatch(x)
    db.ws.fill_(fill)
    db.step()
    torch.cuda.synchronize()
    first = (db.accept_len.clone(), db.out_tok.clone(), db.new_kv_len.clone())
    db.step()
    torch.cuda.synchronize()
    for got, want in zip((db.accept_len, db.out_tok, db.new_kv_len), first):
        assert torch.equal(got, want)
    db.accept()  # two launches, on the step's logits and row log-sum-exps
    torch.cuda.synchronize()
    for got, want in zip((db.accept_len, db.out_tok, db.new_kv_len), first):
        assert torch.equal(got, want)
    ref = accept_resample(to_np(db.logits), to_np(db.lse), x.q_draft, x.draft, x.u, kv_len=x.kv_len)
    assert_accept_parity(to_np(first[0]), to_np(first[1]), to_np(first[2]), ref)
