"""sd_verify_step_static, the step on the library's static per-device
scratch (no workspace argument), against sd_verify_step on the same inputs:
every output identical (the same kernels run in the same order on the same
data), on two calls in a row, the second with a smaller problem, so the
scratch holds the first call's contents when the second starts."""

import pytest
import torch

import paper_2601_21622_amd as sd
from workloads import get_config, make_inputs

from gpu_util import DeviceBatch, announce

pytestmark = pytest.mark.gpu

LARGE = get_config("llama3_8b").replace(batch=6, lengths=("explicit", (5000, 900, 8200, 3100, 64, 12000)))
# 224 projection rows and a large vocabulary: the wide projection schedule.
WIDE = get_config("llama3_8b").replace(batch=32, hidden=256, vocab=100001, lengths=("fixed", 64))
SMALL = get_config("vicuna7b").replace(batch=3, n_q_heads=8, n_kv_heads=8, hidden=1024, vocab=5000,
                                       lengths=("explicit", (40, 300, 1200)))


def _static_outputs(db):
    c = db.cfg
    B, G, M, V = c.batch, c.positions, c.rows, c.vocab
    adt = torch.bfloat16 if c.dtype == "bf16" else torch.float32
    out = {
        "attn": torch.empty((B, G, c.n_q_heads, c.head_dim), dtype=adt, device="cuda"),
        "logits": torch.empty((M, V), dtype=torch.float32, device="cuda"),
        "lse": torch.empty((M,), dtype=torch.float32, device="cuda"),
        "accept_len": torch.empty((B,), dtype=torch.int32, device="cuda"),
        "out_tok": torch.empty((B, G), dtype=torch.int32, device="cuda"),
        "new_kv_len": torch.empty((B,), dtype=torch.int32, device="cuda"),
    }
    sd.sd_verify_step_static(db.dims, db.q, db.k, db.v, db.x.kv_off, db.x.kv_len, db.scale, db.hidden, db.w,
                             db.q_draft, db.draft, db.u, out["attn"], out["logits"], out["lse"], out["accept_len"],
                             out["out_tok"], out["new_kv_len"])
    return out


def _check(cfg, packed):
    x = make_inputs(cfg)
    db = DeviceBatch(x, packed_vocab=packed)
    static = _static_outputs(db)      # first, on whatever the scratch holds
    db.step(use_hidden=True)
    torch.cuda.synchronize()
    ref = {"attn": db.attn, "logits": db.logits, "lse": db.lse, "accept_len": db.accept_len, "out_tok": db.out_tok,
           "new_kv_len": db.new_kv_len}
    for k, v in ref.items():
        assert torch.equal(static[k], v), k
    assert int(static["accept_len"].min()) >= 0
    return int(x.kv_len.sum())


def test_static_scratch_step_matches_workspace_step_twice():
    big = _check(LARGE, packed=True)
    small = _check(SMALL, packed=False)
    assert small < big
    announce(f"static-scratch step: {LARGE.name} ({big} keys) then {SMALL.name} ({small} keys) identical to "
             f"the workspace step")


def test_static_scratch_step_matches_workspace_step_wide_projection():
    """The same, with the wide projection schedule on the static scratch,
    then the small problem again."""
    assert sd.sd_vocab_kernel_name(sd.Dims.of(WIDE, packed_vocab=True)) == "vocab_bf16_wide_kernel"
    wide = _check(WIDE, packed=True)
    small = _check(SMALL, packed=True)
    assert small < wide
    announce(f"static-scratch step (wide projection): identical to the workspace step")
