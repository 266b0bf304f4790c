"""GPU parity: sd_verify_attention against the float64 oracle (tolerance rule:
|gpu - oracle| <= rtol * max(|oracle|, rms of the oracle row); rtol 2e-2 for
bf16, 1e-4 for fp32).  Shapes span several 32-key tiles and 512+-key chunks,
ragged tails, the shortest cache (L = G), GQA groups 1/4/8/16 (1 to 8 blocks
of 16 query rows per KV head), head_dim 64/128, and more requests than one
launch carries."""

import numpy as np
import pytest

from oracle import verify_attention
from workloads import get_config, make_inputs

from gpu_util import RTOL, DeviceBatch, announce, assert_close_rows, to_np

pytestmark = pytest.mark.gpu

CASES = {
    "tiny_f32": get_config("tiny"),
    "mha128_bf16": get_config("vicuna7b").replace(batch=4, n_q_heads=4, n_kv_heads=4, hidden=512, vocab=256,
                                                    lengths=("explicit", (6, 37, 513, 1100))),
    "gqa4_bf16": get_config("llama3_8b").replace(batch=3, n_q_heads=8, n_kv_heads=2, hidden=1024, vocab=256,
                                                 lengths=("explicit", (7, 300, 2100))),
    "gqa8_bf16": get_config("llama70b_share").replace(batch=3, n_q_heads=16, n_kv_heads=2, hidden=2048,
                                                      vocab=256, lengths=("explicit", (9, 1500, 4100))),
    "mha64_bf16": get_config("vicuna7b").replace(batch=3, gamma=3, n_q_heads=4, n_kv_heads=4, head_dim=64,
                                                  hidden=256, vocab=256, lengths=("explicit", (4, 65, 200))),
    "gqa2_f32": get_config("tiny").replace(batch=3, n_q_heads=4, n_kv_heads=2, head_dim=128, hidden=512,
                                           vocab=256, lengths=("explicit", (5, 70, 300))),
    "many_requests_bf16": get_config("pooled").replace(batch=70, n_q_heads=2, n_kv_heads=2, hidden=256,
                                                       vocab=128, lengths=("uniform", 5, 700)),
    # Query rows per KV head = G * group: 40 (3 blocks of 16), 56 (4, head_dim 64), 88 (6 blocks: two row
    # groups of 3 at head_dim 128), 112 (7: groups of 4 and 3), 128 (8: 4 and 4), 120 at head_dim 64 (8
    # blocks in one wave).
    "rows40_bf16": get_config("llama70b_share").replace(batch=2, gamma=4, n_q_heads=16, n_kv_heads=2, hidden=2048,
                                                        vocab=256, lengths=("explicit", (5, 777))),
    "rows56_d64_bf16": get_config("llama70b_share").replace(batch=2, gamma=6, n_q_heads=16, n_kv_heads=2,
                                                            head_dim=64, hidden=1024, vocab=256,
                                                            lengths=("explicit", (600, 7))),
    "rows88_bf16": get_config("llama70b_share").replace(batch=2, gamma=10, n_q_heads=16, n_kv_heads=2,
                                                        hidden=2048, vocab=256, lengths=("explicit", (11, 1030))),
    "rows112_bf16": get_config("llama70b_share").replace(batch=2, gamma=6, n_q_heads=32, n_kv_heads=2,
                                                         hidden=4096, vocab=256, lengths=("explicit", (700, 33))),
    "rows128_bf16": get_config("llama70b_share").replace(batch=2, gamma=7, n_q_heads=32, n_kv_heads=2,
                                                         hidden=4096, vocab=256, lengths=("explicit", (8, 2200))),
    "rows120_d64_bf16": get_config("llama70b_share").replace(batch=2, gamma=14, n_q_heads=16, n_kv_heads=2,
                                                             head_dim=64, hidden=1024, vocab=256,
                                                             lengths=("explicit", (1500, 15))),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_attention_matches_oracle(name):
    cfg = CASES[name]
    announce(f"attention parity case={name} B={cfg.batch} gamma={cfg.gamma} Hq={cfg.n_q_heads} "
             f"Hkv={cfg.n_kv_heads} D={cfg.head_dim} dtype={cfg.dtype}")
    x = make_inputs(cfg)
    db = DeviceBatch(x)
    db.attention()
    got = to_np(db.attn)
    ref = verify_attention(x.f32("q"), x.f32("k_pool"), x.f32("v_pool"), x.kv_off, x.kv_len, cfg.n_kv_heads)
    err = assert_close_rows(got, ref, RTOL[cfg.dtype], f"attention[{name}]")
    announce(f"attention case={name} max scaled err {err:.3e}")


def test_attention_deterministic():
    cfg = CASES["gqa4_bf16"]
    x = make_inputs(cfg)
    db = DeviceBatch(x)
    db.attention()
    a = to_np(db.attn).copy()
    db.attn.zero_()
    db.attention()
    assert np.array_equal(a, to_np(db.attn))
