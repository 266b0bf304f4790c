"""GPU parity: sd_verify_logits (vocabulary projection + row log-sum-exp)
against the float64 oracle.  Shapes cover the shallow bf16 schedule (at most
64 rows) and each deep shape (one or two 32-entry vocabulary blocks per wave,
four or eight waves per workgroup), ragged vocabulary tiles (V not a multiple
of the tile, and not of 4), K not a multiple of the chunk, several M-tiles,
and the tiny fp32 case."""

import numpy as np
import pytest
import torch

from oracle import verify_logits
from workloads import get_config, make_inputs

from gpu_util import RTOL, DeviceBatch, announce, assert_close_rows, to_np

pytestmark = pytest.mark.gpu

_v = get_config("vicuna7b")
CASES = {
    "tiny_f32": get_config("tiny"),
    "m18_k512_v1000": _v.replace(batch=3, n_q_heads=4, n_kv_heads=4, hidden=512, vocab=1000,
                                 lengths=("fixed", 16)),
    "m18_k512_v1003": _v.replace(batch=3, n_q_heads=4, n_kv_heads=4, hidden=512, vocab=1003,
                                 lengths=("fixed", 16)),
    "m100_k256_v777": _v.replace(batch=20, gamma=4, n_q_heads=2, n_kv_heads=2, hidden=256, vocab=777,
                                 lengths=("fixed", 8)),
    "m320_k96_v300": _v.replace(batch=64, gamma=4, n_q_heads=2, n_kv_heads=2, hidden=96, vocab=300,
                                lengths=("fixed", 8)),
    "m336_k256_v130": _v.replace(batch=56, gamma=5, n_q_heads=2, n_kv_heads=2, hidden=256, vocab=130,
                                 lengths=("fixed", 8)),
    # Deep schedule, one 32-entry block per wave, ragged last tile.
    "m80_k128_v65600": _v.replace(batch=16, gamma=4, n_q_heads=2, n_kv_heads=2, hidden=128, vocab=65600,
                                  lengths=("fixed", 8)),
    # Same schedule, K not a multiple of 128, V odd.
    "m272_k96_v65537": _v.replace(batch=34, gamma=7, n_q_heads=2, n_kv_heads=2, hidden=96, vocab=65537,
                                  lengths=("fixed", 8)),
    # Two blocks per wave, four waves (256-wide tiles): one M-tile of 7 row
    # blocks, then two M-tiles; K of 3 and 5 chunks (the 6-stage ring runs
    # past the last chunk), V odd.
    "m224_k96_v32992": _v.replace(batch=32, gamma=6, n_q_heads=2, n_kv_heads=2, hidden=96, vocab=32992,
                                  lengths=("fixed", 8)),
    "m336_k160_v32001": _v.replace(batch=48, gamma=6, n_q_heads=2, n_kv_heads=2, hidden=160, vocab=32001,
                                   lengths=("fixed", 8)),
    # Four blocks per wave, four waves (512-wide tiles, accumulators in both
    # register files, 3-stage ring run in steps of three chunks, the ones
    # past K read as zeros): 7 row blocks with K of 3, 4 and 5 chunks; 200
    # rows (a partial last block) with a ragged last tile; two M-tiles.
    "m224_k96_v100001": _v.replace(batch=32, gamma=6, n_q_heads=2, n_kv_heads=2, hidden=96, vocab=100001,
                                   lengths=("fixed", 8)),
    "m224_k128_v100001": _v.replace(batch=32, gamma=6, n_q_heads=2, n_kv_heads=2, hidden=128, vocab=100001,
                                    lengths=("fixed", 8)),
    # K of one and two chunks: the prologue's second chunk, or the loop's
    # whole second and third, read as zeros.
    "m224_k32_v100001": _v.replace(batch=32, gamma=6, n_q_heads=1, n_kv_heads=1, head_dim=64, hidden=32,
                                   vocab=100001, lengths=("fixed", 8)),
    "m224_k64_v100001": _v.replace(batch=32, gamma=6, n_q_heads=1, n_kv_heads=1, head_dim=64, hidden=64,
                                   vocab=100001, lengths=("fixed", 8)),
    "m200_k160_v70003": _v.replace(batch=25, gamma=7, n_q_heads=2, n_kv_heads=2, hidden=160, vocab=70003,
                                   lengths=("fixed", 8)),
    "m416_k160_v100001": _v.replace(batch=52, gamma=7, n_q_heads=2, n_kv_heads=2, hidden=160, vocab=100001,
                                    lengths=("fixed", 8)),
    # Two blocks per wave, eight waves (512-wide tiles, 3-stage ring), rows
    # not a multiple of 32, V odd.
    "m100_k160_v100003": _v.replace(batch=20, gamma=4, n_q_heads=2, n_kv_heads=2, hidden=160, vocab=100003,
                                    lengths=("fixed", 8)),
    # Degenerate vocabularies (one, two, three entries) on the shallow and
    # the deep schedules and in float32: every tile but the first is empty.
    "m18_k64_v1": _v.replace(batch=3, n_q_heads=2, n_kv_heads=2, hidden=64, vocab=1, lengths=("fixed", 8)),
    "m100_k64_v1": _v.replace(batch=20, gamma=4, n_q_heads=2, n_kv_heads=2, hidden=64, vocab=1,
                              lengths=("fixed", 8)),
    "m48_k64_v2": _v.replace(batch=8, n_q_heads=2, n_kv_heads=2, hidden=64, vocab=2, lengths=("fixed", 8)),
    "m416_k64_v3": _v.replace(batch=52, gamma=7, n_q_heads=2, n_kv_heads=2, hidden=64, vocab=3,
                              lengths=("fixed", 8)),
    # The largest vocabulary the boundary takes (2,097,152 entries).
    "m18_k32_v2097152": _v.replace(batch=3, n_q_heads=2, n_kv_heads=2, hidden=32, vocab=2097152,
                                   lengths=("fixed", 8)),
    "f32_m10_k64_v1": get_config("tiny").replace(batch=2, gamma=4, hidden=64, vocab=1, lengths=("fixed", 8)),
    "f32_m70_k128_v65": get_config("tiny").replace(batch=14, gamma=4, hidden=128, vocab=65, lengths=("fixed", 8)),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_logits_match_oracle(name):
    cfg = CASES[name]
    announce(f"logits parity case={name} M={cfg.rows} K={cfg.hidden} V={cfg.vocab} dtype={cfg.dtype}")
    x = make_inputs(cfg)
    db = DeviceBatch(x)
    db.logits_()
    ref_logits, ref_lse = verify_logits(x.f32("hidden"), x.f32("w"))
    err = assert_close_rows(to_np(db.logits), ref_logits, RTOL[cfg.dtype], f"logits[{name}]")
    lse = to_np(db.lse).astype(np.float64)
    assert np.all(np.abs(lse - ref_lse) <= RTOL[cfg.dtype] * np.maximum(np.abs(ref_lse), 1.0)), (lse, ref_lse)
    # The float32 logits with the float32 lse give distributions that sum to one.
    p = np.exp(to_np(db.logits).astype(np.float64) - lse[:, None])
    assert np.allclose(p.sum(axis=1), 1.0, atol=1e-5)
    announce(f"logits case={name} max scaled err {err:.3e} max |dlse| {np.abs(lse - ref_lse).max():.3e}")


@pytest.mark.parametrize("name", ["m18_k512_v1000", "m18_k512_v1003", "m100_k256_v777", "m336_k256_v130",
                                  "m272_k96_v65537", "m224_k96_v32992", "m416_k160_v100001", "m200_k160_v70003",
                                  "m100_k160_v100003", "m100_k64_v1", "m416_k64_v3"])
def test_packed_vocab_matches_row_major_bitwise(name):
    """The packed layout changes where W is read from, not the arithmetic:
    logits and log-sum-exp must be bit-identical to the row-major path."""
    cfg = CASES[name]
    announce(f"packed vocab case={name}")
    x = make_inputs(cfg)
    a = DeviceBatch(x)
    b = DeviceBatch(x, packed_vocab=True)
    a.logits_()
    b.logits_()
    assert np.array_equal(to_np(a.logits), to_np(b.logits))
    assert np.array_equal(to_np(a.lse), to_np(b.lse))
    # The packed buffer itself: fragment (s, n), lane l holds W[16n + l%16][32s + 8(l/16) .. +8].
    V, K = cfg.vocab, cfg.hidden
    nb = (V + 15) // 16
    w = np.zeros((nb * 16, K), dtype=np.uint16)
    w[:V] = x.w
    want = w.reshape(nb, 16, K // 32, 4, 8).transpose(2, 0, 3, 1, 4).reshape(-1)
    got = b.w.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, want)


def test_logits_deterministic():
    x = make_inputs(CASES["m100_k256_v777"])
    db = DeviceBatch(x)
    db.logits_()
    a, b = to_np(db.logits).copy(), to_np(db.lse).copy()
    db.logits.zero_()
    db.lse.zero_()
    db.logits_()
    assert np.array_equal(a, to_np(db.logits)) and np.array_equal(b, to_np(db.lse))
