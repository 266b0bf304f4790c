"""GPU parity of verification over paged KV caches (sd_verify_attention_paged,
sd_verify_step_paged) against the oracle (oracle.paged: rows gathered through
the block table, then the chain attention definition).

Pages are a seeded permutation of the pool handed out one page per request
in turn, so each request's pages are scattered and interleaved.  Rows past a request's length inside its last page, and pages nobody holds,
are filled with bf16 NaN: any read of them would show up in the output.
Tolerance as for the segment layout (|gpu - oracle| <= 2e-2 * max(|oracle|,
rms of the row)).  Shapes: one and several 16-row blocks per KV head (the
register-staged and the LDS-DMA kernels), head dims 64 and 128, page sizes
64 to 4096, lengths inside, at and one past page boundaries, down to G,
more than 64 requests, and the pooled workload at its full size in the
launch configuration bench.py times.
"""

import numpy as np
import pytest
import torch

import paper_2601_21622_amd as sd
from oracle import accept_resample, paged_attention, verify_logits
from workloads import get_config, make_inputs

from gpu_util import RTOL, DeviceBatch, announce, assert_accept_parity, assert_close_rows, tensor, to_np

pytestmark = pytest.mark.gpu

BF16_NAN = np.uint16(0x7FC0)


def build_pages(x, P, spare=5, seed=0):
    """Scatter the workload's per-request caches into pages; returns (k_pages,
    v_pages, table, num_pages) as host arrays.  Pages are a seeded permutation
    of the pool handed out round-robin, one page per request at a time, so a
    request's pages are scattered and interleaved with the others'."""
    c = x.cfg
    Hkv, D, B = c.n_kv_heads, c.head_dim, c.batch
    need = [(int(L) + P - 1) // P for L in x.kv_len]
    num_pages = sum(need) + spare
    order = iter(np.random.default_rng(seed).permutation(num_pages).tolist())
    max_pages = max(need)
    table = np.full((B, max_pages), -1, dtype=np.int32)
    for j in range(max_pages):
        for b in range(B):
            if j < need[b]:
                table[b, j] = next(order)
    kp = np.full((num_pages, Hkv, P, D), BF16_NAN, dtype=np.uint16)
    vp = np.full_like(kp, BF16_NAN)
    for b in range(B):
        L, off = int(x.kv_len[b]), int(x.kv_off[b])
        segk = x.k_pool[off:off + Hkv * L * D].reshape(Hkv, L, D)
        segv = x.v_pool[off:off + Hkv * L * D].reshape(Hkv, L, D)
        for j in range(need[b]):
            k0, k1 = j * P, min(L, (j + 1) * P)
            kp[table[b, j], :, :k1 - k0] = segk[:, k0:k1]
            vp[table[b, j], :, :k1 - k0] = segv[:, k0:k1]
    return kp, vp, table, num_pages


def f32(a):
    return (a.astype(np.uint32) << 16).view(np.float32)


CASES = {
    "mha_p64": (get_config("vicuna7b").replace(batch=4, n_q_heads=4, n_kv_heads=4, hidden=512, vocab=256,
                                               lengths=("explicit", (6, 65, 700, 1300))), 64),
    "mha_p256": (get_config("vicuna7b").replace(batch=3, n_q_heads=4, n_kv_heads=4, hidden=512, vocab=256,
                                                lengths=("explicit", (256, 257, 1100))), 256),
    "gqa4_p128": (get_config("llama3_8b").replace(batch=3, n_q_heads=8, n_kv_heads=2, hidden=1024, vocab=256,
                                                  lengths=("explicit", (7, 300, 2100))), 128),
    "gqa8_p64": (get_config("llama70b_share").replace(batch=2, n_q_heads=16, n_kv_heads=2, hidden=2048, vocab=256,
                                                      lengths=("explicit", (9, 4100))), 64),
    "mha64_p64": (get_config("vicuna7b").replace(batch=3, gamma=3, n_q_heads=4, n_kv_heads=4, head_dim=64,
                                                 hidden=256, vocab=256, lengths=("explicit", (4, 64, 200))), 64),
    "many_requests_p64": (get_config("pooled").replace(batch=70, n_q_heads=2, n_kv_heads=2, hidden=256, vocab=128,
                                                       lengths=("uniform", 5, 700)), 64),
    "gqa_p4096": (get_config("llama3_8b").replace(batch=2, n_q_heads=8, n_kv_heads=2, hidden=1024, vocab=256,
                                                  lengths=("explicit", (5000, 20))), 4096),
    # 88 rows per KV head: two row groups of 3 blocks.
    "gqa8_rows88_p64": (get_config("llama70b_share").replace(batch=2, gamma=10, n_q_heads=16, n_kv_heads=2,
                                                             hidden=2048, vocab=256, lengths=("explicit", (11, 1030))),
                        64),
}


def _pages_on_device(x, P):
    kp, vp, table, num_pages = build_pages(x, P)
    dt = tensor(table)
    return tensor(kp), tensor(vp), dt, sd.KVPages.of(dt, P, num_pages), (kp, vp, table)


@pytest.mark.parametrize("name", sorted(CASES))
def test_paged_attention_matches_oracle(name):
    cfg, P = CASES[name]
    announce(f"paged attention case={name} B={cfg.batch} G={cfg.positions} Hq={cfg.n_q_heads} Hkv={cfg.n_kv_heads} "
             f"D={cfg.head_dim} page={P}")
    x = make_inputs(cfg)
    db = DeviceBatch(x)
    kd, vd, _t, pages, (kp, vp, table) = _pages_on_device(x, P)
    sd.sd_verify_attention_paged(db.dims, db.q, kd, vd, pages, x.kv_len, db.scale, db.attn, db.ws)
    got = to_np(db.attn)
    assert np.all(np.isfinite(got))
    ref = paged_attention(x.f32("q"), f32(kp), f32(vp), table, x.kv_len, P)
    err = assert_close_rows(got, ref, RTOL[cfg.dtype], f"paged attention[{name}]")
    announce(f"paged attention case={name}: max scaled err {err:.3e}")


def test_paged_step_matches_oracle():
    cfg = get_config("llama3_8b").replace(batch=3, n_q_heads=8, n_kv_heads=2, hidden=1024, vocab=2500,
                                          lengths=("explicit", (7, 900, 130)))
    P = 64
    announce(f"paged step case=gqa_small page={P}")
    x = make_inputs(cfg)
    db = DeviceBatch(x)
    kd, vd, _t, pages, (kp, vp, table) = _pages_on_device(x, P)
    sd.sd_verify_step_paged(db.dims, db.q, kd, vd, pages, x.kv_len, db.scale, db.hidden, db.w, db.q_draft, db.draft,
                            db.u, db.attn, db.logits, db.lse, db.accept_len, db.out_tok, db.new_kv_len, db.ws)
    torch.cuda.synchronize()
    rtol = RTOL[cfg.dtype]
    assert_close_rows(to_np(db.attn), paged_attention(x.f32("q"), f32(kp), f32(vp), table, x.kv_len, P), rtol,
                      "paged step attention")
    logits_ref, _ = verify_logits(x.f32("hidden"), x.f32("w"))
    assert_close_rows(to_np(db.logits), logits_ref, rtol, "paged step logits")
    ref = accept_resample(to_np(db.logits), to_np(db.lse), x.q_draft, x.draft, x.u, kv_len=x.kv_len)
    near = assert_accept_parity(to_np(db.accept_len), to_np(db.out_tok), to_np(db.new_kv_len), ref)
    announce(f"paged step: near-threshold {near}")


def test_paged_step_full_size_pooled():
    cfg = get_config("pooled")
    P = 64
    announce(f"paged full-size step case=pooled B={cfg.batch} page={P}")
    x = make_inputs(cfg)
    db = DeviceBatch(x, packed_vocab=True)
    kd, vd, _t, pages, (kp, vp, table) = _pages_on_device(x, P)
    sd.sd_verify_step_paged(db.dims, db.q, kd, vd, pages, x.kv_len, db.scale, db.hidden, db.w, db.q_draft, db.draft,
                            db.u, db.attn, db.logits, db.lse, db.accept_len, db.out_tok, db.new_kv_len, db.ws)
    torch.cuda.synchronize()
    got = to_np(db.attn)
    assert np.all(np.isfinite(got))
    order = np.argsort(x.kv_len)
    reqs = np.unique([order[0], order[len(order) // 2], order[-1]])
    ref = paged_attention(x.f32("q")[reqs], f32(kp), f32(vp), table[reqs], x.kv_len[reqs], P)
    assert_close_rows(got[reqs], ref, RTOL[cfg.dtype], "paged full-size attention")
    logits, lse = to_np(db.logits), to_np(db.lse)
    ref_acc = accept_resample(logits, lse, x.q_draft, x.draft, x.u, kv_len=x.kv_len)
    near = assert_accept_parity(to_np(db.accept_len), to_np(db.out_tok), to_np(db.new_kv_len), ref_acc)
    announce(f"paged full-size step: near-threshold {near}")
