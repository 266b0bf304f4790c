"""The C-ABI library on the CPU: it loads, exports every function the header
declares, and rejects invalid arguments with the documented status before
enqueuing anything (these calls never reach a kernel launch)."""

import ctypes

import pytest
import torch

import paper_2601_21622_amd as sd

# Fake, suitably aligned device addresses: every call below fails its host
# checks before any pointer is used.
P = 0x100000
cpu_only = pytest.mark.skipif(torch.cuda.is_available(), reason="host-validation tests use fake pointers")


def dims(**kw):
    base = dict(batch=2, gamma=3, n_q_heads=8, n_kv_heads=2, head_dim=128, hidden=1024, vocab=1000, dtype=1)
    base.update(kw)
    return sd.Dims(**base)


def test_library_loads_and_exports_header_symbols():
    lib = sd.library()
    names = sd.exported_symbols()
    assert set(names) == {"sd_workspace_bytes", "sd_verify_attention", "sd_verify_logits", "sd_accept_resample",
                          "sd_verify_step", "sd_status_string", "sd_version", "sd_vocab_packed_bytes",
                          "sd_pack_vocab", "sd_accept_resample_sampled", "sd_verify_step_sampled",
                          "sd_verify_attention_tree", "sd_accept_tree", "sd_verify_step_tree", "sd_tree_commit_kv",
                          "sd_acceptance_rate", "sd_verify_attention_paged", "sd_verify_step_paged",
                          "sd_kv_pool_create", "sd_kv_pool_destroy", "sd_kv_pool_reserve", "sd_kv_pool_truncate",
                          "sd_kv_pool_release", "sd_kv_pool_free_pages", "sd_kv_pool_tag_pages",
                          "sd_kv_pool_block_table", "sd_expand_layer", "sd_verify_step_static",
                          "sd_vocab_kernel_name"}
    for n in names:
        assert hasattr(lib, n), n
    assert sd.sd_version().count(".") == 2


def test_vocab_kernel_name_follows_the_plan():
    """The projection kernel the plan picks: the shallow schedule up to 64
    rows, the wide one where one M-tile of up to 224 rows meets a vocabulary
    large enough for 512-wide tiles to fill the chip, the deep one otherwise."""
    from workloads import get_config

    def name(cfg, **kw):
        d = dict(batch=cfg.batch, gamma=cfg.gamma, n_q_heads=cfg.n_q_heads, n_kv_heads=cfg.n_kv_heads,
                 head_dim=cfg.head_dim, hidden=cfg.hidden, vocab=cfg.vocab, dtype=1 if cfg.dtype == "bf16" else 0)
        d.update(kw)
        return sd.sd_vocab_kernel_name(sd.Dims(**d))

    assert name(get_config("tiny")) == "vocab_f32_kernel"
    assert name(get_config("vicuna7b")) == "vocab_bf16_kernel"
    assert name(get_config("pooled")) == "vocab_bf16_deep_kernel"
    assert name(get_config("llama3_8b")) == "vocab_bf16_wide_kernel"
    assert name(get_config("llama3_8b"), flags=sd.SD_FLAG_PACKED_VOCAB) == "vocab_bf16_wide_kernel"
    assert name(get_config("llama70b_share")) == "vocab_bf16_deep_kernel"
    assert name(get_config("llama3_8b"), vocab=30000) == "vocab_bf16_deep_kernel"
    # W past 4 GB: the wide schedule's 32-bit offsets rule it out.
    assert name(get_config("llama3_8b"), hidden=16384, vocab=2_000_000) == "vocab_bf16_deep_kernel"
    assert name(get_config("llama3_8b"), hidden=8192, vocab=250_000) == "vocab_bf16_wide_kernel"
    assert sd.sd_vocab_kernel_name(dims(head_dim=96)) is None


def test_status_strings():
    for st in (sd.SD_OK, sd.SD_ERR_INVALID_ARGUMENT, sd.SD_ERR_UNSUPPORTED, sd.SD_ERR_WORKSPACE, sd.SD_ERR_HIP):
        assert sd.sd_status_string(st).startswith("SD_")
    assert sd.sd_status_string(12345) == "unknown status"


def test_workspace_bytes():
    d = dims()
    a = sd.sd_workspace_bytes(d, 1000)
    b = sd.sd_workspace_bytes(d, 100000)
    assert 0 < a < b
    assert sd.sd_workspace_bytes(d, 3) == 0           # shorter than gamma + 1
    assert sd.sd_workspace_bytes(dims(head_dim=96), 1000) == 0
    assert sd.sd_workspace_bytes(dims(n_q_heads=7), 1000) == 0


def _attn(d, kv_off=(0, 8 * 128 * 2 * 64), kv_len=(64, 64), ws_bytes=1 << 30, q=P, k=P, v=P, out=P, ws=P,
          scale=0.088):
    lib = sd.library()
    off = (ctypes.c_int64 * len(kv_off))(*kv_off)
    ln = (ctypes.c_int32 * len(kv_len))(*kv_len)
    return lib.sd_verify_attention(ctypes.byref(d), q, k, v, off, ln, scale, out, ws, ws_bytes, None)


@cpu_only
@pytest.mark.parametrize("bad,status", [
    (dict(batch=0), sd.SD_ERR_INVALID_ARGUMENT),
    (dict(gamma=0), sd.SD_ERR_INVALID_ARGUMENT),
    (dict(n_q_heads=6, n_kv_heads=4), sd.SD_ERR_INVALID_ARGUMENT),
    (dict(dtype=7), sd.SD_ERR_INVALID_ARGUMENT),
    (dict(head_dim=96), sd.SD_ERR_UNSUPPORTED),
    (dict(hidden=100), sd.SD_ERR_UNSUPPORTED),
    (dict(gamma=64), sd.SD_ERR_UNSUPPORTED),
    (dict(n_q_heads=68, n_kv_heads=2), sd.SD_ERR_UNSUPPORTED),   # 4 * 34 > 128 rows per KV head
    (dict(vocab=3_000_000), sd.SD_ERR_UNSUPPORTED),
])
def test_attention_rejects_bad_dims(bad, status):
    assert _attn(dims(**bad)) == status


@cpu_only
def test_attention_rejects_bad_pointers_lengths_and_workspace():
    d = dims()
    assert _attn(d, q=None) == sd.SD_ERR_INVALID_ARGUMENT
    assert _attn(d, k=P + 8) == sd.SD_ERR_INVALID_ARGUMENT        # misaligned
    assert _attn(d, kv_len=(3, 64)) == sd.SD_ERR_INVALID_ARGUMENT  # shorter than gamma + 1
    assert _attn(d, kv_off=(0, 3)) == sd.SD_ERR_INVALID_ARGUMENT   # offset not 16-byte aligned
    assert _attn(d, kv_off=(-8, 0)) == sd.SD_ERR_INVALID_ARGUMENT
    assert _attn(d, ws_bytes=16) == sd.SD_ERR_WORKSPACE
    assert _attn(d, scale=float("nan")) == sd.SD_ERR_INVALID_ARGUMENT
    assert _attn(d, scale=0.0) == sd.SD_ERR_INVALID_ARGUMENT
    assert _attn(d, scale=-0.088) == sd.SD_ERR_INVALID_ARGUMENT
    assert _attn(d, scale=float("inf")) == sd.SD_ERR_INVALID_ARGUMENT
    lib = sd.library()
    assert lib.sd_verify_attention(ctypes.byref(d), P, P, P, None, None, 0.1, P, P, 1 << 30, None) == \
        sd.SD_ERR_INVALID_ARGUMENT
    assert lib.sd_verify_attention(None, P, P, P, None, None, 0.1, P, P, 1 << 30, None) == sd.SD_ERR_INVALID_ARGUMENT


@cpu_only
def test_logits_and_accept_reject_bad_arguments():
    lib = sd.library()
    d = dims()
    assert lib.sd_verify_logits(ctypes.byref(d), None, P, P, P, P, 1 << 30, None) == sd.SD_ERR_INVALID_ARGUMENT
    assert lib.sd_verify_logits(ctypes.byref(d), P, P, P + 4, P, P, 1 << 30, None) == sd.SD_ERR_INVALID_ARGUMENT
    assert lib.sd_verify_logits(ctypes.byref(d), P, P, P, P, P, 8, None) == sd.SD_ERR_WORKSPACE
    # new_kv_len without kv_len
    assert lib.sd_accept_resample(ctypes.byref(d), P, P, P, P, P, None, P, P, P, None, 0, None) == \
        sd.SD_ERR_INVALID_ARGUMENT
    assert lib.sd_accept_resample(ctypes.byref(d), P, P, P, P + 2, P, None, P, P, None, None, 0, None) == \
        sd.SD_ERR_INVALID_ARGUMENT
    short = (ctypes.c_int32 * 2)(2, 10)
    assert lib.sd_accept_resample(ctypes.byref(d), P, P, P, P, P, short, P, P, P, None, 0, None) == \
        sd.SD_ERR_INVALID_ARGUMENT


@cpu_only
def test_paged_calls_reject_bad_arguments():
    lib = sd.library()
    d = dims()
    ln = (ctypes.c_int32 * 2)(200, 64)

    def attn(pages, dd=d, lens=ln, ws=1 << 30):
        return lib.sd_verify_attention_paged(ctypes.byref(dd), P, P, P, pages, lens, 0.088, P, P, ws, None)

    good = sd.KVPages(P, 4, 64, 16)
    assert attn(None) == sd.SD_ERR_INVALID_ARGUMENT
    assert attn(ctypes.byref(sd.KVPages(None, 4, 64, 16))) == sd.SD_ERR_INVALID_ARGUMENT
    for bad in (sd.KVPages(P, 4, 32, 16), sd.KVPages(P, 4, 96, 16), sd.KVPages(P, 4, 8192, 16),
                sd.KVPages(P, 0, 64, 16), sd.KVPages(P, 4, 64, 0), sd.KVPages(P + 2, 4, 64, 16),
                sd.KVPages(P, 3, 64, 16)):                      # 3 pages of 64 < kv_len 200
        assert attn(ctypes.byref(bad)) == sd.SD_ERR_INVALID_ARGUMENT
    assert attn(ctypes.byref(good), dd=dims(dtype=0)) == sd.SD_ERR_UNSUPPORTED
    assert attn(ctypes.byref(good), lens=(ctypes.c_int32 * 2)(3, 64)) == sd.SD_ERR_INVALID_ARGUMENT   # < G
    assert attn(ctypes.byref(good), ws=8) == sd.SD_ERR_WORKSPACE
    step = lib.sd_verify_step_paged
    assert step(ctypes.byref(d), P, P, P, None, ln, 0.088, P, P, P, P, P, P, P, P, P, P, None, P, 1 << 30, None,
                None) == sd.SD_ERR_INVALID_ARGUMENT
    assert sd.sd_status_string(sd.SD_ERR_CAPACITY).startswith("SD_ERR_CAPACITY")


@cpu_only
def test_expand_rejects_bad_arguments():
    lib = sd.library()

    def call(**kw):
        base = dict(batch=2, frontier=3, vocab=100, top_k=4, frontier0=1, first_child=4, nodes=16)
        base.update(kw)
        return lib.sd_expand_layer(ctypes.byref(sd.Expand(**base)), P, P, P, P, None)

    assert lib.sd_expand_layer(None, P, P, P, P, None) == sd.SD_ERR_INVALID_ARGUMENT
    assert lib.sd_expand_layer(ctypes.byref(sd.Expand(2, 3, 100, 4, 1, 4, 16)), P + 2, P, P, P, None) == \
        sd.SD_ERR_INVALID_ARGUMENT
    assert call(top_k=0) == sd.SD_ERR_INVALID_ARGUMENT
    assert call(top_k=17) == sd.SD_ERR_UNSUPPORTED
    assert call(vocab=3) == sd.SD_ERR_INVALID_ARGUMENT              # k > V
    assert call(nodes=15) == sd.SD_ERR_INVALID_ARGUMENT             # 4 + 3*4 > 15
    assert call(frontier0=2) == sd.SD_ERR_INVALID_ARGUMENT          # frontier 2..4 overlaps the children at 4
    assert call(frontier0=-2) == sd.SD_ERR_INVALID_ARGUMENT
    assert call(batch=0) == sd.SD_ERR_INVALID_ARGUMENT


@cpu_only
def test_acceptance_rate_rejects_bad_arguments():
    lib = sd.library()
    d = dims()
    call = lib.sd_acceptance_rate
    assert call(ctypes.byref(d), None, P, P, P, P, 1 << 30, None) == sd.SD_ERR_INVALID_ARGUMENT
    assert call(ctypes.byref(d), P, P, None, P, P, 1 << 30, None) == sd.SD_ERR_INVALID_ARGUMENT
    assert call(ctypes.byref(d), P, P, P, None, P, 1 << 30, None) == sd.SD_ERR_INVALID_ARGUMENT
    assert call(ctypes.byref(d), P, P, P, P + 4, P, 1 << 30, None) == sd.SD_ERR_INVALID_ARGUMENT   # beta: 8-byte
    assert call(ctypes.byref(d), P + 2, P, P, P, P, 1 << 30, None) == sd.SD_ERR_INVALID_ARGUMENT
    assert call(ctypes.byref(d), P, P, P, P, P + 8, 1 << 30, None) == sd.SD_ERR_INVALID_ARGUMENT   # ws: 16-byte
    assert call(ctypes.byref(d), P, P, P, P, P, 8, None) == sd.SD_ERR_WORKSPACE
    assert call(ctypes.byref(dims(gamma=0)), P, P, P, P, P, 1 << 30, None) == sd.SD_ERR_INVALID_ARGUMENT
    # The step-sized workspace covers the rate's.
    assert sd.sd_workspace_bytes(d, 1000) >= 8


@cpu_only
def test_sampled_calls_reject_bad_sampling_and_arguments():
    lib = sd.library()
    d = dims()

    def acc(sp, row_min=P, ws_bytes=1 << 30):
        return lib.sd_accept_resample_sampled(ctypes.byref(d), None if sp is None else ctypes.byref(sp), P, P, P, P,
                                              None, P, row_min, P, P, None, P, ws_bytes, None)

    good = sd.Sampling(0.8, 50, 0.9)
    for bad in (None, sd.Sampling(-1.0, 0, 1.0), sd.Sampling(float("nan"), 0, 1.0), sd.Sampling(float("inf"), 0, 1.0),
                sd.Sampling(1.0, -1, 1.0), sd.Sampling(1.0, 0, 0.0), sd.Sampling(1.0, 0, 1.5),
                sd.Sampling(1.0, 0, float("nan"))):
        assert acc(bad) == sd.SD_ERR_INVALID_ARGUMENT
    assert acc(good, row_min=None) == sd.SD_ERR_INVALID_ARGUMENT
    assert acc(good, row_min=P + 2) == sd.SD_ERR_INVALID_ARGUMENT
    assert acc(good, ws_bytes=64) == sd.SD_ERR_WORKSPACE
    off = (ctypes.c_int64 * 2)(0, 8 * 128 * 2 * 64)
    ln = (ctypes.c_int32 * 2)(64, 64)
    args = [P, P, P, off, ln, 0.1, P, P, P, P, P, P, P, P, P, P, P, P, P, 1 << 30, None, None]
    assert lib.sd_verify_step_sampled(ctypes.byref(d), ctypes.byref(sd.Sampling(-2.0, 0, 1.0)), *args) == \
        sd.SD_ERR_INVALID_ARGUMENT
    args_no_min = list(args)
    args_no_min[14] = None  # row_min_logit
    assert lib.sd_verify_step_sampled(ctypes.byref(d), ctypes.byref(good), *args_no_min) == sd.SD_ERR_INVALID_ARGUMENT
    assert sd.sd_workspace_bytes(d, 1000) > 0


@cpu_only
def test_step_rejects_hidden_null_with_mismatched_width():
    lib = sd.library()
    d = dims(hidden=2048)  # != n_q_heads * head_dim = 1024
    off = (ctypes.c_int64 * 2)(0, 8 * 128 * 2 * 64)
    ln = (ctypes.c_int32 * 2)(64, 64)
    st = lib.sd_verify_step(ctypes.byref(d), P, P, P, off, ln, 0.1, None, P, P, P, P, P, P, P, P, P, P, P,
                            1 << 30, None, None)
    assert st == sd.SD_ERR_INVALID_ARGUMENT


@cpu_only
def test_packed_vocab_sizes_and_validation():
    d = dims()
    assert sd.sd_vocab_packed_bytes(d) == 2 * 1024 * 1008   # V rounded up to 16
    assert sd.sd_vocab_packed_bytes(dims(dtype=0)) == 0      # fp32 is not packed
    lib = sd.library()
    assert lib.sd_pack_vocab(ctypes.byref(dims(dtype=0)), P, P + (1 << 24), None) == sd.SD_ERR_UNSUPPORTED
    assert lib.sd_pack_vocab(ctypes.byref(d), P, P + 8, None) == sd.SD_ERR_INVALID_ARGUMENT     # misaligned
    assert lib.sd_pack_vocab(ctypes.byref(d), P, P + 4096, None) == sd.SD_ERR_INVALID_ARGUMENT  # overlap
    assert lib.sd_pack_vocab(ctypes.byref(d), None, P, None) == sd.SD_ERR_INVALID_ARGUMENT
    bad = dims(flags=4)
    assert sd.sd_workspace_bytes(bad, 1000) == 0
    assert sd.sd_workspace_bytes(dims(dtype=0, flags=1), 1000) == 0


def test_binding_requires_device_tensors():
    d = dims()
    with pytest.raises((TypeError, ValueError)):
        sd.sd_verify_logits(d, torch.zeros(4), torch.zeros(4), torch.zeros(4), torch.zeros(4), torch.zeros(4))


@cpu_only
def test_static_step_rejects_before_any_device_work():
    """The no-workspace step checks its arguments and its scratch need on the
    host: a problem beyond the static maximum, a missing length table or a bad
    scale return their status before the device is touched."""
    lib = sd.library()
    args = (P, P, P)

    def call(d, off, ln, scale=0.088):
        return lib.sd_verify_step_static(ctypes.byref(d), *args, off, ln, scale, P, P, P, P, P, P, P, P, P, P, P, None)

    big = dims(batch=64, gamma=8, n_q_heads=64, n_kv_heads=8, hidden=8192, vocab=128256)
    L = 32768
    off = (ctypes.c_int64 * 64)(*[i * 8 * 128 * L for i in range(64)])
    ln = (ctypes.c_int32 * 64)(*([L] * 64))
    assert call(big, off, ln) == sd.SD_ERR_WORKSPACE
    small = dims()
    off2 = (ctypes.c_int64 * 2)(0, 8 * 128 * 2 * 64)
    ln2 = (ctypes.c_int32 * 2)(64, 64)
    assert call(small, off2, None) == sd.SD_ERR_INVALID_ARGUMENT
    assert call(small, off2, ln2, scale=0.0) == sd.SD_ERR_INVALID_ARGUMENT
    assert call(dims(head_dim=96), off2, ln2) == sd.SD_ERR_UNSUPPORTED
