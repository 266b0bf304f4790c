"""Helpers shared by the GPU tests: device upload of generated inputs, the
documented tolerance rule, and the exact-parity rule for acceptance."""

from __future__ import annotations

import math

import numpy as np
import torch

import paper_2601_21622_amd as sd
from oracle import near_threshold

RTOL = {"bf16": 2e-2, "f32": 1e-4}


def gpu_available() -> bool:
    return torch.cuda.is_available()


def announce(msg: str) -> None:
    print(f"[gpu-test] {msg}", flush=True)


def tensor(a: np.ndarray, dev="cuda"):
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


class DeviceBatch:
    """Device copies of a VerifyInputs plus output buffers and the workspace."""

    def __init__(self, x, dev="cuda", packed_vocab=False):
        c = x.cfg
        self.x = x
        self.cfg = c
        self.dims = sd.Dims.of(c, packed_vocab=packed_vocab)
        B, G, M, V = c.batch, c.positions, c.rows, c.vocab
        self.q = tensor(x.q, dev)
        self.k = tensor(x.k_pool, dev)
        self.v = tensor(x.v_pool, dev)
        self.hidden = tensor(x.hidden, dev)
        self.w = tensor(x.w, dev)
        if packed_vocab:
            packed = torch.empty((sd.sd_vocab_packed_bytes(self.dims) // 2,), dtype=torch.bfloat16, device=dev)
            sd.sd_pack_vocab(self.dims, self.w, packed)
            self.w = packed
        self.q_draft = tensor(x.q_draft, dev)
        self.draft = tensor(x.draft, dev)
        self.u = tensor(x.u, dev)
        adt = torch.bfloat16 if c.dtype == "bf16" else torch.float32
        self.attn = torch.empty((B, G, c.n_q_heads, c.head_dim), dtype=adt, device=dev)
        self.logits = torch.empty((M, V), dtype=torch.float32, device=dev)
        self.lse = torch.empty((M,), dtype=torch.float32, device=dev)
        self.accept_len = torch.empty((B,), dtype=torch.int32, device=dev)
        self.out_tok = torch.empty((B, G), dtype=torch.int32, device=dev)
        self.new_kv_len = torch.empty((B,), dtype=torch.int32, device=dev)
        nbytes = sd.sd_workspace_bytes(self.dims, int(x.kv_len.max()))
        assert nbytes > 0
        self.ws = torch.empty((nbytes,), dtype=torch.uint8, device=dev)
        self.scale = 1.0 / math.sqrt(c.head_dim)

    def attention(self):
        sd.sd_verify_attention(self.dims, self.q, self.k, self.v, self.x.kv_off, self.x.kv_len, self.scale,
                               self.attn, self.ws)

    def logits_(self, hidden=None):
        sd.sd_verify_logits(self.dims, self.hidden if hidden is None else hidden, self.w, self.logits, self.lse,
                            self.ws)

    def accept(self, probs=None, lse="own"):
        x = self.logits if probs is None else probs
        l = self.lse if (probs is None and lse == "own") else None
        sd.sd_accept_resample(self.dims, x, l, self.q_draft, self.draft, self.u, self.x.kv_len,
                              self.accept_len, self.out_tok, self.new_kv_len, self.ws)

    def step(self, use_hidden=True, kernel_events=None):
        sd.sd_verify_step(self.dims, self.q, self.k, self.v, self.x.kv_off, self.x.kv_len, self.scale,
                          self.hidden if use_hidden else None, self.w, self.q_draft, self.draft, self.u,
                          self.attn, self.logits, self.lse, self.accept_len, self.out_tok, self.new_kv_len,
                          self.ws, kernel_events=kernel_events)


def to_np(t: torch.Tensor) -> np.ndarray:
    t = t.detach()
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy()


def assert_close_rows(gpu: np.ndarray, ref: np.ndarray, rtol: float, what: str):
    """|gpu - ref| <= rtol * max(|ref|, rms(ref row)), rows along the last axis."""
    g = gpu.astype(np.float64).reshape(-1, gpu.shape[-1])
    r = ref.astype(np.float64).reshape(-1, ref.shape[-1])
    rms = np.sqrt((r * r).mean(axis=1, keepdims=True))
    bound = rtol * np.maximum(np.abs(r), rms)
    err = np.abs(g - r)
    bad = err > bound
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} elements exceed the bound; first at {tuple(i)}: "
                             f"gpu={g[tuple(i)]!r} ref={r[tuple(i)]!r} bound={bound[tuple(i)]!r}; "
                             f"max rel err {float((err / np.maximum(np.abs(r), rms)).max()):.3e}")
    return float((err / np.maximum(np.abs(r), rms)).max())


def max_excluded(batch: int) -> int:
    """Requests a parity test may set aside as near-threshold: a draw falls
    within 1e-6 of a boundary with probability of order 1e-5 per request, so
    more than max(1, 1% of the batch) means the band helper over-fires."""
    return max(1, batch // 100)


def assert_accept_parity(gpu_len, gpu_tok, gpu_new, ref, band=1e-6):
    """Bit-exact accept lengths, emitted tokens and new lengths, excluding
    requests whose draws fall within ``band`` of a decision boundary (at most
    max_excluded of them)."""
    near = np.array([near_threshold(t, band) for t in ref["traces"]])
    assert int(near.sum()) <= max_excluded(len(near)), f"{int(near.sum())} of {len(near)} requests near a boundary"
    keep = ~near
    assert np.array_equal(gpu_len[keep], ref["accept_len"][keep]), (gpu_len, ref["accept_len"])
    assert np.array_equal(gpu_tok[keep], ref["out_tok"][keep]), (gpu_tok, ref["out_tok"])
    if ref["new_kv_len"] is not None and gpu_new is not None:
        assert np.array_equal(gpu_new[keep], ref["new_kv_len"][keep])
    return int(near.sum())
