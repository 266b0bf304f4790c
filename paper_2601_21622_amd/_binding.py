"""ctypes marshalling for libsdverify.so.  Argument conversion only."""

from __future__ import annotations

import ctypes
import os
import re
from typing import Optional, Sequence

import numpy as np
import torch  # loaded first so the library binds to the HIP runtime torch already uses

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_NAME = "libsdverify.so"
_HEADER = os.path.join(os.path.dirname(_HERE), "include", "sdverify.h")

SD_DTYPE_F32 = 0
SD_DTYPE_BF16 = 1
SD_FLAG_PACKED_VOCAB = 1
SD_OK = 0
SD_ERR_INVALID_ARGUMENT = -1
SD_ERR_UNSUPPORTED = -2
SD_ERR_WORKSPACE = -3
SD_ERR_HIP = -4
SD_ERR_CAPACITY = -5


class SdError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {sd_status_string(status)} (status {status})")


class Dims(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("gamma", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("hidden", ctypes.c_int32),
        ("vocab", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("flags", ctypes.c_int32),
    ]

    @classmethod
    def of(cls, cfg, packed_vocab: bool = False) -> "Dims":
        """Dims of a workload description (anything with the same attribute names)."""
        return cls(cfg.batch, cfg.gamma, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.hidden,
                   cfg.vocab, SD_DTYPE_BF16 if cfg.dtype == "bf16" else SD_DTYPE_F32,
                   SD_FLAG_PACKED_VOCAB if packed_vocab else 0)

    def with_flags(self, flags: int) -> "Dims":
        return Dims(self.batch, self.gamma, self.n_q_heads, self.n_kv_heads, self.head_dim, self.hidden,
                    self.vocab, self.dtype, flags)


class Sampling(ctypes.Structure):
    """sd_sampling_t: temperature (0 = greedy), top_k (0 = off), top_p (1 = off)."""
    _fields_ = [
        ("temperature", ctypes.c_float),
        ("top_k", ctypes.c_int32),
        ("top_p", ctypes.c_float),
    ]


class KVPages(ctypes.Structure):
    """sd_kv_pages_t: a paged cache's block table (device int32 [B][max_pages]),
    keys per page and pages per pool.  Build it with KVPages.of(table, ...),
    which keeps the table tensor referenced."""
    _fields_ = [
        ("block_table", ctypes.c_void_p),
        ("max_pages", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("num_pages", ctypes.c_int32),
    ]

    @classmethod
    def of(cls, block_table, page_size: int, num_pages: int) -> "KVPages":
        pg = cls(_ptr(block_table), int(block_table.shape[-1]), int(page_size), int(num_pages))
        pg._table = block_table
        return pg


class Expand(ctypes.Structure):
    """sd_expand_t: one layer of draft-side tree expansion."""
    _fields_ = [(n, ctypes.c_int32) for n in ("batch", "frontier", "vocab", "top_k", "frontier0", "first_child",
                                              "nodes")]


_lib: Optional[ctypes.CDLL] = None


def library_path() -> str:
    return os.environ.get("SDVERIFY_LIB", os.path.join(_HERE, _LIB_NAME))


def library() -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2601_21622_amd.build` "
                           "(there is no fallback implementation)")
    lib = ctypes.CDLL(path)
    P, I32, I64, SZ, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_float
    DP = ctypes.POINTER(Dims)
    lib.sd_workspace_bytes.argtypes = [DP, I32]
    lib.sd_workspace_bytes.restype = SZ
    lib.sd_verify_attention.argtypes = [DP, P, P, P, P, P, F, P, P, SZ, P]
    lib.sd_verify_attention.restype = ctypes.c_int
    lib.sd_verify_logits.argtypes = [DP, P, P, P, P, P, SZ, P]
    lib.sd_verify_logits.restype = ctypes.c_int
    lib.sd_accept_resample.argtypes = [DP, P, P, P, P, P, P, P, P, P, P, SZ, P]
    lib.sd_accept_resample.restype = ctypes.c_int
    lib.sd_verify_step.argtypes = [DP, P, P, P, P, P, F, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P, P]
    lib.sd_verify_step.restype = ctypes.c_int
    lib.sd_verify_step_static.argtypes = [DP, P, P, P, P, P, F, P, P, P, P, P, P, P, P, P, P, P, P]
    lib.sd_verify_step_static.restype = ctypes.c_int
    lib.sd_verify_attention_tree.argtypes = [DP, P, P, P, P, P, P, F, P, P, SZ, P]
    lib.sd_verify_attention_tree.restype = ctypes.c_int
    lib.sd_accept_tree.argtypes = [DP, P, P, P, P, P, P, P, P, P, P, P, SZ, P]
    lib.sd_accept_tree.restype = ctypes.c_int
    lib.sd_verify_step_tree.argtypes = [DP, P, P, P, P, P, P, F, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P, P]
    lib.sd_verify_step_tree.restype = ctypes.c_int
    lib.sd_tree_commit_kv.argtypes = [DP, P, P, P, P, P, P, P]
    lib.sd_tree_commit_kv.restype = ctypes.c_int
    lib.sd_acceptance_rate.argtypes = [DP, P, P, P, P, P, SZ, P]
    lib.sd_acceptance_rate.restype = ctypes.c_int
    KP = ctypes.POINTER(KVPages)
    lib.sd_verify_attention_paged.argtypes = [DP, P, P, P, KP, P, F, P, P, SZ, P]
    lib.sd_verify_attention_paged.restype = ctypes.c_int
    lib.sd_verify_step_paged.argtypes = [DP, P, P, P, KP, P, F, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P, P]
    lib.sd_verify_step_paged.restype = ctypes.c_int
    lib.sd_expand_layer.argtypes = [ctypes.POINTER(Expand), P, P, P, P, P]
    lib.sd_expand_layer.restype = ctypes.c_int
    lib.sd_kv_pool_create.argtypes = [I32, I32]
    lib.sd_kv_pool_create.restype = P
    lib.sd_kv_pool_destroy.argtypes = [P]
    lib.sd_kv_pool_destroy.restype = None
    for name in ("sd_kv_pool_reserve", "sd_kv_pool_truncate"):
        getattr(lib, name).argtypes = [P, I32, I32]
        getattr(lib, name).restype = ctypes.c_int
    lib.sd_kv_pool_release.argtypes = [P, I32]
    lib.sd_kv_pool_release.restype = ctypes.c_int
    lib.sd_kv_pool_free_pages.argtypes = [P]
    lib.sd_kv_pool_free_pages.restype = I32
    lib.sd_kv_pool_tag_pages.argtypes = [P, I32]
    lib.sd_kv_pool_tag_pages.restype = I32
    lib.sd_kv_pool_block_table.argtypes = [P, P, I32, I32, P]
    lib.sd_kv_pool_block_table.restype = ctypes.c_int
    SP = ctypes.POINTER(Sampling)
    lib.sd_accept_resample_sampled.argtypes = [DP, SP, P, P, P, P, P, P, P, P, P, P, P, SZ, P]
    lib.sd_accept_resample_sampled.restype = ctypes.c_int
    lib.sd_verify_step_sampled.argtypes = [DP, SP, P, P, P, P, P, F, P, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P, P]
    lib.sd_verify_step_sampled.restype = ctypes.c_int
    lib.sd_vocab_packed_bytes.argtypes = [DP]
    lib.sd_vocab_packed_bytes.restype = SZ
    lib.sd_pack_vocab.argtypes = [DP, P, P, P]
    lib.sd_pack_vocab.restype = ctypes.c_int
    lib.sd_vocab_kernel_name.argtypes = [DP]
    lib.sd_vocab_kernel_name.restype = ctypes.c_char_p
    lib.sd_status_string.argtypes = [ctypes.c_int]
    lib.sd_status_string.restype = ctypes.c_char_p
    lib.sd_version.argtypes = []
    lib.sd_version.restype = ctypes.c_char_p
    _ = (I64,)
    _lib = lib
    return lib


def exported_symbols() -> list:
    """Names of the functions include/sdverify.h declares."""
    with open(_HEADER) as f:
        text = f.read()
    return re.findall(r"SD_API\s+[\w\s\*]*?\b(sd_\w+)\s*\(", text)


def sd_status_string(status: int) -> str:
    return library().sd_status_string(int(status)).decode()


def sd_version() -> str:
    return library().sd_version().decode()


# ---- marshalling helpers ------------------------------------------------------

def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"expected a torch device tensor, got {type(t).__name__}")
    if not t.is_cuda:
        raise ValueError("device arguments must be GPU tensors")
    if not t.is_contiguous():
        raise ValueError("device arguments must be contiguous")
    return t.data_ptr()


def _host(a, dtype):
    if a is None:
        return None, None
    arr = np.ascontiguousarray(np.asarray(a, dtype=dtype))
    return arr, arr.ctypes.data_as(ctypes.c_void_p)


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def _check(status: int, where: str) -> None:
    if status != SD_OK:
        raise SdError(status, where)


# ---- the C calls ----------------------------------------------------------------

def sd_workspace_bytes(dims: Dims, max_kv_len: int) -> int:
    return int(library().sd_workspace_bytes(ctypes.byref(dims), int(max_kv_len)))


def sd_vocab_kernel_name(dims: Dims):
    name = library().sd_vocab_kernel_name(ctypes.byref(dims))
    return None if name is None else name.decode()


def sd_vocab_packed_bytes(dims: Dims) -> int:
    return int(library().sd_vocab_packed_bytes(ctypes.byref(dims)))


def sd_pack_vocab(dims: Dims, w_vocab, w_packed, stream=None) -> None:
    st = library().sd_pack_vocab(ctypes.byref(dims), _ptr(w_vocab), _ptr(w_packed), _stream(stream))
    _check(st, "sd_pack_vocab")


def _attn_args(dims: Dims, q, k_pool, v_pool, kv_off: Sequence[int], kv_len: Sequence[int], scale: float, out,
               workspace, stream=None):
    _off, off_p = _host(kv_off, np.int64)
    _len, len_p = _host(kv_len, np.int32)
    args = (ctypes.byref(dims), _ptr(q), _ptr(k_pool), _ptr(v_pool), off_p, len_p, float(scale), _ptr(out),
            _ptr(workspace), _nbytes(workspace), _stream(stream))
    return args, (_off, _len)


def sd_verify_attention(dims: Dims, q, k_pool, v_pool, kv_off: Sequence[int], kv_len: Sequence[int],
                        scale: float, out, workspace, stream=None) -> None:
    args, _keep = _attn_args(dims, q, k_pool, v_pool, kv_off, kv_len, scale, out, workspace, stream)
    _check(library().sd_verify_attention(*args), "sd_verify_attention")


def prepare_verify_attention(*a, **kw) -> "PreparedCall":
    """sd_verify_attention with the same arguments, converted once (see PreparedCall)."""
    args, keep = _attn_args(*a, **kw)
    return PreparedCall(library().sd_verify_attention, args, (keep, a, kw), "sd_verify_attention")


def sd_verify_attention_tree(dims: Dims, q, k_pool, v_pool, kv_off: Sequence[int], kv_len: Sequence[int], parent,
                             scale: float, out, workspace, stream=None) -> None:
    _off, off_p = _host(kv_off, np.int64)
    _len, len_p = _host(kv_len, np.int32)
    st = library().sd_verify_attention_tree(ctypes.byref(dims), _ptr(q), _ptr(k_pool), _ptr(v_pool), off_p, len_p,
                                            _ptr(parent), float(scale), _ptr(out), _ptr(workspace),
                                            _nbytes(workspace), _stream(stream))
    _check(st, "sd_verify_attention_tree")


def sd_verify_logits(dims: Dims, hidden, w_vocab, logits, row_lse, workspace, stream=None) -> None:
    st = library().sd_verify_logits(ctypes.byref(dims), _ptr(hidden), _ptr(w_vocab), _ptr(logits),
                                    _ptr(row_lse), _ptr(workspace), _nbytes(workspace), _stream(stream))
    _check(st, "sd_verify_logits")


def sd_accept_resample(dims: Dims, logits_or_probs, row_lse, q_draft, draft_tok, u, kv_len, accept_len,
                       out_tok, new_kv_len, workspace, stream=None) -> None:
    _len, len_p = _host(kv_len, np.int32)
    st = library().sd_accept_resample(ctypes.byref(dims), _ptr(logits_or_probs), _ptr(row_lse), _ptr(q_draft),
                                      _ptr(draft_tok), _ptr(u), len_p, _ptr(accept_len), _ptr(out_tok),
                                      _ptr(new_kv_len), _ptr(workspace), _nbytes(workspace), _stream(stream))
    _check(st, "sd_accept_resample")


def sd_accept_resample_sampled(dims: Dims, sampling: Sampling, logits, q_draft, draft_tok, u, kv_len, row_lse,
                               row_min_logit, accept_len, out_tok, new_kv_len, workspace, stream=None) -> None:
    _len, len_p = _host(kv_len, np.int32)
    st = library().sd_accept_resample_sampled(ctypes.byref(dims), ctypes.byref(sampling), _ptr(logits),
                                              _ptr(q_draft), _ptr(draft_tok), _ptr(u), len_p, _ptr(row_lse),
                                              _ptr(row_min_logit), _ptr(accept_len), _ptr(out_tok),
                                              _ptr(new_kv_len), _ptr(workspace), _nbytes(workspace),
                                              _stream(stream))
    _check(st, "sd_accept_resample_sampled")


def sd_accept_tree(dims: Dims, logits_or_probs, row_lse, tokens, parent, u, kv_len, accept_len, out_tok, out_node,
                   new_kv_len, workspace, stream=None) -> None:
    _len, len_p = _host(kv_len, np.int32)
    st = library().sd_accept_tree(ctypes.byref(dims), _ptr(logits_or_probs), _ptr(row_lse), _ptr(tokens),
                                  _ptr(parent), _ptr(u), len_p, _ptr(accept_len), _ptr(out_tok), _ptr(out_node),
                                  _ptr(new_kv_len), _ptr(workspace), _nbytes(workspace), _stream(stream))
    _check(st, "sd_accept_tree")


def sd_tree_commit_kv(dims: Dims, k_pool, v_pool, kv_off, kv_len, out_node, accept_len, stream=None) -> None:
    _off, off_p = _host(kv_off, np.int64)
    _len, len_p = _host(kv_len, np.int32)
    st = library().sd_tree_commit_kv(ctypes.byref(dims), _ptr(k_pool), _ptr(v_pool), off_p, len_p, _ptr(out_node),
                                     _ptr(accept_len), _stream(stream))
    _check(st, "sd_tree_commit_kv")


def _rate_args(dims, logits_or_probs, row_lse, q_draft, beta, workspace, stream=None):
    return (ctypes.byref(dims), _ptr(logits_or_probs), _ptr(row_lse), _ptr(q_draft), _ptr(beta), _ptr(workspace),
            _nbytes(workspace), _stream(stream))


def sd_acceptance_rate(dims: Dims, logits_or_probs, row_lse, q_draft, beta, workspace, stream=None) -> None:
    _check(library().sd_acceptance_rate(*_rate_args(dims, logits_or_probs, row_lse, q_draft, beta, workspace, stream)),
           "sd_acceptance_rate")


def prepare_acceptance_rate(*a, **kw) -> "PreparedCall":
    """sd_acceptance_rate with the same arguments, converted once (see PreparedCall)."""
    return PreparedCall(library().sd_acceptance_rate, _rate_args(*a, **kw), (a, kw), "sd_acceptance_rate")


def sd_expand_layer(e: Expand, draft_logits, tokens, parent, q_child, stream=None) -> None:
    st = library().sd_expand_layer(ctypes.byref(e), _ptr(draft_logits), _ptr(tokens), _ptr(parent), _ptr(q_child),
                                   _stream(stream))
    _check(st, "sd_expand_layer")


def _event_handles(events):
    if events is None:
        return None
    handles = []
    for e in events:
        if not isinstance(e, int):
            if e.cuda_event == 0:  # torch creates its event lazily, on first record
                e.record()
            e = e.cuda_event
        handles.append(e)
    if len(handles) != 6:
        raise ValueError("kernel_events needs 6 events (start/stop of three kernels)")
    return (ctypes.c_void_p * 6)(*handles)


class PreparedCall:
    """One C call whose arguments were converted once.  Calling it re-issues
    the call with the same pointers, sizes and stream; the caller keeps every
    buffer alive.  (For tight launch loops, where per-call marshalling would
    cost more than the GPU work.)"""

    def __init__(self, fn, args, keep, where):
        self._fn, self._args, self._keep, self._where = fn, args, keep, where

    def __call__(self) -> None:
        st = self._fn(*self._args)
        if st != SD_OK:
            raise SdError(st, self._where)


def _step_args(dims, q, k_pool, v_pool, kv_off, kv_len, scale, hidden, w_vocab, q_draft, draft_tok, u, attn_out,
               logits, row_lse, accept_len, out_tok, new_kv_len, workspace, stream=None, kernel_events=None):
    off, off_p = _host(kv_off, np.int64)
    ln, len_p = _host(kv_len, np.int32)
    ev = _event_handles(kernel_events)
    args = (ctypes.byref(dims), _ptr(q), _ptr(k_pool), _ptr(v_pool), off_p, len_p, float(scale), _ptr(hidden),
            _ptr(w_vocab), _ptr(q_draft), _ptr(draft_tok), _ptr(u), _ptr(attn_out), _ptr(logits), _ptr(row_lse),
            _ptr(accept_len), _ptr(out_tok), _ptr(new_kv_len), _ptr(workspace), _nbytes(workspace),
            _stream(stream), ev)
    return args, (dims, off, ln, ev)


def sd_verify_step(dims: Dims, q, k_pool, v_pool, kv_off, kv_len, scale: float, hidden, w_vocab, q_draft,
                   draft_tok, u, attn_out, logits, row_lse, accept_len, out_tok, new_kv_len, workspace,
                   stream=None, kernel_events=None) -> None:
    args, _keep = _step_args(dims, q, k_pool, v_pool, kv_off, kv_len, scale, hidden, w_vocab, q_draft, draft_tok,
                             u, attn_out, logits, row_lse, accept_len, out_tok, new_kv_len, workspace, stream,
                             kernel_events)
    _check(library().sd_verify_step(*args), "sd_verify_step")


def sd_verify_step_static(dims: Dims, q, k_pool, v_pool, kv_off, kv_len, scale: float, hidden, w_vocab, q_draft,
                          draft_tok, u, attn_out, logits, row_lse, accept_len, out_tok, new_kv_len,
                          stream=None) -> None:
    """sd_verify_step on the library's static per-device scratch (no workspace)."""
    off, off_p = _host(kv_off, np.int64)
    ln, len_p = _host(kv_len, np.int32)
    st = library().sd_verify_step_static(ctypes.byref(dims), _ptr(q), _ptr(k_pool), _ptr(v_pool), off_p, len_p,
                                         float(scale), _ptr(hidden), _ptr(w_vocab), _ptr(q_draft), _ptr(draft_tok),
                                         _ptr(u), _ptr(attn_out), _ptr(logits), _ptr(row_lse), _ptr(accept_len),
                                         _ptr(out_tok), _ptr(new_kv_len), _stream(stream))
    _check(st, "sd_verify_step_static")


def _step_sampled_args(dims, sampling, q, k_pool, v_pool, kv_off, kv_len, scale, hidden, w_vocab, q_draft,
                       draft_tok, u, attn_out, logits, row_lse, row_min_logit, accept_len, out_tok, new_kv_len,
                       workspace, stream=None, kernel_events=None):
    off, off_p = _host(kv_off, np.int64)
    ln, len_p = _host(kv_len, np.int32)
    ev = _event_handles(kernel_events)
    args = (ctypes.byref(dims), ctypes.byref(sampling), _ptr(q), _ptr(k_pool), _ptr(v_pool), off_p, len_p,
            float(scale), _ptr(hidden), _ptr(w_vocab), _ptr(q_draft), _ptr(draft_tok), _ptr(u), _ptr(attn_out),
            _ptr(logits), _ptr(row_lse), _ptr(row_min_logit), _ptr(accept_len), _ptr(out_tok), _ptr(new_kv_len),
            _ptr(workspace), _nbytes(workspace), _stream(stream), ev)
    return args, (dims, sampling, off, ln, ev)


def sd_verify_step_sampled(dims: Dims, sampling: Sampling, q, k_pool, v_pool, kv_off, kv_len, scale: float, hidden,
                           w_vocab, q_draft, draft_tok, u, attn_out, logits, row_lse, row_min_logit, accept_len,
                           out_tok, new_kv_len, workspace, stream=None, kernel_events=None) -> None:
    args, _keep = _step_sampled_args(dims, sampling, q, k_pool, v_pool, kv_off, kv_len, scale, hidden, w_vocab,
                                     q_draft, draft_tok, u, attn_out, logits, row_lse, row_min_logit, accept_len,
                                     out_tok, new_kv_len, workspace, stream, kernel_events)
    _check(library().sd_verify_step_sampled(*args), "sd_verify_step_sampled")


def prepare_verify_step_sampled(*a, **kw) -> PreparedCall:
    """sd_verify_step_sampled with the same arguments, converted once (see PreparedCall)."""
    args, keep = _step_sampled_args(*a, **kw)
    return PreparedCall(library().sd_verify_step_sampled, args, (keep, a, kw), "sd_verify_step_sampled")


def _step_tree_args(dims, q, k_pool, v_pool, kv_off, kv_len, parent, scale, hidden, w_vocab, tokens, u, attn_out,
                    logits, row_lse, accept_len, out_tok, out_node, new_kv_len, workspace, stream=None,
                    kernel_events=None):
    off, off_p = _host(kv_off, np.int64)
    ln, len_p = _host(kv_len, np.int32)
    ev = _event_handles(kernel_events)
    args = (ctypes.byref(dims), _ptr(q), _ptr(k_pool), _ptr(v_pool), off_p, len_p, _ptr(parent), float(scale),
            _ptr(hidden), _ptr(w_vocab), _ptr(tokens), _ptr(u), _ptr(attn_out), _ptr(logits), _ptr(row_lse),
            _ptr(accept_len), _ptr(out_tok), _ptr(out_node), _ptr(new_kv_len), _ptr(workspace), _nbytes(workspace),
            _stream(stream), ev)
    return args, (dims, off, ln, ev)


def sd_verify_step_tree(dims: Dims, q, k_pool, v_pool, kv_off, kv_len, parent, scale: float, hidden, w_vocab, tokens,
                        u, attn_out, logits, row_lse, accept_len, out_tok, out_node, new_kv_len, workspace,
                        stream=None, kernel_events=None) -> None:
    args, _keep = _step_tree_args(dims, q, k_pool, v_pool, kv_off, kv_len, parent, scale, hidden, w_vocab, tokens, u,
                                  attn_out, logits, row_lse, accept_len, out_tok, out_node, new_kv_len, workspace,
                                  stream, kernel_events)
    _check(library().sd_verify_step_tree(*args), "sd_verify_step_tree")


def prepare_verify_step_tree(*a, **kw) -> PreparedCall:
    """sd_verify_step_tree with the same arguments, converted once (see PreparedCall)."""
    args, keep = _step_tree_args(*a, **kw)
    return PreparedCall(library().sd_verify_step_tree, args, (keep, a, kw), "sd_verify_step_tree")


def sd_verify_attention_paged(dims: Dims, q, k_pages, v_pages, pages: KVPages, kv_len, scale: float, out, workspace,
                              stream=None) -> None:
    _len, len_p = _host(kv_len, np.int32)
    st = library().sd_verify_attention_paged(ctypes.byref(dims), _ptr(q), _ptr(k_pages), _ptr(v_pages),
                                             ctypes.byref(pages), len_p, float(scale), _ptr(out), _ptr(workspace),
                                             _nbytes(workspace), _stream(stream))
    _check(st, "sd_verify_attention_paged")


def _step_paged_args(dims, q, k_pages, v_pages, pages, kv_len, scale, hidden, w_vocab, q_draft, draft_tok, u,
                     attn_out, logits, row_lse, accept_len, out_tok, new_kv_len, workspace, stream=None,
                     kernel_events=None):
    ln, len_p = _host(kv_len, np.int32)
    ev = _event_handles(kernel_events)
    args = (ctypes.byref(dims), _ptr(q), _ptr(k_pages), _ptr(v_pages), ctypes.byref(pages), len_p, float(scale),
            _ptr(hidden), _ptr(w_vocab), _ptr(q_draft), _ptr(draft_tok), _ptr(u), _ptr(attn_out), _ptr(logits),
            _ptr(row_lse), _ptr(accept_len), _ptr(out_tok), _ptr(new_kv_len), _ptr(workspace), _nbytes(workspace),
            _stream(stream), ev)
    return args, (dims, pages, ln, ev)


def sd_verify_step_paged(dims: Dims, q, k_pages, v_pages, pages: KVPages, kv_len, scale: float, hidden, w_vocab,
                         q_draft, draft_tok, u, attn_out, logits, row_lse, accept_len, out_tok, new_kv_len, workspace,
                         stream=None, kernel_events=None) -> None:
    args, _keep = _step_paged_args(dims, q, k_pages, v_pages, pages, kv_len, scale, hidden, w_vocab, q_draft,
                                   draft_tok, u, attn_out, logits, row_lse, accept_len, out_tok, new_kv_len,
                                   workspace, stream, kernel_events)
    _check(library().sd_verify_step_paged(*args), "sd_verify_step_paged")


def prepare_verify_step_paged(*a, **kw) -> PreparedCall:
    """sd_verify_step_paged with the same arguments, converted once (see PreparedCall)."""
    args, keep = _step_paged_args(*a, **kw)
    return PreparedCall(library().sd_verify_step_paged, args, (keep, a, kw), "sd_verify_step_paged")


class KVPool:
    """The library's host-side page allocator (sd_kv_pool_*): per-tag page
    lists over num_pages pages of page_size keys."""

    def __init__(self, num_pages: int, page_size: int):
        self._lib = library()
        self._h = self._lib.sd_kv_pool_create(int(num_pages), int(page_size))
        if not self._h:
            raise SdError(SD_ERR_INVALID_ARGUMENT, "sd_kv_pool_create")
        self.num_pages, self.page_size = int(num_pages), int(page_size)

    def close(self) -> None:
        if self._h:
            self._lib.sd_kv_pool_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def reserve(self, tag: int, length: int) -> None:
        _check(self._lib.sd_kv_pool_reserve(self._h, int(tag), int(length)), "sd_kv_pool_reserve")

    def truncate(self, tag: int, length: int) -> None:
        _check(self._lib.sd_kv_pool_truncate(self._h, int(tag), int(length)), "sd_kv_pool_truncate")

    def release(self, tag: int) -> None:
        _check(self._lib.sd_kv_pool_release(self._h, int(tag)), "sd_kv_pool_release")

    def free_pages(self) -> int:
        return int(self._lib.sd_kv_pool_free_pages(self._h))

    def tag_pages(self, tag: int) -> int:
        return int(self._lib.sd_kv_pool_tag_pages(self._h, int(tag)))

    def block_table(self, tags, max_pages: int) -> np.ndarray:
        t, t_p = _host(tags, np.int32)
        out = np.empty((len(t), int(max_pages)), dtype=np.int32)
        _check(self._lib.sd_kv_pool_block_table(self._h, t_p, len(t), int(max_pages),
                                                out.ctypes.data_as(ctypes.c_void_p)), "sd_kv_pool_block_table")
        return out


def prepare_verify_step(*a, **kw) -> PreparedCall:
    """sd_verify_step with the same arguments, converted once (see PreparedCall)."""
    args, keep = _step_args(*a, **kw)
    return PreparedCall(library().sd_verify_step, args, (keep, a, kw), "sd_verify_step")
