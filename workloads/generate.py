"""Seeded generator of verification-step inputs.

Determinism: ``numpy.random.SeedSequence(workload.seed).spawn(10)`` gives ten
fixed streams (lengths, Q, K, V, hidden, W, draft noise, draft sampling,
uniform draws, spare).  Large tensors are drawn in fixed-size chunks, each from
its own spawned child seed, so the bytes do not depend on how many threads
generate them.

bf16 workloads are drawn in float32 and rounded once, round-to-nearest-even, to
bfloat16; the GPU receives the 16-bit patterns and the oracle receives the same
values widened to float32/float64, so both sides see identical numbers.

Uniform draws are fp32 multiples of 2^-24 in [0, 1): ``(uint32 >> 8) * 2^-24``.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Dict, Optional

import numpy as np

from .configs import Workload

_CHUNK = 1 << 22  # elements per independently seeded chunk
_STREAMS = ("lengths", "q", "k", "v", "hidden", "w", "draft_noise", "draft_sample", "u", "spare")


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _normal_f32(ss: np.random.SeedSequence, n: int, std: float) -> np.ndarray:
    """n float32 normals N(0, std^2), drawn in seeded chunks (thread-count independent)."""
    out = np.empty(n, dtype=np.float32)
    nchunks = (n + _CHUNK - 1) // _CHUNK
    seeds = ss.spawn(nchunks) if nchunks else []

    def work(i):
        lo, hi = i * _CHUNK, min(n, (i + 1) * _CHUNK)
        seg = out[lo:hi]
        np.random.default_rng(seeds[i]).standard_normal(out=seg, dtype=np.float32)
        if std != 1.0:
            seg *= np.float32(std)

    if nchunks <= 1:
        for i in range(nchunks):
            work(i)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(work, range(nchunks)))
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest, ties to even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).reshape(-1)
    out = np.empty(u.shape, dtype=np.uint16)
    step = 1 << 24
    for lo in range(0, u.size, step):
        s = u[lo:lo + step]
        out[lo:lo + step] = ((s + np.uint32(0x7FFF) + ((s >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)
    return out.reshape(x.shape)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float32 values (exact widening)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 values rounded to the nearest bfloat16 value, returned as float32."""
    return bf16_bits_to_f32(bf16_bits(x))


@dataclass
class VerifyInputs:
    """One pooled verification batch.

    Tensors whose workload dtype is bf16 are stored as uint16 bit patterns;
    :meth:`f32` widens any of them to float32 values.

    Layouts (row-major):
      q        [B][G][Hq][D]      G = gamma + 1 query positions per request
      k_pool   flat; request b occupies [Hkv][kv_len[b]][D] from element kv_off[b]
      v_pool   same layout as k_pool
      hidden   [B*G][hidden]      row b*G + j feeds target distribution p_{j+1}
      w        [V][hidden]
      q_draft  [B][gamma][V]      q_draft[b][i] is the draft distribution of x_{i+1}
      draft    [B][gamma] int32   draft tokens x_1..x_gamma
      u        [B][G] float32     u[b][i] tests x_{i+1}; u[b][gamma] drives the final sample
    """

    cfg: Workload
    kv_len: np.ndarray
    kv_off: np.ndarray
    q: np.ndarray
    k_pool: np.ndarray
    v_pool: np.ndarray
    hidden: np.ndarray
    w: np.ndarray
    q_draft: np.ndarray
    draft: np.ndarray
    u: np.ndarray
    draft_noise_std: Optional[np.ndarray] = None
    extra: Dict = field(default_factory=dict)

    def f32(self, name: str) -> np.ndarray:
        a = getattr(self, name)
        if a.dtype == np.uint16:
            return bf16_bits_to_f32(a)
        return a

    @property
    def kv_elements(self) -> int:
        c = self.cfg
        return int(c.n_kv_heads * int(self.kv_len.sum()) * c.head_dim)


def _lengths(cfg: Workload, rng: np.random.Generator) -> np.ndarray:
    kind = cfg.lengths[0]
    B, G = cfg.batch, cfg.positions
    if kind == "fixed":
        L = np.full(B, int(cfg.lengths[1]), dtype=np.int64)
    elif kind == "uniform":
        L = rng.integers(int(cfg.lengths[1]), int(cfg.lengths[2]) + 1, size=B)
    elif kind == "lognormal":
        med, sig, clip = cfg.lengths[1], cfg.lengths[2], cfg.lengths[3]
        L = np.rint(np.exp(rng.normal(np.log(med), sig, size=B))).astype(np.int64)
        L = np.clip(L, G, int(clip))
    elif kind == "explicit":
        L = np.asarray(cfg.lengths[1], dtype=np.int64)
        if L.shape != (B,):
            raise ValueError("explicit lengths must have one entry per request")
    else:
        raise ValueError(f"unknown length recipe {kind!r}")
    if np.any(L < G):
        raise ValueError("every kv_len must cover the gamma + 1 positions of the step")
    return L.astype(np.int32)


def draft_logits_f32(hidden_f32: np.ndarray, w_f32: np.ndarray) -> np.ndarray:
    """Stand-in draft model: a float32 product of hidden states and vocabulary
    weights, used only to build draft distributions that resemble the target's.
    It is computed in float32 on purpose (it is synthetic input, not a
    reference value) and neither the oracle nor the kernels use it."""
    out = np.empty((hidden_f32.shape[0], w_f32.shape[0]), dtype=np.float32)
    step = 16384
    for lo in range(0, w_f32.shape[0], step):
        np.matmul(hidden_f32, w_f32[lo:lo + step].T, out=out[:, lo:lo + step])
    return out


def _softmax_rows_f32(z: np.ndarray) -> np.ndarray:
    z = z.astype(np.float64)
    z -= z.max(axis=-1, keepdims=True)
    np.exp(z, out=z)
    z /= z.sum(axis=-1, keepdims=True)
    return z.astype(np.float32)


def make_inputs(cfg: Workload, seed: Optional[int] = None) -> VerifyInputs:
    """Draw one batch for ``cfg`` (optionally overriding its seed)."""
    seed = cfg.seed if seed is None else seed
    ss = dict(zip(_STREAMS, np.random.SeedSequence(seed).spawn(len(_STREAMS))))
    B, gam, G = cfg.batch, cfg.gamma, cfg.positions
    Hq, Hkv, D, Hd, V = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.hidden, cfg.vocab
    bf16 = cfg.dtype == "bf16"
    if cfg.dtype not in ("f32", "bf16"):
        raise ValueError(cfg.dtype)

    kv_len = _lengths(cfg, np.random.default_rng(ss["lengths"]))
    seg = Hkv * kv_len.astype(np.int64) * D
    kv_off = np.concatenate([[0], np.cumsum(seg)[:-1]]).astype(np.int64)
    total = int(seg.sum())

    def draw(name, n, std):
        x = _normal_f32(ss[name], n, std)
        return bf16_bits(x) if bf16 else x

    q = draw("q", B * G * Hq * D, 1.0).reshape(B, G, Hq, D)
    k_pool = draw("k", total, 1.0)
    v_pool = draw("v", total, 1.0)
    hidden = draw("hidden", B * G * Hd, 1.0).reshape(B * G, Hd)
    w = draw("w", V * Hd, cfg.logit_scale / np.sqrt(Hd)).reshape(V, Hd)

    # Draft distributions (stand-in for the draft model M_q).
    kind = cfg.draft[0]
    rng_noise = np.random.default_rng(ss["draft_noise"])
    noise_std = None
    if kind in ("noisy", "noisy_mix", "smoothed_onehot"):
        h32 = bf16_bits_to_f32(hidden) if bf16 else hidden
        w32 = bf16_bits_to_f32(w) if bf16 else w
        rows = np.concatenate([np.arange(b * G, b * G + gam) for b in range(B)])
        tl = draft_logits_f32(h32[rows], w32).reshape(B, gam, V)
        del w32
    if kind == "noisy":
        std = np.sqrt(float(cfg.draft[1]))
        z = tl + rng_noise.standard_normal((B, gam, V), dtype=np.float32) * np.float32(std)
        q_draft = _softmax_rows_f32(z)
    elif kind == "noisy_mix":
        choices = np.asarray(cfg.draft[1], dtype=np.float64)
        noise_std = choices[rng_noise.integers(0, len(choices), size=B)]
        z = tl + rng_noise.standard_normal((B, gam, V), dtype=np.float32) * noise_std[:, None, None].astype(np.float32)
        q_draft = _softmax_rows_f32(z)
    elif kind == "smoothed_onehot":
        mass = float(cfg.draft[1])
        q_draft = np.full((B, gam, V), (1.0 - mass) / (V - 1), dtype=np.float32)
        am = tl.argmax(axis=-1)
        np.put_along_axis(q_draft, am[..., None], np.float32(mass), axis=-1)
    elif kind == "independent":
        var = float(cfg.draft[1])
        z = rng_noise.standard_normal((B, gam, V), dtype=np.float32) * np.float32(np.sqrt(var))
        q_draft = _softmax_rows_f32(z)
    else:
        raise ValueError(f"unknown draft recipe {kind!r}")

    # Draft tokens x_i ~ q_i by inverse CDF of the stored float32 q.
    rng_s = np.random.default_rng(ss["draft_sample"])
    draft = np.empty((B, gam), dtype=np.int32)
    r = rng_s.random((B, gam))
    for b in range(B):
        for i in range(gam):
            c = np.cumsum(q_draft[b, i].astype(np.float64))
            t = int(np.searchsorted(c, r[b, i] * c[-1], side="right"))
            draft[b, i] = min(t, V - 1)

    rng_u = np.random.default_rng(ss["u"])
    u = ((rng_u.integers(0, 1 << 32, size=(B, G), dtype=np.uint64) >> np.uint64(8)).astype(np.float64)
         * 2.0 ** -24).astype(np.float32)

    return VerifyInputs(cfg=cfg, kv_len=kv_len, kv_off=kv_off, q=q, k_pool=k_pool, v_pool=v_pool,
                        hidden=hidden, w=w, q_draft=q_draft, draft=draft, u=u,
                        draft_noise_std=noise_std)
