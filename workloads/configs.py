"""The five synthetic verification workloads and their value recipes.

Each workload is one verifier's pooled batch: ``batch`` requests, each with
``gamma`` draft tokens, verified at ``gamma + 1`` query positions (the root,
i.e. the last verified token, plus the drafts).  Shapes follow the model
families they are named after; values are synthetic (no weights or prompts).

Recipe conventions
------------------
* ``N(0, x)`` in a recipe is a normal with variance ``x``.
* ``logit_scale`` s: the vocabulary weights are drawn N(0, s^2 / hidden) so the
  target logits are roughly N(0, s^2) for N(0, 1) hidden states.
* Lengths ``kv_len`` include the ``gamma + 1`` positions of the current step.
* Draft recipes:
  - ``("noisy", var)``: q = softmax(target logits + N(0, var) noise).
  - ``("noisy_mix", (s1, s2, ...))``: as above, with a per-request noise
    standard deviation drawn uniformly from the list.
  - ``("smoothed_onehot", mass)``: ``mass`` on the target argmax, the rest
    spread evenly over the other tokens.
  - ``("independent", var)``: q = softmax(N(0, var)) independent of p.
"""

from __future__ import annotations

import dataclasses
from dataclasses import dataclass
from typing import Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    gamma: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    hidden: int
    vocab: int
    dtype: str  # "f32" or "bf16": storage type of Q/K/V/hidden/W
    lengths: Tuple  # ("fixed", L) | ("uniform", lo, hi) | ("lognormal", median, sigma_ln, clip)
    draft: Tuple
    logit_scale: float = 1.0
    seed: int = 0

    @property
    def positions(self) -> int:
        """Query positions per request: the root plus the gamma drafts."""
        return self.gamma + 1

    @property
    def rows(self) -> int:
        """Rows of the vocabulary projection: one per (request, position)."""
        return self.batch * self.positions

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    def max_kv_len(self) -> int:
        kind = self.lengths[0]
        if kind == "fixed":
            return int(self.lengths[1])
        if kind == "uniform":
            return int(self.lengths[2])
        if kind == "lognormal":
            return int(self.lengths[3])
        raise ValueError(kind)


CONFIGS = {
    # Tiny fp32 case: MHA, 4 heads of 64, L = 128, vocab 1000.
    "tiny": Workload(
        name="tiny", batch=1, gamma=4, n_q_heads=4, n_kv_heads=4, head_dim=64,
        hidden=256, vocab=1000, dtype="f32", lengths=("fixed", 128),
        draft=("noisy", 0.5), logit_scale=1.0, seed=1001),
    # Vicuna-7B-shaped single layer: 32 heads of 128, hidden 4096, vocab 32000.
    "vicuna7b": Workload(
        name="vicuna7b", batch=8, gamma=5, n_q_heads=32, n_kv_heads=32, head_dim=128,
        hidden=4096, vocab=32000, dtype="bf16", lengths=("uniform", 512, 2048),
        draft=("noisy", 1.0), logit_scale=1.0, seed=1002),
    # Pooled many-client share: 64 requests, log-normal lengths, mixed drafts.
    "pooled": Workload(
        name="pooled", batch=64, gamma=4, n_q_heads=32, n_kv_heads=32, head_dim=128,
        hidden=4096, vocab=32000, dtype="bf16", lengths=("lognormal", 1024, 0.6931471805599453, 8192),
        draft=("noisy_mix", (0.2, 1.0, 3.0)), logit_scale=1.0, seed=1003),
    # Llama-3-8B-shaped GQA: 32 query / 8 KV heads, vocab 128256, L = 4096.
    "llama3_8b": Workload(
        name="llama3_8b", batch=32, gamma=6, n_q_heads=32, n_kv_heads=8, head_dim=128,
        hidden=4096, vocab=128256, dtype="bf16", lengths=("fixed", 4096),
        draft=("smoothed_onehot", 0.9), logit_scale=16.0, seed=1004),
    # Llama-70B-shaped long-context share: 64 query / 8 KV heads, hidden 8192.
    "llama70b_share": Workload(
        name="llama70b_share", batch=16, gamma=8, n_q_heads=64, n_kv_heads=8, head_dim=128,
        hidden=8192, vocab=128256, dtype="bf16", lengths=("uniform", 16384, 32768),
        draft=("independent", 1.0), logit_scale=1.0, seed=1005),
}


def get_config(name: str) -> Workload:
    try:
        return CONFIGS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(CONFIGS)}") from None
