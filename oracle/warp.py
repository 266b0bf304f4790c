"""Warped target distributions for sampled verification, float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper verifies with the target distribution itself (temperature 1, Sec. 2
and Algorithm 2).  Deployments sample from a warped target instead; the
Leviathan formulation the paper adopts stays lossless with respect to whatever
distribution p' replaces p, as long as the drafts were drawn from the draft
model's equally warped q'.  The warps, in the order they are applied to one
row of target logits (readings recorded in the design notes; the paper states
none of them):

* temperature T > 0: z = logit / T;
* top-k (1 <= k < V): keep the tokens whose logit is at least the k-th largest
  logit (every token tied with it is kept);
* top-p (0 < top_p < 1): among the tokens top-k kept, with masses
  w = exp(z - max z), keep the smallest set of the form {logit >= theta} whose
  mass is at least top_p times the kept total;
* p'(v) = exp(z(v)) / sum over kept of exp(z), zero elsewhere;
* T = 0 is greedy decoding: p' is one-hot on the largest logit (the smallest
  token id among equal maxima); top-k and top-p are then irrelevant.

"Order" is the order of float32 values, with -0 below +0 (the order of the
integer keys below), so that ties and thresholds are exact on both sides of
the parity tests.  Logits must be finite.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass
class WarpedRow:
    """One warped row: the distribution and how it was cut."""
    p: np.ndarray            # [V] float64, sums to 1
    theta_key: int           # keep key >= theta_key (0: no cut); greedy: 2**32 - 1
    lse: float               # log sum over kept of exp(logit / T) (greedy: 0)
    argmax: int              # smallest token id holding the largest logit
    near: bool               # the top-p cut lies within the decision band


def order_keys(row32) -> np.ndarray:
    """uint32 keys whose unsigned order is the order of the float32 values
    (negative values bit-inverted, positive ones with the sign bit set)."""
    b = np.asarray(row32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    neg = (b & 0x80000000) != 0
    k = np.where(neg, (~b) & 0xFFFFFFFF, b | 0x80000000)
    return k.astype(np.uint64)


def warp_row(row32, temperature: float, top_k: int = 0, top_p: float = 1.0, band: float = 1e-6) -> WarpedRow:
    """Warp one row of float32 logits (widened to float64 for the arithmetic)."""
    row32 = np.asarray(row32, dtype=np.float32)
    V = row32.shape[0]
    keys = order_keys(row32)
    argmax = int(np.argmax(keys))           # first index of the largest key
    if temperature == 0.0:
        p = np.zeros(V, dtype=np.float64)
        p[argmax] = 1.0
        return WarpedRow(p=p, theta_key=(1 << 32) - 1, lse=0.0, argmax=argmax, near=False)
    if not temperature > 0.0:
        raise ValueError("temperature must be >= 0")
    x = row32.astype(np.float64)
    m = x[argmax]
    w = np.exp((x - m) / temperature)       # masses relative to the largest

    theta = 0
    keep = np.ones(V, dtype=bool)
    if 1 <= top_k < V:
        theta = int(np.sort(keys)[::-1][top_k - 1])      # the k-th largest key
        keep = keys >= theta

    near = False
    if 0.0 < top_p < 1.0:
        total = float(w[keep].sum())
        target = top_p * total
        levels, inv = np.unique(keys[keep], return_inverse=True)   # distinct kept keys, ascending
        mass = np.bincount(inv, weights=w[keep], minlength=len(levels))
        levels, mass = levels[::-1], mass[::-1]                       # largest first
        cum = np.cumsum(mass)
        j = int(np.nonzero(cum >= target)[0][0])
        near = abs(cum[j] - target) < band * total or (j > 0 and abs(cum[j - 1] - target) < band * total)
        theta = max(theta, int(levels[j]))
        keep = keys >= theta

    z = x / temperature
    W = float(w[keep].sum())
    lse = m / temperature + np.log(W)
    p = np.where(keep, np.exp(z - lse), 0.0)
    return WarpedRow(p=p, theta_key=theta, lse=float(lse), argmax=argmax, near=bool(near))


def warped_from_cut(row32, temperature: float, theta_key: int, lse: float, argmax: int) -> np.ndarray:
    """p' of one row given the cut and normaliser another implementation
    chose: the float64 evaluation of exactly the distribution that cut defines
    (used to compare acceptance decisions on identical p')."""
    row32 = np.asarray(row32, dtype=np.float32)
    V = row32.shape[0]
    if temperature == 0.0:
        p = np.zeros(V, dtype=np.float64)
        p[int(argmax)] = 1.0
        return p
    keys = order_keys(row32)
    z = row32.astype(np.float64) * np.float64(np.float32(1.0) / np.float32(temperature))
    return np.where(keys >= theta_key, np.exp(z - np.float64(lse)), 0.0)
