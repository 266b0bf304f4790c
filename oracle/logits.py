"""Vocabulary projection and row log-sum-exp, float64, by definition.

Source: Algorithm 2 of the paper produces the target distributions
p_1(.), ..., p_{d+1}(.) from the target model along the path's prefixes; the
last step of that forward is the language-model head: logits = h W^T and
p = softmax(logits).  Temperature is 1 (the paper states none).

Layout: hidden [M][H] with row m = b * G + j feeding p_{j+1} of request b;
W [V][H] (one row per vocabulary entry, the usual linear-layer layout).
"""

from __future__ import annotations

import numpy as np


def verify_logits(hidden, w_vocab, v_chunk: int = 8192):
    """Return (logits[M][V] float64, lse[M] float64).

    lse[m] = log sum_v exp(logits[m][v]), evaluated with the max shift
    lse = max + log(sum exp(logits - max)).  W is widened to float64 in
    vocabulary chunks only to bound memory; each logit is one full dot product.
    """
    h = np.asarray(hidden, dtype=np.float64)
    w = np.asarray(w_vocab)
    M, H = h.shape
    V, H2 = w.shape
    if H != H2:
        raise ValueError("hidden and w_vocab disagree on the hidden size")
    logits = np.empty((M, V), dtype=np.float64)
    for lo in range(0, V, v_chunk):
        hi = min(V, lo + v_chunk)
        logits[:, lo:hi] = h @ w[lo:hi].astype(np.float64).T
    mx = logits.max(axis=1)
    lse = mx + np.log(np.exp(logits - mx[:, None]).sum(axis=1))
    return logits, lse


def probabilities(logits, lse):
    """p[m][v] = exp(logits[m][v] - lse[m]) in float64 (inputs widened first)."""
    lg = np.asarray(logits, dtype=np.float64)
    ls = np.asarray(lse, dtype=np.float64)
    return np.exp(lg - ls[:, None])
