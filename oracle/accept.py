"""Lossless acceptance test, first rejection and residual resampling, float64.

Source: Algorithm 2 of the paper (EAGLE speculative decoding), verification of
one chain path [x_1..x_d] (branching k = 1; here d is called gamma):
  1. draw r_1..r_d ~ U(0, 1) and let l be the number of leading positions that
     pass the stochastic test;
  2. if l < d, sample one corrected token from norm(max(0, p_{l+1} - q_{l+1}));
  3. return the accepted prefix (plus that token).
The test is the ratio rule of the formulation the paper adopts in Sec. 2
(Leviathan et al.): x_i passes when r_i < p_i(x_i) / q_i(x_i).  Sec. 3.2,
Eq. (1) gives the resulting per-token acceptance probability
beta = sum_x min(p(x), q(x)) = 1 - TV(p, q).

Readings where the algorithm as printed is silent or garbled (each recorded in
the design notes):
* The printed test compares r_i with p_i(x) and omits the division by q_i; the
  ratio p_i(x_i)/q_i(x_i) is used, since only then is the acceptance
  probability Eq. (1) and the output distribution the target's.
* r_i = u[i] in [0, 1); accept iff u < ratio (strict).  ratio = 0 when
  p_i(x_i) = 0 (never accepted) and +inf when q_i(x_i) = 0 < p_i(x_i) (always
  accepted); a NaN ratio rejects.
* When every draft passes (l = gamma), one bonus token is sampled from
  p_{gamma+1}, so each request emits l + 1 tokens.
* The final sample uses its own draw u[gamma]; the rejected test's draw is not
  reused.
* "norm" is L1 normalisation.  The sample is the inverse CDF in ascending
  token-id order: with r the unnormalised distribution, C its inclusive prefix
  sums (float64, sequential) and Z = C[V-1], t = min{k : C[k] > u * Z}.  If
  rounding leaves no such k, t is the largest k with r(k) > 0; if Z is not
  positive (reachable only through rounding when p_{l+1} <= q_{l+1}
  everywhere) r falls back to p_{l+1}.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np


@dataclass
class AcceptTrace:
    """Intermediate values of one request's verification, for the near-threshold band."""
    ratios: List[float] = field(default_factory=list)   # ratio of every evaluated test
    draws: List[float] = field(default_factory=list)    # the u used by each evaluated test
    z: float = 0.0
    threshold: float = 0.0
    c_before: float = 0.0    # C[t-1] (0 when t = 0)
    c_at: float = 0.0        # C[t]
    source: str = ""        # "residual", "bonus", or either with "+fallback"


def _ratio(px: float, qx: float) -> float:
    if px <= 0.0:
        return 0.0
    if qx <= 0.0:
        return math.inf
    return px / qx


def accept_request(p_rows, q_rows, draft, u):
    """Verify one request.

    p_rows  [gamma+1][V] float: p_rows[j] = p_{j+1}, the target distribution
            after the root and the first j drafts
    q_rows  [gamma][V] float: q_rows[i] = q_{i+1}, the draft distribution x_{i+1} was drawn from
    draft   [gamma] int: x_1..x_gamma
    u       [gamma+1] float in [0, 1)

    Returns (l, tokens, trace): l accepted drafts, tokens = x_1..x_l followed by
    the corrected (l < gamma) or bonus (l = gamma) token.
    """
    p_rows = np.asarray(p_rows, dtype=np.float64)
    q_rows = np.asarray(q_rows, dtype=np.float64)
    gamma = len(draft)
    V = p_rows.shape[1]
    tr = AcceptTrace()

    # Step 1: leading positions that pass the stochastic test.
    l = gamma
    for i in range(gamma):
        x = int(draft[i])
        ratio = _ratio(float(p_rows[i, x]), float(q_rows[i, x]))
        tr.ratios.append(ratio)
        tr.draws.append(float(u[i]))
        if not (float(u[i]) < ratio):
            l = i
            break

    # Step 2: the distribution of the appended token.
    if l < gamma:
        r = np.maximum(p_rows[l] - q_rows[l], 0.0)
        tr.source = "residual"
    else:
        r = p_rows[gamma].copy()
        tr.source = "bonus"
    c = np.cumsum(r)
    z = float(c[-1])
    if not z > 0.0:
        r = p_rows[l].copy()
        c = np.cumsum(r)
        z = float(c[-1])
        tr.source += "+fallback"

    # Step 3: inverse CDF with the final draw.
    thr = float(u[gamma]) * z
    t = int(np.searchsorted(c, thr, side="right"))
    if t >= V:
        t = int(np.nonzero(r > 0.0)[0][-1])
    tr.z = z
    tr.threshold = thr
    tr.c_before = float(c[t - 1]) if t > 0 else 0.0
    tr.c_at = float(c[t])
    tokens = [int(x) for x in draft[:l]] + [t]
    return l, tokens, tr


def accept_resample(logits_or_probs, row_lse, q_draft, draft, u, kv_len=None):
    """Batched verification mirroring the library's accept/resample call.

    logits_or_probs [B*G][V]: logits when ``row_lse`` is given (p = exp(logit - lse),
                    evaluated in float64 after widening), else probabilities.
    q_draft [B][gamma][V], draft [B][gamma], u [B][G], kv_len [B] or None.

    Returns dict with accept_len [B] int32, out_tok [B][G] int32 (-1 padded),
    new_kv_len [B] int32 (L_b - gamma + l_b) or None, and per-request traces.
    """
    x = np.asarray(logits_or_probs)
    q_draft = np.asarray(q_draft)
    draft = np.asarray(draft)
    u = np.asarray(u)
    B, gamma = draft.shape
    G = gamma + 1
    if x.shape[0] != B * G:
        raise ValueError("logits_or_probs must have B * (gamma + 1) rows")
    accept_len = np.zeros(B, dtype=np.int32)
    out_tok = np.full((B, G), -1, dtype=np.int32)
    traces = []
    for b in range(B):
        rows = x[b * G:(b + 1) * G].astype(np.float64)
        if row_lse is not None:
            lse = np.asarray(row_lse[b * G:(b + 1) * G], dtype=np.float64)
            rows = np.exp(rows - lse[:, None])
        l, toks, tr = accept_request(rows, q_draft[b], draft[b], u[b])
        accept_len[b] = l
        out_tok[b, :len(toks)] = toks
        traces.append(tr)
    new_kv_len = None
    if kv_len is not None:
        new_kv_len = (np.asarray(kv_len, dtype=np.int64) - gamma + accept_len).astype(np.int32)
    return {"accept_len": accept_len, "out_tok": out_tok, "new_kv_len": new_kv_len, "traces": traces}


def accept_resample_sampled(logits, q_draft, draft, u, temperature, top_k=0, top_p=1.0, kv_len=None, cut=None):
    """Verification against the warped target (``oracle.warp``): each row of
    float32 logits becomes p' (temperature, top-k, top-p, or greedy when
    temperature is 0) and the same test and correction run on p'.

    ``cut`` = (theta_keys [B*G], lse [B*G], argmax [B*G]) makes p' the exact
    distribution another implementation's cut and normaliser define, so that
    acceptance decisions can be compared on identical p'; without it the cut
    is computed here.  Returns the dict of ``accept_resample`` plus per-row
    WarpedRow records (``rows``, only when ``cut`` is None) and ``near_cut``
    [B] (a row of the request has its top-p cut within the decision band).
    """
    from .warp import warp_row, warped_from_cut

    x = np.asarray(logits, dtype=np.float32)
    draft = np.asarray(draft)
    B, gamma = draft.shape
    G = gamma + 1
    if x.shape[0] != B * G:
        raise ValueError("logits must have B * (gamma + 1) rows")
    rows = []
    pw = np.empty(x.shape, dtype=np.float64)
    near_cut = np.zeros(B, dtype=bool)
    for r in range(B * G):
        if cut is None:
            wr = warp_row(x[r], temperature, top_k, top_p)
            rows.append(wr)
            pw[r] = wr.p
            near_cut[r // G] |= wr.near
        else:
            pw[r] = warped_from_cut(x[r], temperature, int(cut[0][r]), float(cut[1][r]), int(cut[2][r]))
    out = accept_resample(pw, None, q_draft, draft, u, kv_len)
    out["rows"] = rows
    out["near_cut"] = near_cut
    return out


# Decision bands of the comparison with another implementation: a ratio test
# whose draw lies within RATIO_BAND of its threshold, or a final draw whose
# u * Z lies within FINAL_BAND * Z of an end of the chosen token's CDF
# interval, may legitimately go either way under a different (correct)
# rounding of p.  The final-draw band covers an inverse CDF built in float64
# from float64 values of p (relative differences of order 1e-13 of Z).
RATIO_BAND = 1e-6
FINAL_BAND = 1e-9


def near_threshold(trace: AcceptTrace, band: float = RATIO_BAND, final_band: float = FINAL_BAND) -> bool:
    """True when a draw lies within a decision band: an evaluated test with
    |u - ratio| < band, or a final draw with u*Z within final_band*Z of the
    chosen token's CDF interval ends."""
    for ui, ri in zip(trace.draws, trace.ratios):
        if math.isfinite(ri) and abs(ui - ri) < band:
            return True
    z = trace.z
    if (trace.threshold - trace.c_before) < final_band * z or (trace.c_at - trace.threshold) < final_band * z:
        return True
    return False
