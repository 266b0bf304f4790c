"""The StarSD performance model (Sec. 3 and Sec. 4.2) and the acceptance rate,
float64, each quantity in its plain definition.

TEST INFRASTRUCTURE ONLY (see the package docstring).

* beta (eq. beta_cond): the acceptance rate of one draft position, the sum over
  the vocabulary of min(p(x), q(x)).
* E[l(d)] for one target (eq. tail_sum_li under the i.i.d. approximation of
  eq. El_closed): the expectation of the number of leading successes among d
  Bernoulli(beta) trials, taken over that count's distribution
  Pr(l = j) = beta^j (1 - beta) for j < d and Pr(l = d) = beta^d.
* The per-iteration time (eqs. Sd, Zd, Tidle, Tgamma_full, Tgamma_under): a
  discrete-event run of the draft server of Algorithm 1 serving N targets.
  The server is work-conserving and first-in first-out, each request taking
  S = d t_s; a target submits its next request Z = t_c + t_v after its
  previous reply left the server.  The run reports the steady-state period
  (one request from every target), the server's idle time per period and the
  queueing wait of a request.
* N_full (Sec. 4.2): the smallest N whose run has no idle time; N_max: the
  largest N whose per-target throughput E[l_i] / T_gamma is at least a given
  standalone rate, found by running every N in turn.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import List

import numpy as np


def acceptance_rate(p, q) -> np.ndarray:
    """beta over the last axis: sum_x min(p(x), q(x)) (eq. beta_cond)."""
    p = np.asarray(p, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    return np.minimum(p, q).sum(axis=-1)


def acceptance_rate_batch(x, row_lse, q_draft, gamma: int) -> np.ndarray:
    """beta[b][i] of draft position i of request b: target row b*(gamma+1)+i of
    x (logits with row_lse, p = exp(logit - lse) after widening to float64;
    probabilities without) against q_draft[b][i]."""
    x = np.asarray(x)
    q_draft = np.asarray(q_draft, dtype=np.float64)
    B = q_draft.shape[0]
    G = gamma + 1
    out = np.empty((B, gamma), dtype=np.float64)
    for b in range(B):
        for i in range(gamma):
            row = x[b * G + i].astype(np.float64)
            if row_lse is not None:
                row = np.exp(row - np.float64(row_lse[b * G + i]))
            out[b, i] = acceptance_rate(row, q_draft[b, i])
    return out


def accept_length_pmf(beta: float, d: int) -> np.ndarray:
    """Pr(l = j), j = 0..d, for the leading successes of d i.i.d. trials."""
    pmf = np.empty(d + 1, dtype=np.float64)
    for j in range(d):
        pmf[j] = beta ** j * (1.0 - beta)
    pmf[d] = beta ** d
    return pmf


def expected_accept_length(beta: float, d: int) -> float:
    """E[l(d)] = sum_j j Pr(l = j)."""
    pmf = accept_length_pmf(beta, d)
    return float(np.dot(np.arange(d + 1, dtype=np.float64), pmf))


@dataclass
class StarRun:
    """Steady state of the draft server with N targets."""
    period: float        # T_gamma: time for one request from every target
    idle: float          # server idle time per period
    wait: float          # mean queueing wait of a request
    load: float          # busy fraction of the server


def simulate_star(N: int, S: float, Z: float, periods: int = 64, warmup: int = 16) -> StarRun:
    """Discrete-event run of the work-conserving FIFO draft server (Algorithm 1)."""
    if N < 1 or not S > 0.0 or Z < 0.0:
        raise ValueError("need N >= 1, S > 0, Z >= 0")
    arrivals = [(0.0, i) for i in range(N)]      # (time, target): all targets submit at t = 0
    server_free = 0.0
    served: List[tuple] = []                     # (end, wait, idle gap before the start)
    for _ in range((periods + warmup) * N):
        arrivals.sort()
        t_arr, tgt = arrivals.pop(0)             # earliest request first (ties: lower target)
        start = max(server_free, t_arr)
        end = start + S
        served.append((end, start - t_arr, start - server_free))
        server_free = end
        arrivals.append((end + Z, tgt))          # reply leaves, target verifies and returns
    window = served[warmup * N:]
    span = window[-1][0] - served[warmup * N - 1][0]
    return StarRun(period=span / periods, idle=sum(g for _, _, g in window) / periods,
                   wait=float(np.mean([w for _, w, _ in window])), load=periods * N * S / span)


def per_target_throughput(el_i: float, N: int, S: float, Z: float) -> float:
    """O_gamma^(i) = E[l_i] / T_gamma with T_gamma from the simulated run."""
    return el_i / simulate_star(N, S, Z).period


def n_full(S: float, Z: float, limit: int = 4096) -> int:
    """Smallest N whose simulated server never idles."""
    for N in range(1, limit + 1):
        if simulate_star(N, S, Z).idle <= 1e-12 * max(S, Z, 1.0):
            return N
    raise ValueError("no N up to the limit keeps the server busy")


def n_max(el_i: float, S: float, Z: float, standalone_rate: float, limit: int = 4096) -> int:
    """Largest N with E[l_i] / T_gamma(N) >= standalone_rate (0 if none)."""
    full = n_full(S, Z, limit)
    best = 0
    for N in range(1, limit + 1):
        if per_target_throughput(el_i, N, S, Z) >= standalone_rate:
            best = N
        elif N >= full:
            break                                # past full load the rate only falls
    return best
