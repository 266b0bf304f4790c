"""The StarSD performance model in closed form (Sec. 3, Sec. 4.2 and the
appendix on round speeds), fed with measured quantities.

One draft server M_q serves N target instances; every iteration it drafts a
depth-d proposal for each of them (service S(d) = d t_s, eq. Sd), and a target
returns its next request Z(d) = t_c + t_v after the reply (eq. Zd), t_v being
the verification time this library measures (one sd_verify_step of the
target's batch) and t_c the transfer time of one iteration.  The acceptance
rate beta of the pair (eq. beta_cond) comes from sd_acceptance_rate over the
target and draft distributions of real steps.

Host arithmetic only: nothing here touches the GPU.  Times are in any one
unit (the report uses milliseconds); throughputs are per that unit.
"""

from __future__ import annotations

import math
from dataclasses import asdict, dataclass
from typing import Iterable, Optional


def expected_accept_length(beta: float, d: int) -> float:
    """E[l(d)] ~ beta (1 - beta^d) / (1 - beta) under i.i.d. acceptance
    (eq. El_closed); d when beta = 1."""
    if not 0.0 <= beta <= 1.0 or d < 0:
        raise ValueError("need 0 <= beta <= 1 and d >= 0")
    if beta == 1.0:
        return float(d)
    return beta * (1.0 - beta ** d) / (1.0 - beta)


def expected_total_accept(betas: Iterable[float], d: int) -> float:
    """E[l]_gamma: the sum over the active targets (eq. El_gamma)."""
    return float(sum(expected_accept_length(b, d) for b in betas))


def service_time(d: int, t_s: float) -> float:
    """S(d) = d t_s (eq. Sd)."""
    return d * t_s


def return_time(t_c: float, t_v: float) -> float:
    """Z(d) = t_c + t_v (eq. Zd)."""
    return t_c + t_v


def non_idling(N: int, S: float, Z: float) -> bool:
    """The sufficient condition Z <= (N - 1) S of the non-idling lemma."""
    return Z <= (N - 1) * S


def idle_gap(N: int, S: float, Z: float) -> float:
    """T_idle = max(0, Z - (N - 1) S) (eq. Tidle)."""
    return max(0.0, Z - (N - 1) * S)


def iteration_time(N: int, S: float, Z: float) -> float:
    """T_gamma = N S + T_idle (eqs. Tgamma_full and Tgamma_under)."""
    return N * S + idle_gap(N, S, Z)


def throughput(el: float, T: float) -> float:
    """O_gamma = E[l]_gamma / T_gamma (eq. Ogamma); with one target's E[l_i]
    it is that target's O_gamma^(i)."""
    return el / T


def n_full(S: float, Z: float) -> int:
    """N_full = ceil(Z / S) + 1, the onset of full load (Sec. 4.2)."""
    return int(math.ceil(Z / S)) + 1


def n_max(el_i: float, S: float, Z: float, standalone_rate: float) -> int:
    """Largest N whose per-target throughput E[l_i] / T_gamma(N) stays at or
    above a standalone target's rate (the admission rule of Sec. 4.2); 0 when
    even the under-loaded plateau E[l_i] / (S + Z) falls short.  Below full
    load T_gamma = S + Z; above it T_gamma = N S, so the bound is
    floor(E[l_i] / (rate S))."""
    if el_i / (S + Z) < standalone_rate:
        return 0
    return int(math.floor(el_i / (standalone_rate * S)))


def round_speeds(N: int, S: float, Z: float):
    """(R_q, R_p): draft rounds and one target's verification rounds per unit
    time in steady state, N / T_gamma and 1 / T_gamma (appendix, round
    speeds; R_q = R_p at N = 1)."""
    T = iteration_time(N, S, Z)
    return N / T, 1.0 / T


@dataclass
class StarReport:
    beta: float
    depth: int
    expected_accept: float      # E[l_i]
    t_s: float
    t_c: float
    t_v: float
    S: float
    Z: float
    n_full: int
    n_targets: int              # N the per-N figures are for (N_full unless given)
    idle: float                 # T_idle at n_targets
    T_gamma: float
    O_gamma: float              # system accepted tokens per unit time
    O_gamma_per_target: float
    R_q: float
    R_p: float
    draft_load: float           # N S / T_gamma
    n_max: Optional[int]

    def as_dict(self) -> dict:
        return asdict(self)


def star_report(betas: Iterable[float], d: int, t_s: float, t_c: float, t_v: float, n_targets: Optional[int] = None,
                standalone_rate: Optional[float] = None) -> StarReport:
    """The model for symmetric targets whose draft positions have the given
    acceptance rates (their mean is the beta of eq. El_closed)."""
    betas = list(betas)
    if not betas:
        raise ValueError("need at least one acceptance rate")
    beta = float(sum(betas) / len(betas))
    el = expected_accept_length(beta, d)
    S = service_time(d, t_s)
    Z = return_time(t_c, t_v)
    nf = n_full(S, Z)
    N = nf if n_targets is None else int(n_targets)
    T = iteration_time(N, S, Z)
    rq, rp = round_speeds(N, S, Z)
    return StarReport(beta=beta, depth=d, expected_accept=el, t_s=t_s, t_c=t_c, t_v=t_v, S=S, Z=Z, n_full=nf,
                      n_targets=N, idle=idle_gap(N, S, Z), T_gamma=T, O_gamma=throughput(N * el, T),
                      O_gamma_per_target=throughput(el, T), R_q=rq, R_p=rp, draft_load=N * S / T,
                      n_max=None if standalone_rate is None else n_max(el, S, Z, standalone_rate))
