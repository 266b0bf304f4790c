"""The closed-form performance model (paper_2601_21622_amd.starsd) against
the oracle's definitions (oracle.model): E[l] from the accept-length
distribution, T_gamma, T_idle and the busy fraction from the discrete-event
run of the draft server, N_full and N_max by running every N, and the round
speeds' N = 1 identity R_q = R_p.  Host arithmetic only (no GPU)."""

import numpy as np
import pytest

from paper_2601_21622_amd import starsd
from oracle import model as om


@pytest.mark.parametrize("beta", [0.0, 0.3, 0.75, 0.999, 1.0])
@pytest.mark.parametrize("d", [0, 1, 5, 12])
def test_expected_accept_length_matches_distribution(beta, d):
    assert abs(starsd.expected_accept_length(beta, d) - om.expected_accept_length(beta, d)) < 1e-12


def test_expected_total_and_argument_checks():
    assert abs(starsd.expected_total_accept([0.5, 0.9], 4) -
               (om.expected_accept_length(0.5, 4) + om.expected_accept_length(0.9, 4))) < 1e-12
    with pytest.raises(ValueError):
        starsd.expected_accept_length(1.2, 3)
    with pytest.raises(ValueError):
        starsd.star_report([], 3, 1.0, 0.0, 1.0)


def test_iteration_time_idle_and_load_match_the_server_run():
    rng = np.random.default_rng(11)
    for _ in range(300):
        N = int(rng.integers(1, 10))
        d = int(rng.integers(1, 9))
        t_s = float(rng.integers(1, 6))
        S = starsd.service_time(d, t_s)
        Z = starsd.return_time(float(rng.integers(0, 30)), float(rng.integers(0, 60)))
        run = om.simulate_star(N, S, Z)
        T = starsd.iteration_time(N, S, Z)
        assert abs(T - run.period) < 1e-9
        assert abs(starsd.idle_gap(N, S, Z) - run.idle) < 1e-9
        assert starsd.non_idling(N, S, Z) == (run.idle == 0.0)
        rep = starsd.star_report([0.6], d, t_s, Z, 0.0, n_targets=N)
        assert abs(rep.draft_load - run.load) < 1e-9


def test_n_full_and_n_max_match_running_every_n():
    rng = np.random.default_rng(12)
    for _ in range(60):
        S = float(rng.integers(1, 8))
        Z = float(rng.integers(0, 50))
        assert starsd.n_full(S, Z) == om.n_full(S, Z)
        el = float(rng.uniform(0.5, 5.0))
        rate = float(rng.uniform(0.01, 0.6))
        assert starsd.n_max(el, S, Z, rate) == om.n_max(el, S, Z, rate)


def test_throughput_and_round_speeds():
    rep = starsd.star_report([0.8, 0.6], 5, t_s=1.5, t_c=2.0, t_v=10.0, standalone_rate=0.1)
    beta = 0.7
    el = om.expected_accept_length(beta, 5)
    run = om.simulate_star(rep.n_full, 7.5, 12.0)
    assert rep.n_full == om.n_full(7.5, 12.0)
    assert abs(rep.O_gamma - rep.n_full * el / run.period) < 1e-9
    assert abs(rep.O_gamma_per_target - om.per_target_throughput(el, rep.n_full, 7.5, 12.0)) < 1e-9
    assert rep.n_max == om.n_max(el, 7.5, 12.0, 0.1)
    rq, rp = starsd.round_speeds(1, 7.5, 12.0)
    assert rq == rp
    rq, rp = starsd.round_speeds(4, 7.5, 12.0)
    assert abs(rq - 4 * rp) < 1e-15
