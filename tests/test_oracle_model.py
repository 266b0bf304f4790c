"""Pins of oracle.model (Sec. 3 and Sec. 4.2) against the mathematics.

* beta: the total-variation identity of eq. beta_cond (1 - half the L1
  distance), the acceptance probability of the ratio test of Sec. 2 written
  as sum_x q(x) min(1, p(x)/q(x)) and estimated by drawing x ~ q and u, and
  the special cases p = q (1) and disjoint supports (0); the batched form is
  checked on rows built to have known, distinct rates.
* E[l]: the closed form of eq. El_closed, the tail-sum identity of the lemma
  (sum over j of Pr(l >= j)), the end points beta = 0 and 1, and a Monte
  Carlo count of leading successes.
* The draft-server run: timelines worked by hand, the sufficient non-idling
  condition of the lemma in Sec. 3.3 (no idle time whenever Z <= (N - 1) S),
  idle time whenever it fails, and the busy fraction N S / T_gamma.
* N_full and N_max on hand-worked cases.
"""

import numpy as np
import pytest

from oracle.model import (accept_length_pmf, acceptance_rate, acceptance_rate_batch, expected_accept_length, n_full,
                          n_max, per_target_throughput, simulate_star)


def _dist(rng, V, alpha=0.3):
    p = rng.gamma(alpha, size=V)
    return p / p.sum()


def test_beta_is_one_minus_total_variation():
    rng = np.random.default_rng(1)
    for V in (2, 17, 1000):
        for _ in range(5):
            p, q = _dist(rng, V), _dist(rng, V)
            assert abs(acceptance_rate(p, q) - (1.0 - 0.5 * np.abs(p - q).sum())) < 1e-12


def test_beta_special_cases():
    rng = np.random.default_rng(2)
    p = _dist(rng, 50)
    assert abs(acceptance_rate(p, p) - 1.0) < 1e-12
    a = np.zeros(10)
    b = np.zeros(10)
    a[:5] = 0.2
    b[5:] = 0.2
    assert acceptance_rate(a, b) == 0.0
    q = _dist(rng, 50)
    assert abs(acceptance_rate(p, q) - acceptance_rate(q, p)) < 1e-15


def test_beta_is_the_ratio_test_acceptance_probability():
    rng = np.random.default_rng(3)
    V = 40
    p, q = _dist(rng, V, 0.8), _dist(rng, V, 0.8)
    exact = float(np.sum(q * np.minimum(1.0, p / q)))
    assert abs(acceptance_rate(p, q) - exact) < 1e-12
    n = 400_000
    x = rng.choice(V, size=n, p=q)
    u = rng.random(n)
    rate = float(np.mean(u < p[x] / q[x]))
    sigma = np.sqrt(exact * (1 - exact) / n)
    assert abs(rate - acceptance_rate(p, q)) < 5 * sigma


def test_beta_batch_rows_and_logits():
    # Row (b, i) has p uniform on 10 tokens and q uniform on 10 tokens shifted
    # by s = b * gamma + i (overlap 10 - s tokens): beta = (10 - s) / 10.
    B, gamma, V = 2, 3, 40
    G = gamma + 1
    probs = np.zeros((B * G, V))
    q = np.zeros((B, gamma, V))
    for b in range(B):
        for i in range(gamma):
            s = b * gamma + i
            probs[b * G + i, :10] = 0.1
            q[b, i, s:s + 10] = 0.1
        probs[b * G + gamma, :] = 1.0 / V
    want = np.array([[(10 - (b * gamma + i)) / 10 for i in range(gamma)] for b in range(B)])
    assert np.allclose(acceptance_rate_batch(probs, None, q, gamma), want, atol=1e-12)
    # The same rows as logits: log p + 3, with row lse 3 (zeros -> -inf -> p = 0).
    with np.errstate(divide="ignore"):
        logits = np.log(probs) + 3.0
    lse = np.full(B * G, 3.0)
    assert np.allclose(acceptance_rate_batch(logits, lse, q, gamma), want, atol=1e-12)


@pytest.mark.parametrize("beta", [0.05, 0.5, 0.8, 0.97])
@pytest.mark.parametrize("d", [1, 4, 9])
def test_expected_accept_length_closed_form_and_tail_sum(beta, d):
    el = expected_accept_length(beta, d)
    assert abs(el - beta * (1 - beta ** d) / (1 - beta)) < 1e-12
    pmf = accept_length_pmf(beta, d)
    assert abs(pmf.sum() - 1.0) < 1e-12
    tail = sum(pmf[j:].sum() for j in range(1, d + 1))
    assert abs(el - tail) < 1e-12
    assert abs(tail - sum(beta ** j for j in range(1, d + 1))) < 1e-12


def test_expected_accept_length_end_points_and_monte_carlo():
    assert expected_accept_length(0.0, 6) == 0.0
    assert expected_accept_length(1.0, 6) == 6.0
    rng = np.random.default_rng(4)
    beta, d, n = 0.7, 5, 200_000
    trials = rng.random((n, d)) < beta
    lead = np.where(trials.all(axis=1), d, np.argmin(trials, axis=1))
    se = lead.std() / np.sqrt(n)
    assert abs(lead.mean() - expected_accept_length(beta, d)) < 5 * se


@pytest.mark.parametrize("N,S,Z,period,idle,wait", [
    (1, 2.0, 5.0, 7.0, 5.0, 0.0),      # one target: serve 2, wait out the 5-unit return
    (2, 2.0, 5.0, 7.0, 3.0, 0.0),      # two targets: each period has one 3-unit gap
    (3, 2.0, 3.0, 6.0, 0.0, 1.0),      # 3 <= 2 * 2: never idle, each request queues 1 unit
    (2, 1.0, 1.0, 2.0, 0.0, 0.0),      # boundary Z = (N - 1) S: busy, no queueing
    (4, 1.5, 2.0, 6.0, 0.0, 2.5),      # queueing (N - 1) S - Z
])
def test_star_run_hand_timelines(N, S, Z, period, idle, wait):
    r = simulate_star(N, S, Z)
    assert abs(r.period - period) < 1e-12
    assert abs(r.idle - idle) < 1e-12
    assert abs(r.wait - wait) < 1e-12
    assert abs(r.load - N * S / period) < 1e-12


def test_star_run_non_idling_lemma():
    rng = np.random.default_rng(5)
    for _ in range(200):
        N = int(rng.integers(1, 9))
        S = float(rng.integers(1, 20))
        Z = float(rng.integers(0, 80))
        r = simulate_star(N, S, Z)
        if Z <= (N - 1) * S:
            assert r.idle == 0.0 and abs(r.load - 1.0) < 1e-12
        else:
            assert r.idle > 0.0 and r.load < 1.0


def test_n_full_and_n_max_hand_cases():
    # S = 2, Z = 5: busy from Z <= (N - 1) S, i.e. N >= 3.5 -> N_full = 4.
    assert n_full(2.0, 5.0) == 4
    # Z a multiple of S: Z = 4, S = 2 -> N = 3 already busy.
    assert n_full(2.0, 4.0) == 3
    assert n_full(1.0, 0.0) == 1
    # E[l_i] = 3, standalone 0.2: 3 / 7 for N <= 3, 3 / (2 N) after -> N_max = 7.
    assert n_max(3.0, 2.0, 5.0, 0.2) == 7
    assert abs(per_target_throughput(3.0, 7, 2.0, 5.0) - 3.0 / 14.0) < 1e-12
    # A standalone rate above the under-loaded plateau 3 / 7: no N qualifies.
    assert n_max(3.0, 2.0, 5.0, 0.5) == 0
