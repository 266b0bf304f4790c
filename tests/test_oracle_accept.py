"""Pins of the oracle's acceptance test and residual resampling (oracle.accept).

What fixes the answers (none of them restates the oracle's code):
* Sec. 3.2, Eq. (1): per-token acceptance probability beta = sum min(p, q);
  its complement is the total-variation distance.
* Sec. 3.2, Eq. (2) (tail-sum identity) and Eq. (3) (closed form of E[l] under
  i.i.d. acceptances), which is exact when p and q do not depend on position.
* Special cases with known outcomes: q == p, disjoint supports, one-hot draft.
* Losslessness (Sec. 1: speculative decoding preserves the target's output
  distribution), checked by brute force in test_oracle_lossless.py.
All probabilities are exact integrals over the draws (tests/exact_law.py).
"""

import json
import math
import os

import numpy as np
import pytest

from oracle.accept import accept_request, accept_resample, near_threshold
from exact_law import exact_law, law_of_l, law_of_last

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _dist(rng, V, zeros=0):
    p = rng.dirichlet(np.ones(V))
    if zeros:
        idx = rng.choice(V, size=zeros, replace=False)
        p[idx] = 0.0
        p /= p.sum()
    return p


def test_q_equals_p_accepts_everything_and_bonus_is_p_last():
    rng = np.random.default_rng(0)
    V, gamma = 6, 3
    p_rows = np.stack([_dist(rng, V) for _ in range(gamma + 1)])
    q_rows = p_rows[:gamma].copy()
    draft = [int(np.argmax(q_rows[i])) for i in range(gamma)]
    law = exact_law(accept_request, p_rows, q_rows, draft)
    assert law_of_l(law) == pytest.approx({gamma: 1.0}, abs=1e-15)
    last = law_of_last(law)
    for v in range(V):
        assert last.get(v, 0.0) == pytest.approx(p_rows[gamma][v], abs=1e-12)


def test_disjoint_supports_reject_first_and_sample_p1():
    V, gamma = 8, 3
    p = np.array([0, 0, 0, 0, .1, .2, .3, .4])
    q = np.array([.25, .25, .25, .25, 0, 0, 0, 0])
    p_rows = np.stack([p] * (gamma + 1))
    q_rows = np.stack([q] * gamma)
    for x0 in range(4):
        law = exact_law(accept_request, p_rows, q_rows, [x0, 1, 2])
        assert law_of_l(law) == pytest.approx({0: 1.0}, abs=1e-15)
        last = law_of_last(law)
        for v in range(V):
            assert last.get(v, 0.0) == pytest.approx(p[v], abs=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_single_position_reject_rate_is_total_variation(seed):
    rng = np.random.default_rng(100 + seed)
    V = 7
    p = _dist(rng, V, zeros=seed % 3)
    q = _dist(rng, V, zeros=(seed + 1) % 3)
    beta = np.minimum(p, q).sum()                      # Eq. (1)
    tv = 0.5 * np.abs(p - q).sum()
    assert beta == pytest.approx(1 - tv, abs=1e-15)
    p_rows = np.stack([p, _dist(rng, V)])
    q_rows = q[None, :]
    # Marginalise over x_1 ~ q.
    rej = 0.0
    for x in range(V):
        if q[x] == 0:
            continue
        law = exact_law(accept_request, p_rows, q_rows, [x])
        rej += q[x] * law_of_l(law).get(0, 0.0)
    assert rej == pytest.approx(tv, abs=1e-12)


@pytest.mark.parametrize("gamma,seed", [(1, 0), (2, 1), (3, 2), (4, 3)])
def test_accept_length_law_iid_case(gamma, seed):
    """Position-independent p and q: P(l = j) = beta^j (1 - beta) for j < gamma,
    P(l = gamma) = beta^gamma, and E[l] equals Eq. (3) and Eq. (2)."""
    rng = np.random.default_rng(200 + seed)
    V = 4
    p = _dist(rng, V, zeros=1)
    q = _dist(rng, V)
    beta = np.minimum(p, q).sum()
    p_rows = np.stack([p] * (gamma + 1))
    q_rows = np.stack([q] * gamma)
    pl = np.zeros(gamma + 1)
    import itertools
    for path in itertools.product(range(V), repeat=gamma):
        w = np.prod([q[x] for x in path])
        if w == 0:
            continue
        for l, pr in law_of_l(exact_law(accept_request, p_rows, q_rows, list(path), final=False)).items():
            pl[l] += w * pr
    for j in range(gamma):
        assert pl[j] == pytest.approx(beta ** j * (1 - beta), abs=1e-12)
    assert pl[gamma] == pytest.approx(beta ** gamma, abs=1e-12)
    el = float(np.dot(np.arange(gamma + 1), pl))
    assert el == pytest.approx(beta * (1 - beta ** gamma) / (1 - beta), abs=1e-12)   # Eq. (3)
    tail = sum(pl[j:].sum() for j in range(1, gamma + 1))                           # Eq. (2)
    assert el == pytest.approx(tail, abs=1e-12)


def test_one_hot_draft():
    """q one-hot on a with p(a) = alpha: accept with probability alpha; the
    correction is p restricted to v != a, renormalised by 1 - alpha."""
    p = np.array([.1, .35, .05, .3, .2])
    a = 3
    q = np.zeros(5)
    q[a] = 1.0
    p_rows = np.stack([p, p])
    law = exact_law(accept_request, p_rows, q[None, :], [a])
    assert law_of_l(law)[1] == pytest.approx(p[a], abs=1e-15)
    rejected = {toks[-1]: pr for (l, toks), pr in law.items() if l == 0}
    total = sum(rejected.values())
    assert total == pytest.approx(1 - p[a], abs=1e-15)
    for v in range(5):
        want = 0.0 if v == a else p[v] / (1 - p[a])
        assert rejected.get(v, 0.0) / total == pytest.approx(want, abs=1e-12)


def test_worked_example_fixture():
    with open(os.path.join(GOLDEN, "worked_example.json")) as f:
        ex = json.load(f)
    p = np.array(ex["p"])
    q = np.array(ex["q"])
    assert np.minimum(p, q).sum() == pytest.approx(ex["beta"], abs=1e-15)
    p_rows = np.stack([p, p])
    res = {}
    total_rej = 0.0
    for x in range(len(q)):
        if q[x] == 0:
            continue
        for (l, toks), pr in exact_law(accept_request, p_rows, q[None, :], [x]).items():
            if l == 0:
                res[toks[-1]] = res.get(toks[-1], 0.0) + q[x] * pr
                total_rej += q[x] * pr
    assert total_rej == pytest.approx(1 - ex["beta"], abs=1e-12)
    for v, want in enumerate(ex["residual"]):
        assert res.get(v, 0.0) / total_rej == pytest.approx(want, abs=1e-12)


def test_boundary_conventions():
    p = np.array([0.0, 0.5, 0.5])
    q = np.array([0.5, 0.0, 0.5])
    p_rows = np.stack([p, np.array([0.2, 0.3, 0.5])])
    # p(x) = 0 is never accepted, even with u = 0 (strict test).
    l, toks, _ = accept_request(p_rows, q[None, :], [0], [0.0, 0.0])
    assert l == 0
    # u = 0 in the inverse CDF never returns a zero-mass token: residual is (0, .5, 0)/.5.
    assert toks == [1]
    # ratio >= 1 always accepts, even at the largest draw 1 - 2^-24.
    l, toks, _ = accept_request(p_rows, q[None, :], [2], [1 - 2 ** -24, 0.0])
    assert l == 1 and toks == [2, 0]
    # Bonus with the largest draw picks the last token with mass.
    l, toks, _ = accept_request(p_rows, q[None, :], [2], [0.5, 1 - 2 ** -24])
    assert toks == [2, 2]


def test_q_zero_at_draft_accepts():
    p = np.array([0.4, 0.6])
    q = np.array([0.0, 1.0])
    l, _, tr = accept_request(np.stack([p, p]), q[None, :], [0], [1 - 2 ** -24, 0.3])
    assert l == 1 and math.isinf(tr.ratios[0])


def test_fallbacks():
    # Residual identically zero (p == q, reachable only by rounding): falls back to p_{l+1}.
    p = np.array([0.25, 0.25, 0.5])
    l, toks, tr = accept_request(np.stack([p, p]), p[None, :], [2], [1.0, 0.6])
    assert l == 0 and tr.source == "residual+fallback"
    assert toks == [2]  # C = (.25, .5, 1.0), thr = .6
    # Threshold at or beyond the last prefix sum: last token with mass.
    r_p = np.array([0.5, 0.5, 0.0])
    l, toks, _ = accept_request(np.stack([r_p, r_p]), np.array([[0.0, 1.0, 0.0]]), [1], [0.0, 1.0])
    assert l == 1 and toks == [1, 1]


def test_batched_wrapper_matches_per_request_and_logits_mode():
    rng = np.random.default_rng(5)
    B, gamma, V = 3, 2, 9
    G = gamma + 1
    logits = rng.normal(size=(B * G, V))
    lse = np.log(np.exp(logits).sum(axis=1))
    p = np.exp(logits - lse[:, None])
    q = np.stack([np.stack([_dist(rng, V) for _ in range(gamma)]) for _ in range(B)])
    draft = rng.integers(0, V, size=(B, gamma))
    u = rng.random((B, G))
    kv_len = np.array([10, 20, 30])
    a = accept_resample(logits, lse, q, draft, u, kv_len=kv_len)
    b = accept_resample(p, None, q, draft, u)
    assert np.array_equal(a["accept_len"], b["accept_len"])
    assert np.array_equal(a["out_tok"], b["out_tok"])
    for i in range(B):
        l, toks, _ = accept_request(p[i * G:(i + 1) * G], q[i], draft[i], u[i])
        assert a["accept_len"][i] == l
        assert list(a["out_tok"][i, :l + 1]) == toks
        assert all(a["out_tok"][i, l + 1:] == -1)
        assert a["new_kv_len"][i] == kv_len[i] - gamma + l


def test_near_threshold_band():
    p = np.array([0.3, 0.7])
    q = np.array([0.6, 0.4])
    p_rows = np.stack([p, p])
    _, _, tr = accept_request(p_rows, q[None, :], [0], [0.5 + 5e-7, 0.1])
    assert near_threshold(tr)
    _, _, tr = accept_request(p_rows, q[None, :], [0], [0.5 + 5e-6, 0.1])
    assert not near_threshold(tr)
