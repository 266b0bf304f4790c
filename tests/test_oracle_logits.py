"""Pins of the oracle's vocabulary projection and log-sum-exp (oracle.logits).

* Integer operands make every float64 logit exact; compared with an int64
  product (exact integer arithmetic, a different number system).
* One-hot weight rows select hidden entries (closed form).
* LSE agrees with scipy.special.logsumexp (an independent library routine).
* p = exp(logits - lse) rows sum to one; adding a constant to a row leaves p
  unchanged and shifts lse by that constant; huge logits do not overflow.
"""

import numpy as np
import pytest
from scipy.special import logsumexp

from oracle.logits import probabilities, verify_logits


def test_integer_operands_exact():
    rng = np.random.default_rng(0)
    h = rng.integers(-50, 50, size=(7, 33))
    w = rng.integers(-50, 50, size=(101, 33))
    logits, _ = verify_logits(h.astype(np.float32), w.astype(np.float32), v_chunk=16)
    assert np.array_equal(logits, (h.astype(np.int64) @ w.astype(np.int64).T).astype(np.float64))


def test_one_hot_rows_select_hidden_entries():
    rng = np.random.default_rng(1)
    h = rng.normal(size=(4, 10))
    cols = rng.integers(0, 10, size=25)
    w = np.zeros((25, 10))
    w[np.arange(25), cols] = 1.0
    logits, _ = verify_logits(h, w)
    assert np.array_equal(logits, h[:, cols])


def test_lse_matches_scipy_and_rows_normalise():
    rng = np.random.default_rng(2)
    h = rng.normal(size=(5, 64))
    w = rng.normal(size=(1000, 64)) * 0.3
    logits, lse = verify_logits(h, w, v_chunk=128)
    assert np.allclose(lse, logsumexp(logits, axis=1), rtol=0, atol=1e-12)
    p = probabilities(logits, lse)
    assert np.allclose(p.sum(axis=1), 1.0, atol=1e-12)


def test_shift_invariance_and_no_overflow():
    rng = np.random.default_rng(3)
    h = rng.normal(size=(3, 8))
    w = rng.normal(size=(50, 8))
    logits, lse = verify_logits(h, w)
    p = probabilities(logits, lse)
    big = logits + 1000.0
    lse_big = np.log(np.exp(big - big.max(axis=1, keepdims=True)).sum(axis=1)) + big.max(axis=1)
    assert np.allclose(probabilities(big, lse_big), p, atol=1e-12)
    # The oracle itself on inputs producing huge logits.
    _, lse2 = verify_logits(h * 1e3, w)
    assert np.all(np.isfinite(lse2))


def test_shape_mismatch_rejected():
    with pytest.raises(ValueError):
        verify_logits(np.zeros((2, 3)), np.zeros((4, 5)))
