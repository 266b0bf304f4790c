"""Pins of the decision-band helpers (``near_threshold`` for chains,
``tree_near_threshold`` for trees): a request is set aside from bit-exact
comparison only when one of its draws lies within 1e-6 of a test threshold,
or its final draw within 1e-9 * Z of an end of the chosen token's CDF
interval.  Draws are planted just inside and just outside the band at each
kind of boundary, and at points far from all of them; planted mistakes in a
helper (always true, the final draw ignored, the tests ignored, a band on
one side only, the final draw held to the wider test band) each fail one of
the checks.
"""

from __future__ import annotations

import math

import numpy as np
import pytest

from oracle import accept_request, accept_tree_request, near_threshold, tree_near_threshold
from oracle.accept import FINAL_BAND, RATIO_BAND

BAND = 1e-6
FINAL = 1e-9

# Chain: one draft position.  p_1 = (0.1, 0.4, 0.3, 0.2), q_1 = (0.1, 0.5, 0.2, 0.2),
# draft token 1: ratio 0.8.  After a rejection the residual is
# max(0, p_1 - q_1) = (0, 0, 0.1, 0) -> only token 2 can be drawn (t = 2,
# C_1 = 0, C_2 = 0.1): its interval covers all of [0, Z).  After an accept the
# bonus comes from p_2 = (0.25, 0.25, 0.25, 0.25): intervals of width 0.25.
P1 = np.array([0.1, 0.4, 0.3, 0.2])
Q1 = np.array([0.1, 0.5, 0.2, 0.2])
P2 = np.full(4, 0.25)


def chain_trace(u_test, u_final):
    _, _, tr = accept_request(np.stack([P1, P2]), Q1[None, :], [1], [u_test, u_final])
    return tr


def check_chain_helper(fn):
    # far from everything: accept (0.3 < 0.8), bonus draw in the middle of token 1's interval
    assert not fn(chain_trace(0.3, 0.375), BAND)
    # test draw just inside the band, on both sides of the ratio
    assert fn(chain_trace(0.8 - 0.4 * BAND, 0.375), BAND)
    assert fn(chain_trace(0.8 + 0.4 * BAND, 0.375), BAND)
    # just outside
    assert not fn(chain_trace(0.8 - 3 * BAND, 0.375), BAND)
    assert not fn(chain_trace(0.8 + 3 * BAND, 0.375), BAND)
    # accepted, final draw just past an interval's start (C_1 = 0.25 of Z = 1)
    assert fn(chain_trace(0.3, 0.25 + 0.4 * FINAL), BAND)
    # ... and just before an interval's end
    assert fn(chain_trace(0.3, 0.5 - 0.4 * FINAL), BAND)
    # ... and outside both, also where the test band would still reach
    assert not fn(chain_trace(0.3, 0.25 + 3 * FINAL), BAND)
    assert not fn(chain_trace(0.3, 0.5 - 3 * FINAL), BAND)
    assert not fn(chain_trace(0.3, 0.25 + 0.5 * BAND), BAND)


def test_band_constants():
    assert RATIO_BAND == BAND and FINAL_BAND == FINAL


def test_chain_band_pins():
    check_chain_helper(near_threshold)


def test_chain_rejection_branch_uses_residual_interval():
    # rejected (0.9 >= 0.8): the residual has mass 0.1 on token 2 only, so the
    # final draw's interval is all of [0, Z) and only draws near 0 are near.
    tr = chain_trace(0.9, 0.5)
    assert tr.source == "residual" and math.isclose(tr.z, 0.1)
    assert not near_threshold(tr, BAND)
    assert near_threshold(chain_trace(0.9, 0.4 * FINAL), BAND)


# Tree: root with children node 0 (token 1) and node 1 (token 2), node 2 a
# child of node 0 (token 0).  p at the root = (0.1, 0.4, 0.3, 0.2); node 0 is
# tested against 0.4, node 1 against 0.3 / (1 - 0.4) = 0.5 after node 0 is
# rejected.  When both are rejected the final draw comes from the root's p
# without tokens 1 and 2: r = (0.1, 0, 0, 0.2), Z = 0.3, intervals
# [0, 0.1) -> token 0 and [0.1, 0.3) -> token 3.
P_ROOT = np.array([0.1, 0.4, 0.3, 0.2])
P_NODE0 = np.full(4, 0.25)
P_OTHER = np.full(4, 0.25)
TOKENS = [1, 2, 0]
PARENT = [-1, -1, 0]


def tree_trace(u0, u1, u2, u_final):
    rows = np.stack([P_ROOT, P_NODE0, P_OTHER, P_OTHER])
    _, _, _, tr = accept_tree_request(rows, TOKENS, PARENT, [u0, u1, u2, u_final])
    return tr


def check_tree_helper(fn):
    # both root children rejected (0.9 >= 0.4, 0.9 >= 0.5), final draw in the
    # middle of token 3's interval: far from every boundary
    assert not fn(tree_trace(0.9, 0.9, 0.5, 2.0 / 3.0), BAND)
    # first child's draw just inside the band around 0.4
    assert fn(tree_trace(0.4 - 0.4 * BAND, 0.9, 0.5, 2.0 / 3.0), BAND)
    assert fn(tree_trace(0.4 + 0.4 * BAND, 0.9, 0.5, 2.0 / 3.0), BAND)
    assert not fn(tree_trace(0.4 + 3 * BAND, 0.9, 0.5, 2.0 / 3.0), BAND)
    # second child's threshold is the renormalised 0.5
    assert fn(tree_trace(0.9, 0.5 + 0.4 * BAND, 0.5, 2.0 / 3.0), BAND)
    assert not fn(tree_trace(0.9, 0.5 + 3 * BAND, 0.5, 2.0 / 3.0), BAND)
    # final draw near the interval boundary at 0.1 / 0.3 = 1/3 (start of token 3)
    assert fn(tree_trace(0.9, 0.9, 0.5, 1.0 / 3.0 + 0.4 * FINAL), BAND)
    assert not fn(tree_trace(0.9, 0.9, 0.5, 1.0 / 3.0 + 3 * FINAL), BAND)
    assert not fn(tree_trace(0.9, 0.9, 0.5, 1.0 / 3.0 + 0.5 * BAND), BAND)
    # ... and near the end of token 0's interval, just below 1/3
    assert fn(tree_trace(0.9, 0.9, 0.5, 1.0 / 3.0 - 0.4 * FINAL), BAND)
    assert not fn(tree_trace(0.9, 0.9, 0.5, 1.0 / 3.0 - 3 * FINAL), BAND)


def test_tree_band_pins():
    check_tree_helper(tree_near_threshold)


def test_tree_duplicate_candidate_is_not_a_boundary():
    # a repeated sibling token has threshold 0: no draw in [0, 1) passes it, so
    # u = 0 there is no boundary case
    # (only token 1 is rejected: r = (0.1, 0, 0.3, 0.2), Z = 0.6; the final
    # draw 0.5 -> 0.3 lies inside token 2's interval [0.1, 0.4))
    rows = np.stack([P_ROOT, P_NODE0, P_OTHER, P_OTHER])
    _, _, _, tr = accept_tree_request(rows, [1, 1, 0], PARENT, [0.9, 0.0, 0.5, 0.5])
    assert any(thr == 0.0 for _, thr in tr["tests"])
    assert not tree_near_threshold(tr, BAND)


def test_tree_walk_through_accepted_node():
    # node 0 accepted (0.1 < 0.4), then node 2 (token 0) tested at node 0's
    # row: p = 0.25, draw 0.25 + 0.4e-6 -> near; 0.6 -> far
    assert tree_near_threshold(tree_trace(0.1, 0.9, 0.25 + 0.4 * BAND, 0.375), BAND)
    assert not tree_near_threshold(tree_trace(0.1, 0.9, 0.6, 0.375), BAND)


# Planted mistakes: each variant must fail its pin.
def _always(trace, band=BAND):
    return True


def _chain_no_final(tr, band=BAND):
    return any(math.isfinite(r) and abs(u - r) < band for u, r in zip(tr.draws, tr.ratios))


def _chain_no_tests(tr, band=BAND):
    return (tr.threshold - tr.c_before) < FINAL * tr.z or (tr.c_at - tr.threshold) < FINAL * tr.z


def _chain_one_sided(tr, band=BAND):
    return (any(math.isfinite(r) and 0 <= u - r < band for u, r in zip(tr.draws, tr.ratios))
            or (tr.threshold - tr.c_before) < FINAL * tr.z)


def _chain_wide_final(tr, band=BAND):
    return near_threshold(tr, band, final_band=band)


def _tree_no_final(tr, band=BAND):
    return any(0.0 < thr and abs(u - thr) < band for u, thr in tr["tests"])


def _tree_no_tests(tr, band=BAND):
    z = tr["z"]
    return (tr["threshold"] - tr["c_before"]) < FINAL * z or (tr["c_at"] - tr["threshold"]) < FINAL * z


def _tree_one_sided(tr, band=BAND):
    return (any(0.0 < thr and 0 <= u - thr < band for u, thr in tr["tests"])
            or (tr["threshold"] - tr["c_before"]) < FINAL * tr["z"])


def _tree_wide_final(tr, band=BAND):
    return tree_near_threshold(tr, band, final_band=band)


@pytest.mark.parametrize("mutant", [_always, _chain_no_final, _chain_no_tests, _chain_one_sided, _chain_wide_final])
def test_chain_pins_reject_planted_mistakes(mutant):
    with pytest.raises(AssertionError):
        check_chain_helper(mutant)


@pytest.mark.parametrize("mutant", [_always, _tree_no_final, _tree_no_tests, _tree_one_sided, _tree_wide_final])
def test_tree_pins_reject_planted_mistakes(mutant):
    with pytest.raises(AssertionError):
        check_tree_helper(mutant)
