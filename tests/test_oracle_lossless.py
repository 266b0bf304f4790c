"""Brute-force losslessness of the oracle's verification (oracle.accept).

Speculative decoding must leave the target model's output distribution
unchanged (Sec. 1 and Sec. 2 of the paper; the property Algorithm 2's
correction step exists for).  With a vocabulary of 8 and gamma = 2, build
prefix-dependent target tables p_1, p_2(.|x_1), p_3(.|x_1, x_2) and draft
tables q_1, q_2(.|x_1), with zeros in both.  Enumerate every draft path, every
acceptance branch (exactly, over the draws) and extend each emitted prefix to
three tokens with exact target samples.  The joint law of the three tokens
must be p_1 p_2 p_3.

The second half plants plausible mistakes in copies of the oracle (on the CPU)
and checks that this pin rejects each of them.
"""

import inspect
import itertools
import textwrap

import numpy as np
import pytest

import oracle.accept as acc
from exact_law import exact_law

V = 8
GAMMA = 2


def _tables(seed):
    rng = np.random.default_rng(seed)

    def dist(zeros):
        p = rng.dirichlet(np.ones(V) * 0.7)
        if zeros:
            p[rng.choice(V, size=zeros, replace=False)] = 0.0
            p /= p.sum()
        return p

    p1 = dist(2)
    p2 = np.stack([dist(1 + (a % 3)) for a in range(V)])
    p3 = np.stack([np.stack([dist((a + b) % 3) for b in range(V)]) for a in range(V)])
    q1 = dist(3)
    q2 = np.stack([dist(2 - (a % 3)) for a in range(V)])
    return p1, p2, p3, q1, q2


def joint_after_verification(fn, tables):
    p1, p2, p3, q1, q2 = tables
    cond = [lambda s: p1, lambda s: p2[s[0]], lambda s: p3[s[0], s[1]]]
    joint = np.zeros((V, V, V))
    for x1, x2 in itertools.product(range(V), repeat=2):
        w = q1[x1] * q2[x1, x2]
        if w == 0:
            continue
        p_rows = np.stack([p1, p2[x1], p3[x1, x2]])
        q_rows = np.stack([q1, q2[x1]])
        for (l, toks), pr in exact_law(fn, p_rows, q_rows, [x1, x2]).items():
            # Extend the emitted prefix with exact target samples.
            prefixes = [(tuple(toks), w * pr)]
            for k in range(len(toks), 3):
                nxt = []
                for s, m in prefixes:
                    row = cond[k](s)
                    for v in range(V):
                        if row[v] > 0:
                            nxt.append((s + (v,), m * row[v]))
                prefixes = nxt
            for s, m in prefixes:
                joint[s[:3]] += m
    return joint


def target_joint(tables):
    p1, p2, p3, _, _ = tables
    return p1[:, None, None] * p2[:, :, None] * p3


@pytest.mark.parametrize("seed", [11, 12, 13])
def test_emitted_tokens_follow_target(seed):
    t = _tables(seed)
    joint = joint_after_verification(acc.accept_request, t)
    assert np.abs(joint - target_joint(t)).max() < 1e-12
    # The first emitted token alone is distributed exactly as p_1.
    assert np.abs(joint.sum(axis=(1, 2)) - t[0]).max() < 1e-12


# ---- planted mistakes -------------------------------------------------------

_MUTATIONS = {
    # The test as printed, without dividing by q_i(x_i).
    "no_division_by_q": ("return px / qx", "return px"),
    # Correction with the draft distribution of the wrong position.
    "residual_wrong_q_index": ("np.maximum(p_rows[l] - q_rows[l], 0.0)",
                               "np.maximum(p_rows[l] - q_rows[max(l - 1, 0)], 0.0)"),
    # Correction from the wrong target row.
    "residual_wrong_p_row": ("np.maximum(p_rows[l] - q_rows[l], 0.0)",
                             "np.maximum(p_rows[min(l + 1, gamma)] - q_rows[l], 0.0)"),
    # Absolute difference instead of the positive part.
    "residual_abs": ("np.maximum(p_rows[l] - q_rows[l], 0.0)", "np.abs(p_rows[l] - q_rows[l])"),
    # Sampling the correction from p instead of the residual.
    "residual_is_p": ("np.maximum(p_rows[l] - q_rows[l], 0.0)", "p_rows[l].copy()"),
    # Reusing the rejected test's draw for the final sample.
    "reuse_rejected_draw": ("thr = float(u[gamma]) * z", "thr = float(u[min(l, gamma)]) * z"),
    # Sign flip in the test.
    "accept_when_above": ("if not (float(u[i]) < ratio):", "if float(u[i]) < ratio:"),
}


def _mutant(name):
    old, new = _MUTATIONS[name]
    src = textwrap.dedent(inspect.getsource(acc.accept_request))
    ratio_src = textwrap.dedent(inspect.getsource(acc._ratio))
    assert old in src or old in ratio_src, f"mutation target for {name} not found in the oracle"
    src = src.replace(old, new)
    ratio_src = ratio_src.replace(old, new)
    ns = dict(vars(acc))
    exec(compile(ratio_src, "<mutant_ratio>", "exec"), ns)
    exec(compile(src, "<mutant>", "exec"), ns)
    return ns["accept_request"]


@pytest.mark.parametrize("name", sorted(_MUTATIONS))
def test_pin_rejects_planted_mistake(name):
    fn = _mutant(name)
    t = _tables(11)
    try:
        joint = joint_after_verification(fn, t)
    except Exception:
        return  # a crash is also a detection
    assert np.abs(joint - target_joint(t)).max() > 1e-6, f"pin did not catch {name}"
