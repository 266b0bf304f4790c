"""Exact output law of a per-request verification function.

The function under test reads each draw u[i] (i < gamma) only through the
comparison u[i] < ratio_{i+1}, and u[gamma] only through the inverse CDF of the
continuation distribution.  It is therefore constant on every box of a grid
whose cuts on each axis include those thresholds.  Evaluating it once at the
centre of every box and weighting by the box volume integrates it over
u ~ U[0, 1)^{gamma+1} exactly (up to float64 rounding).

The cut lists below are a superset of the true discontinuities: the test ratios
p_i(x_i)/q_i(x_i), and the normalised prefix sums of every distribution the
final sample could use (each residual and the bonus row).  Extra cuts only
subdivide boxes.
"""

from __future__ import annotations

import itertools
from collections import defaultdict

import numpy as np


def _cuts_test(p_row, q_row, x):
    px, qx = float(p_row[x]), float(q_row[x])
    c = [0.0, 1.0]
    if qx > 0 and 0.0 < px / qx < 1.0:
        c.append(px / qx)
    return sorted(set(c))


def _cuts_final(p_rows, q_rows):
    gamma = q_rows.shape[0]
    cands = [np.maximum(p_rows[i] - q_rows[i], 0.0) for i in range(gamma)]
    cands += [p_rows[i] for i in range(gamma + 1)]
    c = {0.0, 1.0}
    for r in cands:
        z = r.sum()
        if z > 0:
            for v in np.cumsum(r) / z:
                if 0.0 < v < 1.0:
                    c.add(float(v))
    return sorted(c)


def exact_law(fn, p_rows, q_rows, draft, final=True):
    """Distribution of fn's output over u ~ U[0,1)^{gamma+1}.

    fn(p_rows, q_rows, draft, u) -> (l, tokens, ...).  Returns a dict mapping
    (l, tuple(tokens)) to probability.  With ``final=False`` the last draw is
    fixed at 0.5 and only the law of l is meaningful.
    """
    p_rows = np.asarray(p_rows, dtype=np.float64)
    q_rows = np.asarray(q_rows, dtype=np.float64)
    gamma = len(draft)
    axes = [_cuts_test(p_rows[i], q_rows[i], int(draft[i])) for i in range(gamma)]
    axes.append(_cuts_final(p_rows, q_rows) if final else [0.0, 1.0])
    cells = []
    for cuts in axes:
        cells.append([((a + b) / 2.0, b - a) for a, b in zip(cuts[:-1], cuts[1:]) if b > a])
    law = defaultdict(float)
    for combo in itertools.product(*cells):
        u = np.array([c[0] for c in combo])
        wgt = float(np.prod([c[1] for c in combo]))
        out = fn(p_rows, q_rows, draft, u)
        law[(int(out[0]), tuple(int(t) for t in out[1]))] += wgt
    return dict(law)


def law_of_l(law):
    out = defaultdict(float)
    for (l, _), pr in law.items():
        out[l] += pr
    return dict(out)


def law_of_last(law):
    out = defaultdict(float)
    for (_, toks), pr in law.items():
        out[toks[-1]] += pr
    return dict(out)
