"""Pins of ``oracle.verify_step``, the composition of attention, projection
and acceptance, on cases whose results follow by hand.

With identical keys every score of a row is equal, so each query's attention
weights are uniform over its visible keys and O is the mean of the visible
value rows (the causal window of query j is keys 0 .. L - G + j).  With the
LM head W = c * I, a logit is c times one entry of the projected row.  The
acceptance decisions are built so that each lies far from its threshold:
a ratio of at least one always passes, a ratio near zero fails a draw of 0.9,
and a one-hot draft at the rejected position leaves p without that token as
the residual.
"""

from __future__ import annotations

import numpy as np
import pytest
from scipy.special import softmax

from oracle import verify_step
from oracle.attention import verify_attention

GAMMA = 2
G = GAMMA + 1
HQ = HKV = 2
D = 2
HID = HQ * D
C = 6.0  # logit scale of the one-hot LM head


def _caches(lengths, rng):
    """Identical keys (all zero) and distinct values, [Hkv][L][D] per request."""
    k_parts, v_parts, off = [], [], [0]
    for L in lengths:
        k_parts.append(np.zeros((HKV, L, D)))
        v_parts.append(rng.uniform(-1.0, 1.0, size=(HKV, L, D)))
        off.append(off[-1] + HKV * L * D)
    return (np.concatenate([a.ravel() for a in k_parts]), np.concatenate([a.ravel() for a in v_parts]),
            np.array(off[:-1], dtype=np.int64), v_parts)


def _mean_windows(v_parts, lengths):
    """O[b][j][h] = mean of value rows 0 .. L - G + j of head h."""
    out = np.empty((len(lengths), G, HQ, D))
    for b, (vb, L) in enumerate(zip(v_parts, lengths)):
        for j in range(G):
            for h in range(HQ):
                out[b, j, h] = vb[h, :L - G + j + 1].mean(axis=0)
    return out


def _setup(seed=3, lengths=(G, 7)):
    rng = np.random.default_rng(seed)
    B = len(lengths)
    q = rng.standard_normal((B, G, HQ, D))
    k, v, off, v_parts = _caches(lengths, rng)
    return q, k, v, off, np.array(lengths, dtype=np.int32), v_parts, B


def test_uniform_attention_is_window_mean():
    q, k, v, off, kv_len, v_parts, _ = _setup()
    attn = verify_attention(q, k, v, off, kv_len, HKV)
    assert np.allclose(attn, _mean_windows(v_parts, kv_len), atol=1e-14)
    # the root of a cache holding only this step's tokens sees key 0 alone
    assert np.allclose(attn[0, 0], v_parts[0][:, 0, :], atol=1e-15)


def test_projection_of_attention_output_rows():
    """hidden = None: row b*G + j of the projection is O[b][j] with its heads
    side by side (head-major, then the head dimension)."""
    q, k, v, off, kv_len, v_parts, B = _setup()
    w = C * np.eye(HID)
    qd = np.full((B, GAMMA, HID), 1.0 / HID)
    draft = np.zeros((B, GAMMA), dtype=np.int32)
    u = np.full((B, G), 0.5)
    out = verify_step(q, k, v, off, kv_len, HKV, None, w, qd, draft, u)
    rows = _mean_windows(v_parts, kv_len).reshape(B * G, HID)
    assert np.allclose(out["logits"], C * rows, atol=1e-13)
    lse = np.log(np.exp(C * rows).sum(axis=1))
    assert np.allclose(out["lse"], lse, atol=1e-12)


def _peaked_hidden(B, peaks):
    """Caller rows: row b*G + j is one-hot on peaks[b][j] (so p is peaked there)."""
    h = np.zeros((B * G, HID))
    for b in range(B):
        for j in range(G):
            h[b * G + j, peaks[b][j]] = 1.0
    return h


def test_caller_rows_drive_the_decisions():
    """hidden given: attention is still returned, but p comes from the caller's
    rows.  Request 0: x_1 = the peak of p_1 (ratio >= 1, accepted), x_2 a token
    of small mass under p_2 with a one-hot draft (ratio ~ 0.002, rejected by
    u = 0.9), so the corrected token is drawn from p_2 without x_2; u_2 = 0.5
    lands on the peak of p_2.  Request 1: both drafts are the peaks (accepted)
    and the bonus token comes from p_3."""
    q, k, v, off, kv_len, v_parts, B = _setup()
    peaks = [[3, 1, 0], [2, 0, 3]]
    hidden = _peaked_hidden(B, peaks)
    w = C * np.eye(HID)
    p = softmax(C * hidden, axis=1)               # [B*G][V]
    qd = np.full((B, GAMMA, HID), 1.0 / HID)
    draft = np.array([[3, 2], [2, 0]], dtype=np.int32)
    qd[0, 1] = np.eye(HID)[2]                      # one-hot draft at the rejected position
    u = np.array([[0.3, 0.9, 0.5], [0.99, 0.4, 0.5]])
    out = verify_step(q, k, v, off, kv_len, HKV, hidden, w, qd, draft, u)

    assert np.allclose(out["attn"], _mean_windows(v_parts, kv_len), atol=1e-14)
    assert np.allclose(out["logits"], C * hidden, atol=1e-15)
    # request 0: p_1(3) / (1/4) > 1 passes; p_2(2) / 1 = small fails u = 0.9
    assert p[0, 3] / 0.25 > 1.0 and p[1, 2] < 0.01
    assert out["accept_len"].tolist() == [1, 2]
    # corrected token of request 0: r = p_2 without token 2; u * Z = 0.5 * Z
    # falls inside token 1's interval (the peak of p_2); bonus of request 1
    # from p_3 of request 1, peaked on token 3: 0.5 lands there.
    r = p[1].copy()
    r[2] = 0.0
    cdf = np.cumsum(r)
    assert cdf[0] < 0.5 * cdf[-1] < cdf[1]
    assert p[5, :3].sum() < 0.5 < p[5].sum()
    assert out["out_tok"].tolist() == [[3, 1, -1], [2, 0, 3]]
    assert out["new_kv_len"].tolist() == [int(kv_len[0]) - GAMMA + 1, int(kv_len[1]) - GAMMA + 2]


def test_wrong_row_order_is_caught():
    """A planted mistake: projecting O viewed head-major ([Hq][G][D]) instead of
    row-major changes the logits the pin above compares."""
    q, k, v, off, kv_len, v_parts, B = _setup()
    attn = verify_attention(q, k, v, off, kv_len, HKV)
    wrong = attn.transpose(0, 2, 1, 3).reshape(B * G, HID)
    rows = _mean_windows(v_parts, kv_len).reshape(B * G, HID)
    assert not np.allclose(C * wrong, C * rows, atol=1e-6)


@pytest.mark.parametrize("L", [G, G + 1, 40])
def test_step_tokens_follow_attention_rows(L):
    """hidden = None end to end: with one head's value rows making a single
    entry dominant in every window, the accepted drafts are exactly the
    entries that dominate (ratio >= 1 under a uniform draft)."""
    rng = np.random.default_rng(L)
    B = 1
    q = rng.standard_normal((B, G, HQ, D))
    k = np.zeros(HKV * L * D)
    v = np.zeros((HKV, L, D))
    v[1, :, 0] = 5.0          # head 1, dimension 0 -> hidden entry 2 dominates every row
    out = verify_step(q, k, v.ravel(), np.array([0]), np.array([L], dtype=np.int32), HKV, None, C * np.eye(HID),
                      np.full((B, GAMMA, HID), 1.0 / HID), np.array([[2, 2]], dtype=np.int32),
                      np.array([[0.9, 0.9, 0.5]]))
    assert out["accept_len"].tolist() == [GAMMA]
    assert out["out_tok"].tolist() == [[2, 2, 2]]
