"""Pins of the warped target distributions (oracle.warp) and of verification
against them (oracle.accept.accept_resample_sampled).

Temperature, top-k, top-p and greedy selection replace the target p of the
Leviathan test (Sec. 2) with a warped p'; the pins check each warp against an
independent route (a power of the probabilities, numpy's partition, scipy's
softmax, a hand-worked fixture) and that verification stays lossless with
respect to the warped target (brute force, as for the plain target).
"""

import itertools
import json
import os

import numpy as np
import pytest
from scipy.special import softmax

from oracle import accept_request, accept_resample_sampled, order_keys, warp_row, warped_from_cut
from exact_law import exact_law

HERE = os.path.dirname(os.path.abspath(__file__))


def _row(rng, V, scale=2.0):
    return (rng.standard_normal(V) * scale).astype(np.float32)


def test_order_keys_follow_float_order():
    vals = np.array([-np.inf, -3.4e38, -2.0, -1e-30, -0.0, 0.0, 1e-45, 1e-30, 1.0, 2.0, 3.4e38, np.inf],
                    dtype=np.float32)
    k = order_keys(vals)
    assert np.all(np.diff(k.astype(np.int64)) > 0)


def test_identity_warp_is_softmax():
    rng = np.random.default_rng(1)
    x = _row(rng, 1000)
    wr = warp_row(x, 1.0)
    np.testing.assert_allclose(wr.p, softmax(x.astype(np.float64)), rtol=1e-12, atol=0)
    assert wr.theta_key == 0 and not wr.near


@pytest.mark.parametrize("T", [0.5, 0.7, 2.0])
def test_temperature_is_a_power_of_the_probabilities(T):
    rng = np.random.default_rng(2)
    x = _row(rng, 500)
    p = softmax(x.astype(np.float64))
    want = p ** (1.0 / T)
    want /= want.sum()
    np.testing.assert_allclose(warp_row(x, T).p, want, rtol=1e-10, atol=1e-300)


@pytest.mark.parametrize("k", [1, 7, 100, 499])
def test_top_k_keeps_exactly_the_k_largest(k):
    rng = np.random.default_rng(3)
    x = _row(rng, 500)
    assert len(np.unique(x)) == 500
    wr = warp_row(x, 0.8, top_k=k)
    kept = set(np.nonzero(wr.p > 0)[0].tolist())
    assert kept == set(np.argpartition(-x.astype(np.float64), k - 1)[:k].tolist())
    a, b = sorted(kept)[0], sorted(kept)[-1]
    assert np.isclose(wr.p[a] / wr.p[b], np.exp((float(x[a]) - float(x[b])) / 0.8), rtol=1e-12)
    assert abs(wr.p.sum() - 1.0) < 1e-12


def test_top_k_keeps_every_tie_of_the_kth_logit():
    x = np.array([3.0, 2.0, 2.0, 1.0, 2.0], dtype=np.float32)
    wr = warp_row(x, 1.0, top_k=2)
    assert set(np.nonzero(wr.p > 0)[0].tolist()) == {0, 1, 2, 4}


@pytest.mark.parametrize("top_p,top_k", [(0.5, 0), (0.9, 0), (0.99, 0), (0.9, 40)])
def test_top_p_set_is_sufficient_and_minimal(top_p, top_k):
    rng = np.random.default_rng(4)
    for _ in range(20):
        x = _row(rng, 300, scale=3.0)
        T = 0.9
        wr = warp_row(x, T, top_k=top_k, top_p=top_p)
        if wr.near:
            continue
        base = softmax(x.astype(np.float64) / T)
        if top_k:
            cut = np.sort(x)[::-1][top_k - 1]
            base = np.where(x >= cut, base, 0.0)
            base /= base.sum()
        kept = wr.p > 0
        assert base[kept].sum() >= top_p
        smallest = x[kept].min()
        assert base[kept & (x > smallest)].sum() < top_p
        assert np.all(x[~kept] < smallest)


def test_hand_worked_fixture():
    fx = json.load(open(os.path.join(HERE, "golden", "sampling_example.json")))
    x = np.log(np.array(fx["probabilities"])).astype(np.float32)
    for c in fx["cases"]:
        got = warp_row(x, c["temperature"], c["top_k"], c["top_p"]).p
        np.testing.assert_allclose(got, c["expect"], rtol=1e-6, atol=1e-7, err_msg=c["why"])
    g = fx["greedy_ties"]
    wr = warp_row(np.array(g["logits"], dtype=np.float32), 0.0)
    assert wr.argmax == g["argmax"] and wr.p[g["argmax"]] == 1.0 and wr.p.sum() == 1.0


def test_cut_reproduces_the_warped_row():
    rng = np.random.default_rng(5)
    x = _row(rng, 777)
    for T, k, p in [(1.0, 0, 1.0), (0.6, 50, 0.8), (1.7, 0, 0.95), (0.0, 0, 1.0)]:
        wr = warp_row(x, T, k, p)
        got = warped_from_cut(x, T, wr.theta_key, wr.lse, wr.argmax)
        np.testing.assert_allclose(got, wr.p, rtol=1e-6, atol=1e-12)


def test_greedy_verification_accepts_the_argmax_prefix():
    rng = np.random.default_rng(6)
    B, gamma, V = 30, 5, 40
    G = gamma + 1
    logits = (rng.standard_normal((B * G, V)) * 2).astype(np.float32)
    am = logits.argmax(axis=1).reshape(B, G)
    draft = np.where(rng.random((B, gamma)) < 0.6, am[:, :gamma], rng.integers(0, V, (B, gamma)))
    q = rng.dirichlet(np.ones(V), size=(B, gamma))
    for trial in range(3):
        u = rng.random((B, G)).astype(np.float32)
        out = accept_resample_sampled(logits, q, draft, u, 0.0)
        for b in range(B):
            l = 0
            while l < gamma and draft[b, l] == am[b, l]:
                l += 1
            assert out["accept_len"][b] == l
            assert out["out_tok"][b, l] == am[b, l]


V8, GAMMA = 8, 2


def _warped_tables(seed, T, k, p):
    rng = np.random.default_rng(seed)

    def warp(lg):
        return warp_row(lg.astype(np.float32), T, k, p).p

    def logits():
        return rng.standard_normal(V8) * 1.5

    p1 = warp(logits())
    p2 = np.stack([warp(logits()) for _ in range(V8)])
    p3 = np.stack([np.stack([warp(logits()) for _ in range(V8)]) for _ in range(V8)])
    q1 = warp(logits())
    q2 = np.stack([warp(logits()) for _ in range(V8)])
    return p1, p2, p3, q1, q2


@pytest.mark.parametrize("T,k,p", [(0.7, 5, 0.9), (1.3, 0, 0.8), (0.0, 0, 1.0)])
def test_verification_is_lossless_for_the_warped_target(T, k, p):
    p1, p2, p3, q1, q2 = _warped_tables(21, T, k, p)
    cond = [lambda s: p1, lambda s: p2[s[0]], lambda s: p3[s[0], s[1]]]
    joint = np.zeros((V8, V8, V8))
    for x1, x2 in itertools.product(range(V8), repeat=2):
        w = q1[x1] * q2[x1, x2]
        if w == 0:
            continue
        p_rows = np.stack([p1, p2[x1], p3[x1, x2]])
        q_rows = np.stack([q1, q2[x1]])
        for (l, toks), pr in exact_law(accept_request, p_rows, q_rows, [x1, x2]).items():
            prefixes = [(tuple(toks), w * pr)]
            for kk in range(len(toks), 3):
                nxt = []
                for s, m in prefixes:
                    row = cond[kk](s)
                    for v in range(V8):
                        if row[v] > 0:
                            nxt.append((s + (v,), m * row[v]))
                prefixes = nxt
            for s, m in prefixes:
                joint[s[:3]] += m
    want = p1[:, None, None] * p2[:, :, None] * p3
    np.testing.assert_allclose(joint, want, atol=1e-12)


# ---- planted mistakes in warp_row (on the CPU): each must fail a pin above ----

import inspect
import textwrap

import oracle.warp as warp_mod

_MUTATIONS = {
    "tempered_by_multiplying": ("w = np.exp((x - m) / temperature)", "w = np.exp((x - m) * temperature)"),
    "top_k_off_by_one": ("np.sort(keys)[::-1][top_k - 1]", "np.sort(keys)[::-1][top_k]"),
    "top_k_drops_ties": ("keep = keys >= theta\n", "keep = keys > theta\n"),
    "greedy_last_maximum": ("argmax = int(np.argmax(keys))", "argmax = int(len(keys) - 1 - np.argmax(keys[::-1]))"),
    "top_p_one_level_short": ("theta = max(theta, int(levels[j]))", "theta = max(theta, int(levels[max(j - 1, 0)]))"),
    "top_p_against_whole_row": ("total = float(w[keep].sum())", "total = float(w.sum())"),
    "normaliser_without_top_k": ("W = float(w[keep].sum())", "W = float(w.sum())"),
}


def _mutant(name):
    old, new = _MUTATIONS[name]
    src = textwrap.dedent(inspect.getsource(warp_mod.warp_row))
    assert old in src, f"mutation target for {name} not found in the oracle"
    ns = dict(vars(warp_mod))
    exec(compile(src.replace(old, new), "<mutant>", "exec"), ns)
    return ns["warp_row"]


def _pins_pass(fn):
    rng = np.random.default_rng(7)
    x = _row(rng, 300, scale=3.0)
    fx = json.load(open(os.path.join(HERE, "golden", "sampling_example.json")))
    xs = np.log(np.array(fx["probabilities"])).astype(np.float32)
    for c in fx["cases"]:
        if not np.allclose(fn(xs, c["temperature"], c["top_k"], c["top_p"]).p, c["expect"], rtol=1e-6, atol=1e-7):
            return False
    g = fx["greedy_ties"]
    if fn(np.array(g["logits"], dtype=np.float32), 0.0).argmax != g["argmax"]:
        return False
    for k in (1, 7, 100):
        wr = fn(x, 0.8, top_k=k)
        if set(np.nonzero(wr.p > 0)[0].tolist()) != set(np.argpartition(-x.astype(np.float64), k - 1)[:k].tolist()):
            return False
    p = softmax(x.astype(np.float64))
    want = p ** 2.0
    if not np.allclose(fn(x, 0.5).p, want / want.sum(), rtol=1e-10):
        return False
    for top_p, top_k in [(0.9, 0), (0.9, 40)]:
        wr = fn(x, 0.9, top_k=top_k, top_p=top_p)
        base = softmax(x.astype(np.float64) / 0.9)
        if top_k:
            base = np.where(x >= np.sort(x)[::-1][top_k - 1], base, 0.0)
            base /= base.sum()
        kept = wr.p > 0
        if base[kept].sum() < top_p or base[kept & (x > x[kept].min())].sum() >= top_p:
            return False
        if abs(wr.p.sum() - 1.0) > 1e-9:
            return False
    return True


def test_pins_pass_for_the_oracle():
    assert _pins_pass(warp_row)


@pytest.mark.parametrize("name", sorted(_MUTATIONS))
def test_pins_reject_planted_mistake(name):
    fn = _mutant(name)
    try:
        ok = _pins_pass(fn)
    except Exception:
        return  # a crash is also a detection
    assert not ok, f"pins did not catch {name}"
