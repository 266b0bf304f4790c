"""GPU parity: sd_accept_resample against the oracle on identical inputs.

Accept lengths, emitted tokens and new cache lengths must be bit-exact,
excluding requests whose draws lie within 1e-6 of a decision boundary (those
are counted and reported).  Both modes are covered: probabilities given
directly, and logits with their row log-sum-exp (both sides evaluate
p = exp(logit - lse) from the same float32 numbers)."""

import math
import zlib

import numpy as np
import pytest
import torch

from oracle import accept_resample
from workloads import get_config, make_inputs

from gpu_util import DeviceBatch, announce, assert_accept_parity, tensor, to_np

pytestmark = pytest.mark.gpu


def _synthetic(rng, B, gamma, V, mode="noisy", scale=2.0, noise=1.0):
    """Logits/lse (float32), draft tables and draws for B requests."""
    G = gamma + 1
    logits = (rng.standard_normal((B * G, V)) * scale).astype(np.float32)
    l64 = logits.astype(np.float64)
    mx = l64.max(axis=1, keepdims=True)
    lse = (mx[:, 0] + np.log(np.exp(l64 - mx).sum(axis=1))).astype(np.float32)
    p = np.exp(l64 - lse.astype(np.float64)[:, None]).reshape(B, G, V)
    if mode == "equal":
        q = p[:, :gamma].astype(np.float32)
    elif mode == "independent":
        z = rng.standard_normal((B, gamma, V)) * scale
        q = np.exp(z - z.max(axis=-1, keepdims=True))
        q = (q / q.sum(axis=-1, keepdims=True)).astype(np.float32)
    else:
        z = np.log(p[:, :gamma] + 1e-30) + rng.standard_normal((B, gamma, V)) * noise
        q = np.exp(z - z.max(axis=-1, keepdims=True))
        q = (q / q.sum(axis=-1, keepdims=True)).astype(np.float32)
    draft = np.empty((B, gamma), np.int32)
    for b in range(B):
        for i in range(gamma):
            c = np.cumsum(q[b, i].astype(np.float64))
            draft[b, i] = min(V - 1, int(np.searchsorted(c, rng.random() * c[-1], side="right")))
    u = ((rng.integers(0, 1 << 32, size=(B, G), dtype=np.uint64) >> np.uint64(8)).astype(np.float64)
         * 2.0 ** -24).astype(np.float32)
    kv_len = rng.integers(G, 5000, size=B).astype(np.int32)
    return logits, lse, q, draft, u, kv_len


class _Dims:
    def __init__(self, B, gamma, V):
        self.batch, self.gamma, self.vocab = B, gamma, V
        self.n_q_heads = self.n_kv_heads = 1
        self.head_dim, self.hidden, self.dtype = 64, 64, "f32"


def _run(logits, lse, q, draft, u, kv_len, probs_mode=False, oracle=True):
    import paper_2601_21622_amd as sd
    B, gamma = draft.shape
    V = q.shape[-1]
    dims = sd.Dims.of(_Dims(B, gamma, V))
    G = gamma + 1
    if probs_mode:
        x = np.exp(logits.astype(np.float64) - lse.astype(np.float64)[:, None]).astype(np.float32)
        dx, dl = tensor(x), None
    else:
        x = logits
        dx, dl = tensor(logits), tensor(lse)
    acc = torch.empty((B,), dtype=torch.int32, device="cuda")
    tok = torch.empty((B, G), dtype=torch.int32, device="cuda")
    new = torch.empty((B,), dtype=torch.int32, device="cuda")
    ws = torch.empty((sd.sd_workspace_bytes(dims, int(kv_len.max())),), dtype=torch.uint8, device="cuda")
    sd.sd_accept_resample(dims, dx, dl, tensor(q), tensor(draft), tensor(u), kv_len, acc, tok, new, ws)
    ref = accept_resample(x, None if probs_mode else lse, q, draft, u, kv_len=kv_len) if oracle else None
    return to_np(acc), to_np(tok), to_np(new), ref


CASES = [
    # name, B, gamma, V, mode
    ("noisy_v1000", 40, 4, 1000, "noisy"),
    ("noisy_v513_g1", 50, 1, 513, "noisy"),
    ("independent_v32000", 16, 5, 32000, "independent"),
    ("equal_q_p", 20, 6, 777, "equal"),
    ("many_requests", 70, 3, 300, "noisy"),
    ("v128256", 6, 8, 128256, "noisy"),
    ("single_token_vocab", 5, 2, 1, "equal"),
    ("max_gamma", 3, 63, 300, "noisy"),          # gamma at its limit: 64 positions, one per lane
    ("max_gamma_equal", 2, 63, 300, "equal"),
    ("max_vocab", 2, 1, 2097152, "noisy"),       # the largest vocabulary: 4096 segments of 512
]


@pytest.mark.parametrize("name,B,gamma,V,mode", CASES)
@pytest.mark.parametrize("probs_mode", [False, True])
def test_accept_matches_oracle(name, B, gamma, V, mode, probs_mode):
    announce(f"accept parity case={name} B={B} gamma={gamma} V={V} probs_mode={probs_mode}")
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    args = _synthetic(rng, B, gamma, V, mode)
    acc, tok, new, ref = _run(*args, probs_mode=probs_mode)
    near = assert_accept_parity(acc, tok, new, ref)
    if mode == "equal":
        assert np.all(acc == gamma)
    announce(f"accept case={name}: {B - near} bit-exact, {near} near-threshold excluded, "
             f"mean accept {acc.mean():.2f}")


def test_accept_edge_draws_and_forced_reject():
    rng = np.random.default_rng(7)
    B, gamma, V = 8, 3, 64
    logits, lse, q, draft, u, kv_len = _synthetic(rng, B, gamma, V, "noisy")
    u[0, :] = 0.0                      # smallest draw: every test with ratio > 0 passes
    u[1, :] = 1.0 - 2.0 ** -24         # largest draw
    logits[2 * (gamma + 1), draft[2, 0]] = -1e30   # p(x_1) == 0: forced rejection
    acc, tok, new, ref = _run(logits, lse, q, draft, u, kv_len)
    assert acc[2] == 0
    assert_accept_parity(acc, tok, new, ref)
    # A draft token outside the vocabulary is rejected (never read out of bounds).
    draft[3, 1] = V + 5
    draft[3, 0] = draft[0, 0]
    u[3, 0] = 0.0
    acc, tok, _, _ = _run(logits[:4 * (gamma + 1)], lse[:4 * (gamma + 1)], q[:4], draft[:4], u[:4], kv_len[:4],
                          oracle=False)
    assert acc[3] <= 1 and tok[3, acc[3]] >= 0


def test_accept_on_workload_logits():
    cfg = get_config("vicuna7b").replace(batch=6, n_q_heads=4, n_kv_heads=4, hidden=512, vocab=5000,
                                         lengths=("fixed", 16))
    x = make_inputs(cfg)
    db = DeviceBatch(x)
    db.logits_()
    db.accept()
    ref = accept_resample(to_np(db.logits), to_np(db.lse), x.q_draft, x.draft, x.u, kv_len=x.kv_len)
    near = assert_accept_parity(to_np(db.accept_len), to_np(db.out_tok), to_np(db.new_kv_len), ref)
    announce(f"accept on workload logits: near-threshold {near}")


# Branches of the test and the correction that softmax-made inputs never
# reach (q > 0 everywhere, rows summing to one, finite logits).

def _probs_inputs(rng, B, gamma, V):
    """Probability rows p (float32, [B*G][V]), draft rows q = a noisy copy,
    draft tokens drawn from q and draws u."""
    G = gamma + 1
    z = rng.standard_normal((B * G, V))
    p = np.exp(z - z.max(axis=1, keepdims=True))
    p = (p / p.sum(axis=1, keepdims=True)).astype(np.float32)
    zq = rng.standard_normal((B, gamma, V))
    q = np.exp(zq - zq.max(axis=-1, keepdims=True))
    q = (q / q.sum(axis=-1, keepdims=True)).astype(np.float32)
    draft = rng.integers(0, V, size=(B, gamma)).astype(np.int32)
    u = rng.uniform(0.05, 0.95, size=(B, G)).astype(np.float32)
    return p, q, draft, u


def _run_probs(p, q, draft, u, kv_len):
    import paper_2601_21622_amd as sd
    B, gamma = draft.shape
    V = q.shape[-1]
    G = gamma + 1
    dims = sd.Dims.of(_Dims(B, gamma, V))
    acc = torch.empty((B,), dtype=torch.int32, device="cuda")
    tok = torch.empty((B, G), dtype=torch.int32, device="cuda")
    new = torch.empty((B,), dtype=torch.int32, device="cuda")
    ws = torch.empty((sd.sd_workspace_bytes(dims, int(kv_len.max())),), dtype=torch.uint8, device="cuda")
    sd.sd_accept_resample(dims, tensor(p), None, tensor(q), tensor(draft), tensor(u), kv_len, acc, tok, new, ws)
    ref = accept_resample(p, None, q, draft, u, kv_len=kv_len)
    return to_np(acc), to_np(tok), to_np(new), ref


@pytest.mark.parametrize("V", [64, 4097])
def test_accept_infinite_ratio_when_draft_prob_zero(V):
    """q_i(x_i) = 0 < p_i(x_i): the ratio is +inf and the draft passes for any draw."""
    rng = np.random.default_rng(11 + V)
    B, gamma = 12, 4
    G = gamma + 1
    p, q, draft, u = _probs_inputs(rng, B, gamma, V)
    for b in range(B):
        for i in range(gamma):
            q[b, i, draft[b, i]] = 0.0
            assert p[b * G + i, draft[b, i]] > 0.0
    u[:, :gamma] = np.float32(1.0 - 2.0 ** -24)          # the largest draw still passes
    acc, tok, new, ref = _run_probs(p, q, draft, u, np.full(B, 50, dtype=np.int32))
    assert all(math.isinf(r) for t in ref["traces"] for r in t.ratios)
    assert np.all(acc == gamma)
    assert_accept_parity(acc, tok, new, ref)
    announce(f"ratio +inf case V={V}: all {B} requests accepted every draft")


@pytest.mark.parametrize("V", [100, 9000])
def test_accept_vanishing_residual_falls_back_to_p(V):
    """q = 1.5 p (unnormalised): every ratio is 2/3, a draw of 0.9 rejects, and
    max(0, p - q) is zero everywhere, so the corrected token is drawn from p
    itself."""
    rng = np.random.default_rng(21 + V)
    B, gamma = 10, 3
    G = gamma + 1
    p, _, draft, u = _probs_inputs(rng, B, gamma, V)
    q = np.stack([np.stack([p[b * G + i] * np.float32(1.5) for i in range(gamma)]) for b in range(B)])
    u[:, 0] = np.float32(0.9)
    acc, tok, new, ref = _run_probs(p, q, draft, u, np.full(B, 50, dtype=np.int32))
    assert all(t.source == "residual+fallback" for t in ref["traces"])
    assert np.all(acc == 0)
    assert_accept_parity(acc, tok, new, ref)


def test_accept_final_draw_past_every_prefix_takes_last_token_with_mass():
    """A draw of 1 - 2^-24 with trailing zero-mass tokens: u * Z lies within
    one part in 2^24 of Z, past every prefix sum but the last positive one, so
    the emitted token is the last token with mass (both sides; the draw sits
    inside the decision band, so the value is asserted directly)."""
    rng = np.random.default_rng(5)
    B, gamma, V = 6, 2, 3000
    G = gamma + 1
    p, q, draft, u = _probs_inputs(rng, B, gamma, V)
    last = np.zeros(B, dtype=np.int64)
    for b in range(B):
        cut = 700 + 300 * b                              # tokens from `cut` on have no mass
        for j in range(G):
            p[b * G + j, cut:] = 0.0
        q[b] = p[b * G:b * G + gamma]                    # q = p: every draft passes, bonus from p_{gamma+1}
        last[b] = cut - 1
        draft[b] = rng.integers(0, cut, size=gamma)
    u[:, :gamma] = 0.5
    u[:, gamma] = np.float32(1.0 - 2.0 ** -24)
    acc, tok, new, ref = _run_probs(p, q, draft, u, np.full(B, 50, dtype=np.int32))
    assert np.all(acc == gamma)
    assert np.array_equal(tok[:, gamma], last), (tok[:, gamma], last)
    assert np.array_equal(ref["out_tok"][:, gamma], last)


@pytest.mark.parametrize("mode", ["bonus", "residual"])
def test_accept_masked_logits(mode):
    """Logits with -inf entries (masked tokens) have p = 0 there, on the bonus
    path (q = p, every draft accepted) and on the residual path."""
    rng = np.random.default_rng(31 if mode == "bonus" else 32)
    B, gamma, V = 16, 4, 5000
    G = gamma + 1
    logits, lse, q, draft, u, kv_len = _synthetic(rng, B, gamma, V, "equal" if mode == "bonus" else "noisy")
    mask = rng.random((B * G, V)) < 0.3
    for r in range(B * G):
        mask[r, draft[r // G, min(r % G, gamma - 1)]] = False   # keep the drafts themselves
    logits[mask] = -np.inf
    l64 = logits.astype(np.float64)
    mx = l64.max(axis=1, keepdims=True)
    lse = (mx[:, 0] + np.log(np.exp(l64 - mx).sum(axis=1))).astype(np.float32)
    if mode == "bonus":
        p = np.exp(l64 - lse.astype(np.float64)[:, None]).reshape(B, G, V)
        q = p[:, :gamma].astype(np.float32)
    acc, tok, new, ref = _run(logits, lse, q, draft, u, kv_len)
    assert_accept_parity(acc, tok, new, ref)
    # no emitted token is a masked one
    for b in range(B):
        t = tok[b, acc[b]]
        assert not mask[b * G + acc[b], t], (b, t)
    if mode == "bonus":
        assert np.all(acc == gamma)
