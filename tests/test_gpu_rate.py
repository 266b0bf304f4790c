"""GPU parity of the acceptance rate (sd_acceptance_rate) against the oracle
(oracle.model.acceptance_rate_batch).

Inputs are seeded host arrays: target logits ~ N(0, 2^2) per entry with the
row log-sum-exp taken in float64 from the float32 logits, or the float64
softmax of them rounded to float32 (probability mode); draft distributions
are softmaxes of the target logits plus N(0, s^2) noise, so beta spans
roughly 0.2 to 0.99.  Bound: |gpu - oracle| <= 1e-6 in logit mode (p is
evaluated in float32 within a few ulp of exp(logit - lse), so sum |dp| stays
below about 4e-7; the sums are float64) and <= 1e-12 with probabilities
(the same float32 minima, summed in another order).  Shapes cover ragged and
tiny vocabularies, one token, more than 64 requests, 63 draft positions and
the four bf16 workloads at their full batch, depth and vocabulary.
"""

import zlib

import numpy as np
import pytest
import torch

import paper_2601_21622_amd as sd
from oracle import acceptance_rate_batch
from workloads import get_config

from gpu_util import announce, tensor, to_np

pytestmark = pytest.mark.gpu


def _inputs(seed, B, gamma, V, noise):
    rng = np.random.default_rng(seed)
    G = gamma + 1
    logits = (rng.standard_normal((B * G, V)) * 2.0).astype(np.float32)
    l64 = logits.astype(np.float64)
    mx = l64.max(axis=1, keepdims=True)
    lse = mx[:, 0] + np.log(np.exp(l64 - mx).sum(axis=1))
    q = np.empty((B, gamma, V), dtype=np.float32)
    for b in range(B):
        for i in range(gamma):
            z = l64[b * G + i] + rng.standard_normal(V) * noise[(b * gamma + i) % len(noise)]
            e = np.exp(z - z.max())
            q[b, i] = (e / e.sum()).astype(np.float32)
    return logits, lse.astype(np.float32), q


def _run(B, gamma, V, logits, lse, q, probs_mode):
    cfg = get_config("tiny").replace(batch=B, gamma=gamma, vocab=V, n_q_heads=1, n_kv_heads=1)
    dims = sd.Dims.of(cfg)
    if probs_mode:
        x = np.exp(logits.astype(np.float64) - lse.astype(np.float64)[:, None]).astype(np.float32)
        dx, dl = tensor(x), None
    else:
        x, dx, dl = logits, tensor(logits), tensor(lse)
    beta = torch.empty((B, gamma), dtype=torch.float64, device="cuda")
    ws = torch.empty((sd.sd_workspace_bytes(dims, gamma + 1),), dtype=torch.uint8, device="cuda")
    sd.sd_acceptance_rate(dims, dx, dl, tensor(q), beta, ws)
    torch.cuda.synchronize()
    ref = acceptance_rate_batch(x, None if probs_mode else lse, q, gamma)
    return to_np(beta), ref


CASES = {
    "v1000": (12, 4, 1000),
    "v_ragged": (5, 3, 2049),
    "v7": (3, 2, 7),
    "v1": (2, 3, 1),
    "many_requests": (70, 4, 300),
    "max_gamma": (2, 63, 500),
    "v32000": (8, 5, 32000),
    "v128256": (3, 6, 128256),
}


@pytest.mark.parametrize("probs_mode", [False, True])
@pytest.mark.parametrize("name", sorted(CASES))
def test_rate_matches_oracle(name, probs_mode):
    B, gamma, V = CASES[name]
    announce(f"acceptance rate case={name} B={B} gamma={gamma} V={V} probs_mode={probs_mode}")
    logits, lse, q = _inputs(zlib.crc32(name.encode()), B, gamma, V, (0.3, 1.0, 3.0))
    got, ref = _run(B, gamma, V, logits, lse, q, probs_mode)
    tol = 1e-12 if probs_mode else 1e-6
    err = float(np.abs(got - ref).max())
    assert err <= tol, (name, err)
    assert np.all((got >= -1e-12) & (got <= 1 + 1e-6))
    announce(f"acceptance rate case={name}: max err {err:.2e}, beta range [{ref.min():.3f}, {ref.max():.3f}]")


@pytest.mark.parametrize("workload", ["vicuna7b", "pooled", "llama3_8b", "llama70b_share"])
def test_rate_full_size(workload):
    cfg = get_config(workload)
    B, gamma, V = cfg.batch, cfg.gamma, cfg.vocab
    announce(f"acceptance rate full size workload={workload} B={B} gamma={gamma} V={V}")
    logits, lse, q = _inputs(zlib.crc32(workload.encode()), B, gamma, V, (0.5, 1.5))
    got, ref = _run(B, gamma, V, logits, lse, q, False)
    err = float(np.abs(got - ref).max())
    assert err <= 1e-6, (workload, err)


def test_rate_is_deterministic_and_exact_cases():
    B, gamma, V = 4, 3, 5000
    logits, lse, q = _inputs(7, B, gamma, V, (1.0,))
    a, _ = _run(B, gamma, V, logits, lse, q, False)
    b, _ = _run(B, gamma, V, logits, lse, q, False)
    assert np.array_equal(a, b)
    # q equal to p (probability mode): beta is the sum of p, 1 up to float32 rounding of p.
    G = gamma + 1
    p = np.exp(logits.astype(np.float64) - lse.astype(np.float64)[:, None]).astype(np.float32)
    q_same = np.stack([p[b * G:b * G + gamma] for b in range(B)])
    got, ref = _run(B, gamma, V, logits, lse, q_same, True)
    assert np.abs(got - ref).max() <= 1e-12
    assert np.abs(got - 1.0).max() <= 1e-5


def test_rate_with_masked_logits():
    """-inf logits (masked tokens) have p = 0, so they add nothing to
    sum min(p, q) even where q > 0."""
    B, gamma, V = 6, 4, 3000
    logits, _, q = _inputs(91, B, gamma, V, (0.5, 2.0))
    rng = np.random.default_rng(92)
    logits[rng.random(logits.shape) < 0.35] = -np.inf
    l64 = logits.astype(np.float64)
    mx = l64.max(axis=1, keepdims=True)
    lse = (mx[:, 0] + np.log(np.exp(l64 - mx).sum(axis=1))).astype(np.float32)
    got, ref = _run(B, gamma, V, logits, lse, q, False)
    assert np.all(np.isfinite(got))
    assert float(np.abs(got - ref).max()) <= 1e-6
