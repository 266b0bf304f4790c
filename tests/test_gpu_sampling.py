"""GPU parity of sampled verification (sd_accept_resample_sampled and
sd_verify_step_sampled) against the oracle (oracle.warp, oracle.accept).

Three comparisons per case:
* the cut: the GPU's smallest kept logit equals the oracle's exactly (keys of
  float32 values), except rows whose top-p cut the oracle flags as lying
  within 1e-6 of a cumulative mass (float32 vs float64 masses may differ
  there); the GPU's normaliser matches the oracle's within 1e-5 relative;
* acceptance on identical p': the oracle re-runs the test and correction on
  the GPU's own cut and normaliser (widened to float64), and accept lengths
  and emitted tokens must agree bit for bit outside the 1e-6 decision band;
* the agreement of the fully independent oracle (its own cut) is reported.
Vocabularies 1000, 32000 and 128256; temperature 0 (greedy), below and above
1; top-k 1, 40 and off; top-p 0.5, 0.9 and off.
"""

import zlib

import numpy as np
import pytest
import torch

import paper_2601_21622_amd as sd
from oracle import accept_resample_sampled, order_keys, warp_row
from workloads import get_config, make_inputs

from gpu_util import DeviceBatch, announce, assert_accept_parity, max_excluded, to_np

pytestmark = pytest.mark.gpu

SETTINGS = {
    "identity": (1.0, 0, 1.0),
    "t07": (0.7, 0, 1.0),
    "t13_k40": (1.3, 40, 1.0),
    "t08_p09": (0.8, 0, 0.9),
    "t10_k40_p05": (1.0, 40, 0.5),
    "top1": (0.6, 1, 1.0),
    "greedy": (0.0, 0, 1.0),
}

SHAPES = {
    "v1000": (24, 4, 1000),
    "v32000": (8, 5, 32000),
    "v128256": (4, 3, 128256),
}


def _inputs(B, gamma, V, T, k, p, seed, levels=None):
    """Target logits, warped draft distributions and drafts drawn from them;
    with ``levels``, the target logits are rounded onto that many steps of
    their range, so that large sets of them tie."""
    rng = np.random.default_rng(seed)
    G = gamma + 1
    logits = (rng.standard_normal((B * G, V)) * 2.0).astype(np.float32)
    if levels is not None:
        lo, hi = float(logits.min()), float(logits.max())
        step = (hi - lo) / levels
        logits = (np.round((logits - lo) / step) * step + lo).astype(np.float32)
    q = np.empty((B, gamma, V), dtype=np.float32)
    draft = np.empty((B, gamma), dtype=np.int32)
    for b in range(B):
        for i in range(gamma):
            noisy = (logits[b * G + i] + rng.standard_normal(V).astype(np.float32) * 0.7).astype(np.float32)
            qi = warp_row(noisy, T if T > 0 else 1.0, k, p).p
            q[b, i] = qi
            c = np.cumsum(qi)
            draft[b, i] = min(int(np.searchsorted(c, rng.random() * c[-1], side="right")), V - 1)
    u = ((rng.integers(0, 1 << 32, size=(B, G), dtype=np.uint64) >> 8).astype(np.float64) * 2.0 ** -24).astype(np.float32)
    return logits, q, draft, u


def _check_cut(logits, T, k, p, gpu_lse, gpu_min):
    bad_cut = 0
    flagged = 0
    for r in range(logits.shape[0]):
        wr = warp_row(logits[r], T, k, p)
        if T == 0.0:
            assert np.isposinf(gpu_min[r]) and gpu_lse[r] == 0.0
            continue
        gkey = 0 if np.isneginf(gpu_min[r]) else int(order_keys(np.array([gpu_min[r]], dtype=np.float32))[0])
        if gkey != wr.theta_key:
            if wr.near:
                flagged += 1
                continue
            bad_cut += 1
            continue
        assert abs(float(gpu_lse[r]) - wr.lse) <= 1e-5 * max(1.0, abs(wr.lse)), (r, gpu_lse[r], wr.lse)
    assert bad_cut == 0, f"{bad_cut} rows cut differently from the oracle outside the band"
    assert flagged <= max_excluded(logits.shape[0]), f"{flagged} rows with a top-p cut in the band"
    return flagged


def _gpu_cut(logits, T, gpu_lse, gpu_min):
    keys = np.where(np.isneginf(gpu_min), 0, order_keys(gpu_min.astype(np.float32)).astype(np.int64))
    if T == 0.0:
        keys = np.full(logits.shape[0], (1 << 32) - 1, dtype=np.int64)
    argmax = np.array([int(np.argmax(order_keys(row))) for row in logits])
    return keys, gpu_lse.astype(np.float64), argmax


@pytest.mark.parametrize("shape", sorted(SHAPES))
@pytest.mark.parametrize("setting", sorted(SETTINGS))
def test_sampled_accept_matches_oracle(shape, setting):
    B, gamma, V = SHAPES[shape]
    T, k, p = SETTINGS[setting]
    announce(f"sampled accept case={setting} shape={shape} B={B} gamma={gamma} V={V} T={T} k={k} p={p}")
    logits, q, draft, u = _inputs(B, gamma, V, T, k, p, seed=zlib.crc32(f"{shape}/{setting}".encode()))
    G = gamma + 1
    kv_len = np.full(B, 100, dtype=np.int32)
    cfg = get_config("tiny").replace(batch=B, gamma=gamma, vocab=V)
    dims = sd.Dims.of(cfg)
    dev = "cuda"
    t_logits = torch.from_numpy(logits).to(dev)
    t_q = torch.from_numpy(q).to(dev)
    t_draft = torch.from_numpy(draft).to(dev)
    t_u = torch.from_numpy(u).to(dev)
    lse = torch.empty(B * G, dtype=torch.float32, device=dev)
    mn = torch.empty(B * G, dtype=torch.float32, device=dev)
    acc = torch.empty(B, dtype=torch.int32, device=dev)
    tok = torch.empty((B, G), dtype=torch.int32, device=dev)
    new = torch.empty(B, dtype=torch.int32, device=dev)
    ws = torch.empty(sd.sd_workspace_bytes(dims, 100), dtype=torch.uint8, device=dev)
    sd.sd_accept_resample_sampled(dims, sd.Sampling(T, k, p), t_logits, t_q, t_draft, t_u, kv_len, lse, mn, acc, tok,
                                  new, ws)
    torch.cuda.synchronize()
    g_lse, g_min = to_np(lse), to_np(mn)
    flagged = _check_cut(logits, T, k, p, g_lse, g_min)

    ref = accept_resample_sampled(logits, q, draft, u, T, k, p, kv_len, cut=_gpu_cut(logits, T, g_lse, g_min))
    near = assert_accept_parity(to_np(acc), to_np(tok), to_np(new), ref)
    indep = accept_resample_sampled(logits, q, draft, u, T, k, p, kv_len)
    agree = float(np.mean(np.all(indep["out_tok"] == to_np(tok), axis=1)))
    announce(f"case={setting} shape={shape}: cut rows in band {flagged}, requests in band {near}, "
             f"agreement with the independent oracle {agree:.3f}")
    assert agree >= 0.9


def test_sampled_step_matches_oracle():
    cfg = get_config("vicuna7b").replace(batch=3, n_q_heads=4, n_kv_heads=4, hidden=512, vocab=3001,
                                         lengths=("explicit", (6, 300, 1100)))
    announce(f"sampled step case=vicuna_small B={cfg.batch} gamma={cfg.gamma} V={cfg.vocab}")
    x = make_inputs(cfg)
    db = DeviceBatch(x)
    T, k, p = 0.8, 40, 0.9
    mn = torch.empty_like(db.lse)
    sd.sd_verify_step_sampled(db.dims, sd.Sampling(T, k, p), db.q, db.k, db.v, x.kv_off, x.kv_len, db.scale,
                              db.hidden, db.w, db.q_draft, db.draft, db.u, db.attn, db.logits, db.lse, mn,
                              db.accept_len, db.out_tok, db.new_kv_len, db.ws)
    torch.cuda.synchronize()
    logits = to_np(db.logits)
    g_lse, g_min = to_np(db.lse), to_np(mn)
    _check_cut(logits, T, k, p, g_lse, g_min)
    ref = accept_resample_sampled(logits, x.q_draft, x.draft, x.u, T, k, p, x.kv_len,
                                  cut=_gpu_cut(logits, T, g_lse, g_min))
    near = assert_accept_parity(to_np(db.accept_len), to_np(db.out_tok), to_np(db.new_kv_len), ref)
    announce(f"sampled step: requests in band {near}")


@pytest.mark.parametrize("levels,k,p", [(3, 40, 0.9), (12, 40, 0.9), (12, 64, 1.0), (3000, 64, 0.5), (12, 0, 0.9),
                                        (3, 0, 0.5)])
def test_sampled_ties_match_oracle(levels, k, p):
    """Target logits on a few levels, so that the cut falls inside a large
    tie: kept sets above 64 entries (the top-p cut by radix descent),
    candidate sets above 2048 (the top-k cut by radix descent), the small-k
    selection, and top-p with no top-k (the row's mass from the first radix
    level)."""
    B, gamma, V = 4, 3, 32000
    T = 0.9
    G = gamma + 1
    announce(f"sampled ties case levels={levels} k={k} p={p} B={B} gamma={gamma} V={V}")
    logits, q, draft, u = _inputs(B, gamma, V, T, k, p, seed=levels * 131 + k, levels=levels)
    kv_len = np.full(B, 100, dtype=np.int32)
    cfg = get_config("tiny").replace(batch=B, gamma=gamma, vocab=V)
    dims = sd.Dims.of(cfg)
    dev = "cuda"
    lse = torch.empty(B * G, dtype=torch.float32, device=dev)
    mn = torch.empty(B * G, dtype=torch.float32, device=dev)
    acc = torch.empty(B, dtype=torch.int32, device=dev)
    tok = torch.empty((B, G), dtype=torch.int32, device=dev)
    new = torch.empty(B, dtype=torch.int32, device=dev)
    ws = torch.empty(sd.sd_workspace_bytes(dims, 100), dtype=torch.uint8, device=dev)
    sd.sd_accept_resample_sampled(dims, sd.Sampling(T, k, p), torch.from_numpy(logits).to(dev),
                                  torch.from_numpy(q).to(dev), torch.from_numpy(draft).to(dev),
                                  torch.from_numpy(u).to(dev), kv_len, lse, mn, acc, tok, new, ws)
    torch.cuda.synchronize()
    g_lse, g_min = to_np(lse), to_np(mn)
    _check_cut(logits, T, k, p, g_lse, g_min)
    ref = accept_resample_sampled(logits, q, draft, u, T, k, p, kv_len, cut=_gpu_cut(logits, T, g_lse, g_min))
    assert_accept_parity(to_np(acc), to_np(tok), to_np(new), ref)
    kept = [int(np.sum(logits[r] >= g_min[r])) for r in range(B * G)]
    announce(f"ties levels={levels} k={k} p={p}: kept set sizes {min(kept)}..{max(kept)}")


def test_sampled_accept_is_deterministic():
    B, gamma, V = 8, 4, 32000
    T, k, p = 0.9, 0, 0.9
    logits, q, draft, u = _inputs(B, gamma, V, T, k, p, seed=99)
    cfg = get_config("tiny").replace(batch=B, gamma=gamma, vocab=V)
    dims = sd.Dims.of(cfg)
    dev = "cuda"
    args = [torch.from_numpy(a).to(dev) for a in (logits, q, draft, u)]
    outs = []
    for _ in range(2):
        lse = torch.empty(B * (gamma + 1), dtype=torch.float32, device=dev)
        mn = torch.empty_like(lse)
        acc = torch.empty(B, dtype=torch.int32, device=dev)
        tok = torch.empty((B, gamma + 1), dtype=torch.int32, device=dev)
        ws = torch.empty(sd.sd_workspace_bytes(dims, 100), dtype=torch.uint8, device=dev)
        sd.sd_accept_resample_sampled(dims, sd.Sampling(T, k, p), *args, None, lse, mn, acc, tok, None, ws)
        torch.cuda.synchronize()
        outs.append([to_np(t) for t in (lse, mn, acc, tok)])
    for a, b in zip(*outs):
        assert np.array_equal(a, b)
