"""GPU parity of tree verification against the oracle (oracle.tree).

Attention: sd_verify_attention_tree against the float64 tree-masked oracle
(tolerance rule of the chain path: |gpu - oracle| <= rtol * max(|oracle|, rms
of the row), rtol 2e-2 bf16 / 1e-4 fp32) on random trees of 4 to 63 nodes,
multi-head and grouped-query shapes, bf16 and fp32, ragged cache lengths;
a chain tree must reproduce sd_verify_attention bit for bit.
"""

import zlib

import numpy as np
import pytest
import torch

import paper_2601_21622_amd as sd
from oracle import tree_attention
from workloads import get_config, make_inputs

from gpu_util import RTOL, DeviceBatch, announce, assert_close_rows, tensor, to_np

pytestmark = pytest.mark.gpu


def random_parents(rng, B, N, kind="random"):
    par = np.empty((B, N), dtype=np.int32)
    for b in range(B):
        for i in range(N):
            if kind == "chain":
                par[b, i] = i - 1
            elif kind == "star":
                par[b, i] = -1
            else:
                par[b, i] = rng.integers(-1, i) if i > 0 else -1
    return par


TREE_CASES = {
    "f32_n4": (get_config("tiny").replace(batch=2, gamma=4, lengths=("explicit", (5, 140))), "random"),
    "f32_n63_star": (get_config("tiny").replace(batch=1, gamma=63, n_q_heads=2, n_kv_heads=2, hidden=128,
                                                lengths=("explicit", (300,))), "star"),
    "mha_n6": (get_config("vicuna7b").replace(batch=3, gamma=6, n_q_heads=4, n_kv_heads=4, hidden=512, vocab=256,
                                              lengths=("explicit", (7, 600, 1300))), "random"),
    "gqa4_n7": (get_config("llama3_8b").replace(batch=2, gamma=7, n_q_heads=8, n_kv_heads=2, hidden=1024,
                                                vocab=256, lengths=("explicit", (8, 2000))), "random"),
    "gqa8_n8": (get_config("llama70b_share").replace(batch=2, gamma=8, n_q_heads=16, n_kv_heads=2, hidden=2048,
                                                     vocab=256, lengths=("explicit", (700, 9))), "random"),
    "mha_n63": (get_config("vicuna7b").replace(batch=2, gamma=63, n_q_heads=2, n_kv_heads=2, hidden=256,
                                               vocab=256, lengths=("explicit", (64, 900))), "random"),
}


@pytest.mark.parametrize("name", sorted(TREE_CASES))
def test_tree_attention_matches_oracle(name):
    cfg, kind = TREE_CASES[name]
    announce(f"tree attention case={name} B={cfg.batch} nodes={cfg.gamma} Hq={cfg.n_q_heads} Hkv={cfg.n_kv_heads} "
             f"dtype={cfg.dtype}")
    x = make_inputs(cfg)
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    parent = random_parents(rng, cfg.batch, cfg.gamma, kind)
    db = DeviceBatch(x)
    sd.sd_verify_attention_tree(db.dims, db.q, db.k, db.v, x.kv_off, x.kv_len, tensor(parent), db.scale, db.attn,
                                db.ws)
    got = to_np(db.attn)
    ref = tree_attention(x.f32("q"), x.f32("k_pool"), x.f32("v_pool"), x.kv_off, x.kv_len, cfg.n_kv_heads, parent)
    err = assert_close_rows(got, ref, RTOL[cfg.dtype], f"tree attention[{name}]")
    announce(f"tree attention case={name} max scaled err {err:.3e}")


@pytest.mark.parametrize("name", ["mha_n6", "gqa8_n8", "f32_n4"])
def test_chain_tree_equals_chain_attention(name):
    cfg, _ = TREE_CASES[name]
    x = make_inputs(cfg)
    parent = random_parents(None, cfg.batch, cfg.gamma, "chain")
    db = DeviceBatch(x)
    db.attention()
    chain = to_np(db.attn).copy()
    db.attn.zero_()
    sd.sd_verify_attention_tree(db.dims, db.q, db.k, db.v, x.kv_off, x.kv_len, tensor(parent), db.scale, db.attn,
                                db.ws)
    assert np.array_equal(chain, to_np(db.attn))
