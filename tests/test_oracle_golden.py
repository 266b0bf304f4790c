"""The oracle still reproduces its stored verification of the tiny workload
(tests/golden/tiny_reference.json, written by make_tiny_reference.py from the
oracle alone).  A change here must come with a reason in the commit message."""

import json
import os

import numpy as np

from golden.make_tiny_reference import compute

HERE = os.path.join(os.path.dirname(__file__), "golden")


def test_tiny_reference_unchanged():
    with open(os.path.join(HERE, "tiny_reference.json")) as f:
        ref = json.load(f)
    now = compute()
    for k in ("accept_len", "out_tok", "new_kv_len", "near_threshold", "seed"):
        assert now[k] == ref[k], k
    for k in ("lse", "logits_first8", "attn_first8"):
        assert np.allclose(now[k], ref[k], rtol=1e-12, atol=1e-12), k
    assert abs(now["attn_sum"] - ref["attn_sum"]) < 1e-9
