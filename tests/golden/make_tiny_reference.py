"""Writes tiny_reference.json: the oracle's verification of the tiny fp32
workload (seeded), kept as a regression fixture of the oracle itself.

Calls only the oracle and the input generator.  Run from the repository root:
    python tests/golden/make_tiny_reference.py
"""

import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from oracle import near_threshold, verify_step  # noqa: E402
from workloads import get_config, make_inputs  # noqa: E402


def compute():
    x = make_inputs(get_config("tiny"))
    c = x.cfg
    out = verify_step(x.q, x.k_pool, x.v_pool, x.kv_off, x.kv_len, c.n_kv_heads, x.hidden, x.w,
                      x.q_draft, x.draft, x.u)
    return {
        "workload": "tiny",
        "seed": c.seed,
        "accept_len": out["accept_len"].tolist(),
        "out_tok": out["out_tok"].tolist(),
        "new_kv_len": out["new_kv_len"].tolist(),
        "near_threshold": [bool(near_threshold(t)) for t in out["traces"]],
        "lse": [float(v) for v in out["lse"]],
        "logits_first8": [float(v) for v in out["logits"][:, :8].reshape(-1)],
        "attn_first8": [float(v) for v in out["attn"].reshape(-1)[:8]],
        "attn_sum": float(out["attn"].sum()),
    }


if __name__ == "__main__":
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_reference.json")
    with open(path, "w") as f:
        json.dump(compute(), f, indent=1)
        f.write("\n")
    print("wrote", path)
