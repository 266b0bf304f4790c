"""One pooled verification step: attention, vocabulary projection, acceptance.

Source: the target side of Algorithm 1 (one-for-many serving loop) verifies a
received proposal with the target model; Algorithm 2 (verification of one
path) defines what that verification returns.  The step here verifies B
pooled requests at once, each isolated to its own KV segment (the per-tag
isolation of Algorithm 1's design properties).

``hidden`` is caller-supplied by default; ``hidden=None`` projects the
attention output itself, viewed as [B*G][Hq*D] (a decoder-like dataflow).
"""

from __future__ import annotations

import numpy as np

from .attention import verify_attention
from .logits import verify_logits
from .accept import accept_resample


def verify_step(q, k_pool, v_pool, kv_off, kv_len, n_kv_heads, hidden, w_vocab,
                q_draft, draft, u, scale=None):
    B, G, Hq, D = np.asarray(q).shape
    attn = verify_attention(q, k_pool, v_pool, kv_off, kv_len, n_kv_heads, scale)
    h = attn.reshape(B * G, Hq * D) if hidden is None else hidden
    logits, lse = verify_logits(h, w_vocab)
    acc = accept_resample(logits, lse, q_draft, draft, u, kv_len=kv_len)
    return {"attn": attn, "logits": logits, "lse": lse, **acc}
