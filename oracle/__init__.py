"""Plain float64 CPU oracle for batched speculative verification.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call, link
or execute this package: it is used by ``tests/``, by the smoke check of the
build entry point and by the CPU-baseline leg of the benchmark.  It shares no
code with the HIP library (no kernels, headers, helpers, tables or constant
generators) and imports nothing from it.

What it computes (StarSD, "One-for-Many Speculative Decoding"):

* :mod:`oracle.attention` -- causal multi-query attention of the gamma + 1
  verification queries of each request over that request's KV cache: the
  target forward along the path's prefixes, which Algorithm 2 (EAGLE
  speculative decoding, verification loop) says may run in parallel, and the
  batched tree/path scoring of Sec. 2 ("Tree-based proposals").
  Reached exactly by its textbook definition.
* :mod:`oracle.logits` -- vocabulary projection and row log-sum-exp giving the
  target distributions p_1..p_{gamma+1} of Algorithm 2.  Textbook definition.
* :mod:`oracle.accept` -- the stochastic acceptance test, first rejection,
  residual correction norm(max(0, p_{l+1} - q_{l+1})) and the final sample of
  Algorithm 2, with the ratio rule of the Leviathan et al. formulation the
  paper adopts in Sec. 2 and whose acceptance probability is Eq. (1) of
  Sec. 3.2.  Followed step by step.
* :mod:`oracle.warp` -- warped target distributions for sampled verification
  (temperature, top-k, top-p, greedy), with which the same test and
  correction stay lossless with respect to the warped target.  By definition.
* :mod:`oracle.tree` -- tree verification: tree-masked attention (each node
  sees the prefix, the root and its ancestors) and lossless acceptance of a
  candidate tree (candidates as point-mass proposals of the Sec. 2 test, in
  place of the longest-path rule of Algorithm 2, which is not lossless).
  Attention by definition; acceptance step by step.
* :mod:`oracle.step` -- the composition of the three for one pooled batch.
* :mod:`oracle.paged` -- attention of requests whose KV rows live in pages
  of a shared pool (per-tag state, Algorithm 1): the rows gathered key by key
  through the block table, then the chain attention above.  By definition.
* :mod:`oracle.expand` -- the draft side's layer expansion (Algorithm 2,
  ExpandLayer): top-k children per frontier node with their draft
  probabilities.  By definition.
* :mod:`oracle.model` -- the performance model of Sec. 3 and Sec. 4.2: the
  acceptance rate beta (sum of min(p, q)), the expected accept length from
  the distribution of the accept length, and the per-iteration time, idle
  time, N_full and N_max from a discrete-event run of the draft server of
  Algorithm 1.  By definition.

Every function is pinned by ``tests/test_oracle_*.py`` against closed forms,
special cases, library routines of other packages and brute-force enumeration;
see those files for which pin covers which function.
"""

from .attention import verify_attention
from .logits import verify_logits, probabilities
from .accept import accept_request, accept_resample, accept_resample_sampled, near_threshold
from .warp import order_keys, warp_row, warped_from_cut
from .tree import (accept_tree, accept_tree_request, ancestor_masks, tree_attention, tree_commit_kv,
                   tree_near_threshold)
from .step import verify_step
from .paged import gather_request, paged_attention
from .expand import expand_layer, full_tree_layout, top_k_tokens
from .model import (acceptance_rate, acceptance_rate_batch, accept_length_pmf, expected_accept_length, n_full, n_max,
                    per_target_throughput, simulate_star)

__all__ = [
    "expand_layer",
    "full_tree_layout",
    "top_k_tokens",
    "gather_request",
    "paged_attention",
    "acceptance_rate",
    "acceptance_rate_batch",
    "accept_length_pmf",
    "expected_accept_length",
    "n_full",
    "n_max",
    "per_target_throughput",
    "simulate_star",
    "verify_attention",
    "verify_logits",
    "probabilities",
    "accept_request",
    "accept_resample",
    "accept_resample_sampled",
    "near_threshold",
    "order_keys",
    "warp_row",
    "warped_from_cut",
    "accept_tree",
    "accept_tree_request",
    "ancestor_masks",
    "tree_attention",
    "tree_commit_kv",
    "tree_near_threshold",
    "verify_step",
]
