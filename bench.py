#!/usr/bin/env python3
"""Throughput of the batched speculative-verification step on one MI355X.

A step is one pass of the whole hot path over one pooled batch: causal
multi-query attention over every request's KV cache, the vocabulary
projection with its softmax statistics, and the acceptance test with residual
resampling (sd_verify_step).  The default workload is the largest one that
is one GPU's share at real shape, the Llama-70B-shaped long-context verify:
B = 16 requests, gamma = 8 drafts, 64 query / 8 KV heads of 128, hidden
8192, vocabulary 128256, kv_len ~ U[16384, 32768], bf16, drafts independent
of the target (frequent early rejection).

Inputs are synthetic and seeded (no weights or prompts exist here).  They are
resident in HBM before timing starts, and the timed steps rotate over several
identical copies placed at different addresses, so that each step streams its
KV cache and vocabulary weights from HBM rather than from the 256 MB Infinity
Cache.

Prints one JSON line.  `value` is verified (emitted) tokens per second: each
request emits its accepted drafts plus one corrected or bonus token.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16
INFINITY_CACHE_BYTES = 256 << 20
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


CSRC = os.path.join(ROOT, "paper_2601_21622_amd", "csrc")


def source_files(name: str):
    """The kernel source and every local header it includes (recursively,
    each once, in include order)."""
    seen = []

    def add(fname):
        if fname in seen:
            return
        seen.append(fname)
        with open(os.path.join(CSRC, fname), errors="replace") as f:
            for line in f:
                line = line.strip()
                if line.startswith('#include "') and line.endswith('"'):
                    inc = line[len('#include "'):-1]
                    if os.path.exists(os.path.join(CSRC, inc)):
                        add(inc)

    add(name)
    return seen


def source_digest(name: str) -> str:
    """SHA-256 over source_files(name), names and contents."""
    h = hashlib.sha256()
    for fname in source_files(name):
        with open(os.path.join(CSRC, fname), "rb") as f:
            h.update(fname.encode() + b"\0" + f.read())
    return h.hexdigest()


def counter_entry(kernel: str, workload: str, source: str):
    """The committed rocprofv3 counter record of a kernel on a workload, or
    None when there is none or the kernel source changed since it was taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            entries = json.load(f)
    except (OSError, ValueError):
        return None
    for e in entries:
        if e.get("kernel") == kernel and e.get("workload") == workload:
            return e if e.get("source_sha256") == source_digest(source) else None
    return None


def counter_traffic(kernel: str, workload: str, source: str):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, calibrated), or None."""
    e = counter_entry(kernel, workload, source)
    return float(e["bytes_per_launch"]) if e is not None else None


def counter_mfma_busy(kernel: str, workload: str, source: str):
    """MFMA busy share of the kernel's SIMD cycles from its SQ counter run
    (SQ_VALU_MFMA_BUSY_CYCLES over 1024 SIMDs x GRBM_GUI_ACTIVE / 8), or None."""
    e = counter_entry(kernel, workload, source)
    return float(e["sq_mfma_busy"]) if e is not None and "sq_mfma_busy" in e else None


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(x, budget_s: float):
    """The oracle (plain float64 numpy) on a bounded sample of the same batch:
    requests in order, each through attention over its own cache, the
    projection of its G rows and its acceptance, until about budget_s seconds
    of CPU work have been spent (at least one request).  BLAS runs with one
    thread per core of this process's affinity mask.  Returns emitted tokens
    per second over the sample, with the time of each stage."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import accept_resample, verify_attention, verify_logits
    from workloads.generate import bf16_bits_to_f32

    c = x.cfg
    G, Hkv, D = c.positions, c.n_kv_heads, c.head_dim
    cores = len(os.sched_getaffinity(0))

    def f32(a):
        return bf16_bits_to_f32(a) if a.dtype == np.uint16 else np.asarray(a, dtype=np.float32)

    w = f32(x.w)          # converted once, outside the timed stages
    stage = {"attention": 0.0, "logits_softmax": 0.0, "accept": 0.0}
    emitted = accepted = n = 0
    with threadpool_limits(limits=cores, user_api="blas"):
        blas = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] + [1])
        for b in range(c.batch):
            L, off = int(x.kv_len[b]), int(x.kv_off[b])
            seg = slice(off, off + Hkv * L * D)
            kb, vb, qb = f32(x.k_pool[seg]), f32(x.v_pool[seg]), f32(x.q[b:b + 1])
            hb = f32(x.hidden[b * G:(b + 1) * G])
            t0 = time.perf_counter()
            verify_attention(qb, kb, vb, np.array([0]), np.array([L]), Hkv)
            t1 = time.perf_counter()
            logits, lse = verify_logits(hb, w)
            t2 = time.perf_counter()
            out = accept_resample(logits, lse, x.q_draft[b:b + 1], x.draft[b:b + 1], x.u[b:b + 1])
            t3 = time.perf_counter()
            stage["attention"] += t1 - t0
            stage["logits_softmax"] += t2 - t1
            stage["accept"] += t3 - t2
            emitted += int(out["accept_len"][0]) + 1
            accepted += int(out["accept_len"][0])
            n += 1
            if sum(stage.values()) >= budget_s:
                break
    total = sum(stage.values())
    return {
        "value": emitted / total,
        "unit": "tokens/s",
        "cores": cores,
        "blas_threads": int(blas),
        "cpu_model": cpu_model(),
        "kind": "oracle",
        "sample": f"requests 0..{n - 1} of the {c.batch}-request {c.name} batch (attention over each request's "
                  f"own cache, its {G} projection rows, its acceptance), {total:.1f} s of CPU work, float64 numpy",
        "requests": n,
        "stage_s": stage,
        "accepted_tokens_per_s": accepted / total,
    }


# The paper's own system-level figures, for context only: they measure the
# whole StarSD system (EAGLE-2 draft + targets) on MT-Bench, not this
# verification step, on other hardware.
PAPER_CONTEXT = {
    "source": "Table 1 (system throughput O_gamma, MT-Bench, EAGLE-2 backend)",
    "hardware": "draft on one RTX 4090; targets 1-3 on RTX 4090, 4-6 on A100 (two servers, LAN)",
    "colocated_eagle_tok_s": 94.3,
    "starsd_n6_tok_s": 288.7,
    "speedup_n6_vs_colocated": 288.7 / 94.3,
    "speedup_n6_vs_n1": 288.7 / 79.9,
    "note": "context, not a target: whole-system throughput of the paper's star deployment",
}


def paged_caches(sd, cfg, x, k_pool, v_pool, P):
    """The workload's caches moved into pools of P-key pages.  Page ids come
    from the library's allocator (sd_kv_pool_*), every request (tag) growing
    one page at a time in turn, as sessions that advance together do."""
    import numpy as np
    import torch

    Hkv, D, B = cfg.n_kv_heads, cfg.head_dim, cfg.batch
    need = [(int(L) + P - 1) // P for L in x.kv_len]
    num_pages = sum(need)
    pool = sd.KVPool(num_pages, P)
    for j in range(max(need)):
        for b in range(B):
            if j < need[b]:
                pool.reserve(b, min(int(x.kv_len[b]), (j + 1) * P))
    table = pool.block_table(list(range(B)), max(need))
    pool.close()
    kp = torch.zeros((num_pages, Hkv, P, D), dtype=k_pool.dtype, device="cuda")
    vp = torch.zeros_like(kp)
    for b in range(B):
        L, off = int(x.kv_len[b]), int(x.kv_off[b])
        segk = k_pool[off:off + Hkv * L * D].view(Hkv, L, D)
        segv = v_pool[off:off + Hkv * L * D].view(Hkv, L, D)
        for j in range(need[b]):
            k0, k1 = j * P, min(L, (j + 1) * P)
            kp[int(table[b, j]), :, :k1 - k0] = segk[:, k0:k1]
            vp[int(table[b, j]), :, :k1 - k0] = segv[:, k0:k1]
    torch.cuda.synchronize()
    log(f"paged caches: {num_pages} pages of {P} keys")
    return kp, vp, torch.from_numpy(np.ascontiguousarray(table)).cuda(), num_pages


def expand_leg(sd, cfg, args) -> dict:
    """Draft-side tree expansion for the workload's B requests: a full K-ary
    tree of depth D grown layer by layer from synthetic draft logits."""
    import numpy as np
    import torch

    k, depth = (int(v) for v in args.expand.split(","))
    B, V = cfg.batch, cfg.vocab
    layers, first, F = [], 0, 1
    f0 = -1
    for _ in range(depth):
        layers.append((f0, first, F))
        f0, first, F = first, first + F * k, F * k
    N = first
    gen = torch.Generator(device="cuda").manual_seed(7)
    logits = [torch.randn((B, L[2], V), device="cuda", generator=gen) * 2.0 for L in layers]
    tok = torch.empty((B, N), dtype=torch.int32, device="cuda")
    par = torch.empty_like(tok)
    q = torch.empty((B, N), dtype=torch.float32, device="cuda")
    specs = [sd.Expand(B, F_, V, k, f0_, first_, N) for (f0_, first_, F_) in layers]

    def grow():
        for e, x in zip(specs, logits):
            sd.sd_expand_layer(e, x, tok, par, q)

    for _ in range(3):
        grow()
    torch.cuda.synchronize()
    n = max(10, min(args.steps, 100))
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s0.record()
    for _ in range(n):
        grow()
    s1.record()
    torch.cuda.synchronize()
    ms = s0.elapsed_time(s1) / n
    nbytes = sum(B * L[2] * V * 4 for L in layers)
    par_h = par.cpu().numpy()
    if not all(np.all(par_h[:, j] < j) for j in range(N)):
        raise RuntimeError("expanded tree has a parent after its child")
    log(f"expansion: {N} nodes per request, {ms * 1e3:.1f} us per tree ({nbytes / (ms * 1e-3) / 1e9:.0f} GB/s)")
    return {"top_k": k, "depth": depth, "nodes": N, "requests": B, "ms_per_tree": ms, "bytes_per_tree": nbytes,
            "hbm_gbps": nbytes / (ms * 1e-3) / 1e9, "launches_per_tree": depth}


def starsd_leg(sd, dims, cfg, copies, ms_step, args) -> dict:
    """Acceptance rates of the step's own target and draft distributions
    (sd_acceptance_rate, timed on its own), then the performance model with
    t_v = the measured step time."""
    import numpy as np
    import torch
    from paper_2601_21622_amd import starsd

    parts = [float(v) for v in args.starsd.split(",")]
    t_s, t_c = parts[0], parts[1]
    rate = parts[2] if len(parts) > 2 else None
    B, gamma, V = cfg.batch, cfg.gamma, cfg.vocab
    betas = [torch.empty((B, gamma), dtype=torch.float64, device="cuda") for _ in copies]
    for t, b in zip(copies, betas):
        sd.sd_acceptance_rate(dims, t["logits"], t["lse"], t["q_draft"], b, t["ws"])
    torch.cuda.synchronize()
    n = max(20, min(args.steps, 200))
    calls = [sd.prepare_acceptance_rate(dims, t["logits"], t["lse"], t["q_draft"], b, t["ws"])
             for t, b in zip(copies, betas)]
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s0.record()
    for i in range(n):
        calls[i % len(calls)]()
    s1.record()
    torch.cuda.synchronize()
    ms = s0.elapsed_time(s1) / n
    beta = betas[0].cpu().numpy()
    if not all(np.array_equal(beta, b.cpu().numpy()) for b in betas):
        raise RuntimeError("input copies disagree on the acceptance rates")
    nbytes = B * gamma * V * 8 + B * (gamma + 1) * 4    # p (logits) and q read once, lse
    gbps = nbytes / (ms * 1e-3) / 1e9
    rep = starsd.star_report(beta.ravel().tolist(), gamma, t_s, t_c, ms_step, standalone_rate=rate)
    log(f"acceptance rate: {ms * 1e3:.1f} us per call, host launches included ({gbps:.0f} GB/s), "
        f"mean beta {rep.beta:.4f}")
    # Back-to-back calls of two launches each: for small shapes the host's
    # launch time, not the kernels, sets this rate.
    return {"rate_kernel": {"ms_per_call": ms, "host_inclusive": True, "bytes_per_call": nbytes, "hbm_gbps": gbps,
                            "hbm_frac": gbps / HBM_PEAK_GBPS},
            "beta_per_position": beta.mean(axis=0).tolist(),
            "time_unit": "ms", "standalone_rate": rate, "model": rep.as_dict()}


def workload_config(args, get_config):
    """The workload of this run and its mode checks: (config, None), or
    (None, message) when the options do not go together."""
    if args.tree_nodes and args.sampling is not None:
        return None, "--tree-nodes and --sampling are separate modes"
    if args.paged and (args.tree_nodes or args.sampling is not None):
        return None, "--paged applies to the plain verification step"
    if args.starsd is not None and (args.tree_nodes or args.sampling is not None):
        return None, "--starsd applies to the plain verification step"
    cfg = get_config(args.workload)
    if args.tree_nodes:
        cfg = cfg.replace(gamma=args.tree_nodes)
    return cfg, None


def parser() -> argparse.ArgumentParser:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--warmup-ms", type=float, default=200.0,
                    help="keep warming up (untimed steps) until the warm-up has run at least this long")
    ap.add_argument("--workload", default="llama70b_share")
    ap.add_argument("--copies", type=int, default=0, help="input copies to rotate over (0: enough to exceed "
                                                           "4x the Infinity Cache)")
    ap.add_argument("--vocab-layout", choices=["packed", "row-major"], default="packed",
                    help="LM-head weight layout: repacked once before timing (sd_pack_vocab), or [V][hidden]")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sampling", default=None, metavar="T,K,P",
                    help="time sd_verify_step_sampled with temperature T, top-k K (0: off), top-p P (1: off) "
                         "instead of the plain step (T = 0: greedy)")
    ap.add_argument("--tree-nodes", type=int, default=0, metavar="N",
                    help="time sd_verify_step_tree on a binary candidate tree of N nodes (two children per node, "
                         "breadth first) instead of the chain; the workload's draft length becomes N")
    ap.add_argument("--paged", type=int, default=0, metavar="P",
                    help="keep the KV caches in a paged pool of P-key pages (sd_verify_step_paged); pages come "
                         "from the library's allocator with the requests growing in turn, so they interleave")
    ap.add_argument("--expand", default=None, metavar="K,D",
                    help="also time the draft-side expansion of a full K-ary tree of depth D for the workload's "
                         "requests and vocabulary (sd_expand_layer, D launches per tree; synthetic draft logits)")
    ap.add_argument("--starsd", default=None, metavar="T_S,T_C[,RATE]",
                    help="also time sd_acceptance_rate on the step's distributions and evaluate the StarSD model "
                         "with the measured t_v: draft time per layer t_s and transfer time t_c in ms, and "
                         "optionally a standalone target rate in tokens/ms (gives N_max)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a device copy of known size (counter calibration)")
    return ap


def main() -> int:
    args = parser().parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the verification step "
              "runs on a single GPU and does not shard across GPUs)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2601_21622_amd as sd
    from workloads import get_config, make_inputs

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    torch.cuda.set_device(0)
    cfg, problem = workload_config(args, get_config)
    if problem is not None:
        print(problem, file=sys.stderr)
        return 2
    B, G, M, V, K = cfg.batch, cfg.positions, cfg.rows, cfg.vocab, cfg.hidden
    log(f"generating workload {cfg.name}")
    x = make_inputs(cfg)
    packed = args.vocab_layout == "packed" and cfg.dtype == "bf16"
    dims = sd.Dims.of(cfg, packed_vocab=packed)
    scale = 1.0 / math.sqrt(cfg.head_dim)

    def dev(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()

    big_bytes = x.k_pool.nbytes + x.v_pool.nbytes + x.w.nbytes
    ncopies = args.copies or max(2, math.ceil(4 * INFINITY_CACHE_BYTES / big_bytes) + 1)
    adt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    ws_bytes = sd.sd_workspace_bytes(dims, int(x.kv_len.max()))
    copies = []
    base = {n: dev(getattr(x, n)) for n in ("q", "k_pool", "v_pool", "hidden", "w", "q_draft", "draft", "u")}
    if packed:
        # Weight-load-time repacking of the LM head (not part of a step).
        wp = torch.empty((sd.sd_vocab_packed_bytes(dims) // 2,), dtype=torch.bfloat16, device="cuda")
        sd.sd_pack_vocab(dims, base["w"], wp)
        torch.cuda.synchronize()
        base["w"] = wp
    pages = None
    if args.paged:
        base["k_pool"], base["v_pool"], table, num_pages = paged_caches(sd, cfg, x, base["k_pool"], base["v_pool"],
                                                                        args.paged)
        pages = sd.KVPages.of(table, args.paged, num_pages)
    for i in range(ncopies):
        t = {n: (a if i == 0 else a.clone()) for n, a in base.items()}
        t["attn"] = torch.empty((B, G, cfg.n_q_heads, cfg.head_dim), dtype=adt, device="cuda")
        t["logits"] = torch.empty((M, V), dtype=torch.float32, device="cuda")
        t["lse"] = torch.empty((M,), dtype=torch.float32, device="cuda")
        t["acc"] = torch.full((B,), -7, dtype=torch.int32, device="cuda")
        t["tok"] = torch.empty((B, G), dtype=torch.int32, device="cuda")
        t["node"] = torch.empty((B, G), dtype=torch.int32, device="cuda")
        t["new"] = torch.empty((B,), dtype=torch.int32, device="cuda")
        t["rmin"] = torch.empty((M,), dtype=torch.float32, device="cuda")
        t["ws"] = torch.empty((ws_bytes,), dtype=torch.uint8, device="cuda")
        copies.append(t)
    log(f"{ncopies} input copies of {big_bytes / 1e6:.0f} MB each")

    # Binary candidate tree: nodes 0 and 1 hang from the root, node i >= 2 from node (i - 2) // 2.
    parent = torch.tensor([[-1 if i < 2 else (i - 2) // 2 for i in range(cfg.gamma)]] * B, dtype=torch.int32,
                          device="cuda")
    sampling = None
    if args.sampling is not None:
        s_t, s_k, s_p = args.sampling.split(",")
        sampling = sd.Sampling(float(s_t), int(s_k), float(s_p))

    def prepared(t, events=None):
        if args.tree_nodes:
            return sd.prepare_verify_step_tree(dims, t["q"], t["k_pool"], t["v_pool"], x.kv_off, x.kv_len, parent,
                                               scale, t["hidden"], t["w"], t["draft"], t["u"], t["attn"],
                                               t["logits"], t["lse"], t["acc"], t["tok"], t["node"], t["new"],
                                               t["ws"], kernel_events=events)
        if sampling is not None:
            return sd.prepare_verify_step_sampled(dims, sampling, t["q"], t["k_pool"], t["v_pool"], x.kv_off,
                                                  x.kv_len, scale, t["hidden"], t["w"], t["q_draft"], t["draft"],
                                                  t["u"], t["attn"], t["logits"], t["lse"], t["rmin"], t["acc"],
                                                  t["tok"], t["new"], t["ws"], kernel_events=events)
        if pages is not None:
            return sd.prepare_verify_step_paged(dims, t["q"], t["k_pool"], t["v_pool"], pages, x.kv_len, scale,
                                                t["hidden"], t["w"], t["q_draft"], t["draft"], t["u"], t["attn"],
                                                t["logits"], t["lse"], t["acc"], t["tok"], t["new"], t["ws"],
                                                kernel_events=events)
        return sd.prepare_verify_step(dims, t["q"], t["k_pool"], t["v_pool"], x.kv_off, x.kv_len, scale, t["hidden"],
                                      t["w"], t["q_draft"], t["draft"], t["u"], t["attn"], t["logits"], t["lse"],
                                      t["acc"], t["tok"], t["new"], t["ws"], kernel_events=events)

    calls = [prepared(t) for t in copies]

    if args.calibrate_copy:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # Warm-up: the requested steps, then more untimed steps until the warm-up
    # has kept the GPU busy for --warmup-ms.  From idle, the first ~10 ms of
    # steps run slower (llama70b_share: 736 us per step over 20 steps after 5
    # warm-up steps, 671 after 20, 647 over 200); the timed steps should see
    # the clocks a busy server runs at.
    nwarm = 0
    w0 = time.perf_counter()
    while nwarm < args.warmup or (time.perf_counter() - w0) * 1e3 < args.warmup_ms:
        calls[nwarm % ncopies]()
        nwarm += 1
        if nwarm >= args.warmup and nwarm % 8 == 0:
            torch.cuda.synchronize()
        if nwarm >= 100000:
            break
    torch.cuda.synchronize()
    warm_ms = (time.perf_counter() - w0) * 1e3
    log(f"warm-up: {nwarm} steps, {warm_ms:.1f} ms")

    # Headline: steps back to back, nothing else on the stream.
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    w0 = time.perf_counter()
    for i in range(args.steps):
        calls[(nwarm + i) % ncopies]()
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms_total = start.elapsed_time(end)
    ms_step = ms_total / args.steps
    log(f"timed {args.steps} steps: {ms_total:.3f} ms on the GPU clock, {wall * 1e3:.3f} ms wall")

    # Per-kernel times: the same steps again, each kernel launch recording its
    # own start/stop events (hipExtLaunchKernelGGL), which adds no stream work.
    nev = min(args.steps, 200)
    kev = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(nev)]
    kcalls = [prepared(copies[i % ncopies], kev[i]) for i in range(nev)]
    torch.cuda.synchronize()
    s2, e2 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s2.record()
    for c in kcalls:
        c()
    e2.record()
    torch.cuda.synchronize()
    ms_step_ev = s2.elapsed_time(e2) / nev
    stage = np.array([[ev[2 * j].elapsed_time(ev[2 * j + 1]) for j in range(3)] for ev in kev])  # ms
    st_mean = stage.mean(axis=0)

    # Attention with its split-KV merge: standalone sd_verify_attention calls
    # (partials kernel, then the merge kernel) back to back.  In the step the
    # merge rides in the acceptance launch, so the attention kernel's
    # own time above leaves it out.
    att_calls = [sd.prepare_verify_attention(dims, t["q"], t["k_pool"], t["v_pool"], x.kv_off, x.kv_len, scale,
                                             t["attn"], t["ws"])
                 for t in copies] if pages is None and not args.tree_nodes else []
    ms_attn_merged = None
    if att_calls:
        for i in range(3):
            att_calls[i % ncopies]()
        torch.cuda.synchronize()
        a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        natt = max(10, min(args.steps, 100))
        a0.record()
        for i in range(natt):
            att_calls[i % ncopies]()
        a1.record()
        torch.cuda.synchronize()
        ms_attn_merged = a0.elapsed_time(a1) / natt

    acc = [t["acc"].cpu().numpy() for t in copies]
    if not all(np.array_equal(acc[0], a) for a in acc):
        raise RuntimeError("input copies disagree on the accept lengths")
    emitted = int((acc[0] + 1).sum())
    accepted = int(acc[0].sum())

    # Roofline of each kernel stage (algorithmic bytes / flops per launch).
    kv_bytes = 2 * int(x.kv_len.astype(np.int64).sum()) * cfg.n_kv_heads * cfg.head_dim * (2 if cfg.dtype == "bf16" else 4)
    esz = 2 if cfg.dtype == "bf16" else 4
    attn_bytes = kv_bytes + 2 * B * G * cfg.n_q_heads * cfg.head_dim * esz
    vocab_bytes = V * K * esz + M * K * esz + M * V * 4  # W and hidden read, fp32 logits written
    vocab_flops = 2.0 * M * K * V
    attn_gbps = attn_bytes / (st_mean[0] * 1e-3) / 1e9
    attn_merged_gbps = attn_bytes / (ms_attn_merged * 1e-3) / 1e9 if ms_attn_merged else None
    vocab_gbps = vocab_bytes / (st_mean[1] * 1e-3) / 1e9
    vocab_tflops = vocab_flops / (st_mean[1] * 1e-3) / 1e12
    # Kernel names as rocprofv3 lists them: the library names the projection
    # kernel its plan picks; attention runs the register-staged kernel for a
    # single 16-row block per KV head.
    vocab_kernel = sd.sd_vocab_kernel_name(dims)
    rows = G * (cfg.n_q_heads // cfg.n_kv_heads)
    attn_kernel = "attn_bf16_reg_kernel" if rows <= 16 else "attn_bf16_kernel"
    roof_attn = {"bound": "hbm", "achieved": attn_gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                 "frac": attn_gbps / HBM_PEAK_GBPS, "traffic": counter_traffic(attn_kernel, cfg.name, "attention.hip"),
                 "kernel": attn_kernel, "bytes_per_launch": attn_bytes, "ms_per_launch": float(st_mean[0])}
    roof_vocab = {"bound": "hbm", "achieved": vocab_gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                  "frac": vocab_gbps / HBM_PEAK_GBPS, "traffic": counter_traffic(vocab_kernel, cfg.name, "vocab.hip"),
                  "kernel": vocab_kernel, "bytes_per_launch": vocab_bytes, "ms_per_launch": float(st_mean[1]),
                  "mfma_frac": vocab_tflops / BF16_MFMA_PEAK_TFLOPS,
                  "mfma_busy_counters": counter_mfma_busy(vocab_kernel, cfg.name, "vocab.hip")}
    dominant = "vocab" if st_mean[1] >= st_mean[0] else "attention"
    roof = roof_vocab if dominant == "vocab" else roof_attn

    result = {
        "metric": "verified tokens/sec per MI355X",
        "value": emitted / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_run": {"steps": nwarm, "ms": warm_ms},
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {
            "workload": cfg.name,
            "batch": B, "gamma": cfg.gamma, "n_q_heads": cfg.n_q_heads, "n_kv_heads": cfg.n_kv_heads,
            "head_dim": cfg.head_dim, "hidden": K, "vocab": V,
            "kv_len": list(cfg.lengths), "kv_tokens": int(x.kv_len.sum()), "draft": list(cfg.draft),
            "input_copies": ncopies, "vocab_layout": "packed" if packed else "row-major",
            **({"sampling": {"temperature": sampling.temperature, "top_k": sampling.top_k, "top_p": sampling.top_p}}
               if sampling is not None else {}),
            **({"tree": {"nodes": args.tree_nodes, "shape": "binary"}} if args.tree_nodes else {}),
            **({"kv_cache": {"layout": "paged", "page_size": args.paged}} if args.paged else {}),
        },
        "roofline": roof,
        "roofline_attention": roof_attn,
        "roofline_vocab": roof_vocab,
        "scored_tokens_per_s": B * G / (ms_step * 1e-3),
        "accepted_tokens_per_s": accepted / (ms_step * 1e-3),
        "emitted_per_step": emitted,
        "kernel_ms": {"attention": float(st_mean[0]), "vocab_projection": float(st_mean[1]),
                      "accept": float(st_mean[2])},
        "ms_per_step_with_kernel_events": ms_step_ev,
        "attention_hbm_gbps": attn_gbps,
        "attention_with_merge_ms": ms_attn_merged,
        "attention_with_merge_hbm_gbps": attn_merged_gbps,
        "vocab_hbm_gbps": vocab_gbps,
        "vocab_mfma_frac": vocab_tflops / BF16_MFMA_PEAK_TFLOPS,
        "vocab_attainable_frac": vocab_tflops / min(BF16_MFMA_PEAK_TFLOPS, vocab_flops / vocab_bytes * HBM_PEAK_GBPS / 1e3),
        "wall_ms_per_step": wall * 1e3 / args.steps,
    }
    if args.starsd is not None:
        result["starsd"] = starsd_leg(sd, dims, cfg, copies, ms_step, args)
    if args.expand is not None:
        result["expand"] = expand_leg(sd, cfg, args)
    if not args.no_cpu_baseline and sampling is None and not args.tree_nodes and not args.paged:
        # the CPU leg times the plain step
        log("timing the CPU oracle on the same batch")
        result["cpu_baseline"] = cpu_baseline(x, args.cpu_seconds)
    result["paper_context"] = PAPER_CONTEXT
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
