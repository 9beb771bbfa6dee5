"""Benchmark of the PreLRShared hot path on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input at
the 32k-context, 8B-shaped layer (hidden 4096, 32 q / 8 KV heads, head dim 128,
8 agents, LoRA rank 16 on k and v):
  1. LR-cache precompute of a new 4096-token segment for all 8 agents
     (X[4096x4096] . A_stack[4096x256] -> 16 LR planes);
  2. prefill of that segment: 4096 queries at positions 32768..36863 over the
     shared base cache plus the agent's LR cache (kv_len 36864);
  3. decode of 16 concurrent agent requests, each with its own 32768-token base
     cache, LR cache and up-projections.
Inputs are resident in HBM before the timed region.  Each stage is timed with
HIP events on the stream the kernels run on.

The reported value is decode HBM throughput (algorithmic bytes / decode time);
prefill and precompute throughput (algorithmic flop / time) sit beside it, with
a roofline per stage.  The materialise-then-attend reference (write each
request's full per-agent K/V, then run plain attention) is timed on the same
inputs.  The fp64 oracle is timed on a bounded sample of the same workload on
the host cores (rank 0, N = 1 only).

After the step the same run times the 8k-context 8B-shaped layer and the
64k-context 14B-shaped rank-64 layer (precompute, prefill, decode, each against
materialise-then-attend) and the achievable HBM read rate (the library's
streaming-read kernel over 2 GiB), reported beside the stage rooflines.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline] [--no-workloads]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "LR-shared attention decode HBM GB/s + prefill TFLOP/s at 32k ctx, 1 GPU"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, TFLOP/s


# --------------------------------------------------------------- the workload
def workload_dims(index=3):
    from workload import CONFIGS
    cfg = CONFIGS[index]
    S = cfg.context
    return cfg, dict(
        S=S, seg=cfg.precompute_rows, n_pre=cfg.prefill_tokens, B=cfg.decode_batch,
        hidden=cfg.hidden, n_q=cfg.n_q, n_kv=cfg.n_kv, d=cfg.head_dim, r=cfg.rank, N=cfg.n_agents,
        theta=cfg.theta)


def algorithmic_work(w, lk=True, lv=True):
    """Bytes and flops the method must move/do (each counted once); lk / lv
    say which projections carry an LR part (both for the k-and-v workload,
    only lv for the paper's QV setting)."""
    S, d, n_q, n_kv, r, B = w["S"], w["d"], w["n_q"], w["n_kv"], w["r"], w["B"]
    n_lr = int(lk) + int(lv)
    # Decode: read each request's base K and V and its agent's L_k, L_v rows
    # once, plus Q, B_k, B_v, and write O.
    dec_bytes_req = (S * n_kv * d * 2 * 2 + S * r * 2 * n_lr + n_q * d * 2 + n_lr * n_kv * d * r * 2
                     + n_q * d * 2)
    dec_flops_req = (4 * n_q * d * S                        # Q K^T and P V
                     + int(lk) * 2 * r * d * n_kv * S       # key-side expansion L_k B_k
                     + int(lv) * 2 * n_q * r * S            # P L_v
                     + int(lv) * 2 * n_q * r * d)           # (P L_v) B_v
    # Prefill: 4096 queries at positions S..S+n-1, causal.
    n = w["n_pre"]
    kv = S + n
    vis = sum(S + i + 1 for i in range(n))
    pre_flops = 4 * n_q * d * vis + n_lr * 2 * r * d * n_kv * kv
    pre_bytes = kv * n_kv * d * 2 * 2 + kv * r * 2 * n_lr + 2 * n * n_q * d * 2 + n_lr * n_kv * d * r * 2
    # Precompute: X[seg x hidden] . A[hidden x 2Nr].
    cols = 2 * w["N"] * r
    pc_flops = 2 * w["seg"] * w["hidden"] * cols
    pc_bytes = (w["seg"] * w["hidden"] + cols * w["hidden"] + w["seg"] * cols) * 2
    return dict(decode_bytes=B * dec_bytes_req, decode_flops=B * dec_flops_req, decode_bytes_per_request=dec_bytes_req,
                prefill_flops=pre_flops, prefill_bytes=pre_bytes, precompute_flops=pc_flops,
                precompute_bytes=pc_bytes)


def make_inputs(w, dev, seed=3000):
    """Seeded synthetic inputs, generated directly in HBM."""
    import torch
    g = torch.Generator(device=dev).manual_seed(seed)

    def nrm(shape, std=1.0):
        x = torch.randn(*shape, generator=g, device=dev, dtype=torch.float32)
        if std != 1.0:
            x.mul_(std)
        return x.to(torch.bfloat16)

    S, d, n_q, n_kv, r, B, N = w["S"], w["d"], w["n_q"], w["n_kv"], w["r"], w["B"], w["N"]
    bstd = math.sqrt(0.02)
    kv_pre = S + w["n_pre"]
    x = {}
    # Precompute: 4 rotating segment buffers so every step reads X from HBM.
    x["X"] = [nrm((w["seg"], w["hidden"])) for _ in range(4)]
    x["A_stack"] = nrm((w["hidden"], 2 * N * r), 1.0 / math.sqrt(w["hidden"]))
    x["L_planes"] = torch.zeros((2, N, kv_pre, r), dtype=torch.bfloat16, device=dev)
    # Prefill: one request (agent 0) over the shared trajectory.
    x["pre"] = dict(
        Q=nrm((1, w["n_pre"], n_q, d)), K_base=nrm((1, kv_pre, n_kv, d)), V_base=nrm((1, kv_pre, n_kv, d)),
        L_k=nrm((1, kv_pre, r)), L_v=nrm((1, kv_pre, r)),
        B_k=nrm((1, r, n_kv * d), bstd), B_v=nrm((1, r, n_kv * d), bstd),
        positions=torch.arange(S, kv_pre, dtype=torch.int32, device=dev)[None],
        kv_len=torch.tensor([kv_pre], dtype=torch.int32, device=dev))
    # Decode: 16 requests, each its own base cache, LR plane (agent b mod N)
    # and up-projections.
    x["dec"] = dict(
        Q=nrm((B, 1, n_q, d)), K_base=nrm((B, S, n_kv, d)), V_base=nrm((B, S, n_kv, d)),
        L_k=nrm((B, S, r)), L_v=nrm((B, S, r)),
        B_k=nrm((B, r, n_kv * d), bstd), B_v=nrm((B, r, n_kv * d), bstd),
        positions=torch.full((B, 1), S - 1, dtype=torch.int32, device=dev),
        kv_len=torch.full((B,), S, dtype=torch.int32, device=dev))
    return x


# ------------------------------------------------------------ GPU timing loop
def attn(prc, c, theta, O, ws, tile_cache=True):
    return prc.lr_shared_attention(c["Q"], c["K_base"], c["V_base"], c["L_k"], c["L_v"], c["B_k"],
                                   c["B_v"], c["positions"], c["kv_len"], rope_theta=theta, O=O,
                                   workspace=ws, tile_cache=tile_cache)


def run_fused(prc, x, w, steps, warmup):
    import torch
    theta = w["theta"]
    O_pre = torch.empty_like(x["pre"]["Q"])
    O_dec = torch.empty_like(x["dec"]["Q"])
    dims = prc.make_dims(x["dec"]["Q"], x["dec"]["K_base"], x["dec"]["L_k"], x["dec"]["L_v"], x["dec"]["B_k"],
                         x["dec"]["B_v"], theta)
    ws = torch.empty(max(1, prc.workspace_size(dims)), dtype=torch.uint8, device=O_dec.device)
    # The prefill's workspace (its tile cache), allocated once outside the
    # timed region like the decode's.
    dims_pre = prc.make_dims(x["pre"]["Q"], x["pre"]["K_base"], x["pre"]["L_k"], x["pre"]["L_v"], x["pre"]["B_k"],
                             x["pre"]["B_v"], theta)
    ws_pre = torch.empty(max(1, prc.workspace_size(dims_pre)), dtype=torch.uint8, device=O_dec.device)

    def step(i, ev=None):
        if ev is not None:
            ev[0].record()
        prc.precompute_lr_cache(x["X"][i % 4], x["A_stack"], 2, w["N"], w["r"], x["L_planes"], tok_offset=w["S"])
        if ev is not None:
            ev[1].record()
        attn(prc, x["pre"], theta, O_pre, ws_pre)
        if ev is not None:
            ev[2].record()
        attn(prc, x["dec"], theta, O_dec, ws)
        if ev is not None:
            ev[3].record()

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        step(i, evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = stage_times(evs)
    total = sum(evs[i][0].elapsed_time(evs[i][3]) for i in range(steps))
    return {k: sum(v) / steps for k, v in per.items()}, total / steps, wall / steps * 1e3, per


def stage_times(evs):
    """Per-step times (ms) of the three stages from four events per step."""
    per = {"precompute": [], "prefill": [], "decode": []}
    for e in evs:
        per["precompute"].append(e[0].elapsed_time(e[1]))
        per["prefill"].append(e[1].elapsed_time(e[2]))
        per["decode"].append(e[2].elapsed_time(e[3]))
    return per


def percentiles(v):
    import numpy as np
    p10, p50, p90 = np.percentile(np.asarray(v, dtype=np.float64), [10, 50, 90])
    return {"p10": round(float(p10), 4), "median": round(float(p50), 4), "p90": round(float(p90), 4)}


def torch_copy_rate(dev, gib=1.0, reps=10):
    """HBM rate of torch's device copy (read + write of `gib` GiB each), for
    context beside the 8 TB/s spec peak; torch's own kernels, not a ceiling
    (the decode kernel reads faster than this copy moves data)."""
    import torch
    n = int(gib * (1 << 30)) // 4
    a = torch.empty(n, dtype=torch.float32, device=dev).fill_(1.0)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    for _ in range(reps):
        b.copy_(a)
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / reps
    del a, b
    return round(2 * n * 4 / (ms * 1e-3) / 1e9, 1)


def library_reference(w, dev, prefill_flops, plain_prefill_ms, precompute_ms):
    """Vendor-library reference points, for context only (never the product
    path): hipBLASLt (through torch.matmul) on the precompute's GEMM shape,
    X [seg, hidden] . A_stack [hidden, 2 N r], and torch's flash attention on
    the plain prefill shape (4096 queries over all S + 4096 keys, GQA heads
    expanded, without a causal mask: it does about 6% more work than the
    causal prefill, which its rate below accounts for)."""
    import torch
    import torch.nn.functional as F
    g = torch.Generator(device=dev)
    g.manual_seed(77)

    def timed(fn, reps, warm=3):
        for _ in range(warm):
            fn()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(reps):
            fn()
        ev[1].record()
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / reps

    X = [torch.randn((w["seg"], w["hidden"]), generator=g, device=dev).to(torch.bfloat16) for _ in range(4)]
    A = torch.randn((w["hidden"], 2 * w["N"] * w["r"]), generator=g, device=dev).to(torch.bfloat16)
    C = torch.empty((w["seg"], A.shape[1]), dtype=torch.bfloat16, device=dev)
    it = [0]

    def gemm():
        it[0] += 1
        torch.matmul(X[it[0] % 4], A, out=C)
    t_gemm = timed(gemm, 100)
    del X, A, C
    n_q, n_kv, d, n, S = w["n_q"], w["n_kv"], w["d"], w["n_pre"], w["S"]
    q = torch.randn((1, n_q, n, d), generator=g, device=dev).to(torch.bfloat16)
    k = torch.randn((1, n_q, S + n, d), generator=g, device=dev).to(torch.bfloat16)
    v = torch.randn((1, n_q, S + n, d), generator=g, device=dev).to(torch.bfloat16)
    sdpa_flops = 4.0 * n_q * d * n * (S + n)
    try:
        from torch.nn.attention import SDPBackend, sdpa_kernel
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
            t_sdpa = timed(lambda: F.scaled_dot_product_attention(q, k, v), 5, 2)
        sdpa = {"ms": round(t_sdpa, 4), "tflops": round(sdpa_flops / (t_sdpa * 1e-3) / 1e12, 1),
                "plain_prefill_kernel_speedup": round(t_sdpa / plain_prefill_ms * prefill_flops / sdpa_flops, 3)}
    except Exception as ex:  # a torch build without the flash backend
        sdpa = {"unavailable": repr(ex)[:200]}
    del q, k, v
    torch.cuda.empty_cache()
    return {"precompute_gemm_hipblaslt_ms": round(t_gemm, 4),
            "precompute_kernel_speedup_vs_hipblaslt": round(t_gemm / precompute_ms, 3),
            "plain_prefill_torch_flash_sdpa": sdpa}


def run_materialized(prc, x, w, steps, warmup):
    """Reference point: materialise each request's full K/V, then attend."""
    import torch
    theta = w["theta"]
    p, dcs = x["pre"], x["dec"]
    Kp = torch.empty_like(p["K_base"]); Vp = torch.empty_like(p["V_base"])
    Kd = torch.empty_like(dcs["K_base"]); Vd = torch.empty_like(dcs["V_base"])
    O_pre = torch.empty_like(p["Q"]); O_dec = torch.empty_like(dcs["Q"])
    plain_pre = dict(p, K_base=Kp, V_base=Vp, L_k=None, L_v=None, B_k=None, B_v=None)
    plain_dec = dict(dcs, K_base=Kd, V_base=Vd, L_k=None, L_v=None, B_k=None, B_v=None)
    dims = prc.make_dims(dcs["Q"], Kd, None, None, None, None, theta)
    ws = torch.empty(max(1, prc.workspace_size(dims)), dtype=torch.uint8, device=O_dec.device)

    def step(i, ev=None):
        if ev is not None:
            ev[0].record()
        prc.precompute_lr_cache(x["X"][i % 4], x["A_stack"], 2, w["N"], w["r"], x["L_planes"], tok_offset=w["S"])
        if ev is not None:
            ev[1].record()
        prc.materialize_agent_kv(p["K_base"], p["V_base"], p["L_k"], p["L_v"], p["B_k"], p["B_v"],
                                 p["kv_len"], rope_theta=theta, K_full=Kp, V_full=Vp)
        attn(prc, plain_pre, theta, O_pre, None)
        if ev is not None:
            ev[2].record()
        prc.materialize_agent_kv(dcs["K_base"], dcs["V_base"], dcs["L_k"], dcs["L_v"], dcs["B_k"],
                                 dcs["B_v"], dcs["kv_len"], rope_theta=theta, K_full=Kd, V_full=Vd)
        attn(prc, plain_dec, theta, O_dec, ws)
        if ev is not None:
            ev[3].record()

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for i in range(steps):
        step(i, evs[i])
    torch.cuda.synchronize()
    return {k: sum(v) / steps for k, v in stage_times(evs).items()}


# ------------------------------------------------------------- CPU baseline
def hbm_read_ceiling(prc, dev, gib=2.0, reps=10):
    """Achievable HBM read rate: the library's streaming-read kernel over a
    buffer 8 times the Infinity Cache, best of a few grid sizes (median of
    `reps` timed runs each)."""
    import torch
    n = int(gib * (1 << 30))
    buf = torch.empty(n, dtype=torch.uint8, device=dev)
    buf.fill_(1)
    best = (0.0, 0)
    for grid in (512, 1024, 2048, 4096):
        sink = torch.empty(grid, dtype=torch.int32, device=dev)
        prc.stream_read(buf, sink, grid)
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            prc.stream_read(buf, sink, grid)
            e1.record()
            ts.append((e0, e1))
        torch.cuda.synchronize()
        ms = sorted(a.elapsed_time(b) for a, b in ts)[reps // 2]
        gbs = n / (ms * 1e-3) / 1e9
        if gbs > best[0]:
            best = (gbs, grid)
    del buf
    torch.cuda.empty_cache()
    return {"gbs": round(best[0], 1), "grid": best[1], "bytes": n, "kernel": "stream_read_kernel"}


def cpu_baseline(w, budget_s=20.0):
    """Time the fp64 oracle on a bounded sample of the same workload.

    Sample: decode of whole requests (all 32 q heads, full 32768-token context)
    until about half the budget is spent, then prefill of query tokens (all
    heads, over their full causal range) for the rest.  Reported in the
    metric's unit (GB/s of the decode's algorithmic bytes), with the prefill
    rate in TFLOP/s beside it.
    """
    import numpy as np
    import oracle
    from workload import attention_case
    cfg, _ = workload_dims()
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = 1
    f64 = lambda t: None if t is None else t.double().numpy()
    S, work = w["S"], algorithmic_work(w)
    dec_t, dec_n = 0.0, 0
    while dec_t < budget_s / 2 and dec_n < w["B"]:
        c = attention_case(cfg, batch=1, n_tok=1, kv_len=[S], positions=[[S - 1]], s_cap=S,
                           seed_base=50_000 + dec_n, poison_tail=False)
        t0 = time.perf_counter()
        oracle.lr_shared_attention(f64(c["Q"]), f64(c["K_base"]), f64(c["V_base"]), f64(c["L_k"]),
                                   f64(c["L_v"]), f64(c["B_k"]), f64(c["B_v"]), c["positions"].numpy(),
                                   c["kv_len"].numpy(), cfg.theta)
        dec_t += time.perf_counter() - t0
        dec_n += 1
    # Prefill sample: n_s query tokens at the end of the segment.
    n_s = 384
    kv = S + w["n_pre"]
    pos = list(range(kv - n_s, kv))
    c = attention_case(cfg, batch=1, n_tok=n_s, kv_len=[kv], positions=[pos], s_cap=kv, seed_base=60_000,
                       poison_tail=False)
    t0 = time.perf_counter()
    oracle.lr_shared_attention(f64(c["Q"]), f64(c["K_base"]), f64(c["V_base"]), f64(c["L_k"]), f64(c["L_v"]),
                               f64(c["B_k"]), f64(c["B_v"]), c["positions"].numpy(), c["kv_len"].numpy(),
                               cfg.theta)
    pre_t = time.perf_counter() - t0
    pre_flops = 4 * w["n_q"] * w["d"] * sum(p + 1 for p in pos)
    return {
        "value": round(dec_n * work["decode_bytes_per_request"] / dec_t / 1e9, 4),
        "unit": "GB/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": (f"decode of {dec_n} of {w['B']} requests (32 q heads, {S}-token context) in {dec_t:.1f} s; "
                   f"prefill of the last {n_s} of {w['n_pre']} queries (over {kv} keys) in {pre_t:.1f} s"),
        "prefill_tflops": round(pre_flops / pre_t / 1e12, 6),
        "host_cpus": os.cpu_count(),
    }


def pmc_pass(prc, x, w, dev):
    """One calibration copy of exactly 2^30 bytes (read 1 GiB, write 1 GiB; it
    fills the 256 MB Infinity Cache several times over), then one launch of
    each hot-path kernel, each followed by a synchronisation."""
    import torch
    src = torch.ones(2 ** 29, dtype=torch.bfloat16, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    theta = w["theta"]
    O_pre = torch.empty_like(x["pre"]["Q"])
    O_dec = torch.empty_like(x["dec"]["Q"])
    prc.precompute_lr_cache(x["X"][0], x["A_stack"], 2, w["N"], w["r"], x["L_planes"], tok_offset=w["S"])
    torch.cuda.synchronize()
    attn(prc, x["pre"], theta, O_pre, None)
    torch.cuda.synchronize()
    attn(prc, x["dec"], theta, O_dec, None)
    torch.cuda.synchronize()
    print("pmc pass done", file=sys.stderr, flush=True)


def source_digest(*names):
    """Digest of the kernel sources' code: comments and white space are
    dropped, so a comment edit does not orphan the counters taken on it."""
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2609_34054_amd", "csrc", n), encoding="utf-8") as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        src = re.sub(r"//[^\n]*", "", src)
        h.update(re.sub(r"\s+", "", src).encode())
    return h.hexdigest()[:16]


def traffic_for(kernel_file, launches_per_stage=1):
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(kernel_file)
    except Exception:
        return None
    if not rec or rec.get("source_digest") != source_digest(kernel_file, "common.hpp", "rebuild.hpp"):
        return None
    return rec.get("hbm_bytes_per_launch")


def rank_sweep(prc, w, dev, steps, warmup):
    """Throughput of the fused prefill and decode over LoRA ranks 8..64, with
    LR on k and v (the workload's setting) and on v only (the paper's QV
    setting), plus plain attention over the base cache; one JSON line each.
    Same shapes as the main workload; only the rank and the adapted
    projections change."""
    import torch
    g = torch.Generator(device=dev).manual_seed(4000)

    def nrm(shape, std=1.0):
        x = torch.randn(*shape, generator=g, device=dev, dtype=torch.float32)
        if std != 1.0:
            x.mul_(std)
        return x.to(torch.bfloat16)

    S, d, n_q, n_kv, B = w["S"], w["d"], w["n_q"], w["n_kv"], w["B"]
    kv_pre = S + w["n_pre"]
    base = dict(
        pre=dict(Q=nrm((1, w["n_pre"], n_q, d)), K_base=nrm((1, kv_pre, n_kv, d)), V_base=nrm((1, kv_pre, n_kv, d)),
                 positions=torch.arange(S, kv_pre, dtype=torch.int32, device=dev)[None],
                 kv_len=torch.tensor([kv_pre], dtype=torch.int32, device=dev)),
        dec=dict(Q=nrm((B, 1, n_q, d)), K_base=nrm((B, S, n_kv, d)), V_base=nrm((B, S, n_kv, d)),
                 positions=torch.full((B, 1), S - 1, dtype=torch.int32, device=dev),
                 kv_len=torch.full((B,), S, dtype=torch.int32, device=dev)))

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    runs = [("plain", 16, False, False)] + [(m, r, m == "kv", True) for m in ("qv", "kv") for r in (8, 16, 32, 64)]
    bstd = math.sqrt(0.02)
    recs = []
    for mode, r, lk, lv in runs:
        cases = {}
        for st, nb, ntok in (("pre", 1, kv_pre), ("dec", B, S)):
            c = dict(base[st])
            c["L_k"] = nrm((nb, ntok, r)) if lk else None
            c["L_v"] = nrm((nb, ntok, r)) if lv else None
            c["B_k"] = nrm((nb, r, n_kv * d), bstd) if lk else None
            c["B_v"] = nrm((nb, r, n_kv * d), bstd) if lv else None
            cases[st] = c
        O_pre = torch.empty_like(cases["pre"]["Q"])
        O_dec = torch.empty_like(cases["dec"]["Q"])
        cd = cases["dec"]
        dims = prc.make_dims(cd["Q"], cd["K_base"], cd["L_k"], cd["L_v"], cd["B_k"], cd["B_v"], w["theta"])
        ws = torch.empty(max(1, prc.workspace_size(dims)), dtype=torch.uint8, device=dev)
        cp = cases["pre"]
        dims_p = prc.make_dims(cp["Q"], cp["K_base"], cp["L_k"], cp["L_v"], cp["B_k"], cp["B_v"], w["theta"])
        ws_p = torch.empty(max(1, prc.workspace_size(dims_p)), dtype=torch.uint8, device=dev)
        t_pre = timed(lambda: attn(prc, cases["pre"], w["theta"], O_pre, ws_p))
        t_dec = timed(lambda: attn(prc, cases["dec"], w["theta"], O_dec, ws))
        work = algorithmic_work(dict(w, r=r), lk, lv)
        pre_tf = work["prefill_flops"] / (t_pre * 1e-3) / 1e12
        dec_gbs = work["decode_bytes"] / (t_dec * 1e-3) / 1e9
        recs.append({"sweep": "rank", "mode": mode, "rank": r if (lk or lv) else 0,
                          "prefill_ms": round(t_pre, 4), "prefill_tflops": round(pre_tf, 2),
                          "prefill_mfma_frac": round(pre_tf / MFMA_BF16_PEAK_TFLOPS, 4),
                          "decode_ms": round(t_dec, 4), "decode_gbs": round(dec_gbs, 1),
                          "decode_hbm_frac": round(dec_gbs / HBM_PEAK_GBS, 4),
                          "decode_bytes": work["decode_bytes"], "prefill_flops": work["prefill_flops"]})
        del cases, O_pre, O_dec, ws
    return recs


def shared_base_decode(prc, w, dev, steps, warmup):
    """Decode of all N agents at the end of one shared 32k-token trajectory:
    one base cache, each agent its own LR plane, up-projections and query.
    The shared-base kernel reads every base tile once for all agents; the
    reference is the per-request kernel over per-agent copies of the base
    (what decoding the agents as independent requests costs).  One JSON line."""
    import torch
    g = torch.Generator(device=dev).manual_seed(5000)

    def nrm(shape, std=1.0):
        x = torch.randn(*shape, generator=g, device=dev, dtype=torch.float32)
        if std != 1.0:
            x.mul_(std)
        return x.to(torch.bfloat16)

    S, d, n_q, n_kv, r, N = w["S"], w["d"], w["n_q"], w["n_kv"], w["r"], w["N"]
    bstd = math.sqrt(0.02)
    c = dict(Q=nrm((N, 1, n_q, d)), K_base=nrm((1, S, n_kv, d)), V_base=nrm((1, S, n_kv, d)),
             L_k=nrm((N, S, r)), L_v=nrm((N, S, r)), B_k=nrm((N, r, n_kv * d), bstd),
             B_v=nrm((N, r, n_kv * d), bstd),
             positions=torch.full((N, 1), S - 1, dtype=torch.int32, device=dev),
             kv_len=torch.full((N,), S, dtype=torch.int32, device=dev))
    O = torch.empty_like(c["Q"])

    def timed(case):
        dims = prc.make_dims(case["Q"], case["K_base"], case["L_k"], case["L_v"], case["B_k"],
                             case["B_v"], w["theta"])
        ws = torch.empty(max(1, prc.workspace_size(dims)), dtype=torch.uint8, device=dev)
        for _ in range(warmup):
            attn(prc, case, w["theta"], O, ws)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            attn(prc, case, w["theta"], O, ws)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps, O.clone()

    t_shared, O_shared = timed(c)
    rep = dict(c, K_base=c["K_base"].expand(N, -1, -1, -1).contiguous(),
               V_base=c["V_base"].expand(N, -1, -1, -1).contiguous())
    t_rep, O_rep = timed(rep)
    diff = (O_shared.float() - O_rep.float()).abs().max().item()
    del rep, c
    base_bytes = S * n_kv * d * 2 * 2
    lr_bytes = N * (S * r * 2 * 2 + 2 * n_kv * d * r * 2 + 2 * n_q * d * 2)
    algo = base_bytes + lr_bytes
    gbs = algo / (t_shared * 1e-3) / 1e9
    return {
        "bench": "shared_base_decode", "agents": N, "context": S, "rank": r,
        "workload": (f"decode of {N} agents at position {S - 1} over one shared {S}-token base cache "
                     f"({n_q} q / {n_kv} KV heads, d {d}), each with its own rank-{r} k and v LR plane"),
        "ms": round(t_shared, 4), "algorithmic_bytes": algo, "gbs": round(gbs, 1),
        "hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
        "per_request_copies_ms": round(t_rep, 4), "speedup_vs_per_request_copies": round(t_rep / t_shared, 3),
        "max_abs_diff_vs_per_request": diff}


def fused_projection(prc, w, dev, steps, warmup):
    """The base projection of a 4096-token segment (K_base with RoPE, V_base)
    and every agent's LR rows in one GEMM over X, against the base projection
    and the LR precompute as two calls.  One JSON line."""
    import torch
    g = torch.Generator(device=dev).manual_seed(6000)

    def nrm(shape, std=1.0):
        x = torch.randn(*shape, generator=g, device=dev, dtype=torch.float32)
        if std != 1.0:
            x.mul_(std)
        return x.to(torch.bfloat16)

    S, T, hid, n_kv, d, r, N = w["S"], w["seg"], w["hidden"], w["n_kv"], w["d"], w["r"], w["N"]
    s_cap = S + T
    X = nrm((T, hid))
    W = nrm((hid, 2 * n_kv * d), 1.0 / math.sqrt(hid))
    A_stack = nrm((hid, 2 * N * r), 1.0 / math.sqrt(hid))
    K = torch.empty((s_cap, n_kv, d), dtype=torch.bfloat16, device=dev)
    V = torch.empty_like(K)
    L = torch.empty((2, N, s_cap, r), dtype=torch.bfloat16, device=dev)

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    th = w["theta"]
    t_fused = timed(lambda: prc.project_kv_and_lr_cache(X, W, A_stack, n_kv, d, 2, N, r, K, V, L,
                                                        rope_theta=th, tok_offset=S))
    t_base = timed(lambda: prc.project_kv_and_lr_cache(X, W, None, n_kv, d, 2, 0, r, K, V, None,
                                                       rope_theta=th, tok_offset=S))
    t_pre = timed(lambda: prc.precompute_lr_cache(X, A_stack, 2, N, r, L, tok_offset=S))
    cols = 2 * n_kv * d + 2 * N * r
    flops = 2 * T * hid * cols
    byts = (T * hid + cols * hid + T * cols) * 2
    tf = flops / (t_fused * 1e-3) / 1e12
    return {
        "bench": "fused_projection",
        "workload": (f"{T}-token segment, hidden {hid}: K_base (RoPE) and V_base for {n_kv} KV heads x {d} plus "
                     f"rank-{r} k and v LR rows of {N} agents, one GEMM of {cols} columns"),
        "ms": round(t_fused, 4), "tflops": round(tf, 1), "mfma_frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4),
        "algorithmic_flops": flops, "algorithmic_bytes": byts,
        "base_projection_alone_ms": round(t_base, 4), "precompute_alone_ms": round(t_pre, 4),
        "separate_ms": round(t_base + t_pre, 4),
        "lr_cost_in_fused_ms": round(t_fused - t_base, 4)}


def paged(prc, w, dev, steps, warmup):
    """The step's decode, prefill and segment projection over paged caches
    (pools of fixed-size blocks in a random order, reached through block
    tables), against the same calls over contiguous caches.  One JSON line
    per stage and block size."""
    import torch
    x = make_inputs(w, dev)
    theta = w["theta"]
    g = torch.Generator(device="cpu").manual_seed(7000)

    def table(n_req, mb):
        ids = torch.randperm(n_req * mb, generator=g)
        return ids.reshape(n_req, mb).to(torch.int32).to(dev)

    def to_pool(cache, tbl, blk):
        B, S = cache.shape[:2]
        pool = torch.empty((B * S // blk, blk) + tuple(cache.shape[2:]), dtype=cache.dtype, device=dev)
        pool[tbl.reshape(-1).long()] = cache.reshape((B * S // blk, blk) + tuple(cache.shape[2:]))
        return pool

    def timeit(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    work = algorithmic_work(w)
    recs = []
    for stage in ("decode", "prefill"):
        c = x["dec" if stage == "decode" else "pre"]
        O = torch.empty_like(c["Q"])
        O2 = torch.empty_like(c["Q"])
        dims = prc.make_dims(c["Q"], c["K_base"], c["L_k"], c["L_v"], c["B_k"], c["B_v"], theta)
        ws = torch.empty(max(1, prc.workspace_size(dims)), dtype=torch.uint8, device=dev)
        # Paged calls take no tile cache: the contiguous reference runs without
        # it too (same tile order, so the results must be bitwise equal), and
        # with it for the record.
        t_c = timeit(lambda: attn(prc, c, theta, O, ws, tile_cache=False))
        t_ctc = timeit(lambda: attn(prc, c, theta, O2, ws))
        attn(prc, c, theta, O, ws, tile_cache=False)
        S = c["K_base"].shape[1]
        for blk in (64, 256):
            if S % blk:
                continue
            B, mb = c["K_base"].shape[0], S // blk
            tk, tl = table(B, mb), table(B, mb)
            Kp, Vp = to_pool(c["K_base"], tk, blk), to_pool(c["V_base"], tk, blk)
            Lkp, Lvp = to_pool(c["L_k"], tl, blk), to_pool(c["L_v"], tl, blk)

            def run():
                prc.lr_shared_attention_paged(c["Q"], Kp, Vp, Lkp, Lvp, c["B_k"], c["B_v"],
                                              c["positions"], c["kv_len"], tk, lr_block_table=tl,
                                              rope_theta=theta, O=O2, workspace=ws)
            t_p = timeit(run)
            rec = {"bench": "paged", "stage": stage, "block_size": blk, "requests": B, "context": S,
                   "ms_paged": round(t_p, 4), "ms_contiguous": round(t_c, 4),
                   "paged_over_contiguous": round(t_p / t_c, 4), "bitwise_equal": bool(torch.equal(O, O2)),
                   "ms_contiguous_tile_cache": round(t_ctc, 4)}
            if stage == "decode":
                rec["hbm_frac_paged"] = round(work["decode_bytes"] / (t_p * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
            else:
                rec["mfma_frac_paged"] = round(work["prefill_flops"] / (t_p * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)
            recs.append(rec)
            del Kp, Vp, Lkp, Lvp

    # Segment projection (base K/V + all agents' LR rows) into paged pools.
    T, hid, n_kv, d, r, N, S = w["seg"], w["hidden"], w["n_kv"], w["d"], w["r"], w["N"], w["S"]
    X = x["X"][0]
    W = (torch.randn((hid, 2 * n_kv * d), generator=torch.Generator(device=dev).manual_seed(7001),
                     device=dev) / math.sqrt(hid)).to(torch.bfloat16)
    s_cap = S + T
    K = torch.empty((s_cap, n_kv, d), dtype=torch.bfloat16, device=dev)
    V = torch.empty_like(K)
    L = torch.empty((2, N, s_cap, r), dtype=torch.bfloat16, device=dev)
    t_c = timeit(lambda: prc.project_kv_and_lr_cache(X, W, x["A_stack"], n_kv, d, 2, N, r, K, V, L,
                                                     rope_theta=theta, tok_offset=S))
    for blk in (64, 256):
        mb = s_cap // blk
        tbl = table(1, mb)[0]
        Kp = torch.empty((mb, blk, n_kv, d), dtype=torch.bfloat16, device=dev)
        Vp = torch.empty_like(Kp)
        Lp = torch.empty((2, N, mb, blk, r), dtype=torch.bfloat16, device=dev)
        t_p = timeit(lambda: prc.project_kv_and_lr_cache_paged(X, W, x["A_stack"], n_kv, d, 2, N, r, Kp, Vp,
                                                               Lp, tbl, rope_theta=theta, tok_offset=S))
        rows = torch.arange(S, s_cap, device=dev)
        same = torch.equal(Kp[tbl[rows // blk].long(), rows % blk], K[S:])
        recs.append({"bench": "paged", "stage": "projection", "block_size": blk, "tokens": T,
                     "ms_paged": round(t_p, 4), "ms_contiguous": round(t_c, 4),
                     "paged_over_contiguous": round(t_p / t_c, 4), "bitwise_equal": bool(same)})
        del Kp, Vp, Lp
    del x
    return recs


def stack_bench(prc, dev):
    """The 32-layer stack over 16 turns (8B-shaped layers, 8 agents, rank 16
    on k and v): turn k (k = 1..16, T = 4096 k, agent k mod 8) precomputes
    every layer's LR rows of the newest 4096-token segment [T - 4096, T),
    prefills 256 tokens at [T, T + 256) (a 256-row precompute, then
    attention), computes the LR rows of the turn's 128 decode tokens in one
    128-row precompute per layer (their synthetic hidden states are known in
    advance, as the reference below also uses), and runs 128 decode steps
    attending over [0, pos].  Each layer has its own base cache, LR planes, A
    and B; the base rows are synthetic.  The cost of appending a decode
    token's LR rows step by step instead (a 1-row precompute per layer and
    step) is timed separately and reported beside the run.

    The 128 x 32 decode steps of a turn are launch-bound at short contexts, so
    each turn's decode loop is captured once into a HIP graph (before the
    timed region) and replayed; precompute and prefill launch directly.  The
    reference materialises each layer's agent K/V once per turn (after
    computing that turn's LR rows in one pass), then runs the same schedule
    with plain attention.  One JSON line."""
    import torch
    cfg, w = workload_dims(5)
    ex = cfg.extra
    n_layers, turns, turn, n_pre, n_dec = cfg.layers, ex["turns"], ex["turn_tokens"], cfg.prefill_tokens, \
        ex["decode_steps"]
    hid, n_q, n_kv, d, r, N, theta = w["hidden"], w["n_q"], w["n_kv"], w["d"], w["r"], w["N"], w["theta"]
    S_cap = turns * turn + n_pre + n_dec
    g = torch.Generator(device=dev).manual_seed(5005)

    def nrm(shape, std=1.0):
        x = torch.randn(*shape, generator=g, device=dev, dtype=torch.float32)
        if std != 1.0:
            x.mul_(std)
        return x.to(torch.bfloat16)

    print(f"bench: stack: {n_layers} layers x {S_cap} tokens of base cache", file=sys.stderr, flush=True)
    bstd = math.sqrt(0.02)
    K = [nrm((1, S_cap, n_kv, d)) for _ in range(n_layers)]
    V = [nrm((1, S_cap, n_kv, d)) for _ in range(n_layers)]
    Lp = [torch.zeros((2, N, S_cap, r), dtype=torch.bfloat16, device=dev) for _ in range(n_layers)]
    A = [nrm((hid, 2 * N * r), 1.0 / math.sqrt(hid)) for _ in range(n_layers)]
    Bk = [nrm((N, r, n_kv * d), bstd) for _ in range(n_layers)]
    Bv = [nrm((N, r, n_kv * d), bstd) for _ in range(n_layers)]
    X_seg = [nrm((turn, hid)) for _ in range(4)]
    X_pre = [nrm((n_pre, hid)) for _ in range(2)]
    X_dec = nrm((n_dec, hid))
    Q_pre = nrm((1, n_pre, n_q, d))
    Q_dec = nrm((n_dec, 1, n_q, d))
    O_pre = torch.empty_like(Q_pre)
    O_dec = torch.empty((1, 1, n_q, d), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(64 << 20, dtype=torch.uint8, device=dev)
    Kf = [torch.empty_like(K[0]) for _ in range(n_layers)]
    Vf = [torch.empty_like(V[0]) for _ in range(n_layers)]

    def i32(v):
        return torch.tensor(v, dtype=torch.int32, device=dev)

    T_of = {k: turn * k for k in range(1, turns + 1)}
    cap = {k: T_of[k] + n_pre + n_dec for k in T_of}
    pos_pre = {k: i32([list(range(T_of[k], T_of[k] + n_pre))]) for k in T_of}
    kvl_pre = {k: i32([T_of[k] + n_pre]) for k in T_of}
    pos_dec = {k: i32([[T_of[k] + n_pre + j] for j in range(n_dec)]) for k in T_of}
    kvl_dec = {k: i32([T_of[k] + n_pre + j + 1 for j in range(n_dec)]) for k in T_of}
    kvl_cap = {k: i32([cap[k]]) for k in T_of}

    def views(k, l, fused):
        s, a = cap[k], k % N
        if fused:
            return (K[l][:, :s], V[l][:, :s], Lp[l][0, a, :s][None], Lp[l][1, a, :s][None], Bk[l][a:a + 1],
                    Bv[l][a:a + 1])
        return Kf[l][:, :s], Vf[l][:, :s], None, None, None, None

    def segment(k):
        for l in range(n_layers):
            prc.precompute_lr_cache(X_seg[(l + k) % 4], A[l], 2, N, r, Lp[l], tok_offset=T_of[k] - turn)

    def prefill(k, fused):
        for l in range(n_layers):
            if fused:
                prc.precompute_lr_cache(X_pre[(l + k) % 2], A[l], 2, N, r, Lp[l], tok_offset=T_of[k])
            Kv, Vv, Lk, Lv, B_k, B_v = views(k, l, fused)
            prc.lr_shared_attention(Q_pre, Kv, Vv, Lk, Lv, B_k, B_v, pos_pre[k], kvl_pre[k], rope_theta=theta,
                                    O=O_pre, workspace=ws)

    def decode_rows(k):
        # The LR rows of every agent for the turn's decode tokens, one pass.
        for l in range(n_layers):
            prc.precompute_lr_cache(X_dec, A[l], 2, N, r, Lp[l], tok_offset=T_of[k] + n_pre)

    def decode(k, fused):
        for j in range(n_dec):
            for l in range(n_layers):
                Kv, Vv, Lk, Lv, B_k, B_v = views(k, l, fused)
                prc.lr_shared_attention(Q_dec[j:j + 1], Kv, Vv, Lk, Lv, B_k, B_v, pos_dec[k][j:j + 1],
                                        kvl_dec[k][j:j + 1], rope_theta=theta, O=O_dec, workspace=ws)

    def materialise(k):
        # The reference computes the turn's LR rows in one pass, then writes
        # each layer's agent K/V over [0, cap).
        for l in range(n_layers):
            prc.precompute_lr_cache(X_pre[(l + k) % 2], A[l], 2, N, r, Lp[l], tok_offset=T_of[k])
            prc.precompute_lr_cache(X_dec, A[l], 2, N, r, Lp[l], tok_offset=T_of[k] + n_pre)
            Kv, Vv, Lk, Lv, B_k, B_v = views(k, l, True)
            prc.materialize_agent_kv(Kv, Vv, Lk, Lv, B_k, B_v, kvl_cap[k], rope_theta=theta,
                                     K_full=Kf[l][:, :cap[k]], V_full=Vf[l][:, :cap[k]])

    def capture(fused):
        graphs = {}
        for k in T_of:
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr):
                decode(k, fused)
            graphs[k] = gr
            print(f"bench: stack: captured decode of turn {k} ({'LR-shared' if fused else 'materialised'})",
                  file=sys.stderr, flush=True)
        return graphs

    def run(fused, graphs):
        ev = {ph: [] for ph in ("segment", "materialise", "prefill", "decode_rows", "decode")}
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        for k in T_of:
            for ph, fn in (("segment", lambda: segment(k)),
                           ("materialise", (lambda: None) if fused else (lambda: materialise(k))),
                           ("prefill", lambda: prefill(k, fused)),
                           ("decode_rows", (lambda: decode_rows(k)) if fused else (lambda: None)),
                           ("decode", lambda: graphs[k].replay())):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                fn()
                e1.record()
                ev[ph].append((e0, e1))
        t1.record()
        torch.cuda.synchronize()
        out = {ph: round(sum(a.elapsed_time(b) for a, b in v), 3) for ph, v in ev.items()}
        out["total"] = round(t0.elapsed_time(t1), 3)
        return out

    # Warm-up outside capture (first calls load kernels), then capture.
    segment(1)
    prefill(1, True)
    decode_rows(1)
    decode(1, True)
    materialise(1)
    prefill(1, False)
    decode(1, False)
    torch.cuda.synchronize()
    g_fused = capture(True)
    # A replay reproduces the eager result (last turn's last step).
    g_fused[turns].replay()
    torch.cuda.synchronize()
    o_graph = O_dec.clone()
    decode(turns, True)
    torch.cuda.synchronize()
    same = torch.equal(o_graph, O_dec)
    print("bench: stack: timing the LR-shared run", file=sys.stderr, flush=True)
    fused = run(True, g_fused)
    del g_fused
    g_mat = capture(False)
    print("bench: stack: timing the materialised run", file=sys.stderr, flush=True)
    mat = run(False, g_mat)
    del g_mat

    dec_bytes = 0
    for k in T_of:
        for j in range(n_dec):
            kv = T_of[k] + n_pre + j + 1
            dec_bytes += n_layers * (kv * n_kv * d * 4 + kv * r * 4 + 2 * n_q * d * 2 + 2 * n_kv * d * r * 2)
    # Appending the LR rows step by step instead: one 1-row precompute per
    # layer and decode step (32 layers' A in rotation).
    def append_step(i):
        prc.precompute_lr_cache(X_dec[i % n_dec:i % n_dec + 1], A[i % n_layers], 2, N, r, Lp[i % n_layers],
                                tok_offset=T_of[turns] + n_pre + i % n_dec)
    for i in range(n_layers):
        append_step(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(20 * n_layers):
        append_step(i)
    e1.record()
    torch.cuda.synchronize()
    append_us = e0.elapsed_time(e1) / (20 * n_layers) * 1e3
    del K, V, Lp, Kf, Vf
    return {
        "bench": "workload", "index": 5, "workload": cfg.name,
        "shape": {"layers": n_layers, "hidden": hid, "n_q_heads": n_q, "n_kv_heads": n_kv, "head_dim": d,
                  "agents": N, "rank": r, "turns": turns, "turn_tokens": turn, "prefill_tokens": n_pre,
                  "decode_steps": n_dec, "s_cap": S_cap},
        "lr_shared_ms": fused, "materialised_ms": mat,
        "speedup_total": round(mat["total"] / fused["total"], 3),
        "speedup_decode": round((mat["decode"] + mat["materialise"]) / (fused["decode"] + fused["decode_rows"]), 3),
        "per_step_lr_append_us": round(append_us, 2),
        "decode_algorithmic_bytes": dec_bytes,
        "decode_gbs": round(dec_bytes / (fused["decode"] * 1e-3) / 1e9, 1),
        "decode_hbm_frac": round(dec_bytes / (fused["decode"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "graph_replay_equals_eager": bool(same),
        "resident_gb": {"base_cache": round(2 * n_layers * S_cap * n_kv * d * 2 / 1e9, 2),
                        "lr_planes": round(n_layers * 2 * N * S_cap * r * 2 / 1e9, 2),
                        "materialised_copy": round(2 * n_layers * S_cap * n_kv * d * 2 / 1e9, 2)},
    }


def workload_bench(prc, index, dev, steps, warmup):
    """Precompute, prefill and decode at the shapes of another workload (the
    8B-shaped layer at 8k context, or the 14B-shaped one at 64k with rank 64),
    each against the materialise-then-attend reference; one JSON line.  Every
    timed call reads a different input set, with enough sets that one pass
    over them exceeds the 256 MB Infinity Cache, so decode is timed from HBM
    even where one request's caches would fit in the cache."""
    import torch
    cfg, w = workload_dims(index)
    g = torch.Generator(device=dev).manual_seed(5000 + index)

    def nrm(shape, std=1.0):
        x = torch.randn(*shape, generator=g, device=dev, dtype=torch.float32)
        if std != 1.0:
            x.mul_(std)
        return x.to(torch.bfloat16)

    S, d, n_q, n_kv, r, B, N = w["S"], w["d"], w["n_q"], w["n_kv"], w["r"], w["B"], w["N"]
    kv_pre = S + w["n_pre"]
    work = algorithmic_work(w)
    bstd = math.sqrt(0.02)
    mall = 256 << 20
    n_dec = max(1, -(-2 * mall // work["decode_bytes"]))
    n_pre = max(1, -(-2 * mall // (kv_pre * n_kv * d * 4)))

    def case(nb, n_tok, kv, pos0):
        return dict(Q=nrm((nb, n_tok, n_q, d)), K_base=nrm((nb, kv, n_kv, d)), V_base=nrm((nb, kv, n_kv, d)),
                    L_k=nrm((nb, kv, r)), L_v=nrm((nb, kv, r)), B_k=nrm((nb, r, n_kv * d), bstd),
                    B_v=nrm((nb, r, n_kv * d), bstd),
                    positions=(torch.arange(pos0, pos0 + n_tok, dtype=torch.int32, device=dev)[None]
                               .repeat(nb, 1).contiguous()),
                    kv_len=torch.full((nb,), kv, dtype=torch.int32, device=dev))

    print(f"bench: workload {index}: {n_dec} decode and {n_pre} prefill input sets", file=sys.stderr, flush=True)
    dec = [case(B, 1, S, S - 1) for _ in range(n_dec)]
    pre = [case(1, w["n_pre"], kv_pre, S) for _ in range(n_pre)]
    X = [nrm((w["seg"], w["hidden"])) for _ in range(4)]
    A_stack = nrm((w["hidden"], 2 * N * r), 1.0 / math.sqrt(w["hidden"]))
    L = torch.zeros((2, N, w["seg"], r), dtype=torch.bfloat16, device=dev)
    O_dec = torch.empty_like(dec[0]["Q"])
    O_pre = torch.empty_like(pre[0]["Q"])
    dims = prc.make_dims(dec[0]["Q"], dec[0]["K_base"], dec[0]["L_k"], dec[0]["L_v"], dec[0]["B_k"],
                         dec[0]["B_v"], w["theta"])
    ws = torch.empty(max(1, prc.workspace_size(dims)), dtype=torch.uint8, device=dev)
    Kd, Vd = torch.empty_like(dec[0]["K_base"]), torch.empty_like(dec[0]["V_base"])
    Kp, Vp = torch.empty_like(pre[0]["K_base"]), torch.empty_like(pre[0]["V_base"])

    def plain(c, K, V):
        return dict(c, K_base=K, V_base=V, L_k=None, L_v=None, B_k=None, B_v=None)

    def materialised(c, K, V, O, wsp):
        prc.materialize_agent_kv(c["K_base"], c["V_base"], c["L_k"], c["L_v"], c["B_k"], c["B_v"],
                                 c["kv_len"], rope_theta=w["theta"], K_full=K, V_full=V)
        attn(prc, plain(c, K, V), w["theta"], O, wsp)

    def timed(fn, n_sets):
        # Eager warm-up (kernels loaded, workspaces settled), then one HIP
        # graph holding a call per input set, replayed back to back: the GPU
        # time per call without the host's launch overhead between calls
        # (short calls, such as a batch-1 decode, take less GPU time than
        # their launches take on the host).
        for i in range(max(warmup, n_sets)):
            fn(i % n_sets)
        torch.cuda.synchronize()
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            for i in range(n_sets):
                fn(i)
        gr.replay()
        torch.cuda.synchronize()
        reps = max(2, -(-steps // n_sets))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            gr.replay()
        e1.record()
        torch.cuda.synchronize()
        del gr
        return e0.elapsed_time(e1) / (reps * n_sets)

    # The prefill's workspace (split partials and its tile cache), also used
    # by the plain prefill of the reference.
    dims_pre = prc.make_dims(pre[0]["Q"], pre[0]["K_base"], pre[0]["L_k"], pre[0]["L_v"], pre[0]["B_k"],
                             pre[0]["B_v"], w["theta"])
    ws_pre = torch.empty(max(1, prc.workspace_size(dims_pre)), dtype=torch.uint8, device=dev)
    t_pc = timed(lambda i: prc.precompute_lr_cache(X[i % 4], A_stack, 2, N, r, L), 4)
    t_pre = timed(lambda i: attn(prc, pre[i], w["theta"], O_pre, ws_pre), n_pre)
    t_dec = timed(lambda i: attn(prc, dec[i], w["theta"], O_dec, ws), n_dec)
    t_pre_m = timed(lambda i: materialised(pre[i], Kp, Vp, O_pre, ws_pre), n_pre)
    t_dec_m = timed(lambda i: materialised(dec[i], Kd, Vd, O_dec, ws), n_dec)
    pre_tf = work["prefill_flops"] / (t_pre * 1e-3) / 1e12
    dec_gbs = work["decode_bytes"] / (t_dec * 1e-3) / 1e9
    pc_gbs = work["precompute_bytes"] / (t_pc * 1e-3) / 1e9
    pc_tf = work["precompute_flops"] / (t_pc * 1e-3) / 1e12
    return {
        "bench": "workload", "index": index, "workload": cfg.name,
        "shape": {"hidden": w["hidden"], "n_q_heads": n_q, "n_kv_heads": n_kv, "head_dim": d, "agents": N,
                  "rank": r, "context": S, "decode_batch": B, "prefill_tokens": w["n_pre"],
                  "precompute_rows": w["seg"]},
        "input_sets": {"decode": n_dec, "prefill": n_pre},
        "precompute": {"ms": round(t_pc, 4), "gbs": round(pc_gbs, 1), "hbm_frac": round(pc_gbs / HBM_PEAK_GBS, 4),
                       "tflops": round(pc_tf, 1), "mfma_frac": round(pc_tf / MFMA_BF16_PEAK_TFLOPS, 4)},
        "prefill": {"ms": round(t_pre, 4), "tflops": round(pre_tf, 1),
                    "mfma_frac": round(pre_tf / MFMA_BF16_PEAK_TFLOPS, 4),
                    "materialise_ms": round(t_pre_m, 4), "speedup": round(t_pre_m / t_pre, 3)},
        "decode": {"ms": round(t_dec, 4), "gbs": round(dec_gbs, 1), "hbm_frac": round(dec_gbs / HBM_PEAK_GBS, 4),
                   "materialise_ms": round(t_dec_m, 4), "speedup": round(t_dec_m / t_dec, 3)},
        "algorithmic": {"decode_bytes": work["decode_bytes"], "prefill_flops": work["prefill_flops"],
                        "precompute_bytes": work["precompute_bytes"]},
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-materialize", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="leave out the rank sweep, shared-base decode, joined projection, paged caches and the "
                         "32-layer stack from the default line")
    ap.add_argument("--no-workloads", action="store_true",
                    help="leave out the 8k (8B-shaped) and 64k (14B-shaped, rank 64) layers that the default run "
                         "times after the step")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--pmc-pass", action="store_true",
                    help="for hardware-counter runs: one 1 GiB calibration copy, then exactly one launch of "
                         "each hot-path kernel, no timing")
    ap.add_argument("--rank-sweep", action="store_true",
                    help="instead of the step: prefill and decode throughput over ranks 8..64 with LR on k and v "
                         "and on v only (the paper's QV setting), one JSON line each")
    ap.add_argument("--shared-base", action="store_true",
                    help="instead of the step: decode of all agents over one shared base cache, against the "
                         "same agents decoded as independent requests over per-agent copies")
    ap.add_argument("--fused-projection", action="store_true",
                    help="instead of the step: the base K/V projection and the LR precompute of a segment as "
                         "one GEMM, against the two as separate calls")
    ap.add_argument("--paged", action="store_true",
                    help="instead of the step: decode, prefill and segment projection over paged (block-table) "
                         "caches, against the same calls over contiguous caches")
    ap.add_argument("--workload", type=int, choices=(2, 4, 5), default=None,
                    help="instead of the step: precompute, prefill and decode at the 8k-context 8B-shaped (2) or "
                         "64k-context 14B-shaped rank-64 (4) workload, against materialise-then-attend")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              "(the multi-GPU sharding of the path is described in DESIGN.md).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_34054_amd as prc
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    prc.lib()
    dev = torch.device("cuda:0")
    cfg, w = workload_dims()
    if args.rank_sweep:
        for rec in rank_sweep(prc, w, dev, max(3, args.steps // 2), args.warmup):
            print(json.dumps(rec), flush=True)
        return
    if args.shared_base:
        print(json.dumps(shared_base_decode(prc, w, dev, args.steps, args.warmup)), flush=True)
        return
    if args.fused_projection:
        print(json.dumps(fused_projection(prc, w, dev, args.steps, args.warmup)), flush=True)
        return
    if args.paged:
        for rec in paged(prc, w, dev, args.steps, args.warmup):
            print(json.dumps(rec), flush=True)
        return
    if args.workload == 5:
        print(json.dumps(stack_bench(prc, dev)), flush=True)
        return
    if args.workload is not None:
        print(json.dumps(workload_bench(prc, args.workload, dev, args.steps, args.warmup)), flush=True)
        return
    work = algorithmic_work(w)
    print(f"bench: generating inputs ({w['B']} x {w['S']}-token decode caches)", file=sys.stderr, flush=True)
    x = make_inputs(w, dev)
    torch.cuda.synchronize()
    if args.pmc_pass:
        pmc_pass(prc, x, w, dev)
        return
    print("bench: timing fused path", file=sys.stderr, flush=True)
    stage, ms_step, wall_ms, per_step = run_fused(prc, x, w, args.steps, args.warmup)

    dec_gbs = work["decode_bytes"] / (stage["decode"] * 1e-3) / 1e9
    pre_tf = work["prefill_flops"] / (stage["prefill"] * 1e-3) / 1e12
    pc_tf = work["precompute_flops"] / (stage["precompute"] * 1e-3) / 1e12
    pc_gbs = work["precompute_bytes"] / (stage["precompute"] * 1e-3) / 1e9

    def roof(bound, achieved, peak, unit, traffic):
        return {"bound": bound, "achieved": round(achieved, 3), "peak": peak, "unit": unit,
                "frac": round(achieved / peak, 4), "traffic": traffic}

    rooflines = {
        "decode": dict(roof("hbm", dec_gbs, HBM_PEAK_GBS, "GB/s", traffic_for("lrsa_decode.hip")),
                       kernel="lrsa_decode_kernel + lrsa_merge_kernel", ms=round(stage["decode"], 4),
                       algorithmic_bytes=work["decode_bytes"]),
        "prefill": dict(roof("mfma", pre_tf, MFMA_BF16_PEAK_TFLOPS, "TFLOP/s", traffic_for("lrsa_prefill.hip")),
                        kernel="lrsa_prefill_kernel", ms=round(stage["prefill"], 4),
                        algorithmic_flops=work["prefill_flops"]),
        "precompute": dict(roof("hbm", pc_gbs, HBM_PEAK_GBS, "GB/s", traffic_for("precompute_gemm.hip")),
                           kernel="precompute_kernel", ms=round(stage["precompute"], 4),
                           algorithmic_bytes=work["precompute_bytes"], tflops=round(pc_tf, 3),
                           mfma_frac=round(pc_tf / MFMA_BF16_PEAK_TFLOPS, 4)),
    }
    dominant = max(("decode", "prefill", "precompute"), key=lambda k: stage[k])
    out = {
        "metric": METRIC,
        "value": round(dec_gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": ("8B-shaped layer at 32k context: precompute of a 4096-token segment for 8 agents "
                         "(rank 16, k and v); prefill of 4096 queries at positions 32768-36863; decode of 16 "
                         "requests at 32768 tokens"),
            "hidden": w["hidden"], "n_q_heads": w["n_q"], "n_kv_heads": w["n_kv"], "head_dim": w["d"],
            "agents": w["N"], "rank": w["r"], "context": w["S"], "decode_batch": w["B"],
            "prefill_tokens": w["n_pre"], "rope_theta": w["theta"],
        },
        "prefill_tflops": round(pre_tf, 3),
        "precompute_tflops": round(pc_tf, 3),
        "stages_ms": {k: round(v, 4) for k, v in stage.items()},
        "roofline": dict(rooflines[dominant], stage=dominant),
        "rooflines": rooflines,
        "host_ms_per_step": round(wall_ms, 4),
        "stage_ms_percentiles": {k: percentiles(v) for k, v in per_step.items()},
    }
    if not args.no_materialize:
        print("bench: timing materialise-then-attend reference", file=sys.stderr, flush=True)
        ref = run_materialized(prc, x, w, max(3, args.steps // 2), args.warmup)
        out["materialize_baseline"] = {
            "stages_ms": {k: round(v, 4) for k, v in ref.items()},
            "speedup_decode": round(ref["decode"] / stage["decode"], 3),
            "speedup_prefill": round(ref["prefill"] / stage["prefill"], 3),
            "speedup_step": round(sum(ref.values()) / sum(stage.values()), 3),
        }
    del x
    torch.cuda.empty_cache()
    if "materialize_baseline" in out:
        print("bench: timing library reference points", file=sys.stderr, flush=True)
        out["library_reference"] = library_reference(w, dev, work["prefill_flops"],
                                                     out["materialize_baseline"]["stages_ms"]["prefill"],
                                                     stage["precompute"])
    out["torch_copy_gbs"] = torch_copy_rate(dev)
    ceil = hbm_read_ceiling(prc, dev)
    out["hbm_read_ceiling"] = ceil
    for k in ("decode", "precompute"):
        r = rooflines[k]
        r["frac_of_measured_read_ceiling"] = round(r["achieved"] / ceil["gbs"], 4)
    if not args.no_workloads:
        out["workloads"] = {}
        for idx, key in ((2, "8k_8B_layer"), (4, "64k_14B_layer_rank64")):
            print(f"bench: timing workload {idx}", file=sys.stderr, flush=True)
            res = workload_bench(prc, idx, dev, args.steps, args.warmup)
            res["decode"]["frac_of_measured_read_ceiling"] = round(res["decode"]["gbs"] / ceil["gbs"], 4)
            out["workloads"][key] = res
            torch.cuda.empty_cache()
    if not args.no_extras:
        # The other measurements of the hot path, so that one default run
        # carries them all: the rank sweep (both wirings), the shared-base
        # decode, the joined projection, paged caches and the 32-layer stack.
        steps_x = max(3, args.steps // 2)
        extras = {}
        for key, fn in (("rank_sweep", lambda: rank_sweep(prc, w, dev, steps_x, args.warmup)),
                        ("shared_base_decode", lambda: shared_base_decode(prc, w, dev, steps_x, args.warmup)),
                        ("fused_projection", lambda: fused_projection(prc, w, dev, steps_x, args.warmup)),
                        ("paged", lambda: paged(prc, w, dev, steps_x, args.warmup)),
                        ("stack_32_layers", lambda: stack_bench(prc, dev))):
            print(f"bench: timing {key}", file=sys.stderr, flush=True)
            extras[key] = fn()
            torch.cuda.empty_cache()
        out["extras"] = extras
    if not args.no_cpu_baseline:
        print("bench: timing the fp64 oracle on a host sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
