#!/usr/bin/env python3
"""Benchmark of the action-expert denoising loop on one MI355X.

One "step" is one phyai_denoise call: the whole K-step Euler loop of one
batch (all transformer layers, attention over the frozen prefix, readout and
Euler update), i.e. one action chunk per request.

Headline (value): pi0-shaped expert, bf16 weights, batch 1 -- ms per chunk.
Also measured in the same run and reported in the same JSON line:
  * chunk_roofline: algorithmic bytes of a chunk (weights, prefix K/V,
    small per-step weights and boundary I/O; setup-only work excluded) over
    the chunk time, against the HBM datasheet roof and the measured copy roof.
  * batch64: the pi0-shaped expert at rollout batch 64 with ragged prefixes
    and fp8 weights -- chunks/s = B / T_sync (the paper's Q(B)), with the
    whole batch's MFMA fraction of the bf16 peak.
  * legs: the pi0.5-shaped and DiT-shaped batch-1 workloads and the tiny
    fp32 expert, ms per chunk each with its chunk roofline.
  * prefill: the prefix LM that produces the prefix K/V (Gemma-class, 816
    prefix tokens, batch 1): ms per call and its MFMA fraction.
  * vision: the vision tower before it (SigLIP-class ViT, three 256-patch
    images per request, batch 1, and batch 32): ms per call and its MFMA
    fraction.
  * pipeline: one pi0 chunk from the observation at batch 1 (tower -> prefix
    LM -> expert, back to back on one stream): ms per chunk.
  * roofline: the dominant kernel of the batch-1 leg, its algorithmic bytes
    per launch over its average duration, timed with HIP events on the stream
    it runs on.
  * cpu_baseline: the oracle on this host's cores (float64, the parity
    reference, and its float32 timing mode), with the CPU model and BLAS.

Inputs are seeded synthetic tensors resident in HBM before the timed region.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA

# HBM bytes moved by one launch of a block stage, from two rocprofv3 --pmc
# passes (FETCH_SIZE, WRITE_SIZE) over the leg (`--no-batch64 --no-stages` for
# batch 1, `--no-batch1 --no-stages` for batch 64), each scaled by what the
# counter reads for the 4 GiB device copy in the same run (profiles/
# traffic_pi0_b1_fetch_write.md, profiles/traffic_pi0_fp8_b64_fetch_write.md).
# Reported only while the code the counters were taken on is unchanged
# (sha256 prefix over the listed files with comments and blank lines removed).
_ATTN_SRC = ("paper_2608_03682_amd/csrc/attention.hip", "paper_2608_03682_amd/csrc/kernels.hpp",
             "paper_2608_03682_amd/csrc/common.hpp", "paper_2608_03682_amd/csrc/runtime.hip")
_GEMM_SRC = ("paper_2608_03682_amd/csrc/gemm.hip", "paper_2608_03682_amd/csrc/kernels.hpp",
             "paper_2608_03682_amd/csrc/common.hpp", "paper_2608_03682_amd/csrc/runtime.hip")
_MERGE_SRC = _GEMM_SRC + ("paper_2608_03682_amd/csrc/attention.hip",)
MEASURED_TRAFFIC = {
    ("pi0_bf16_b1", "attn"): {"bytes": 6240129, "sources": _ATTN_SRC, "sha256": "fc85730cbaeea999"},
    ("pi0_bf16_b1", "qkv"): {"bytes": 6536714, "sources": _GEMM_SRC, "sha256": "4fa368c185b08404"},
    ("pi0_bf16_b1", "oproj"): {"bytes": 9340935, "sources": _MERGE_SRC, "sha256": "2a06dd1a5a827dc6"},
    ("pi0_bf16_b1", "mlp_up"): {"bytes": 18212884, "sources": _GEMM_SRC, "sha256": "4fa368c185b08404"},
    ("pi0_bf16_b1", "mlp_down"): {"bytes": 12464135, "sources": _GEMM_SRC, "sha256": "4fa368c185b08404"},
    ("pi0_fp8_b64", "mlp_up"): {"bytes": 90550049, "sources": _GEMM_SRC, "sha256": "4fa368c185b08404"},
    ("pi0_fp8_b64", "qkv"): {"bytes": 107004929, "sources": _GEMM_SRC, "sha256": "4fa368c185b08404"},
    ("pi0_fp8_b64", "attn"): {"bytes": 84646916, "sources": _ATTN_SRC, "sha256": "fc85730cbaeea999"},
}


def code_digest(sources):
    """sha256 prefix of the sources' code: comments, trailing blanks and blank
    lines removed, so that a comment edit does not retire a measurement."""
    import hashlib
    import re
    h = hashlib.sha256()
    for src in sources:
        with open(os.path.join(ROOT, src), encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        lines = (re.sub(r"//.*$", "", ln).rstrip() for ln in text.splitlines())
        h.update("\n".join(ln for ln in lines if ln).encode())
    return h.hexdigest()[:16]


def measured_traffic(workload, stage):
    ent = MEASURED_TRAFFIC.get((workload, stage))
    if ent is None:
        return None
    return ent["bytes"] if code_digest(ent["sources"]) == ent["sha256"] else None


def _log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def _upload(case):
    import torch
    pre = case.prefix
    prefix = torch.from_numpy(pre.view(np.int16) if pre.dtype == np.uint16 else pre).cuda()
    noise = torch.from_numpy(case.noise).cuda()
    state = None if case.state is None else torch.from_numpy(case.state).cuda()
    return prefix, noise, state


def stage_bytes_flops(cfg, B, plen_sum):
    """Algorithmic HBM bytes and FLOPs of one launch of each block stage
    (one layer), following the phase-roofline accounting of weights +
    activations + K/V + boundary I/O.  Rows: the B*M suffix tokens."""
    d, F, D, nq, nkv = cfg.d_model, cfg.d_mlp, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
    M = cfg.tokens
    R = B * M
    # fp4: half a byte per weight plus one E8M0 exponent byte per 32 weights
    wb = {"fp8": 1.0, "fp4": 0.5 + 1.0 / 32}.get(cfg.weight_dtype, 2.0)
    scale = 4 if cfg.weight_dtype == "fp8" else 0
    qd, kd = nq * D, nkv * D
    Nqkv = qd + 2 * kd
    rows_alg = B * cfg.horizon            # state-token recompute excluded from FLOPs
    out = {
        "norm1": (R * d * 4 + R * d * 2, 0.0),
        "qkv": (d * Nqkv * wb + Nqkv * scale + R * d * 2 + R * Nqkv * 2, 2.0 * rows_alg * d * Nqkv),
        "attn": (plen_sum * 2 * kd * 2 + R * 2 * kd * 2 + 2 * R * qd * 2,
                 4.0 * rows_alg * nq * (plen_sum / B + M) * D),
        "oproj": (qd * d * wb + d * scale + R * qd * 2 + 2 * R * d * 4, 2.0 * rows_alg * qd * d),
        "norm2": (R * d * 4 + R * d * 2, 0.0),
        "mlp_up": (d * 2 * F * wb + 2 * F * scale + R * d * 2 + R * F * 2, 2.0 * rows_alg * d * 2 * F),
        "mlp_down": (F * d * wb + d * scale + R * F * 2 + 2 * R * d * 4, 2.0 * rows_alg * F * d),
    }
    return out


def chunk_bytes(cfg, B, plen_sum):
    """Algorithmic bytes of one phyai_denoise call (K steps), counted as in
    the paper's phase roofline (weights + K/V + boundary I/O; setup-only work
    and redundant recompute excluded): every step streams the trunk weights,
    the prefix K/V of every layer and the small per-step weights (time-MLP
    action half and second layer, input and output projections); activations
    that a fused implementation keeps on chip are not counted.  DiT: the
    cross-attention K/V projection of the features runs once per call (its
    weights and the features are counted once), and every step reads the
    projected K/V of each cross block."""
    d, A, F, L, K = cfg.d_model, cfg.action_dim, cfg.d_mlp, cfg.n_layers, cfg.n_steps
    D, nq, nkv = cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
    qd, kd = nq * D, nkv * D
    # weight bytes per parameter (fp4: the codes plus one E8M0 exponent per 32)
    wb = {"fp8": 1.0, "fp4": 0.5 + 1.0 / 32, "f32": 4.0}.get(cfg.weight_dtype, 2.0)
    sb = 4 if cfg.weight_dtype == "fp8" else 0          # per-column fp32 scales
    ab = 4 if cfg.weight_dtype == "f32" else 2          # small weights and K/V
    io = B * cfg.horizon * A * 4 * 2 + (B * A * 4 if cfg.state_token else 0)
    if cfg.variant == "dit":
        step_w = 0
        for l in range(L):
            cross = l % 2 == 0
            n_qkv = qd if cross else qd + 2 * kd
            step_w += (d * n_qkv + qd * d + d * F + F * d) * wb
        cross_kv_read = (L // 2) * plen_sum * 2 * kd * ab
        small = 2 * A * d * ab + cfg.horizon * d * 4
        per_call = (L // 2) * cfg.d_feat * 2 * kd * wb + plen_sum * cfg.d_feat * ab
        return K * (step_w + cross_kv_read + small) + per_call + io
    step_w = L * ((d * (qd + 2 * kd) + qd * d + d * 2 * F + F * d) * wb
                  + ((qd + 2 * kd) + d + 2 * F + d) * sb)
    prefix_kv = L * plen_sum * 2 * kd * ab
    small = 2 * A * d * ab + (2 * d * d * ab if cfg.variant == "pi0" else 0)
    return K * (step_w + prefix_kv + small) + io


def time_calls(fn, steps, warmup):
    import torch
    short = steps + warmup <= 8            # counter passes: one progress line per call
    for i in range(warmup):
        fn()
        if short:
            torch.cuda.synchronize()
            _log(f"warm-up call {i + 1} done")
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record()
    for i in range(steps):
        fn()
        evs[i + 1].record()
        if short:
            torch.cuda.synchronize()
            _log(f"timed call {i + 1} done")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(steps)])
    return wall, per


def time_stages(ex, reps=5):
    """Average duration of one launch of each block stage: `reps` passes over
    all layers of the stage are captured into a graph (as the denoising loop
    runs), and HIP events on the replay stream time one replay."""
    import torch
    res = {}
    L = ex.cfg.n_layers
    cap = torch.cuda.Stream()
    for st in ("norm1", "qkv", "attn", "oproj", "norm2", "mlp_up", "mlp_down"):
        ex.profile_stage(st, 1)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap):
            ex.profile_stage(st, reps)
        g.replay()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        g.replay()
        b.record()
        torch.cuda.synchronize()
        res[st] = a.elapsed_time(b) * 1e3 / (reps * L)     # microseconds per launch
        del g
    return res


def _host_info():
    """Threads the oracle's BLAS uses, the CPU model and the BLAS library."""
    cores, blas = os.cpu_count() or 1, "unknown"
    try:
        from threadpoolctl import threadpool_info
        pools = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        if pools:
            cores = max(p.get("num_threads", 1) for p in pools)
            blas = ", ".join(f"{p.get('internal_api')} {p.get('version')}" for p in pools)
    except Exception:
        pass
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return int(cores), model, blas


def _time_oracle(cfg, case, dtype, budget_s, max_runs=3, prefix=None, n_req=None):
    """Median wall time of oracle.denoise over up to max_runs runs (at least
    one; stops adding runs once budget_s is spent).  With n_req, only the
    first n_req requests run, against `prefix` holding just their slots."""
    import oracle
    W = oracle.DecodedWeights(case.weights, dtype)
    n = case.noise.shape[0] if n_req is None else n_req
    pre = case.prefix if prefix is None else prefix
    runs, spent = [], 0.0
    while len(runs) < max_runs and (spent < budget_s or not runs):
        t0 = time.perf_counter()
        oracle.denoise(cfg, case.weights, pre, case.prefix_len[:n], case.noise[:n], case.timesteps,
                       None if case.state is None else case.state[:n], decoded=W, dtype=dtype)
        dt = time.perf_counter() - t0
        runs.append(dt)
        spent += dt
    return float(np.median(runs)), len(runs)


def cpu_baseline(cfg, case):
    """The oracle on the host cores: float64 (the parity reference, `value`)
    and its float32 timing mode, full chunks of the batch-1 pi0 workload."""
    cores, model, blas = _host_info()
    t64, n64 = _time_oracle(cfg, case, np.float64, 8.0)
    t32, n32 = _time_oracle(cfg, case, np.float32, 6.0)
    return {"value": round(t64 * 1e3, 1), "unit": "ms/chunk", "cores": cores, "kind": "oracle",
            "sample": f"{n64} full chunk(s) of the batch-1 pi0 workload (K={cfg.n_steps} Euler steps, "
                      f"L={cfg.n_layers}), float64 NumPy oracle, median; float32 mode {n32} chunk(s)",
            "fp32_ms_per_chunk": round(t32 * 1e3, 1), "cpu_model": model, "blas": blas}


def cpu_baseline_batch(cfg, case, seed, n_req=2):
    """The float64 oracle on the first n_req requests of a batch, scaled to
    the batch (requests are independent, so the oracle's time is linear in
    them): chunks/s and ms per batch."""
    import workloads as wl
    cores, model, blas = _host_info()
    pre = wl.make_prefix(cfg, case.prefix_len, seed, requests=list(range(n_req)))
    t, _ = _time_oracle(cfg, case, np.float64, 0.0, max_runs=1, prefix=pre, n_req=n_req)
    per_req = t / n_req
    return {"value": round(1.0 / per_req, 3), "unit": "chunks/s", "cores": cores,
            "kind": "oracle", "ms_per_batch": round(per_req * cfg.batch * 1e3, 1),
            "sample": f"{n_req} of the {cfg.batch} requests (prefix lengths "
                      f"{', '.join(str(int(p)) for p in case.prefix_len[:n_req])}), one run, float64 NumPy "
                      f"oracle, scaled to the batch", "cpu_model": model, "blas": blas}


def cpu_baseline_prefill(cfg, case):
    """The float64 prefix-LM oracle on a bounded sample of the call: one layer's
    K/V projection alone (the last layer's work) and a full layer plus that
    projection, over the whole prefix; a call is (L - 1) full layers plus one
    K/V projection."""
    import oracle
    cores, model, blas = _host_info()
    t0 = time.perf_counter()
    oracle.prefill(cfg, case.weights, case.embeds, case.prefix_len, n_layers=1)
    t_kv = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.prefill(cfg, case.weights, case.embeds, case.prefix_len, n_layers=2)
    t_full = max(time.perf_counter() - t0 - t_kv, 0.0)
    call = (cfg.n_layers - 1) * t_full + t_kv
    return {"value": round(call * 1e3, 1), "unit": "ms/call", "cores": cores, "kind": "oracle",
            "sample": f"layer 0 in full and one K/V projection over the {int(case.prefix_len.sum())}-token prefix, "
                      f"float64 NumPy oracle, scaled to {cfg.n_layers - 1} full layers + the last layer's K/V",
            "cpu_model": model, "blas": blas}


def cpu_baseline_vision(cfg, weights, patches):
    """The float64 vision-tower oracle on one image (all blocks, the projector),
    scaled to the call's images (images are independent)."""
    import oracle
    cores, model, blas = _host_info()
    t0 = time.perf_counter()
    oracle.encode_images(cfg, weights, patches[:1, :1])
    t = time.perf_counter() - t0
    n = patches.shape[0] * patches.shape[1]
    return {"value": round(t * n * 1e3, 1), "unit": "ms/call", "cores": cores, "kind": "oracle",
            "sample": f"1 of the {n} images ({cfg.n_layers} blocks and the projector), float64 NumPy oracle, "
                      f"scaled to the call", "cpu_model": model, "blas": blas}


def measured_roofs():
    """The paper's roof measurement, on this GPU: best of 50 after 10 warm-up
    iterations of a 4 GiB device copy (memory roof) and an 8192^2 bf16 GEMM
    (compute roof, torch/hipBLASLt used only as a measuring stick)."""
    import torch
    n = (4 << 30) // 4
    src = torch.empty(n, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    a = torch.randn(8192, 8192, dtype=torch.bfloat16, device="cuda")
    b = torch.randn(8192, 8192, dtype=torch.bfloat16, device="cuda")

    def best(fn):
        for _ in range(10):
            fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(50):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3)
        return min(ts)

    t_copy = best(lambda: dst.copy_(src))
    t_gemm = best(lambda: torch.matmul(a, b))
    out = {"copy_GBs": round(2 * n * 4 / t_copy / 1e9, 1), "copy_bytes_per_launch": 2 * n * 4,
           "bf16_gemm_TFLOPs": round(2 * 8192 ** 3 / t_gemm / 1e12, 1)}
    del src, dst, a, b
    torch.cuda.empty_cache()
    return out


def chunk_roofline(cfg, B, plen_sum, ms, copy_gbs=None):
    cb = chunk_bytes(cfg, B, plen_sum)
    ach = cb / (ms * 1e-3) / 1e9
    out = {"bytes_per_chunk": int(cb), "achieved_GBs": round(ach, 1), "frac_of_hbm_peak": round(ach / HBM_PEAK_GBS, 4)}
    if copy_gbs:
        out["frac_of_measured_copy"] = round(ach / copy_gbs, 4)
    return out


def leg_batch1(args, px, wl, K, W):
    import torch
    cfg = wl.CONFIGS["pi0_bf16_b1"]
    _log(f"generating {cfg.name}")
    case = wl.make_case(cfg, seed=args.seed)
    ex = px.Expert(cfg, case.weights)
    prefix, noise, state = _upload(case)
    out = torch.empty_like(noise)
    ex.prepare(1, cfg.n_steps)
    fn = lambda: ex.denoise(prefix, case.prefix_len, noise, case.timesteps, state, out=out)
    _log(f"timing {cfg.name}: {W} warmup + {K} timed")
    wall, per = time_calls(fn, K, W)
    ms = wall * 1e3 / K
    assert np.isfinite(out.cpu().numpy()).all()
    plen_sum = int(case.prefix_len.sum())
    roof, stages = None, {}
    if not args.no_stages:
        stages = time_stages(ex)
        sb = stage_bytes_flops(cfg, 1, plen_sum)
        dom = max(("qkv", "attn", "oproj", "mlp_up", "mlp_down"), key=lambda s: stages[s])
        dom_bytes = sb[dom][0]
        ach = dom_bytes / (stages[dom] * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": measured_traffic(cfg.name, dom),
                "kernel": dom, "bytes_per_launch": int(dom_bytes), "avg_us": round(stages[dom], 2),
                "timing": "graph replay of the stage over all layers, HIP events on the replay stream"}
    rec = {
        "metric": "pi0-shape action-chunk latency ms @B=1 + chunks/s @B=64; % HBM / MFMA peak",
        "value": round(ms, 4), "unit": "ms/chunk", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": round(ms, 4), "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded N(0,0.02) weights, N(0,1) prefix K/V and noise)",
        "config": {"workload": "pi0_bf16_b1: 18 layers, width 1024, 8 q heads + 1 kv head, head_dim 256, "
                               "GeGLU 4096, RoPE, prefix 816, H=50 + state token, A=32, K=10 Euler steps, B=1",
                   "batch": 1, "prefix_len": int(case.prefix_len[0]), "euler_steps": cfg.n_steps},
        "latency_ms": {"mean": round(float(per.mean()), 4), "p50": round(float(np.median(per)), 4),
                       "p99": round(float(np.percentile(per, 99)), 4)},
        "chunks_per_s": round(1e3 / ms, 1),
        "stage_us_per_launch": {k: round(v, 2) for k, v in stages.items()},
        "roofline": roof,
    }
    if not args.no_roofs:
        _log("measuring the copy and GEMM roofs")
        rec["measured_roofs"] = measured_roofs()
    copy = rec.get("measured_roofs", {}).get("copy_GBs")
    rec["chunk_roofline"] = chunk_roofline(cfg, 1, plen_sum, ms, copy)
    if not args.no_cpu_baseline:
        _log("timing the CPU oracle baseline")
        rec["cpu_baseline"] = cpu_baseline(cfg, case)
    ex.close()
    del prefix, noise, state, out, case
    torch.cuda.empty_cache()
    return rec


def leg_plain(args, px, wl, name, K, W, copy_gbs, env=None):
    """ms per chunk of another batch-1 workload, with its chunk roofline
    (`env`: library switches set for the leg, e.g. the persistent loop)."""
    import os
    import torch
    env = env or {}
    for k, v in env.items():
        os.environ[k] = v
    try:
        return _leg_plain(args, px, wl, name, K, W, copy_gbs, env)
    finally:
        for k in env:
            del os.environ[k]


def _leg_plain(args, px, wl, name, K, W, copy_gbs, env):
    import torch
    cfg = wl.CONFIGS[name]
    _log(f"generating {name}")
    case = wl.make_case(cfg, seed=args.seed)
    ex = px.Expert(cfg, case.weights)
    prefix, noise, state = _upload(case)
    out = torch.empty_like(noise)
    ex.prepare(cfg.batch, cfg.n_steps)
    fn = lambda: ex.denoise(prefix, case.prefix_len, noise, case.timesteps, state, out=out)
    _log(f"timing {name}: {W} warmup + {K} timed")
    wall, per = time_calls(fn, K, W)
    ms = wall * 1e3 / K
    assert np.isfinite(out.cpu().numpy()).all()
    rec = {"ms_per_chunk": round(ms, 4), "p50_ms": round(float(np.median(per)), 4), "steps": K, "warmup": W,
           "dtype": "f32" if cfg.weight_dtype == "f32" else "bf16",
           "weights": cfg.weight_dtype,
           "chunk_roofline": chunk_roofline(cfg, cfg.batch, int(case.prefix_len.sum()), ms, copy_gbs)}
    if env:
        rec["env"] = dict(env)
    ex.close()
    del prefix, noise, state, out, case
    torch.cuda.empty_cache()
    return rec


def prefill_flops(cfg, plen):
    """MFMA work of one prefix-LM call: every layer's GEMMs over the valid
    prefix rows (the last layer only its QKV projection) and attention of
    each request over its own prefix (Q K^T and P V: 4 P^2 n_q d_h per
    layer)."""
    d, F, D, nq, nkv, L = cfg.d_model, cfg.d_mlp, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads, cfg.n_layers
    qkv = 2 * d * (nq + 2 * nkv) * D
    full = qkv + 2 * nq * D * d + 2 * d * 2 * F + 2 * F * d
    rows = int(np.sum(plen))
    attn = sum(4 * int(p) ** 2 * nq * D for p in plen)
    return rows * (full * (L - 1) + qkv) + (L - 1) * attn


def stage_mfma_roofline(stage_us, flops):
    """The MFMA roofline of a leg's dominant GEMM or attention stage: its
    algorithmic FLOPs per launch over its replayed per-launch time."""
    dom = max((s for s in flops if s in stage_us), key=lambda s: stage_us[s])
    ach = flops[dom] / (stage_us[dom] * 1e-6) / 1e12
    return {"bound": "mfma", "achieved": round(ach, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(ach / BF16_PEAK_TFLOPS, 4), "traffic": None, "kernel": dom,
            "flops_per_launch": int(flops[dom]), "avg_us": stage_us[dom],
            "timing": "graph replay of the stage over all layers, HIP events on the replay stream"}


def leg_prefill(args, px, wl, K, W):
    """The prefix LM (the VLM's language part producing the prefix K/V) on
    the Gemma-class workload over the pi0 prefix (816 tokens, batch 1): ms
    per call, MFMA throughput, and per-stage launch times (graph replays)."""
    import torch
    cfg = wl.CONFIGS["plm_gemma_bf16_b1"]
    _log(f"generating {cfg.name}")
    case = wl.make_prefill_case(cfg, seed=args.seed)
    m = px.PrefixLM(cfg, case.weights)
    emb = torch.from_numpy(case.embeds).cuda()
    out = torch.empty((cfg.n_layers, 2, cfg.batch, cfg.prefix_cap, cfg.n_kv_heads * cfg.head_dim),
                      dtype=torch.int16, device="cuda")
    _log(f"timing {cfg.name}")
    wall, per = time_calls(lambda: m.prefill(emb, case.prefix_len, out=out), K, W)
    ms = float(np.median(per))
    fl = prefill_flops(cfg, case.prefix_len)
    tf = fl / (ms * 1e-3) / 1e12
    rec = {"config": {"workload": "prefix LM, Gemma-class (18 layers, width 2048, 8 query heads + 1 K/V head "
                                  "of 256, GeGLU 16384), pi0 prefix of 816 tokens, batch 1",
                      "weights": "bf16"},
           "ms_per_call": round(ms, 3), "p99_ms": round(float(np.percentile(per, 99)), 3),
           "tokens_per_s": round(float(np.sum(case.prefix_len)) / (ms * 1e-3), 1),
           "flops_per_call": int(fl), "TFLOPs": round(tf, 1),
           "frac_of_bf16_peak": round(tf / BF16_PEAK_TFLOPS, 4)}
    if not args.no_stages:
        stages = {}
        Lf = cfg.n_layers - 1                  # stages run over the layers with an MLP
        cap = torch.cuda.Stream()
        for st in ("norm1", "qkv", "attn", "oproj", "norm2", "mlp_up", "mlp_down"):
            m.profile_stage(st, 1)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=cap):
                m.profile_stage(st, 2)
            g.replay()
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            g.replay()
            b.record()
            torch.cuda.synchronize()
            stages[st] = round(a.elapsed_time(b) * 1e3 / (2 * Lf), 2)
            del g
        rec["stage_us"] = stages
        d, F, D, nq, nkv = cfg.d_model, cfg.d_mlp, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
        rows = int(np.sum(case.prefix_len))
        rec["roofline"] = stage_mfma_roofline(stages, {
            "qkv": 2 * rows * d * (nq + 2 * nkv) * D, "attn": sum(4 * int(p) ** 2 * nq * D for p in case.prefix_len),
            "oproj": 2 * rows * nq * D * d, "mlp_up": 2 * rows * d * 2 * F, "mlp_down": 2 * rows * F * d})
    m.close()
    del emb, out
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        _log("timing the prefix-LM oracle")
        rec["cpu_baseline"] = cpu_baseline_prefill(cfg, case)
    del case
    return rec


def vision_flops(cfg, B):
    """MFMA work of one vision-tower call over B requests: per image the
    patch embedding, every block's QKV, O and MLP GEMMs and attention (Q K^T
    and P V: 4 N^2 n_heads d_h per block), and the projector."""
    d, F, D, H, L, N = cfg.d_model, cfg.d_mlp, cfg.head_dim, cfg.n_q_heads, cfg.n_layers, cfg.n_patches
    per_row = 2 * cfg.patch_dim * d + L * (2 * d * 3 * H * D + 2 * H * D * d + 2 * d * F * 2) + 2 * d * cfg.d_out
    per_img = N * per_row + L * 4 * N * N * H * D
    return B * cfg.n_images * per_img


def leg_vision(args, px, wl, K, W):
    """The vision tower (image patches to the image tokens that open the
    prefix) on the SigLIP-class workload, batch 1: ms per call, MFMA
    throughput, and per-stage launch times (graph replays)."""
    import torch
    cfg = wl.CONFIGS["vit_siglip_bf16_b1"]
    _log(f"generating {cfg.name}")
    case = wl.make_vision_case(cfg, seed=args.seed)
    m = px.VisionTower(cfg, case.weights)
    pt = torch.from_numpy(case.patches).cuda()
    out = torch.empty((cfg.batch, cfg.n_images * cfg.n_patches, cfg.d_out), dtype=torch.float32, device="cuda")
    _log(f"timing {cfg.name}")
    wall, per = time_calls(lambda: m.encode(pt, out=out), K, W)
    ms = float(np.median(per))
    fl = vision_flops(cfg, cfg.batch)
    tf = fl / (ms * 1e-3) / 1e12
    rec = {"config": {"workload": "vision tower, SigLIP-class ViT (24 blocks of width 1024, 16 heads of 64, GELU "
                                  "MLP 4096), 3 images of 256 patches of 768 values, projected to 2048, batch 1",
                      "weights": "bf16"},
           "ms_per_call": round(ms, 3), "p99_ms": round(float(np.percentile(per, 99)), 3),
           "images_per_s": round(cfg.batch * cfg.n_images / (ms * 1e-3), 1),
           "flops_per_call": int(fl), "TFLOPs": round(tf, 1),
           "frac_of_bf16_peak": round(tf / BF16_PEAK_TFLOPS, 4)}
    if not args.no_stages:
        stages = {}
        cap = torch.cuda.Stream()
        for st in ("norm1", "qkv", "attn", "oproj", "norm2", "mlp_up", "mlp_down"):
            m.profile_stage(st, 1)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=cap):
                m.profile_stage(st, 2)
            g.replay()
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            g.replay()
            b.record()
            torch.cuda.synchronize()
            stages[st] = round(a.elapsed_time(b) * 1e3 / (2 * cfg.n_layers), 2)
            del g
        rec["stage_us"] = stages
        d, F, D, H, N = cfg.d_model, cfg.d_mlp, cfg.head_dim, cfg.n_q_heads, cfg.n_patches
        R = cfg.batch * cfg.n_images * N
        rec["roofline"] = stage_mfma_roofline(stages, {
            "qkv": 2 * R * d * 3 * H * D, "attn": cfg.batch * cfg.n_images * 4 * N * N * H * D,
            "oproj": 2 * R * H * D * d, "mlp_up": 2 * R * d * F, "mlp_down": 2 * R * F * d})
    m.close()
    del pt, out
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        _log("timing the vision oracle")
        rec["cpu_baseline"] = cpu_baseline_vision(cfg, case.weights, case.patches)
    del case
    # the same tower at batch 32 (96 images), the batch of the paper's phase analysis
    c32 = wl.CONFIGS["vit_siglip_bf16_b32"]
    _log(f"timing {c32.name}")
    m = px.VisionTower(c32, wl.make_weights(c32, args.seed))
    pt = torch.from_numpy(wl.make_patches(c32, args.seed)).cuda()
    out = torch.empty((c32.batch, c32.n_images * c32.n_patches, c32.d_out), dtype=torch.float32, device="cuda")
    wall, per = time_calls(lambda: m.encode(pt, out=out), max(1, K // 2), max(1, W))
    ms32 = float(np.median(per))
    tf32 = vision_flops(c32, c32.batch) / (ms32 * 1e-3) / 1e12
    rec["batch32"] = {"ms_per_call": round(ms32, 3), "images_per_s": round(c32.batch * c32.n_images / (ms32 * 1e-3), 1),
                      "TFLOPs": round(tf32, 1), "frac_of_bf16_peak": round(tf32 / BF16_PEAK_TFLOPS, 4)}
    m.close()
    del pt, out
    torch.cuda.empty_cache()
    return rec


def leg_pipeline(args, px, wl, K, W):
    """One pi0 chunk from the observation at batch 1, every phase on the
    GPU back to back on one stream: the vision tower writes the 768 image
    tokens into the prefix embeddings (48 text rows after them), the prefix
    LM turns the 816 rows into the per-layer K/V, and the denoising loop
    reads that cache.  ms per chunk (the paper's end-to-end figure, with its
    own vision and language models, is context only)."""
    import torch
    vc, pc, ec = (wl.CONFIGS[n] for n in ("vit_siglip_bf16_b1", "plm_gemma_bf16_b1", "pi0_bf16_b1"))
    _log("generating the pipeline's three models")
    tower = px.VisionTower(vc, wl.make_weights(vc, args.seed))
    lm = px.PrefixLM(pc, wl.make_weights(pc, args.seed))
    ecase = wl.make_case(ec, seed=args.seed)
    ex = px.Expert(ec, ecase.weights)
    del ecase.weights
    pcase_len = wl.make_prefix_lengths(pc, args.seed)
    emb = torch.from_numpy(wl.make_prefix_embeds(pc, pcase_len, args.seed)).cuda()
    patches = torch.from_numpy(wl.make_patches(vc, args.seed)).cuda()
    kv = torch.empty((pc.n_layers, 2, 1, pc.prefix_cap, pc.n_kv_heads * pc.head_dim), dtype=torch.int16,
                     device="cuda")
    noise = torch.from_numpy(ecase.noise).cuda()
    state = torch.from_numpy(ecase.state).cuda()
    out = torch.empty_like(noise)
    ex.prepare(1, ec.n_steps)

    def chunk():
        tower.encode(patches, out=emb)
        lm.prefill(emb, pcase_len, out=kv)
        ex.denoise(kv, pcase_len, noise, ecase.timesteps, state, out=out)

    _log("timing the pipeline")
    wall, per = time_calls(chunk, K, W)
    assert np.isfinite(out.cpu().numpy()).all()
    ms = float(np.median(per))
    rec = {"config": {"workload": "pi0 chunk from the observation, batch 1: SigLIP-class tower over 3 images "
                                  "-> Gemma-class prefix LM over 816 tokens -> pi0 expert, 10 steps",
                      "weights": "bf16"},
           "ms_per_chunk": round(ms, 3), "p99_ms": round(float(np.percentile(per, 99)), 3)}
    tower.close()
    lm.close()
    ex.close()
    del emb, patches, kv, noise, state, out
    torch.cuda.empty_cache()
    return rec


def leg_batch64(args, px, wl, K, W):
    import torch
    cfg = wl.CONFIGS["pi0_fp8_b64"]
    _log(f"generating {cfg.name}")
    case = wl.make_case(cfg, seed=args.seed)
    ex = px.Expert(cfg, case.weights)
    prefix, noise, state = _upload(case)
    out = torch.empty_like(noise)
    ex.prepare(cfg.batch, cfg.n_steps)
    fn = lambda: ex.denoise(prefix, case.prefix_len, noise, case.timesteps, state, out=out)
    K64 = K if K < 5 else max(5, K // 5)
    W64 = W if W < 2 else max(2, W // 5)
    _log(f"timing {cfg.name}: {W64} warmup + {K64} timed")
    wall, per = time_calls(fn, K64, W64)
    ms64 = wall * 1e3 / K64
    assert np.isfinite(out.cpu().numpy()).all()
    plen_sum = int(case.prefix_len.sum())
    sb = stage_bytes_flops(cfg, cfg.batch, plen_sum)
    chunk_flops = sum(v[1] for v in sb.values()) * cfg.n_layers * cfg.n_steps
    roof, stages = None, {}
    if not args.no_stages:
        stages = time_stages(ex, reps=2)
        dom = max(("qkv", "attn", "oproj", "mlp_up", "mlp_down"), key=lambda s: stages[s])
        fl = sb[dom][1]
        ach = fl / (stages[dom] * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(ach / BF16_PEAK_TFLOPS, 4), "traffic": measured_traffic(cfg.name, dom),
                "kernel": dom, "flops_per_launch": int(fl), "avg_us": round(stages[dom], 2)}
    tf = chunk_flops / (ms64 * 1e-3) / 1e12
    rec = {
        "workload": "pi0_fp8_b64: pi0 shape, B=64, ragged prefixes U[600,1000], fp8 e4m3 trunk weights "
                    "(per-output-channel scales), bf16 prefix K/V, K=10",
        "steps": K64, "warmup": W64, "ms_per_batch": round(ms64, 3),
        "chunks_per_s": round(cfg.batch / (ms64 * 1e-3), 1),
        "stage_us_per_launch": {k: round(v, 2) for k, v in stages.items()},
        "roofline": roof,
        "batch_roofline": {"bound": "mfma", "flops_per_batch": int(chunk_flops), "achieved_TFLOPs": round(tf, 1),
                           "peak": BF16_PEAK_TFLOPS, "frac_of_bf16_peak": round(tf / BF16_PEAK_TFLOPS, 4)},
        "batch_TFLOPs": round(tf, 1),
    }
    if not args.no_cpu_baseline:
        _log("timing the CPU oracle baseline on a sample of the batch")
        rec["cpu_baseline"] = cpu_baseline_batch(cfg, case, args.seed)
    ex.close()
    del prefix, noise, state, out, case
    torch.cuda.empty_cache()
    return rec


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-batch64", action="store_true")
    ap.add_argument("--no-batch1", action="store_true",
                    help="only the batch-64 leg (for counter passes; the line then has no batch-1 value)")
    ap.add_argument("--no-legs", action="store_true", help="skip the pi0.5, DiT and tiny fp32 workloads")
    ap.add_argument("--no-prefill", action="store_true", help="skip the prefix-LM workload")
    ap.add_argument("--no-vision", action="store_true", help="skip the vision-tower workload")
    ap.add_argument("--no-pipeline", action="store_true",
                    help="skip the chunk-from-observation pipeline (tower -> prefix LM -> expert)")
    ap.add_argument("--no-stages", action="store_true",
                    help="skip the per-stage graph timings and the rooflines built on them (counter passes)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-roofs", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU only (the expert loop shards as independent "
              f"requests per GPU, with no cross-GPU step); --gpus {args.gpus} is not run.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_03682_amd as px
    import workloads as wl

    torch.cuda.set_device(0)
    K, W = args.steps, args.warmup

    rec = {}
    if not args.no_batch1:
        rec = leg_batch1(args, px, wl, K, W)
    elif not args.no_roofs:
        _log("measuring the copy and GEMM roofs")
        rec["measured_roofs"] = measured_roofs()      # counter passes calibrate on its copy
    copy = rec.get("measured_roofs", {}).get("copy_GBs")
    if not args.no_legs:
        Kl, Wl = max(1, min(K, 20)), min(W, 5)
        rec["legs"] = {n: leg_plain(args, px, wl, n, Kl, Wl, copy)
                       for n in ("pi05_bf16_b1", "dit_bf16_b1", "tiny_fp32", "pi0_fp4_b1")}
        # the persistent batch-1 loop (opt-in) on the pi0 workload
        rec["legs"]["pi0_bf16_b1_persistent"] = leg_plain(args, px, wl, "pi0_bf16_b1", Kl, Wl, copy,
                                                           env={"PHYAI_PERSIST": "1"})
    if not args.no_prefill:
        rec["prefill"] = leg_prefill(args, px, wl, max(1, min(K, 20)), min(W, 3))
    if not args.no_vision:
        rec["vision"] = leg_vision(args, px, wl, max(1, min(K, 20)), min(W, 3))
    if not args.no_pipeline:
        rec["pipeline"] = leg_pipeline(args, px, wl, max(1, min(K, 20)), min(W, 3))
        parts = [rec.get("cpu_baseline"), rec.get("prefill", {}).get("cpu_baseline"),
                 rec.get("vision", {}).get("cpu_baseline")]
        if all(parts):
            rec["pipeline"]["cpu_baseline"] = {
                "value": round(sum(p["value"] for p in parts), 1), "unit": "ms/chunk", "cores": parts[0]["cores"],
                "kind": "oracle", "sample": "the sum of the three phases' oracle timings (expert chunk, prefix-LM "
                                            "call, vision call) reported with their legs"}
    if not args.no_batch64:
        rec["batch64"] = leg_batch64(args, px, wl, K, W)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
