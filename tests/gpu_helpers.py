"""Shared helpers for the GPU parity tests: small workloads, device upload,
the tolerance rule and the parity report."""
from __future__ import annotations

import sys

import numpy as np

import workloads as wl


def small_cfg(variant: str, **kw) -> wl.ExpertConfig:
    """Small shapes that still cover several MFMA tiles and ragged tails:
    51 suffix rows (one 64-row tile, ragged), 4 query heads x 51 tokens of
    attention rows, ragged prefixes that end mid key-tile."""
    base = dict(n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=1, head_dim=64, d_mlp=512,
                horizon=50, action_dim=32, n_steps=3, prefix_cap=100, prefix_min=37, prefix_max=100,
                batch=3, weight_dtype="bf16", kv_dtype="bf16")
    if variant == "pi0":
        base.update(state_token=True, rope=True)
    elif variant == "pi05":
        base.update(state_token=False, rope=True, head_dim=128, n_q_heads=2)
    elif variant == "dit":
        base.update(n_q_heads=2, n_kv_heads=2, head_dim=128, horizon=16, state_token=True, rope=False,
                    d_feat=128, time_dim=256, prefix_cap=40, prefix_min=23, prefix_max=40, batch=2)
    base.update(kw)
    base.setdefault("time_dim", base["d_model"])
    return wl.ExpertConfig(name=f"small_{variant}", cfg_id=50, variant=variant, **base)


def tolerance(cfg) -> float:
    """Max-abs bar on the final actions (relative to max(1, rms(oracle)))."""
    # fp4 weights decode exactly to bf16 on both sides, so only the bf16
    # activations separate the GPU from the oracle: the bf16 bar
    return {"f32": 1e-4, "bf16": 2e-2, "fp8": 5e-2, "fp4": 2e-2}[cfg.weight_dtype]


def to_device(case):
    import torch
    pre = case.prefix
    if pre.dtype == np.uint16:
        prefix = torch.from_numpy(pre.view(np.int16)).cuda()
    else:
        prefix = torch.from_numpy(np.ascontiguousarray(pre)).cuda()
    noise = torch.from_numpy(case.noise).cuda()
    state = None if case.state is None else torch.from_numpy(case.state).cuda()
    return prefix, noise, state


def run_gpu(expert, case, dev=None, out=None):
    import torch
    prefix, noise, state = dev if dev is not None else to_device(case)
    y = expert.denoise(prefix, case.prefix_len, noise, case.timesteps, state, out=out)
    torch.cuda.synchronize()
    return y.cpu().numpy().astype(np.float64)


def compare(name, gpu, ref, cfg):
    err = np.abs(gpu - ref)
    rms = float(np.sqrt(np.mean(ref ** 2)))
    bar = tolerance(cfg) * max(1.0, rms)
    print(f"[parity] {name}: max_abs={err.max():.3e} mean_abs={err.mean():.3e} rms_ref={rms:.3f} "
          f"bar={bar:.1e}", flush=True)
    sys.stdout.flush()
    assert np.isfinite(gpu).all(), f"{name}: non-finite GPU output"
    assert err.max() <= bar, f"{name}: max abs error {err.max():.3e} > {bar:.3e}"
    return err.max()
