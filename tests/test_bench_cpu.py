"""The benchmark's host-side contract and accounting, CPU only.

The roofline fields of the bench line divide algorithmic bytes or FLOPs by a
measured time; these tests tie the accounting functions to an independent
enumeration (the workload's own tensor shapes), check the traffic figures'
source-digest gate, and the one-GPU refusal of `--gpus N`.
"""
import os
import subprocess
import sys

import numpy as np
import pytest

import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _matrices(cfg):
    """(name, rows, cols) of every weight matrix of a workload (vectors and
    the position table excluded)."""
    return [(n, r, c) for n, (r, c) in wl.weight_specs(cfg).items() if r > 1 and n != "pos_emb"]


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_chunk_bytes_counts_the_trunk_weights_and_prefix_once_per_step():
    cfg = wl.CONFIGS["pi0_bf16_b1"]
    plen = 816
    trunk = sum(r * c for n, r, c in _matrices(cfg) if n.startswith("layers."))
    kv = cfg.n_layers * plen * 2 * cfg.n_kv_heads * cfg.head_dim
    # per step: bf16 trunk weights and prefix K/V, the action in/out
    # projections and the time MLP's action half and second layer
    small = 2 * cfg.action_dim * cfg.d_model + 2 * cfg.d_model * cfg.d_model
    io = cfg.horizon * cfg.action_dim * 4 * 2 + cfg.action_dim * 4
    want = cfg.n_steps * 2 * (trunk + kv + small) + io
    got = bench.chunk_bytes(cfg, 1, plen)
    assert got == want
    # 10 steps of 18 layers of bf16 trunk weights and 816-row prefix K/V: 6.42 GB per chunk
    assert abs(got / 6.42e9 - 1) < 0.005


def test_vision_flops_are_the_gemms_of_the_weight_shapes_plus_attention():
    cfg = wl.CONFIGS["vit_siglip_bf16_b1"]
    rows = cfg.n_images * cfg.n_patches
    gemm = sum(2 * rows * r * c for n, r, c in _matrices(cfg))
    attn = cfg.n_layers * cfg.n_images * 4 * cfg.n_patches ** 2 * cfg.n_q_heads * cfg.head_dim
    assert bench.vision_flops(cfg, 1) == gemm + attn
    assert bench.vision_flops(cfg, 32) == 32 * (gemm + attn)


def test_prefill_flops_are_the_gemms_of_the_weight_shapes_plus_attention():
    cfg = wl.CONFIGS["plm_gemma_bf16_b1"]
    plen = np.array([816])
    gemm = sum(2 * 816 * r * c for n, r, c in _matrices(cfg))
    attn = (cfg.n_layers - 1) * 4 * 816 ** 2 * cfg.n_q_heads * cfg.head_dim
    assert bench.prefill_flops(cfg, plen) == gemm + attn


def test_traffic_is_reported_only_for_the_sources_it_was_measured_on(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("int f() { return 1; }  // a comment\n\n/* block */\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    digest = bench.code_digest(("k.hip",))
    monkeypatch.setitem(bench.MEASURED_TRAFFIC, ("w", "s"), {"bytes": 123, "sources": ("k.hip",), "sha256": digest})
    assert bench.measured_traffic("w", "s") == 123
    # comments and blank lines do not retire a measurement
    src.write_text("int f() { return 1; }  // another comment\n")
    assert bench.measured_traffic("w", "s") == 123
    # a code change does
    src.write_text("int f() { return 2; }\n")
    assert bench.measured_traffic("w", "s") is None
    assert bench.measured_traffic("w", "unknown stage") is None
