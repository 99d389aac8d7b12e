"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the
same seeded inputs.  Bars: max-abs <= tol * max(1, rms(oracle)) with tol
1e-4 (fp32 path), 2e-2 (bf16, and fp4 weights, which both sides decode
exactly), 5e-2 (fp8 weights)."""
import dataclasses
import os

import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_helpers import compare, run_gpu, small_cfg, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _expert(cfg, case, **kw):
    import paper_2608_03682_amd as px
    return px.Expert(cfg, case.weights, **kw)


def _oracle(cfg, case):
    return oracle.denoise(cfg, case.weights, case.prefix, case.prefix_len, case.noise, case.timesteps,
                          case.state)


def test_fp8_decode_all_codes_bit_exact():
    import paper_2608_03682_amd as px
    codes = torch.arange(256, dtype=torch.uint8, device="cuda")
    bits = px.fp8_to_bf16(codes).cpu().numpy().view(np.uint16)
    vals = oracle.decode_bf16(bits)
    ref = oracle.E4M3FN_TABLE
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(vals), nan)
    assert np.array_equal(vals[~nan], ref[~nan])
    assert np.array_equal(np.signbit(vals[~nan]), np.signbit(ref[~nan]))


@pytest.mark.parametrize("variant,kw", [
    ("pi0", {}),
    ("pi0", dict(head_dim=256, n_q_heads=2)),
    ("pi0", dict(weight_dtype="fp8", batch=4)),
    ("pi0", dict(batch=7)),                         # 357 rows: the tiled GEMM with a ragged row tile
    ("pi0", dict(weight_dtype="fp8", batch=7)),
    ("pi0", dict(batch=21)),                        # 1071 rows, 1050 action rows: the row-blocked
                                                    # embedding and readout, each with a partial last block
    ("pi0", dict(d_model=1024, batch=2)),           # width 1024: the four-column norm kernel
    ("pi05", {}),
    ("pi05", dict(d_model=1024)),                   # the same with adaRMS shift and compensated output
    ("dit", {}),
    ("pi0", dict(weight_dtype="f32", kv_dtype="f32", state_token=False, rope=False)),
    ("pi0", dict(weight_dtype="fp4")),              # 4-bit weights: the small-row GEMMs and the merge GEMM
    ("pi0", dict(weight_dtype="fp4", batch=7)),     # 357 rows: fp4 keeps the small-row kernels
    ("pi05", dict(weight_dtype="fp4")),
    ("dit", dict(weight_dtype="fp4")),
])
def test_small_parity(variant, kw):
    cfg = small_cfg(variant, **kw)
    print(f"[case] small {variant} {kw}", flush=True)
    case = wl.make_case(cfg, seed=3)
    ex = _expert(cfg, case)
    gpu = run_gpu(ex, case)
    compare(f"small_{variant}_{kw}", gpu, _oracle(cfg, case), cfg)


@pytest.mark.parametrize("variant,kw", [
    ("pi0", {}),
    ("pi0", dict(head_dim=256, n_q_heads=2, weight_dtype="fp8")),
    ("dit", {}),
])
def test_separate_attention_merge(variant, kw):
    """At small row counts the output projection merges the attention's key
    splits itself; PHYAI_ATTN_MERGE=kernel keeps the separate merge kernel,
    which must agree with the oracle as well."""
    cfg = small_cfg(variant, **kw)
    print(f"[case] separate merge {variant} {kw}", flush=True)
    case = wl.make_case(cfg, seed=5)
    os.environ["PHYAI_ATTN_MERGE"] = "kernel"
    try:
        ex = _expert(cfg, case)
        gpu = run_gpu(ex, case)
    finally:
        del os.environ["PHYAI_ATTN_MERGE"]
    compare(f"separate merge {variant} {kw}", gpu, _oracle(cfg, case), cfg)


@pytest.mark.parametrize("variant,kw,plen", [
    ("pi0", {}, [0, 1, 100, 64]),
    ("pi0", dict(weight_dtype="fp8"), [0, 1, 100, 64]),
    ("pi0", dict(batch=7), [0, 100, 1, 64, 63, 65, 0]),   # 357 rows: the many-row GEMMs, no key split
    ("pi05", {}, [0, 1, 100, 64]),
    ("dit", {}, [1, 40]),
])
def test_edge_prefix_lengths(variant, kw, plen):
    """Prefix lengths at the edges of the key range: none (the suffix keys
    only; a DiT request needs at least one feature row), a single key, the
    full capacity, and whole 64-key tiles with one key more or less."""
    kw = dict(kw)
    kw.setdefault("batch", len(plen))
    cfg = small_cfg(variant, **kw)
    pl = np.array(plen, np.int32)
    print(f"[case] edge prefixes {variant} {kw} {plen}", flush=True)
    case = wl.make_case(cfg, seed=6)
    case = dataclasses.replace(case, prefix_len=pl, prefix=wl.make_prefix(cfg, pl, 6))
    ex = _expert(cfg, case)
    gpu = run_gpu(ex, case)
    compare(f"edge prefixes {variant} {kw} {plen}", gpu, _oracle(cfg, case), cfg)


def test_tiny_fp32_full_config():
    cfg = wl.CONFIGS["tiny_fp32"]
    print("[case] tiny_fp32", flush=True)
    case = wl.make_case(cfg, seed=0)
    ex = _expert(cfg, case)
    compare("tiny_fp32", run_gpu(ex, case), _oracle(cfg, case), cfg)


@pytest.mark.parametrize("name", ["pi0_bf16_b1", "pi05_bf16_b1", "dit_bf16_b1", "pi0_fp4_b1"])
def test_full_size_batch1(name):
    cfg = wl.CONFIGS[name]
    print(f"[case] {name}", flush=True)
    case = wl.make_case(cfg, seed=0)
    ex = _expert(cfg, case)
    gpu = run_gpu(ex, case)
    compare(name, gpu, _oracle(cfg, case), cfg)


def test_full_size_batch64_fp8_sampled():
    """The rollout batch: all 64 requests run on the GPU in the benchmark's
    launch configuration.  The oracle runs a sample of requests live (the
    shortest and the longest prefix, plus the first and last slots) and every
    request is compared with the oracle's stored output for this workload."""
    cfg = wl.CONFIGS["pi0_fp8_b64"]
    print("[case] pi0_fp8_b64 sampled", flush=True)
    case = wl.make_case(cfg, seed=0)
    ex = _expert(cfg, case)
    gpu = run_gpu(ex, case)
    assert np.isfinite(gpu).all()
    pl = case.prefix_len
    sample = sorted({0, cfg.batch - 1, int(np.argmin(pl)), int(np.argmax(pl))})
    W = oracle.DecodedWeights(case.weights)
    pre = wl.make_prefix(cfg, pl, 0, requests=sample)
    ref = oracle.denoise(cfg, case.weights, pre, pl[sample], case.noise[sample], case.timesteps,
                         case.state[sample], decoded=W, slots=list(range(len(sample))))
    compare(f"pi0_fp8_b64 requests {sample}", gpu[sample], ref, cfg)
    # every request against the oracle's stored output (tests/golden/make_c5_expected.py,
    # which runs only the oracle on the same seeded workload)
    gold = np.load(os.path.join(os.path.dirname(__file__), "golden", "c5_expected.npz"))
    assert str(gold["config"]) == cfg.name and int(gold["seed"]) == 0
    # (equal up to BLAS summation order, which depends on the thread count)
    assert np.allclose(gold["actions"][sample], ref, rtol=0, atol=1e-9), "stored oracle output is stale"
    compare("pi0_fp8_b64 all 64 requests", gpu, gold["actions"], cfg)


@pytest.mark.parametrize("variant,kw", [
    ("pi0", {}),
    ("pi0", dict(batch=7)),
    ("dit", {}),
])
def test_attention_128_row_blocks(variant, kw):
    """Attention with four-wave, 128-row blocks and key splits (small batches
    default to two-wave, 64-row blocks; the rollout batch uses 128-row blocks
    without splits).  The switch is set after the expert is loaded, so its
    buffers were sized without it."""
    cfg = small_cfg(variant, **kw)
    print(f"[case] attention 128-row blocks {variant} {kw}", flush=True)
    case = wl.make_case(cfg, seed=8)
    ex = _expert(cfg, case)
    os.environ["PHYAI_ATTN_ROWS"] = "128"
    try:
        gpu = run_gpu(ex, case)
    finally:
        del os.environ["PHYAI_ATTN_ROWS"]
    compare(f"attention 128-row blocks {variant} {kw}", gpu, _oracle(cfg, case), cfg)


@pytest.mark.parametrize("variant,kw", [
    ("pi0", {}),
    ("pi0", dict(weight_dtype="fp8", batch=4)),
    ("pi05", {}),
])
@pytest.mark.parametrize("mt", ["2", "4"])
def test_small_row_gemm_row_blocks(variant, kw, mt):
    """The small-row GEMMs with 32- and 64-row blocks forced (the default
    picks 16-row blocks for these shapes): rows 153 and 204 leave a partial
    last block either way."""
    cfg = small_cfg(variant, **kw)
    print(f"[case] small-row blocks {mt} x 16 rows {variant} {kw}", flush=True)
    case = wl.make_case(cfg, seed=7)
    os.environ["PHYAI_SMALL_MT"] = mt
    try:
        ex = _expert(cfg, case)
        gpu = run_gpu(ex, case)
    finally:
        del os.environ["PHYAI_SMALL_MT"]
    compare(f"small-row blocks {mt} {variant} {kw}", gpu, _oracle(cfg, case), cfg)


@pytest.mark.parametrize("wdt", ["bf16", "fp8"])
@pytest.mark.parametrize("tile", ["ring", "deep", "strided"])
def test_many_row_gemm_tiles(tile, wdt):
    """Each many-row GEMM kernel, forced in turn for every projection: 357
    rows (a ragged last row tile), QKV 512 columns, GeGLU 2 x 512, output and
    down projections 256 columns.  "deep" (the four-stage ring) leaves the
    QKV projection on the two-stage ring."""
    cfg = small_cfg("pi0", n_q_heads=6, batch=7, weight_dtype=wdt)
    print(f"[case] gemm tile {tile} {wdt}", flush=True)
    case = wl.make_case(cfg, seed=4)
    os.environ["PHYAI_GEMM_TILE"] = tile
    try:
        ex = _expert(cfg, case)
        gpu = run_gpu(ex, case)
    finally:
        del os.environ["PHYAI_GEMM_TILE"]
    compare(f"gemm tile {tile} {wdt}", gpu, _oracle(cfg, case), cfg)


@pytest.mark.parametrize("wdt", ["bf16", "fp8"])
def test_many_row_split_k_residual(wdt):
    """The one-tile-per-CU ring GEMM with K split over blocks (few output
    tiles, long K): 408 rows, down projection K = 2048 over 6 tiles, split
    in two; the slices are added by the next norm and by the readout."""
    cfg = small_cfg("pi0", batch=8, d_mlp=2048, weight_dtype=wdt)
    print(f"[case] split-K residual {wdt}", flush=True)
    case = wl.make_case(cfg, seed=6)
    ex = _expert(cfg, case)
    compare(f"split-K residual {wdt}", run_gpu(ex, case), _oracle(cfg, case), cfg)


def test_fp4_scales_must_be_powers_of_two():
    """The fp4 format's scales are applied by the hardware conversion, which
    uses only their exponent: a scale that is not a power of two is refused
    at load (PHYAI_EINVAL) instead of being silently rounded."""
    import paper_2608_03682_amd as px
    cfg = small_cfg("pi0", weight_dtype="fp4", batch=1)
    case = wl.make_case(cfg, seed=3)
    w = dict(case.weights)
    t = w["layers.0.wo"]
    bad = t.scale.copy()
    bad[0, 0] *= 1.5
    w["layers.0.wo"] = dataclasses.replace(t, scale=bad)
    with pytest.raises(px.PhyaiError) as ei:
        px.Expert(cfg, w)
    assert ei.value.code == px.PHYAI_EINVAL and "power of two" in str(ei.value)


@pytest.mark.parametrize("name,kw", [
    ("pi0_b1", dict(batch=1)),
    ("pi0_b3", dict(batch=3)),
    ("pi0_fp8_b2", dict(batch=2, weight_dtype="fp8")),
    ("pi0_fp4_b1_d1024", dict(batch=1, weight_dtype="fp4", d_model=1024, n_layers=3)),
])
def test_folded_norms_match_oracle_and_norm_kernels(name, kw):
    """With PHYAI_NORM_FOLD=1, pi0 at small batch folds the RMSNorms into the
    GEMMs when every residual GEMM is split over K (here: head_dim 128, so
    that the merging output projection takes two 256-wide slices): the
    residual GEMMs finish their split-K tiles and the QKV and gate/up GEMMs
    scale rows by 1/rms; by default the separate norm kernels run.  Both
    paths against the oracle; they must differ (the fold is taken) and the
    folded path must be deterministic."""
    cfg = small_cfg("pi0", head_dim=128, **kw)
    print(f"[case] folded norms {name}", flush=True)
    case = wl.make_case(cfg, seed=12)
    ref = _oracle(cfg, case)
    # path switches are read when a graph is captured: one handle per path
    os.environ["PHYAI_NORM_FOLD"] = "1"
    try:
        ex = _expert(cfg, case)
        folded = run_gpu(ex, case)
        again = run_gpu(ex, case)
    finally:
        del os.environ["PHYAI_NORM_FOLD"]
    compare(f"folded norms {name}", folded, ref, cfg)
    assert np.array_equal(again, folded), "folded path is not deterministic"
    ex.close()
    ex2 = _expert(cfg, case)
    plain = run_gpu(ex2, case)
    ex2.close()
    compare(f"norm kernels {name}", plain, ref, cfg)
    assert not np.array_equal(folded, plain), "the two paths should differ in rounding"
