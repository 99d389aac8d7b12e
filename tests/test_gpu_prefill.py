"""The prefix LM (phyai_prefill) against the oracle, through the C ABI.

The output is the prefix K/V cache [L][2][B][P_cap][n_kv*d_h].  Bar: the
GPU keeps the residual stream in fp32 and rounds every GEMM operand and the
output to bf16 (unit roundoff u = 2^-8); one layer's rounding errors are
random in sign, so they add in quadrature over the L + 1 rounding stages a
cache entry has passed (its own output rounding included), and the largest
error over the cache stays within about six standard deviations: max-abs <=
6 u sqrt(L + 1) max(1, rms) (0.041 at 2 layers, 0.10 at 18).  The fp32 path
keeps the actions' fp32 bar (1e-4).  Fed into the expert, the cache must give
actions within the actions' own bar
(test_prefill_then_denoise_matches_the_oracle_chain).
"""
import ctypes
import math
import sys

import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_helpers import compare, small_cfg

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _px():
    import paper_2608_03682_amd as px
    return px


def plm_cfg(**kw) -> wl.ExpertConfig:
    base = dict(name="small_plm", cfg_id=60, variant="prefix_lm", n_layers=2, d_model=256, n_q_heads=4,
                n_kv_heads=1, head_dim=64, d_mlp=512, horizon=0, action_dim=0, n_steps=0, prefix_cap=100,
                prefix_min=37, prefix_max=100, batch=3, state_token=False, rope=True, weight_dtype="bf16",
                kv_dtype="bf16", time_dim=0)
    base.update(kw)
    return wl.ExpertConfig(**base)


def kv_bar(cfg, ref) -> float:
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    if cfg.weight_dtype == "f32":
        return 1e-4 * max(1.0, rms)
    return 6 * 2.0 ** -8 * math.sqrt(cfg.n_layers + 1) * max(1.0, rms)


def run_prefill(cfg, case, batch=None, model=None):
    px = _px()
    m = model or px.PrefixLM(cfg, case.weights, max_batch=batch or len(case.prefix_len))
    emb = torch.from_numpy(np.ascontiguousarray(case.embeds)).cuda()
    out = m.prefill(emb, case.prefix_len)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    if model is None:
        m.close()
    if got.dtype == np.int16:
        got = oracle.decode_bf16(got.view(np.uint16))
    return got.astype(np.float64)


def check_kv(name, cfg, got, ref, plen):
    bar = kv_bar(cfg, ref)
    err = np.abs(got - ref)
    print(f"[parity] {name}: max_abs={err.max():.3e} mean_abs={err.mean():.3e} "
          f"rms_ref={np.sqrt(np.mean(ref ** 2)):.3f} bar={bar:.2e}", flush=True)
    sys.stdout.flush()
    assert np.isfinite(got).all(), f"{name}: non-finite output"
    for b, n in enumerate(plen):
        assert not got[:, :, b, n:].any(), f"{name}: request {b} rows past its prefix are not zero"
    assert err.max() <= bar, f"{name}: max abs error {err.max():.3e} > {bar:.2e}"


SMALL = [
    ("bf16_dh64_ragged3", dict()),
    ("bf16_dh256_mqa", dict(head_dim=256, n_q_heads=2, d_model=512, prefix_cap=130, prefix_min=70,
                            prefix_max=130, batch=2)),
    ("bf16_dh128_gqa", dict(head_dim=128, n_q_heads=4, n_kv_heads=2, n_layers=3)),
    ("bf16_no_rope", dict(rope=False)),
    # fewer than 256 rows: split-K residual GEMMs, key-split attention merged
    # in the output projection
    ("bf16_small_rows", dict(prefix_cap=40, prefix_min=40, prefix_max=40, batch=1, n_layers=3)),
    # many rows, a long-K down projection over few tiles: K split over blocks
    ("bf16_split_k_down", dict(d_mlp=2048)),
    ("fp8_split_k_down", dict(d_mlp=2048, weight_dtype="fp8")),
    # more than 1,024 query rows per request: 128-row attention blocks with key
    # splits and their merge kernel, ragged prefixes ending mid-tile
    ("bf16_long_queries_ragged", dict(head_dim=256, n_q_heads=4, d_model=512, prefix_cap=300, prefix_min=270,
                                      prefix_max=300, batch=3)),
    ("fp8", dict(weight_dtype="fp8")),
    ("fp4", dict(weight_dtype="fp4")),
    ("f32", dict(weight_dtype="f32", kv_dtype="f32")),
]


@pytest.mark.parametrize("name,kw", SMALL)
def test_prefill_small_parity(name, kw):
    cfg = plm_cfg(**kw)
    print(f"[case] prefill {name} {kw}", flush=True)
    case = wl.make_prefill_case(cfg, seed=31)
    got = run_prefill(cfg, case)
    ref = oracle.prefill(cfg, case.weights, case.embeds, case.prefix_len)
    check_kv(f"prefill {name}", cfg, got, ref, case.prefix_len)


@pytest.mark.parametrize("plen", [0, 1, 63, 64, 65, 100])
def test_prefill_edge_prefix_lengths(plen):
    """An empty prefix, one token, lengths at the edges of a 64-key tile, the
    full capacity; NaN in every row past the prefix must not be read."""
    cfg = plm_cfg(batch=1)
    print(f"[case] prefill prefix {plen}", flush=True)
    pl = np.array([plen], np.int32)
    case = wl.PrefillCase(cfg, wl.make_weights(cfg, 33), wl.make_prefix_embeds(cfg, pl, 33, pad_value=np.nan), pl)
    got = run_prefill(cfg, case)
    ref = oracle.prefill(cfg, case.weights, case.embeds, case.prefix_len)
    check_kv(f"prefill prefix {plen}", cfg, got, ref, pl)


def test_prefill_is_deterministic_and_requests_independent():
    cfg = plm_cfg(batch=3)
    print("[case] prefill determinism / independence", flush=True)
    case = wl.make_prefill_case(cfg, seed=35)
    a = run_prefill(cfg, case)
    b = run_prefill(cfg, case)
    assert np.array_equal(a, b)
    # the others' embeddings changed: request 1's cache keeps every bit (same
    # shapes, so the same kernels and summation orders)
    emb = case.embeds.copy()
    emb[0] += 1.0
    emb[2] *= -1.0
    d = run_prefill(cfg, wl.PrefillCase(cfg, case.weights, emb, case.prefix_len))
    assert np.array_equal(d[:, :, 1], a[:, :, 1])


def test_prefill_then_denoise_matches_the_oracle_chain():
    """The cache the prefix LM writes is the expert's prefix argument as it
    stands: GPU prefill -> GPU denoise against oracle prefill -> oracle
    denoise, on the actions' own bar."""
    px = _px()
    ecfg = small_cfg("pi0")
    pcfg = plm_cfg(n_layers=ecfg.n_layers, n_kv_heads=ecfg.n_kv_heads, head_dim=ecfg.head_dim,
                   prefix_cap=ecfg.prefix_cap, batch=ecfg.batch, d_model=512, n_q_heads=8, d_mlp=1024)
    print("[case] prefill -> denoise chain", flush=True)
    pcase = wl.make_prefill_case(pcfg, seed=37)
    ecase = wl.make_case(ecfg, seed=37)
    plen = pcase.prefix_len
    # the expert runs on the LM's cache: on the GPU straight from its output
    lm = px.PrefixLM(pcfg, pcase.weights, max_batch=ecfg.batch)
    emb = torch.from_numpy(pcase.embeds).cuda()
    kv = lm.prefill(emb, plen)
    ex = px.Expert(ecfg, ecase.weights)
    noise = torch.from_numpy(ecase.noise).cuda()
    state = torch.from_numpy(ecase.state).cuda()
    y = ex.denoise(kv, plen, noise, ecase.timesteps, state)
    torch.cuda.synchronize()
    got = y.cpu().numpy().astype(np.float64)
    # the oracle chain: its own cache, rounded to the cache's storage format
    ref_kv = oracle.prefill(pcfg, pcase.weights, pcase.embeds, plen)
    stored = wl.bf16_bits_from_f32(ref_kv.astype(np.float32))
    ref = oracle.denoise(ecfg, ecase.weights, stored, plen, ecase.noise, ecase.timesteps, ecase.state)
    compare("prefill -> denoise", got, ref, ecfg)
    lm.close()
    ex.close()


def test_prefix_lm_handle_and_arguments_are_checked():
    px = _px()
    cfg = plm_cfg(batch=1)
    case = wl.make_prefill_case(cfg, seed=39)
    m = px.PrefixLM(cfg, case.weights)
    emb = torch.from_numpy(case.embeds).cuda()
    out = torch.zeros((cfg.n_layers, 2, 1, cfg.prefix_cap, cfg.head_dim), dtype=torch.int16, device="cuda")
    L = px.lib()
    big = np.array([cfg.prefix_cap + 1], np.int32)
    assert L.phyai_prefill(m._h, emb.data_ptr(), big.ctypes.data, out.data_ptr(), 1, None) == px.PHYAI_EINVAL
    ok = np.array([5], np.int32)
    assert L.phyai_prefill(m._h, emb.data_ptr() + 4, ok.ctypes.data, out.data_ptr(), 1, None) == px.PHYAI_EINVAL
    assert b"aligned" in L.phyai_last_error()
    assert L.phyai_prefill(m._h, emb.data_ptr(), ok.ctypes.data, out.data_ptr(), 2, None) == px.PHYAI_EINVAL
    # the denoising entry points refuse the handle
    assert L.phyai_denoise(m._h, out.data_ptr(), ok.ctypes.data, emb.data_ptr(), ok.ctypes.data, 1, 1, None,
                           emb.data_ptr(), None) == px.PHYAI_EINVAL
    assert b"prefix-LM" in L.phyai_last_error()
    torch.cuda.synchronize()
    assert not out.any().item(), "a refused call wrote its output"
    m.close()


def test_gemma_prefill_full_size():
    """The Gemma-class prefix LM over the pi0 prefix of 816 tokens (18
    layers, width 2048, MLP 16384): the first two layers' K/V against the
    oracle element by element (layer l depends only on layers below it), and
    every layer finite and deterministic."""
    cfg = wl.CONFIGS["plm_gemma_bf16_b1"]
    print("[case] prefill gemma full size", flush=True)
    case = wl.make_prefill_case(cfg, seed=0)
    m = _px().PrefixLM(cfg, case.weights)
    print("[prefill] loaded", flush=True)
    got = run_prefill(cfg, case, model=m)
    again = run_prefill(cfg, case, model=m)
    m.close()
    assert np.isfinite(got).all()
    assert np.array_equal(got, again)
    ref = oracle.prefill(cfg, case.weights, case.embeds, case.prefix_len, n_layers=2)
    check_kv("prefill gemma layers 0-1", cfg.replace(n_layers=2), got[:2], ref, case.prefix_len)
    rms = np.sqrt(np.mean(got ** 2, axis=(1, 2, 3, 4)))
    print("[prefill] per-layer K/V rms:", np.round(rms, 3), flush=True)
