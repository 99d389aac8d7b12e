"""The vision tower (phyai_encode_images) against the oracle, through the C ABI.

Output: the image tokens [B][out_rows][d_out] (float32), rows 0 ..
n_images*n_patches-1 of each request.  Bar: the GPU keeps the residual stream
in fp32 and rounds every GEMM operand to bf16 (unit roundoff u = 2^-8); one
stage's rounding errors are random in sign, so they add in quadrature over the
L + 2 stages a token has passed (patch embedding, L blocks, projector), and
the largest error over the output stays within about six standard deviations:
max-abs <= 6 u sqrt(L + 2) max(1, rms) (0.047 at 2 blocks, 0.12 at 24).  The
same model bounds the error's rms: a rounding to nearest leaves a relative
error of rms u/sqrt(3), each stage maps it through a well-conditioned
product, and with a factor 2 for the norms and softmax in between, rms(err)
<= 2 u sqrt((L + 2) / 3) rms(ref) (0.9% at 2 blocks, 2.3% at 24).  That second
bound is the one small systematic mistakes cannot pass: in the oracle,
dropping any one residual-path bias (patch, O, MLP-out, projector) moves the
2-block tokens by 6-9% rms, a LayerNorm bias by 1.2%.  The query bias of the
synthetic weights moves them by only 0.05% (and the key bias, a per-query
constant under softmax, not at all), so one case raises the query biases to
3 and the value biases to 0.5, so that the QKV epilogue's bias path decides
the result (dropping the query biases then moves the tokens by 6%).  The fp32 path
keeps the actions' fp32 bar (1e-4 max(1, rms)).
"""
import math
import sys

import numpy as np
import pytest

import oracle
import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _px():
    import paper_2608_03682_amd as px
    return px


def vit_cfg(**kw) -> wl.ExpertConfig:
    base = dict(name="small_vit", cfg_id=70, variant="vision", n_layers=2, d_model=256, n_q_heads=4,
                n_kv_heads=4, head_dim=64, d_mlp=512, horizon=0, action_dim=0, n_steps=0, prefix_cap=0,
                prefix_min=0, prefix_max=0, batch=2, state_token=False, rope=False, weight_dtype="bf16",
                kv_dtype="bf16", time_dim=0, n_images=2, n_patches=40, patch_dim=128, d_out=96)
    base.update(kw)
    return wl.ExpertConfig(**base)


def tok_bar(cfg, ref) -> float:
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    if cfg.weight_dtype == "f32":
        return 1e-4 * max(1.0, rms)
    return 6 * 2.0 ** -8 * math.sqrt(cfg.n_layers + 2) * max(1.0, rms)


def run_encode(cfg, case, model=None, out_rows=None, sentinel=None):
    px = _px()
    m = model or px.VisionTower(cfg, case.weights, max_batch=case.patches.shape[0])
    pt = torch.from_numpy(np.ascontiguousarray(case.patches)).cuda()
    out = None
    if out_rows is not None:
        out = torch.full((pt.shape[0], out_rows, cfg.d_out), sentinel, dtype=torch.float32, device="cuda")
    out = m.encode(pt, out=out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    if model is None:
        m.close()
    return got


def check_tokens(name, cfg, got, ref):
    bar = tok_bar(cfg, ref)
    err = np.abs(got - ref)
    print(f"[parity] {name}: max_abs={err.max():.3e} mean_abs={err.mean():.3e} "
          f"rms_ref={np.sqrt(np.mean(ref ** 2)):.3f} bar={bar:.2e}", flush=True)
    sys.stdout.flush()
    assert np.isfinite(got).all(), f"{name}: non-finite output"
    assert err.max() <= bar, f"{name}: max abs error {err.max():.3e} > {bar:.2e}"
    if cfg.weight_dtype != "f32":
        rel = float(np.sqrt(np.mean(err ** 2)) / np.sqrt(np.mean(ref ** 2)))
        rel_bar = 2 * 2.0 ** -8 * math.sqrt((cfg.n_layers + 2) / 3)
        print(f"[parity] {name}: rel_rms={rel:.2e} bar={rel_bar:.2e}", flush=True)
        assert rel <= rel_bar, f"{name}: relative rms error {rel:.2e} > {rel_bar:.2e}"


SMALL = [
    # 160 rows: split-K residual GEMMs, key-split attention merged in the O
    # projection; 40 patches end mid-way through a 64-key tile
    ("bf16_small_rows", dict()),
    # 600 rows: the many-row GEMMs and attention blocks
    ("bf16_many_rows", dict(n_patches=100, n_images=3)),
    ("bf16_dh128", dict(n_q_heads=2, n_kv_heads=2, head_dim=128, n_patches=70, n_layers=3)),
    # width 1024 over 256 rows: 16 GEMM tiles, so the O and MLP-out
    # projections split K into four slices of four k-blocks
    ("bf16_wide_split_k", dict(d_model=1024, n_q_heads=16, n_kv_heads=16, d_mlp=1024, n_patches=64)),
    ("bf16_one_image_wide_patch", dict(n_images=1, n_patches=64, patch_dim=768, d_out=2048, batch=3)),
    ("fp8", dict(weight_dtype="fp8", n_patches=100)),
    ("fp4", dict(weight_dtype="fp4", n_patches=100)),
    ("f32", dict(weight_dtype="f32", kv_dtype="f32")),
]


def test_vision_large_qv_biases():
    """Query biases ~ N(0, 3^2) and value biases ~ N(0, 0.5^2): a mis-indexed
    or dropped bias in the fused QKV epilogue moves the tokens far past the
    bar."""
    cfg = vit_cfg(n_patches=100)
    print("[case] vision large q/v biases", flush=True)
    g = np.random.default_rng(51)
    ov = {f"layers.{l}.{b}": g.standard_normal((1, cfg.d_model)).astype(np.float32) * {"bq": 3.0, "bv": 0.5}[b]
          for l in range(cfg.n_layers) for b in ("bq", "bv")}
    w = wl.make_weights(cfg, 51, overrides=ov)
    case = wl.make_vision_case(cfg, seed=51, weights=w)
    got = run_encode(cfg, case)
    ref = oracle.encode_images(cfg, case.weights, case.patches)
    w0 = dict(case.weights)
    for l in range(cfg.n_layers):
        w0[f"layers.{l}.bq"] = wl.StoredTensor(w[f"layers.{l}.bq"].dtype, np.zeros_like(w[f"layers.{l}.bq"].data))
    moved = oracle.encode_images(cfg, w0, case.patches)
    # the query biases alone move the tokens far outside the rms bar
    assert np.sqrt(np.mean((moved - ref) ** 2)) > 4 * 2 * 2.0 ** -8 * math.sqrt(4 / 3) * np.sqrt(np.mean(ref ** 2))
    check_tokens("vision large q/v biases", cfg, got, ref)


@pytest.mark.parametrize("name,kw", SMALL)
def test_vision_small_parity(name, kw):
    cfg = vit_cfg(**kw)
    print(f"[case] vision {name} {kw}", flush=True)
    case = wl.make_vision_case(cfg, seed=41)
    got = run_encode(cfg, case)
    ref = oracle.encode_images(cfg, case.weights, case.patches)
    check_tokens(f"vision {name}", cfg, got, ref)


def test_vision_writes_only_its_rows_of_a_larger_slab():
    """Tokens land at rows 0 .. n_images*n_patches-1 of each request's slab
    of out_rows rows; the rows after them (the text's place in a prefix
    embedding buffer) keep what they held."""
    cfg = vit_cfg()
    print("[case] vision out_rows slab", flush=True)
    case = wl.make_vision_case(cfg, seed=43)
    n_tok = cfg.n_images * cfg.n_patches
    got = run_encode(cfg, case, out_rows=n_tok + 13, sentinel=7.25)
    ref = oracle.encode_images(cfg, case.weights, case.patches)
    check_tokens("vision slab", cfg, got[:, :n_tok], ref)
    assert (got[:, n_tok:] == 7.25).all()


def test_vision_is_deterministic_and_images_independent():
    cfg = vit_cfg(n_patches=64)
    print("[case] vision determinism / independence", flush=True)
    case = wl.make_vision_case(cfg, seed=45)
    a = run_encode(cfg, case)
    b = run_encode(cfg, case)
    assert np.array_equal(a, b)
    # other images changed (same shapes, so the same kernels and summation
    # orders): request 0's image 0 keeps every bit
    p = case.patches.copy()
    p[0, 1] += 1.0
    p[1] *= -1.0
    d = run_encode(cfg, wl.VisionCase(cfg, case.weights, p))
    N = cfg.n_patches
    assert np.array_equal(d[0, :N], a[0, :N])
    assert not np.allclose(d[0, N:], a[0, N:])


def test_vision_then_prefill_matches_the_oracle_chain():
    """The tower's tokens are the prefix LM's input rows as they stand: GPU
    encode into the embedding buffer, text rows after them, GPU prefill ->
    against oracle encode -> oracle prefill, on the K/V bar."""
    px = _px()
    from test_gpu_prefill import check_kv, plm_cfg
    vcfg = vit_cfg(d_out=256)
    n_tok = vcfg.n_images * vcfg.n_patches
    pcfg = plm_cfg(prefix_cap=n_tok + 20, prefix_min=n_tok + 5, prefix_max=n_tok + 20, batch=vcfg.batch)
    print("[case] vision -> prefill chain", flush=True)
    vcase = wl.make_vision_case(vcfg, seed=47)
    pcase = wl.make_prefill_case(pcfg, seed=47)
    plen = pcase.prefix_len
    tower = px.VisionTower(vcfg, vcase.weights)
    lm = px.PrefixLM(pcfg, pcase.weights, max_batch=vcfg.batch)
    emb = torch.from_numpy(pcase.embeds).cuda()            # text rows from n_tok on
    tower.encode(torch.from_numpy(vcase.patches).cuda(), out=emb)
    kv = lm.prefill(emb, plen)
    torch.cuda.synchronize()
    got = oracle.decode_bf16(kv.cpu().numpy().view(np.uint16)).astype(np.float64)
    ref_emb = pcase.embeds.astype(np.float64).copy()
    ref_emb[:, :n_tok] = oracle.encode_images(vcfg, vcase.weights, vcase.patches)
    ref = oracle.prefill(pcfg, pcase.weights, ref_emb, plen)
    # the tower's own error enters the LM's input: one more stage of the bar
    check_kv("vision -> prefill", pcfg.replace(n_layers=pcfg.n_layers + vcfg.n_layers + 2), got, ref, plen)
    tower.close()
    lm.close()


def test_vision_handle_and_arguments_are_checked():
    px = _px()
    cfg = vit_cfg(batch=1)
    case = wl.make_vision_case(cfg, seed=49)
    m = px.VisionTower(cfg, case.weights)
    pt = torch.from_numpy(case.patches).cuda()
    n_tok = cfg.n_images * cfg.n_patches
    out = torch.zeros((1, n_tok, cfg.d_out), dtype=torch.float32, device="cuda")
    L = px.lib()
    assert L.phyai_encode_images(m._h, pt.data_ptr(), out.data_ptr(), n_tok - 1, 1, None) == px.PHYAI_EINVAL
    assert b"out_rows" in L.phyai_last_error()
    assert L.phyai_encode_images(m._h, pt.data_ptr() + 4, out.data_ptr(), n_tok, 1, None) == px.PHYAI_EINVAL
    assert b"aligned" in L.phyai_last_error()
    assert L.phyai_encode_images(m._h, pt.data_ptr(), out.data_ptr(), n_tok, 2, None) == px.PHYAI_EINVAL
    # the other entry points refuse the handle
    ok = np.array([5], np.int32)
    assert L.phyai_prefill(m._h, pt.data_ptr(), ok.ctypes.data, out.data_ptr(), 1, None) == px.PHYAI_EINVAL
    assert L.phyai_denoise(m._h, out.data_ptr(), ok.ctypes.data, pt.data_ptr(), ok.ctypes.data, 1, 1, None,
                           pt.data_ptr(), None) == px.PHYAI_EINVAL
    assert b"vision" in L.phyai_last_error()
    torch.cuda.synchronize()
    assert not out.any().item(), "a refused call wrote its output"
    m.close()


def test_siglip_class_tower_full_size():
    """The SigLIP-class tower at full size (24 blocks of width 1024, 16 heads
    of 64, MLP 4096, three images of 256 patches of 768 values, projected to
    2048): every token against the oracle, and deterministic."""
    cfg = wl.CONFIGS["vit_siglip_bf16_b1"]
    print("[case] vision siglip full size", flush=True)
    case = wl.make_vision_case(cfg, seed=0)
    m = _px().VisionTower(cfg, case.weights)
    print("[vision] loaded", flush=True)
    got = run_encode(cfg, case, model=m)
    again = run_encode(cfg, case, model=m)
    m.close()
    assert np.array_equal(got, again)
    ref = oracle.encode_images(cfg, case.weights, case.patches)
    check_tokens("vision siglip full size", cfg, got, ref)


def test_siglip_class_tower_batch32_sampled():
    """The tower at batch 32 (96 images, 24,576 rows: the many-tile GEMM and
    attention launches): the first and last requests' tokens against the
    oracle, every token finite."""
    cfg = wl.CONFIGS["vit_siglip_bf16_b32"]
    print("[case] vision siglip batch 32", flush=True)
    w = wl.make_weights(cfg, 0)
    patches = wl.make_patches(cfg, 0)
    m = _px().VisionTower(cfg, w)
    got = run_encode(cfg, wl.VisionCase(cfg, w, patches), model=m)
    m.close()
    assert np.isfinite(got).all()
    for b in (0, cfg.batch - 1):
        ref = oracle.encode_images(cfg, w, patches[b:b + 1])
        check_tokens(f"vision siglip batch 32 request {b}", cfg, got[b:b + 1], ref)


def test_vision_prefill_denoise_chain():
    """The whole observation-to-action path at small sizes, every phase on the
    GPU (tower -> prefix LM -> expert), against the oracle's chain; the
    actions on their own bar."""
    px = _px()
    from gpu_helpers import compare, small_cfg
    from test_gpu_prefill import plm_cfg
    ecfg = small_cfg("pi0")
    vcfg = vit_cfg(n_images=2, n_patches=30, batch=ecfg.batch, d_out=512)
    n_tok = vcfg.n_images * vcfg.n_patches
    pcfg = plm_cfg(n_layers=ecfg.n_layers, n_kv_heads=ecfg.n_kv_heads, head_dim=ecfg.head_dim,
                   prefix_cap=ecfg.prefix_cap, prefix_min=n_tok + 1, prefix_max=ecfg.prefix_cap,
                   batch=ecfg.batch, d_model=512, n_q_heads=8, d_mlp=1024)
    print("[case] vision -> prefill -> denoise chain", flush=True)
    vcase = wl.make_vision_case(vcfg, seed=53)
    pcase = wl.make_prefill_case(pcfg, seed=53)
    ecase = wl.make_case(ecfg, seed=53)
    plen = pcase.prefix_len
    tower = px.VisionTower(vcfg, vcase.weights)
    lm = px.PrefixLM(pcfg, pcase.weights, max_batch=ecfg.batch)
    ex = px.Expert(ecfg, ecase.weights)
    emb = torch.from_numpy(pcase.embeds).cuda()
    tower.encode(torch.from_numpy(vcase.patches).cuda(), out=emb)
    kv = lm.prefill(emb, plen)
    y = ex.denoise(kv, plen, torch.from_numpy(ecase.noise).cuda(), ecase.timesteps,
                   torch.from_numpy(ecase.state).cuda())
    torch.cuda.synchronize()
    got = y.cpu().numpy().astype(np.float64)
    ref_emb = pcase.embeds.astype(np.float64).copy()
    ref_emb[:, :n_tok] = oracle.encode_images(vcfg, vcase.weights, vcase.patches)
    ref_kv = oracle.prefill(pcfg, pcase.weights, ref_emb, plen)
    stored = wl.bf16_bits_from_f32(ref_kv.astype(np.float32))
    ref = oracle.denoise(ecfg, ecase.weights, stored, plen, ecase.noise, ecase.timesteps, ecase.state)
    compare("vision -> prefill -> denoise", got, ref, ecfg)
    tower.close()
    lm.close()
    ex.close()
