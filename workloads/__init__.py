"""Seeded synthetic workloads for the action-expert denoising loop.

This module is shared by the tests, the benchmark and the oracle's callers.
It holds shapes, seeds and storage formats only: none of the expert's
arithmetic lives here.  Every tensor is drawn from its own counter-keyed
PCG64 stream, so a single request's inputs can be regenerated without
generating the whole batch.

Storage formats produced here (what the library and the oracle consume):
  * ``f32``  -- float32 values.
  * ``bf16`` -- uint16 bit patterns, rounded to nearest-even from float32.
  * ``fp8``  -- uint8 OCP e4m3fn codes plus one float32 scale per output
               column (round-to-nearest weight quantisation, as in the
               paper's offline RTN quantiser, Section "Optimization Methods",
               paragraph "Quantization").
  * ``fp4``  -- 4-bit weights (the paper's W4A16): OCP e2m1 codes, two per
               byte along the output dimension (even column in the low
               nibble), with one power-of-two float32 scale per group of 32
               input rows and output column, chosen so that no code
               saturates; codes are the round-to-nearest (ties to even)
               e2m1 values of W / scale.

Linear weights are stored ``[in][out]`` (``y = x @ W + b``).
"""
from __future__ import annotations

import dataclasses
import zlib
from typing import Dict, Optional

import numpy as np

__all__ = [
    "ExpertConfig", "CONFIGS", "StoredTensor", "weight_specs", "make_weights",
    "make_prefix", "make_prefix_lengths", "make_noise", "make_state",
    "default_timesteps", "make_case", "bf16_bits_from_f32", "e4m3fn_encode",
    "quantize_fp8_per_column", "e2m1_encode", "quantize_fp4_groups", "FP4_GROUP", "TRUNK_LINEARS",
    "make_prefix_embeds", "PrefillCase", "make_prefill_case", "make_patches", "VisionCase", "make_vision_case",
]


@dataclasses.dataclass(frozen=True)
class ExpertConfig:
    """Shape and format of one expert workload.

    variant: ``pi0`` (time mixed into action tokens by an MLP), ``pi05``
    (adaRMSNorm time conditioning) or ``dit`` (DiT head with adaLN-zero,
    alternating cross/self attention); ``prefix_lm`` is the vision-language
    model's language part run over the prefix tokens, which produces the
    prefix K/V an expert reads (horizon, action_dim and n_steps are 0);
    ``vision`` is the vision tower that turns each request's image patches
    into the image tokens at the head of that prefix (n_images images of
    n_patches patches of patch_dim values each, tokens of width d_out).
    """
    name: str
    cfg_id: int
    variant: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_mlp: int
    horizon: int
    action_dim: int
    n_steps: int
    prefix_cap: int           # rows reserved per request in the prefix buffer
    prefix_min: int           # ragged prefix lengths drawn uniform in [min, max]
    prefix_max: int
    batch: int
    state_token: bool
    rope: bool
    weight_dtype: str         # f32 | bf16 | fp8 | fp4
    kv_dtype: str             # f32 | bf16
    d_feat: int = 0           # DiT: width of the VLM feature tokens
    time_dim: int = 0         # width of the sinusoidal timestep embedding
    rms_eps: float = 1e-6
    sin_min_period: float = 4e-3
    sin_max_period: float = 4.0
    rope_base: float = 10000.0
    init_std: float = 0.02
    n_images: int = 0         # vision: images per request
    n_patches: int = 0        # vision: patches (tokens) per image
    patch_dim: int = 0        # vision: values per patch
    d_out: int = 0            # vision: width of the projected image tokens

    @property
    def tokens(self) -> int:
        """Suffix tokens per request (state token, if any, plus actions)."""
        return self.horizon + (1 if self.state_token else 0)

    @property
    def ragged(self) -> bool:
        return self.prefix_min != self.prefix_max

    @property
    def prefix_width(self) -> int:
        """Columns of one prefix row: n_kv*head_dim, or d_feat for DiT."""
        return self.d_feat if self.variant == "dit" else self.n_kv_heads * self.head_dim

    def replace(self, **kw) -> "ExpertConfig":
        return dataclasses.replace(self, **kw)


def _cfg(**kw) -> ExpertConfig:
    kw.setdefault("time_dim", kw["d_model"])
    return ExpertConfig(**kw)


# The five workloads: a tiny fp32 expert, the pi0-shaped expert at batch 1,
# the pi0.5-shaped expert (adaRMSNorm), a DiT-style action head, and the
# pi0-shaped expert at rollout batch 64 with ragged prefixes and fp8 weights;
# plus the batch-1 pi0 shape with 4-bit weights.
CONFIGS: Dict[str, ExpertConfig] = {
    "tiny_fp32": _cfg(
        name="tiny_fp32", cfg_id=1, variant="pi0", n_layers=2, d_model=256,
        n_q_heads=4, n_kv_heads=1, head_dim=64, d_mlp=1024, horizon=16,
        action_dim=7, n_steps=4, prefix_cap=64, prefix_min=64, prefix_max=64,
        batch=1, state_token=False, rope=False, weight_dtype="f32", kv_dtype="f32"),
    "pi0_bf16_b1": _cfg(
        name="pi0_bf16_b1", cfg_id=2, variant="pi0", n_layers=18, d_model=1024,
        n_q_heads=8, n_kv_heads=1, head_dim=256, d_mlp=4096, horizon=50,
        action_dim=32, n_steps=10, prefix_cap=816, prefix_min=816, prefix_max=816,
        batch=1, state_token=True, rope=True, weight_dtype="bf16", kv_dtype="bf16"),
    "pi05_bf16_b1": _cfg(
        name="pi05_bf16_b1", cfg_id=3, variant="pi05", n_layers=18, d_model=1024,
        n_q_heads=8, n_kv_heads=1, head_dim=256, d_mlp=4096, horizon=50,
        action_dim=32, n_steps=10, prefix_cap=968, prefix_min=968, prefix_max=968,
        batch=1, state_token=False, rope=True, weight_dtype="bf16", kv_dtype="bf16"),
    "dit_bf16_b1": _cfg(
        name="dit_bf16_b1", cfg_id=4, variant="dit", n_layers=16, d_model=1536,
        n_q_heads=12, n_kv_heads=12, head_dim=128, d_mlp=6144, horizon=16,
        action_dim=32, n_steps=4, prefix_cap=300, prefix_min=300, prefix_max=300,
        batch=1, state_token=True, rope=False, weight_dtype="bf16", kv_dtype="bf16",
        d_feat=2048, time_dim=256),
    "pi0_fp8_b64": _cfg(
        name="pi0_fp8_b64", cfg_id=5, variant="pi0", n_layers=18, d_model=1024,
        n_q_heads=8, n_kv_heads=1, head_dim=256, d_mlp=4096, horizon=50,
        action_dim=32, n_steps=10, prefix_cap=1000, prefix_min=600, prefix_max=1000,
        batch=64, state_token=True, rope=True, weight_dtype="fp8", kv_dtype="bf16"),
    # the pi0-shaped expert at batch 1 with 4-bit weights (the paper's W4A16
    # quantised path): the trunk linears in fp4, everything else as C2
    "pi0_fp4_b1": _cfg(
        name="pi0_fp4_b1", cfg_id=6, variant="pi0", n_layers=18, d_model=1024,
        n_q_heads=8, n_kv_heads=1, head_dim=256, d_mlp=4096, horizon=50,
        action_dim=32, n_steps=10, prefix_cap=816, prefix_min=816, prefix_max=816,
        batch=1, state_token=True, rope=True, weight_dtype="fp4", kv_dtype="bf16"),
    # The language part of the vision-language model over the prefix tokens
    # (image tokens and text), producing the prefix K/V the expert reads: a
    # tiny fp32 one whose output fits the tiny expert, and a Gemma-class one
    # (18 layers of width 2048, 8 query heads and one K/V head of 256, GeGLU
    # MLP 16384) over the pi0 prefix of 816 tokens, whose output fits the
    # pi0-shaped expert.
    "plm_tiny_fp32": _cfg(
        name="plm_tiny_fp32", cfg_id=7, variant="prefix_lm", n_layers=2, d_model=256,
        n_q_heads=4, n_kv_heads=1, head_dim=64, d_mlp=1024, horizon=0,
        action_dim=0, n_steps=0, prefix_cap=64, prefix_min=64, prefix_max=64,
        batch=1, state_token=False, rope=True, weight_dtype="f32", kv_dtype="f32", time_dim=0),
    # The vision tower before it: a SigLIP-L/16-class ViT (24 layers of width
    # 1024, 16 heads of 64, GELU MLP 4096, LayerNorm, biases everywhere) over 3
    # images of 256 patches of 16 x 16 x 3 values, whose tokens are projected
    # to the Gemma-class LM's width 2048.
    "vit_siglip_bf16_b1": _cfg(
        name="vit_siglip_bf16_b1", cfg_id=9, variant="vision", n_layers=24, d_model=1024,
        n_q_heads=16, n_kv_heads=16, head_dim=64, d_mlp=4096, horizon=0,
        action_dim=0, n_steps=0, prefix_cap=768, prefix_min=768, prefix_max=768,
        batch=1, state_token=False, rope=False, weight_dtype="bf16", kv_dtype="bf16", time_dim=0,
        n_images=3, n_patches=256, patch_dim=768, d_out=2048),
    # the same tower at batch 32, the batch of the paper's phase analysis (96 images)
    "vit_siglip_bf16_b32": _cfg(
        name="vit_siglip_bf16_b32", cfg_id=10, variant="vision", n_layers=24, d_model=1024,
        n_q_heads=16, n_kv_heads=16, head_dim=64, d_mlp=4096, horizon=0,
        action_dim=0, n_steps=0, prefix_cap=768, prefix_min=768, prefix_max=768,
        batch=32, state_token=False, rope=False, weight_dtype="bf16", kv_dtype="bf16", time_dim=0,
        n_images=3, n_patches=256, patch_dim=768, d_out=2048),
    "plm_gemma_bf16_b1": _cfg(
        name="plm_gemma_bf16_b1", cfg_id=8, variant="prefix_lm", n_layers=18, d_model=2048,
        n_q_heads=8, n_kv_heads=1, head_dim=256, d_mlp=16384, horizon=0,
        action_dim=0, n_steps=0, prefix_cap=816, prefix_min=816, prefix_max=816,
        batch=1, state_token=False, rope=True, weight_dtype="bf16", kv_dtype="bf16", time_dim=0),
}

# Per-layer linears that carry the fp8 / fp4 format when weight_dtype is one of those.
TRUNK_LINEARS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down", "mlp_w1", "mlp_w2")


@dataclasses.dataclass
class StoredTensor:
    dtype: str                 # f32 | bf16 | fp8 | fp4
    data: np.ndarray           # float32 | uint16 | uint8, shape [rows][cols] (fp4: [rows][cols / 2])
    scale: Optional[np.ndarray] = None   # fp8: float32 [cols]; fp4: float32 [rows / 32][cols]

    @property
    def rows(self) -> int:
        return int(self.data.shape[0])

    @property
    def cols(self) -> int:
        return int(self.data.shape[1]) * (2 if self.dtype == "fp4" else 1)


# ----------------------------------------------------------------------------
# Storage-format conversions (input preparation, pinned against torch's casts)
# ----------------------------------------------------------------------------

def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    out = (rounded >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = np.uint16(0x7FC0)
    return out


def e4m3fn_encode(v: np.ndarray) -> np.ndarray:
    """Encode float values as OCP e4m3fn codes: saturate to +-448, then round
    to nearest with ties to even.  (No NaN/inf inputs.)

    With a = |v| in the binade [2^E, 2^(E+1)) (E clamped below at -6, where
    the subnormals share the quantum of the lowest binade), the representable
    values are n * 2^(E-3); n = rint(a / 2^(E-3)) lies in [8, 16] for normals
    (n = 16 is the next binade) and in [0, 8] below 2^-6, and in every case
    the code is 8*E + 48 + n."""
    v = np.asarray(v, dtype=np.float32)
    sign = np.signbit(v)
    a = np.minimum(np.abs(v), np.float32(448.0))
    _, e = np.frexp(a)                                  # a = m * 2^e, m in [0.5, 1)
    E = np.maximum(np.where(a > 0, e - 1, -6), -6).astype(np.int32)
    n = np.rint(np.ldexp(a, 3 - E)).astype(np.int32)   # exact scaling by a power of two
    code = 8 * E + 48 + n
    return (code | (sign.astype(np.int32) << 7)).astype(np.uint8)


def quantize_fp8_per_column(w: np.ndarray):
    """Round-to-nearest fp8 weight quantisation with one scale per output column.

    scale_j = max_i |W_ij| / 448 (1 for an all-zero column); codes encode
    W_ij / scale_j.  Returns (codes uint8 [rows][cols], scales float32 [cols]).
    """
    w = np.asarray(w, dtype=np.float32)
    amax = np.abs(w).max(axis=0).astype(np.float32)
    scale = np.where(amax > 0, amax / np.float32(448.0), np.float32(1.0)).astype(np.float32)
    codes = e4m3fn_encode(w / scale[None, :])
    return codes, scale


FP4_GROUP = 32          # input rows sharing one fp4 scale


def e2m1_encode(v: np.ndarray) -> np.ndarray:
    """Encode float values (|v| <= 6) as OCP e2m1 codes, round to nearest with
    ties to even.  The non-negative values are the multiples of 0.5 up to 2,
    of 1 up to 4 and 6 (codes 0..7: 0, 0.5, 1, 1.5, 2, 3, 4, 6); the sign is
    bit 3.  With a = |v| the quantum is 0.5 below 2, 1 in [2, 4) and 2 in
    [4, 6], so a / quantum rounded to even gives the value, and the code
    follows from the value by the ordering above."""
    v = np.asarray(v, dtype=np.float64)
    a = np.abs(v)
    q = np.where(a < 2.0, 0.5, np.where(a < 4.0, 1.0, 2.0))
    val = np.rint(a / q) * q                      # numpy rint rounds ties to even
    # rounding up across a binade boundary lands on the boundary value, which
    # the table below holds
    table = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])
    code = np.searchsorted(table, val).astype(np.uint8)
    assert np.all(table[code] == val), "value outside the e2m1 grid"
    return (code | (np.signbit(v).astype(np.uint8) << 3)).astype(np.uint8)


def quantize_fp4_groups(w: np.ndarray):
    """Round-to-nearest 4-bit weight quantisation (W4A16): for each group of
    FP4_GROUP input rows and each output column, scale = 2^ceil(log2(amax / 6))
    (1 for an all-zero group), so |W / scale| <= 6 and no code saturates; the
    codes are the e2m1 encodings of W / scale.  Returns (packed codes uint8
    [rows][cols / 2], even column in the low nibble; scales float32
    [rows / FP4_GROUP][cols])."""
    w = np.asarray(w, dtype=np.float32)
    rows, cols = w.shape
    assert rows % FP4_GROUP == 0 and cols % 2 == 0
    g = w.reshape(rows // FP4_GROUP, FP4_GROUP, cols)
    amax = np.abs(g).max(axis=1).astype(np.float64)
    e = np.where(amax > 0, np.ceil(np.log2(np.where(amax > 0, amax, 1.0) / 6.0)), 0.0)
    scale = np.ldexp(1.0, e.astype(np.int32)).astype(np.float32)
    # an amax just above a power of two times 6 can round log2 down: bump the
    # exponent until the group fits
    while True:
        over = amax > 6.0 * scale.astype(np.float64)
        if not over.any():
            break
        scale = np.where(over, scale * np.float32(2.0), scale).astype(np.float32)
    codes = e2m1_encode(g / scale[:, None, :].astype(np.float64)).reshape(rows, cols)
    packed = (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)
    return packed, scale


# ----------------------------------------------------------------------------
# Parameter inventory
# ----------------------------------------------------------------------------

def weight_specs(cfg: ExpertConfig) -> Dict[str, tuple]:
    """Name -> (rows, cols) of every parameter, in a fixed order.

    Vectors (biases, norm weights) are stored as one row.
    """
    d, A, F = cfg.d_model, cfg.action_dim, cfg.d_mlp
    qd = cfg.n_q_heads * cfg.head_dim
    kd = cfg.n_kv_heads * cfg.head_dim
    s: Dict[str, tuple] = {}
    if cfg.variant == "vision":
        # LayerNorm scales are stored as their deviation from one (the (1 + w)
        # convention of the norms elsewhere here)
        s["patch_w"] = (cfg.patch_dim, d)
        s["patch_b"] = (1, d)
        s["pos_emb"] = (cfg.n_patches, d)
        for l in range(cfg.n_layers):
            p = f"layers.{l}."
            s[p + "ln1_w"] = (1, d)
            s[p + "ln1_b"] = (1, d)
            for nm in ("wq", "wk", "wv"):
                s[p + nm] = (d, d)
                s[p + "b" + nm[1]] = (1, d)
            s[p + "wo"] = (d, d)
            s[p + "bo"] = (1, d)
            s[p + "ln2_w"] = (1, d)
            s[p + "ln2_b"] = (1, d)
            s[p + "mlp_w1"] = (d, F)
            s[p + "mlp_b1"] = (1, F)
            s[p + "mlp_w2"] = (F, d)
            s[p + "mlp_b2"] = (1, d)
        s["post_ln_w"] = (1, d)
        s["post_ln_b"] = (1, d)
        s["proj_w"] = (d, cfg.d_out)
        s["proj_b"] = (1, cfg.d_out)
        return s
    if cfg.variant == "prefix_lm":
        # the last layer's K/V depend only on its input: its output
        # projection and MLP are never needed and not listed
        for l in range(cfg.n_layers):
            p = f"layers.{l}."
            s[p + "attn_norm"] = (1, d)
            s[p + "wq"] = (d, qd)
            s[p + "wk"] = (d, kd)
            s[p + "wv"] = (d, kd)
            if l + 1 < cfg.n_layers:
                s[p + "wo"] = (qd, d)
                s[p + "mlp_norm"] = (1, d)
                s[p + "w_gate"] = (d, F)
                s[p + "w_up"] = (d, F)
                s[p + "w_down"] = (F, d)
        return s
    s["in_w"] = (A, d)
    s["in_b"] = (1, d)
    if cfg.variant == "pi0":
        s["time_w1"] = (d + cfg.time_dim, d)
        s["time_b1"] = (1, d)
        s["time_w2"] = (d, d)
        s["time_b2"] = (1, d)
    else:
        s["cond_w1"] = (cfg.time_dim, d)
        s["cond_b1"] = (1, d)
        s["cond_w2"] = (d, d)
        s["cond_b2"] = (1, d)
    if cfg.state_token:
        s["state_w"] = (A, d)
        s["state_b"] = (1, d)
    if cfg.variant == "dit":
        s["pos_emb"] = (cfg.horizon, d)
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        if cfg.variant == "pi0":
            s[p + "attn_norm"] = (1, d)
        elif cfg.variant == "pi05":
            s[p + "attn_mod_w"] = (d, 2 * d)
            s[p + "attn_mod_b"] = (1, 2 * d)
        else:
            s[p + "ada_w"] = (d, 6 * d)
            s[p + "ada_b"] = (1, 6 * d)
        s[p + "wq"] = (d, qd)
        kin = cfg.d_feat if (cfg.variant == "dit" and l % 2 == 0) else d
        s[p + "wk"] = (kin, kd)
        s[p + "wv"] = (kin, kd)
        s[p + "wo"] = (qd, d)
        if cfg.variant == "pi0":
            s[p + "mlp_norm"] = (1, d)
        elif cfg.variant == "pi05":
            s[p + "mlp_mod_w"] = (d, 2 * d)
            s[p + "mlp_mod_b"] = (1, 2 * d)
        if cfg.variant == "dit":
            s[p + "mlp_w1"] = (d, F)
            s[p + "mlp_b1"] = (1, F)
            s[p + "mlp_w2"] = (F, d)
            s[p + "mlp_b2"] = (1, d)
        else:
            s[p + "w_gate"] = (d, F)
            s[p + "w_up"] = (d, F)
            s[p + "w_down"] = (F, d)
    if cfg.variant == "pi0":
        s["final_norm"] = (1, d)
    elif cfg.variant == "pi05":
        s["final_mod_w"] = (d, 2 * d)
        s["final_mod_b"] = (1, 2 * d)
    else:
        s["final_ada_w"] = (d, 2 * d)
        s["final_ada_b"] = (1, 2 * d)
    s["out_w"] = (d, A)
    s["out_b"] = (1, A)
    return s


def storage_dtype(cfg: ExpertConfig, name: str) -> str:
    if cfg.weight_dtype in ("fp8", "fp4"):
        leaf = name.rsplit(".", 1)[-1]
        return cfg.weight_dtype if (name.startswith("layers.") and leaf in TRUNK_LINEARS) else "bf16"
    return cfg.weight_dtype


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def _store(x: np.ndarray, dtype: str) -> StoredTensor:
    if dtype == "f32":
        return StoredTensor("f32", np.ascontiguousarray(x, dtype=np.float32))
    if dtype == "bf16":
        return StoredTensor("bf16", bf16_bits_from_f32(x))
    if dtype == "fp4":
        codes, scale = quantize_fp4_groups(x)
        return StoredTensor("fp4", codes, scale)
    codes, scale = quantize_fp8_per_column(x)
    return StoredTensor("fp8", codes, scale)


def make_weights(cfg: ExpertConfig, seed: int = 0,
                 overrides: Optional[Dict[str, np.ndarray]] = None) -> Dict[str, StoredTensor]:
    """Every parameter ~ N(0, init_std) in float32, then stored in the config's
    format.  ``overrides`` replaces named float32 masters before storage (used
    by tests that zero or plant specific weights)."""
    overrides = overrides or {}
    specs = weight_specs(cfg)

    def one(name):
        r, c = specs[name]
        if name in overrides:
            x = np.asarray(overrides[name], dtype=np.float32).reshape(r, c)
        else:
            g = _rng(seed, cfg.cfg_id, 0, zlib.crc32(name.encode()))
            x = g.standard_normal((r, c), dtype=np.float32) * np.float32(cfg.init_std)
        return _store(x, storage_dtype(cfg, name))

    # each tensor has its own stream, so the order of generation does not
    # matter; NumPy's generators and array kernels release the GIL
    from concurrent.futures import ThreadPoolExecutor
    import os
    with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
        stored = list(ex.map(one, specs))
    return dict(zip(specs, stored))


def make_prefix_lengths(cfg: ExpertConfig, seed: int = 0, batch: Optional[int] = None) -> np.ndarray:
    B = cfg.batch if batch is None else batch
    if not cfg.ragged:
        return np.full(B, cfg.prefix_max, dtype=np.int32)
    g = _rng(seed, cfg.cfg_id, 5)
    return g.integers(cfg.prefix_min, cfg.prefix_max + 1, size=B).astype(np.int32)


def _prefix_block(cfg, seed, l, kv, b, n):
    g = _rng(seed, cfg.cfg_id, 1, l, kv, b)
    return g.standard_normal((n, cfg.prefix_width), dtype=np.float32)


def make_prefix(cfg: ExpertConfig, prefix_len: np.ndarray, seed: int = 0,
                requests=None, pad_value: float = 0.0) -> np.ndarray:
    """Prefix buffer for the requests listed (default: all).

    pi0/pi0.5: the frozen prefix K/V cache, layout [L][2][B][P_cap][n_kv*d_h].
    DiT: the VLM feature tokens, layout [B][P_cap][d_feat].
    Valid rows ~ N(0, 1); rows at or beyond prefix_len[b] hold ``pad_value``.
    Returns uint16 bf16 bits or float32 according to kv_dtype.
    """
    reqs = list(range(len(prefix_len))) if requests is None else list(requests)
    P, W = cfg.prefix_cap, cfg.prefix_width
    bf = cfg.kv_dtype == "bf16"
    dt = np.uint16 if bf else np.float32
    if cfg.variant == "dit":
        buf = np.empty((len(reqs), P, W), dtype=dt)
    else:
        buf = np.empty((cfg.n_layers, 2, len(reqs), P, W), dtype=dt)
    pad = bf16_bits_from_f32(np.float32([pad_value]))[0] if bf else np.float32(pad_value)
    for i, b in enumerate(reqs):
        n = int(prefix_len[b])
        if cfg.variant == "dit":
            blk = _prefix_block(cfg, seed, 0, 0, b, n)
            buf[i, :n] = bf16_bits_from_f32(blk) if bf else blk
            buf[i, n:] = pad
        else:
            for l in range(cfg.n_layers):
                for kv in range(2):
                    blk = _prefix_block(cfg, seed, l, kv, b, n)
                    buf[l, kv, i, :n] = bf16_bits_from_f32(blk) if bf else blk
                    buf[l, kv, i, n:] = pad
    return buf


def make_prefix_embeds(cfg: ExpertConfig, prefix_len: np.ndarray, seed: int = 0,
                       requests=None, pad_value: float = 0.0) -> np.ndarray:
    """Input of a prefix LM: the prefix token embeddings, float32
    [B][P_cap][d_model]; valid rows ~ N(0, 1), rows at or beyond
    prefix_len[b] hold ``pad_value``."""
    reqs = list(range(len(prefix_len))) if requests is None else list(requests)
    out = np.empty((len(reqs), cfg.prefix_cap, cfg.d_model), dtype=np.float32)
    for i, b in enumerate(reqs):
        n = int(prefix_len[b])
        out[i, :n] = _rng(seed, cfg.cfg_id, 6, b).standard_normal((n, cfg.d_model), dtype=np.float32)
        out[i, n:] = pad_value
    return out


def make_noise(cfg: ExpertConfig, seed: int = 0, requests=None, batch=None) -> np.ndarray:
    B = cfg.batch if batch is None else batch
    reqs = list(range(B)) if requests is None else list(requests)
    out = np.empty((len(reqs), cfg.horizon, cfg.action_dim), dtype=np.float32)
    for i, b in enumerate(reqs):
        out[i] = _rng(seed, cfg.cfg_id, 3, b).standard_normal(
            (cfg.horizon, cfg.action_dim), dtype=np.float32)
    return out


def make_state(cfg: ExpertConfig, seed: int = 0, requests=None, batch=None) -> Optional[np.ndarray]:
    if not cfg.state_token:
        return None
    B = cfg.batch if batch is None else batch
    reqs = list(range(B)) if requests is None else list(requests)
    out = np.empty((len(reqs), cfg.action_dim), dtype=np.float32)
    for i, b in enumerate(reqs):
        out[i] = _rng(seed, cfg.cfg_id, 4, b).standard_normal(cfg.action_dim, dtype=np.float32)
    return out


def default_timesteps(n_steps: int) -> np.ndarray:
    """Uniform schedule t_k = 1 - k/K, k = 0..K (from noise at t=1 to t=0)."""
    return (1.0 - np.arange(n_steps + 1, dtype=np.float64) / n_steps).astype(np.float32)


@dataclasses.dataclass
class Case:
    cfg: ExpertConfig
    weights: Dict[str, StoredTensor]
    prefix: np.ndarray
    prefix_len: np.ndarray
    noise: np.ndarray
    state: Optional[np.ndarray]
    timesteps: np.ndarray


def make_case(cfg: ExpertConfig, seed: int = 0, batch: Optional[int] = None,
              weights: Optional[Dict[str, StoredTensor]] = None) -> Case:
    B = cfg.batch if batch is None else batch
    plen = make_prefix_lengths(cfg, seed, B)
    return Case(cfg=cfg,
                weights=weights if weights is not None else make_weights(cfg, seed),
                prefix=make_prefix(cfg, plen, seed),
                prefix_len=plen,
                noise=make_noise(cfg, seed, batch=B),
                state=make_state(cfg, seed, batch=B),
                timesteps=default_timesteps(cfg.n_steps))


@dataclasses.dataclass
class PrefillCase:
    cfg: ExpertConfig
    weights: Dict[str, StoredTensor]
    embeds: np.ndarray
    prefix_len: np.ndarray


def make_prefill_case(cfg: ExpertConfig, seed: int = 0, batch: Optional[int] = None,
                      weights: Optional[Dict[str, StoredTensor]] = None) -> PrefillCase:
    B = cfg.batch if batch is None else batch
    plen = make_prefix_lengths(cfg, seed, B)
    return PrefillCase(cfg=cfg,
                       weights=weights if weights is not None else make_weights(cfg, seed),
                       embeds=make_prefix_embeds(cfg, plen, seed),
                       prefix_len=plen)


def make_patches(cfg: ExpertConfig, seed: int = 0, batch: Optional[int] = None, requests=None) -> np.ndarray:
    """Input of a vision tower: normalised pixel patches ~ N(0, 1), float32
    [B][n_images][n_patches][patch_dim]."""
    B = cfg.batch if batch is None else batch
    reqs = list(range(B)) if requests is None else list(requests)
    out = np.empty((len(reqs), cfg.n_images, cfg.n_patches, cfg.patch_dim), dtype=np.float32)
    for i, b in enumerate(reqs):
        out[i] = _rng(seed, cfg.cfg_id, 7, b).standard_normal(out.shape[1:], dtype=np.float32)
    return out


@dataclasses.dataclass
class VisionCase:
    cfg: ExpertConfig
    weights: Dict[str, StoredTensor]
    patches: np.ndarray


def make_vision_case(cfg: ExpertConfig, seed: int = 0, batch: Optional[int] = None,
                     weights: Optional[Dict[str, StoredTensor]] = None) -> VisionCase:
    return VisionCase(cfg=cfg, weights=weights if weights is not None else make_weights(cfg, seed),
                      patches=make_patches(cfg, seed, batch))
