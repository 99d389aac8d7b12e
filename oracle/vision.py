"""The oracle for the vision tower: the image encoder that turns each
request's camera images into the image tokens at the head of the prefix, in
plain float64 NumPy.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code
with the HIP library and imports nothing from it.

What is computed (PhyAI, arXiv 2608.03682):
  * The pi-family encodes the observation once per chunk: the vision tower,
    then the language prefix, whose K/V the action expert reads at every
    step (Section "PhyAI Architecture", the runner's per-chunk flow).  The
    paper's phase analysis times these three phases separately and reports
    vision as about a third of the time at batch 32 (Section "Evaluation",
    batch analysis); this module is the vision phase.
  * Input: per request, n_images images, each already cut into n_patches
    patches of patch_dim normalised pixel values (the patchify step is the
    preprocessing outside the online path).  Output: per request, the
    n_images * n_patches image tokens of width d_out, image-major, ready to
    be the first rows of the language model's prefix embeddings.

The paper names no architecture for the tower; this oracle takes a
SigLIP-class vision transformer (the pi-family's image encoder family):
  * patch embedding: a linear map of each patch plus a bias, plus a learned
    position embedding per patch index (no class token);
  * pre-norm blocks: LayerNorm (gain stored as its deviation from one, the
    (1 + w) convention of the other norms here, plus a bias; eps from the
    config), multi-head self-attention with biased q/k/v/o projections over
    the patches of one image only (every patch sees every patch of its own
    image, no positions beyond the learned embedding, scale 1/sqrt(d_h)),
    residual add; LayerNorm, MLP W2 gelu_tanh(W1 a + b1) + b2, residual add;
  * a final LayerNorm, then a linear projector (with bias) to the language
    model's width d_out.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np

from .numerics import attention, decode_stored, gelu_tanh, layer_normalize


class _Weights:
    """Decoded weights, each decoded once (stored formats -> float64)."""

    def __init__(self, stored: Dict[str, object], dtype=np.float64):
        self._stored, self._dtype, self._cache = stored, dtype, {}

    def __call__(self, name: str) -> np.ndarray:
        if name not in self._cache:
            self._cache[name] = decode_stored(self._stored[name]).astype(self._dtype, copy=False)
        return self._cache[name]

    def vec(self, name: str) -> np.ndarray:
        return self(name)[0]


def _layer_norm(W: _Weights, h: np.ndarray, wname: str, bname: str, eps: float) -> np.ndarray:
    return layer_normalize(h, eps) * (1.0 + W.vec(wname)) + W.vec(bname)


def encode_image(cfg, W: _Weights, patches: np.ndarray, n_layers: Optional[int] = None) -> np.ndarray:
    """One image: patches [n_patches, patch_dim] -> tokens [n_patches, d_out].
    ``n_layers`` runs only the first blocks (default all) before the final
    norm and projector."""
    L = cfg.n_layers if n_layers is None else n_layers
    H, D, eps = cfg.n_q_heads, cfg.head_dim, cfg.rms_eps
    n = patches.shape[0]
    h = patches @ W("patch_w") + W.vec("patch_b") + W("pos_emb")[:n]
    everyone = np.ones((n, n), dtype=bool)
    for l in range(L):
        p = f"layers.{l}."
        a = _layer_norm(W, h, p + "ln1_w", p + "ln1_b", eps)
        q = (a @ W(p + "wq") + W.vec(p + "bq")).reshape(n, H, D)
        k = (a @ W(p + "wk") + W.vec(p + "bk")).reshape(n, H, D)
        v = (a @ W(p + "wv") + W.vec(p + "bv")).reshape(n, H, D)
        o = attention(q, k, v, everyone).reshape(n, H * D)
        h = h + o @ W(p + "wo") + W.vec(p + "bo")
        m = _layer_norm(W, h, p + "ln2_w", p + "ln2_b", eps)
        h = h + gelu_tanh(m @ W(p + "mlp_w1") + W.vec(p + "mlp_b1")) @ W(p + "mlp_w2") + W.vec(p + "mlp_b2")
    z = _layer_norm(W, h, "post_ln_w", "post_ln_b", eps)
    return z @ W("proj_w") + W.vec("proj_b")


def encode_images(cfg, weights: Dict[str, object], patches: np.ndarray, n_layers: Optional[int] = None,
                  dtype=np.float64) -> np.ndarray:
    """A batch: patches [B][n_images][n_patches][patch_dim] -> image tokens
    [B][n_images * n_patches][d_out] (float64), image-major."""
    W = _Weights(weights, dtype)
    B, I, N = patches.shape[:3]
    out = np.empty((B, I * N, cfg.d_out), dtype=dtype)
    for b in range(B):
        for i in range(I):
            out[b, i * N:(i + 1) * N] = encode_image(cfg, W, np.asarray(patches[b, i], dtype=dtype), n_layers)
    return out
