"""The oracle for the prefix K/V producer: the vision-language model's
language part run over the prefix tokens, in plain float64 NumPy.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code
with the HIP library and imports nothing from it.

What is computed (PhyAI, arXiv 2608.03682):
  * For the pi-family the observation (images and the instruction) is
    encoded once per chunk into the prefix, whose per-layer K/V tensors the
    action expert then reads at every denoising step (Section "PhyAI
    Architecture", paragraph "Graph replay").  The paper's phase analysis
    times the vision tower, the language prefix and the action expert
    separately (Section "Evaluation", batch analysis); this module is the
    language-prefix phase.
  * The input is the prefix token embeddings (the vision tower's projected
    image tokens followed by the text embeddings); the output is, for every
    layer, the keys and values of every prefix token, in the layout the
    expert reads: [L][2][B][P_cap][n_kv * d_h].

Where the paper is silent this oracle takes the public Gemma-style
language model the pi-family uses, with the same readings as the expert:
pre-norm blocks with RMSNorm gain (1 + w) and eps from the config; fused
q/k/v projections without bias; RoPE (half-split) on queries and keys at
positions 0 .. prefix_len-1; the prefix tokens attend to one another
bidirectionally (a prefix-LM block: every valid prefix token sees every
valid prefix token); scale 1/sqrt(d_h); GeGLU MLP gelu_tanh(n W_gate) *
(n W_up) then W_down; residual adds.  The embeddings arrive already scaled.
Layer l's K/V depend only on the input of layer l, so the last layer stops
after its K/V projection.  Rows at or beyond prefix_len[b] are zero.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np

from .numerics import attention, decode_stored, gelu_tanh, rms_normalize, rope


def prefill_request(cfg, weights: Dict[str, object], x: np.ndarray, n_layers: Optional[int] = None,
                    dtype=np.float64) -> np.ndarray:
    """K/V of one request's prefix.  x: [n, d] embeddings of its n valid
    tokens.  Returns [L', 2, n, n_kv * d_h] for the first L' = n_layers
    layers (default all)."""
    L = cfg.n_layers if n_layers is None else n_layers
    nq, nkv, D = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    n = x.shape[0]
    cache: Dict[str, np.ndarray] = {}

    def W(name):
        if name not in cache:
            cache[name] = decode_stored(weights[name]).astype(dtype, copy=False)
        return cache[name]

    out = np.zeros((L, 2, n, nkv * D), dtype=dtype)
    h = np.asarray(x, dtype=dtype)
    pos = np.arange(n)
    allowed = np.ones((n, n), dtype=bool)
    for l in range(L):
        p = f"layers.{l}."
        a = rms_normalize(h, cfg.rms_eps) * (1.0 + W(p + "attn_norm")[0])
        q = (a @ W(p + "wq")).reshape(n, nq, D)
        k = (a @ W(p + "wk")).reshape(n, nkv, D)
        v = (a @ W(p + "wv")).reshape(n, nkv, D)
        if cfg.rope:
            q = rope(q, pos, cfg.rope_base)
            k = rope(k, pos, cfg.rope_base)
        out[l, 0] = k.reshape(n, nkv * D)
        out[l, 1] = v.reshape(n, nkv * D)
        if l + 1 == cfg.n_layers or l + 1 == L:
            break
        if n > 0:
            o = attention(q, k, v, allowed)
            h = h + o.reshape(n, nq * D) @ W(p + "wo")
        m = rms_normalize(h, cfg.rms_eps) * (1.0 + W(p + "mlp_norm")[0])
        h = h + (gelu_tanh(m @ W(p + "w_gate")) * (m @ W(p + "w_up"))) @ W(p + "w_down")
    return out


def prefill(cfg, weights: Dict[str, object], embeds: np.ndarray, prefix_len: Sequence[int],
            n_layers: Optional[int] = None, dtype=np.float64) -> np.ndarray:
    """The prefix K/V cache of a batch: [L'][2][B][P_cap][n_kv * d_h] (float64;
    rows at or beyond prefix_len[b] zero).  embeds: [B][P_cap][d]; rows past
    prefix_len[b] are never read."""
    B = len(prefix_len)
    L = cfg.n_layers if n_layers is None else n_layers
    out = np.zeros((L, 2, B, cfg.prefix_cap, cfg.n_kv_heads * cfg.head_dim), dtype=dtype)
    for b in range(B):
        n = int(prefix_len[b])
        out[:, :, b, :n] = prefill_request(cfg, weights, np.asarray(embeds[b, :n]), L, dtype)
    return out
