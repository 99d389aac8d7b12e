"""The oracle: the action-expert denoising loop in plain float64 NumPy.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code
with the HIP library and imports nothing from it.

What is computed (PhyAI, arXiv 2608.03682):
  * A policy request maps an observation to an H-action chunk by refining an
    action latent over several steps (Section "Embodied Task Formulation",
    subsection "From Observation to Action", the equation a = pi(x)).
  * For the pi-family the refinement is a fixed number of Euler steps of a
    flow-matching velocity field; the vision-language prefix is computed once
    per chunk and its K/V tensors stay fixed across the steps, while only the
    action tokens change (paragraph "Graph replay").
  * The velocity field is a compact action expert: a transformer over the
    action tokens whose attention reads the frozen prefix K/V and the action
    tokens' own K/V (paragraph "Profiled operator selection": 50 action-token
    queries against a longer prefix with head dimension 256), built from
    RMSNorm / AdaRMSNorm, one QKV projection, a gate+up projection with the
    GeGLU activation, and residual adds (paragraph "Kernel fusion").
  * Timestep dependence enters through a sinusoidal timestep table and, for
    pi0.5, per-layer AdaRMS modulation (paragraph "Graph replay").
  * Batches are independent requests (Section "Cloud Batching", throughput
    Q(B) = B / T_sync(B)); each request has its own prefix and noise.

The paper does not print the expert's layer equations.  Where it is silent
this oracle takes the public pi0 / pi0.5 / DiT designs it cites, as follows:
  * Gemma-style pre-norm blocks; RMSNorm gain is (1 + w); eps = 1e-6; input
    embeddings are not rescaled by sqrt(d).
  * pi0: action token u = W2 swish(W1 [W_in x + b_in ; tau(t)] + b1) + b2; an
    optional state token W_s s + b_s is prepended.  Block attention mask:
    the state token sees the prefix and itself; action tokens see the
    prefix, the state token and every action token.
  * pi0.5: action token W_in x + b_in; condition c = swish(W_c2 swish(W_c1
    tau(t) + b_c1) + b_c2); every norm is h / rms(h) * (1 + scale) + shift
    with [scale; shift] = c W_mod + b_mod; no residual gate.
  * RoPE (half-split, base 1e4) on suffix queries and keys at positions
    P_b + i; the prefix keys arrive already rotated.
  * Attention scale 1/sqrt(d_h), fp64 softmax, no soft-cap.
  * Readout from the last H suffix tokens: v = W_out norm(h) + b_out.
  * Trunk projections (q, k, v, o, gate, up, down) have no bias; the input,
    time, state, modulation and output projections do.
  * DiT head: c = W_c2 SiLU(W_c1 tau_256(t) + b_c1) + b_c2; per block
    [sh1, sc1, g1, sh2, sc2, g2] = SiLU(c) W_ada + b_ada; LayerNorm without
    affine; even blocks cross-attend to the projected VLM features, odd
    blocks self-attend over all tokens (no mask, no RoPE); GELU(tanh) MLP
    with biases; final (shift, scale) modulation before the readout; action
    tokens carry a learned position embedding.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np

from .numerics import (attention, decode_stored, euler, gelu_tanh, layer_normalize,
                       rms_normalize, rope, sinusoid, swish)


class DecodedWeights:
    """float64 view of the stored weights (decoded once).  dtype=float32 gives
    the timing-only single-precision mode (the decode is exact in float64,
    then rounded once to float32)."""

    def __init__(self, stored: Dict[str, object], dtype=np.float64):
        self.dtype = np.dtype(dtype)
        self.w = {k: decode_stored(v).astype(dtype, copy=False) for k, v in stored.items()}

    def __getitem__(self, k):
        return self.w[k]

    def vec(self, k):
        return self.w[k][0]


def _prefix_rows(cfg, prefix: np.ndarray, i: int, P: int, l: int):
    """Frozen K and V of request slot i at layer l: [P, n_kv, d_h] each."""
    k = np.asarray(prefix[l, 0, i, :P], dtype=np.float64)
    v = np.asarray(prefix[l, 1, i, :P], dtype=np.float64)
    sh = (P, cfg.n_kv_heads, cfg.head_dim)
    return k.reshape(sh), v.reshape(sh)


def _suffix_mask(cfg) -> np.ndarray:
    """allowed[i, j] between suffix tokens (block mask, see module doc)."""
    M = cfg.tokens
    if not cfg.state_token:
        return np.ones((M, M), dtype=bool)
    blk = np.array([1] + [2] * cfg.horizon)
    return blk[None, :] <= blk[:, None]


def _trunk(cfg, W: DecodedWeights, h: np.ndarray, P: int, kv_rows, norm_fn) -> np.ndarray:
    """The L pre-norm transformer blocks of the pi0 / pi0.5 expert.

    norm_fn(site, h) returns the normalised activations for norm site
    ('attn', l) or ('mlp', l)."""
    M = h.shape[0]
    nq, nkv, D = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    pos = P + np.arange(M)
    allowed = np.concatenate([np.ones((M, P), dtype=bool), _suffix_mask(cfg)], axis=1)
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        n = norm_fn(("attn", l), h)
        q = (n @ W[p + "wq"]).reshape(M, nq, D)
        k = (n @ W[p + "wk"]).reshape(M, nkv, D)
        v = (n @ W[p + "wv"]).reshape(M, nkv, D)
        if cfg.rope:
            q = rope(q, pos, cfg.rope_base)
            k = rope(k, pos, cfg.rope_base)
        kp, vp = kv_rows(l)
        o = attention(q, np.concatenate([kp, k]), np.concatenate([vp, v]), allowed)
        h = h + o.reshape(M, nq * D) @ W[p + "wo"]
        n = norm_fn(("mlp", l), h)
        h = h + (gelu_tanh(n @ W[p + "w_gate"]) * (n @ W[p + "w_up"])) @ W[p + "w_down"]
    return h


def velocity_pi0(cfg, W: DecodedWeights, x, t, kv_rows, P, state=None) -> np.ndarray:
    """pi0 expert velocity v(x, t) for one request.  x: [H, A]."""
    d = cfg.d_model
    a = x @ W["in_w"] + W.vec("in_b")
    tau = sinusoid(t, cfg.time_dim, cfg.sin_min_period, cfg.sin_max_period).astype(W.dtype)
    z = np.concatenate([a, np.broadcast_to(tau, (a.shape[0], cfg.time_dim))], axis=1)
    u = swish(z @ W["time_w1"] + W.vec("time_b1")) @ W["time_w2"] + W.vec("time_b2")
    if cfg.state_token:
        e = np.concatenate([(state @ W["state_w"] + W.vec("state_b"))[None, :], u])
    else:
        e = u

    def norm_fn(site, h):
        kind, l = site
        w = W.vec(f"layers.{l}.{kind}_norm")
        return rms_normalize(h, cfg.rms_eps) * (1.0 + w)

    h = _trunk(cfg, W, e, P, kv_rows, norm_fn)
    n = rms_normalize(h, cfg.rms_eps) * (1.0 + W.vec("final_norm"))
    off = 1 if cfg.state_token else 0
    assert n.shape[1] == d
    return n[off:] @ W["out_w"] + W.vec("out_b")


def pi05_condition(cfg, W: DecodedWeights, t) -> np.ndarray:
    tau = sinusoid(t, cfg.time_dim, cfg.sin_min_period, cfg.sin_max_period).astype(W.dtype)
    return swish(swish(tau @ W["cond_w1"] + W.vec("cond_b1")) @ W["cond_w2"] + W.vec("cond_b2"))


def velocity_pi05(cfg, W: DecodedWeights, x, t, kv_rows, P, state=None) -> np.ndarray:
    """pi0.5 expert velocity: adaRMSNorm conditioning in every norm."""
    d = cfg.d_model
    e = x @ W["in_w"] + W.vec("in_b")
    c = pi05_condition(cfg, W, t)

    def ada(h, wname, bname):
        mod = c @ W[wname] + W.vec(bname)
        scale, shift = mod[:d], mod[d:]
        return rms_normalize(h, cfg.rms_eps) * (1.0 + scale) + shift

    def norm_fn(site, h):
        kind, l = site
        return ada(h, f"layers.{l}.{kind}_mod_w", f"layers.{l}.{kind}_mod_b")

    h = _trunk(cfg, W, e, P, kv_rows, norm_fn)
    n = ada(h, "final_mod_w", "final_mod_b")
    return n @ W["out_w"] + W.vec("out_b")


def velocity_dit(cfg, W: DecodedWeights, x, t, feats, P, state=None) -> np.ndarray:
    """DiT action-head velocity.  feats: [P, d_feat] VLM features."""
    d, nh, D = cfg.d_model, cfg.n_q_heads, cfg.head_dim
    tau = sinusoid(t, cfg.time_dim, cfg.sin_min_period, cfg.sin_max_period).astype(W.dtype)
    c = swish(tau @ W["cond_w1"] + W.vec("cond_b1")) @ W["cond_w2"] + W.vec("cond_b2")
    sc = swish(c)
    act = x @ W["in_w"] + W.vec("in_b") + W["pos_emb"]
    h = np.concatenate([(state @ W["state_w"] + W.vec("state_b"))[None, :], act])
    M = h.shape[0]
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        ada = sc @ W[p + "ada_w"] + W.vec(p + "ada_b")
        sh1, sc1, g1, sh2, sc2, g2 = (ada[i * d:(i + 1) * d] for i in range(6))
        xh = layer_normalize(h, cfg.rms_eps) * (1.0 + sc1) + sh1
        q = (xh @ W[p + "wq"]).reshape(M, nh, D)
        src = feats if l % 2 == 0 else xh
        k = (src @ W[p + "wk"]).reshape(src.shape[0], cfg.n_kv_heads, D)
        v = (src @ W[p + "wv"]).reshape(src.shape[0], cfg.n_kv_heads, D)
        o = attention(q, k, v, np.ones((M, src.shape[0]), dtype=bool))
        h = h + g1 * (o.reshape(M, nh * D) @ W[p + "wo"])
        xh = layer_normalize(h, cfg.rms_eps) * (1.0 + sc2) + sh2
        h = h + g2 * (gelu_tanh(xh @ W[p + "mlp_w1"] + W.vec(p + "mlp_b1")) @ W[p + "mlp_w2"]
                      + W.vec(p + "mlp_b2"))
    fin = sc @ W["final_ada_w"] + W.vec("final_ada_b")
    shf, scf = fin[:d], fin[d:]
    n = layer_normalize(h, cfg.rms_eps) * (1.0 + scf) + shf
    return n[1:] @ W["out_w"] + W.vec("out_b")


_VELOCITY = {"pi0": velocity_pi0, "pi05": velocity_pi05, "dit": velocity_dit}


def denoise(cfg, weights, prefix: np.ndarray, prefix_len: Sequence[int], noise: np.ndarray,
            timesteps, state: Optional[np.ndarray] = None, decoded: Optional[DecodedWeights] = None,
            slots: Optional[Sequence[int]] = None, dtype=np.float64) -> np.ndarray:
    """Run the K-step denoising loop for each request.

    prefix: the prefix buffer in the library's layout ([L][2][B][P_cap][n_kv*d_h]
    K/V for pi0/pi0.5, [B][P_cap][d_feat] features for DiT), already decoded to
    float or still in its stored bits (uint16 bf16 bits are decoded here).
    prefix_len[b], noise[b], state[b] belong to request b.  ``slots`` maps
    request b to its slot in ``prefix`` (default: identity), so a subset of a
    large batch can be checked without materialising the rest.
    ``dtype`` float64 is the parity reference; float32 runs the same steps in
    single precision (a CPU timing baseline only, never a parity reference).
    Returns x_K: [B, H, A] in ``dtype``.
    """
    from .numerics import decode_bf16
    W = decoded if decoded is not None else DecodedWeights(weights, dtype)
    vel = _VELOCITY[cfg.variant]
    B = noise.shape[0]
    out = np.empty(noise.shape, dtype=dtype)
    pre = (decode_bf16(prefix) if prefix.dtype == np.uint16 else np.asarray(prefix, np.float64)).astype(
        dtype, copy=False)
    for b in range(B):
        i = b if slots is None else slots[b]
        P = int(prefix_len[b])
        s = None if state is None else np.asarray(state[b], dtype)
        if cfg.variant == "dit":
            ctx = pre[i, :P]
        else:
            def ctx(l, i=i, P=P):
                return _prefix_rows(cfg, pre, i, P, l)
        out[b] = euler(lambda x, t: vel(cfg, W, x, t, ctx, P, s), noise[b], timesteps, dtype)
    return out
