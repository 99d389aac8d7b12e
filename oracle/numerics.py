"""Scalar building blocks of the oracle, in float64.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this package; the product path
(the HIP library and its binding) never does.

Each function is the plain textbook definition of one operation.  The paper
(PhyAI, arXiv 2608.03682) names the operations -- RMSNorm and AdaRMSNorm,
the GeGLU activation, the sinusoidal timestep table, attention of action
tokens against a frozen prefix -- in Section "PhyAI Architecture", subsection
"Optimization Methods" (paragraphs "Kernel fusion", "Graph replay",
"Profiled operator selection", "Quantization"), but does not print their
constants; the constants used here are those of the public pi0 design the
paper cites and are stated next to each function.
"""
from __future__ import annotations

import math

import numpy as np


# ----------------------------------------------------------------------------
# Storage decoders (exact)
# ----------------------------------------------------------------------------

def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float64 (exact: bf16 is the top half of f32)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):
        return u.view(np.float32).astype(np.float64)


def _e4m3fn_value(code: int) -> float:
    """Value of one OCP FP8 E4M3FN code: 1 sign, 4 exponent (bias 7), 3 mantissa
    bits; exponent field 0 is subnormal (m/8 * 2^-6); S.1111.111 is NaN; there
    are no infinities."""
    s = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        return float("nan")
    if e == 0:
        return s * (m / 8.0) * 2.0 ** -6
    return s * (1.0 + m / 8.0) * 2.0 ** (e - 7)


E4M3FN_TABLE = np.array([_e4m3fn_value(c) for c in range(256)], dtype=np.float64)


def decode_fp8(codes: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """W_ij = value(code_ij) * scale_j (one scale per output column), the
    weight format of round-to-nearest W8 quantisation (paragraph
    "Quantization")."""
    return E4M3FN_TABLE[np.asarray(codes, dtype=np.uint8)] * np.asarray(scale, np.float64)[None, :]


def _e2m1_value(code: int) -> float:
    """Value of one OCP FP4 E2M1 code: 1 sign, 2 exponent (bias 1), 1 mantissa
    bit; exponent field 0 is subnormal (m/2); no infinities or NaN."""
    s = -1.0 if code & 0x8 else 1.0
    e = (code >> 1) & 0x3
    m = code & 0x1
    if e == 0:
        return s * m / 2.0
    return s * (1.0 + m / 2.0) * 2.0 ** (e - 1)


E2M1_TABLE = np.array([_e2m1_value(c) for c in range(16)], dtype=np.float64)
FP4_GROUP = 32


def decode_fp4(packed: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """4-bit weights (paragraph "Quantization", W4A16): byte (i, j) of `packed`
    holds the codes of columns 2j (low nibble) and 2j + 1 (high nibble) of row
    i; W_ij = value(code_ij) * scale[i / 32][j]."""
    packed = np.asarray(packed, dtype=np.uint8)
    rows = packed.shape[0]
    codes = np.empty((rows, packed.shape[1] * 2), dtype=np.uint8)
    codes[:, 0::2] = packed & 0xF
    codes[:, 1::2] = packed >> 4
    sc = np.repeat(np.asarray(scale, np.float64), FP4_GROUP, axis=0)
    return E2M1_TABLE[codes] * sc


def decode_stored(t) -> np.ndarray:
    """Decode a stored tensor (dtype, data[, scale]) to float64."""
    if t.dtype == "f32":
        return np.asarray(t.data, dtype=np.float64)
    if t.dtype == "bf16":
        return decode_bf16(t.data)
    if t.dtype == "fp8":
        return decode_fp8(t.data, t.scale)
    if t.dtype == "fp4":
        return decode_fp4(t.data, t.scale)
    raise ValueError(f"unknown storage dtype {t.dtype!r}")


# ----------------------------------------------------------------------------
# Elementwise / row-wise operations
# ----------------------------------------------------------------------------

def sinusoid(t: float, n: int, min_period: float, max_period: float) -> np.ndarray:
    """Sinusoidal timestep embedding of width n (the "sinusoidal timestep
    table" of paragraph "Graph replay").  Periods are geometric from
    min_period to max_period over the n/2 frequencies; the sine block comes
    first, then the cosine block."""
    half = n // 2
    frac = np.arange(half, dtype=np.float64) / (half - 1)
    period = min_period * (max_period / min_period) ** frac
    ang = 2.0 * math.pi * float(t) / period
    return np.concatenate([np.sin(ang), np.cos(ang)])


def rms_normalize(h: np.ndarray, eps: float) -> np.ndarray:
    """Row-wise h / sqrt(mean(h^2) + eps) (RMSNorm without its gain)."""
    return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps)


def layer_normalize(h: np.ndarray, eps: float) -> np.ndarray:
    """Row-wise (h - mean) / sqrt(var + eps), no affine (DiT adaLN input)."""
    mu = np.mean(h, axis=-1, keepdims=True)
    c = h - mu
    return c / np.sqrt(np.mean(c * c, axis=-1, keepdims=True) + eps)


def gelu_tanh(z: np.ndarray) -> np.ndarray:
    """GELU, tanh approximation: z/2 * (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3)))."""
    return 0.5 * z * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (z + 0.044715 * z ** 3)))


def swish(z: np.ndarray) -> np.ndarray:
    """swish(z) = z * sigmoid(z) (also called SiLU)."""
    return z / (1.0 + np.exp(-z))


def rope(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """Rotary position embedding, half-split pairing.

    x: [M, ..., D]; pos: [M].  Dimension i < D/2 is paired with i + D/2 and the
    pair is rotated by theta_i = pos * base^(-2i/D):
      (x1, x2) -> (x1 cos - x2 sin, x2 cos + x1 sin).
    """
    D = x.shape[-1]
    half = D // 2
    inv = base ** (-2.0 * np.arange(half, dtype=np.float64) / D)
    theta = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]        # [M, half]
    shape = (x.shape[0],) + (1,) * (x.ndim - 2) + (half,)
    c = np.cos(theta).reshape(shape).astype(x.dtype, copy=False)
    s = np.sin(theta).reshape(shape).astype(x.dtype, copy=False)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


# ----------------------------------------------------------------------------
# Attention
# ----------------------------------------------------------------------------

def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, allowed: np.ndarray) -> np.ndarray:
    """Masked softmax attention with grouped query heads.

    q: [M, n_q, D]; k, v: [N, n_kv, D]; allowed: bool [M, N] (query token i may
    see key j).  Query head g reads key/value head g // (n_q // n_kv).  Scores
    are q.k / sqrt(D) with disallowed entries removed; no soft-capping.
    Returns [M, n_q, D].
    """
    M, nq, D = q.shape
    nkv = k.shape[1]
    G = nq // nkv
    out = np.empty_like(q)
    for g in range(nq):
        kh = k[:, g // G, :]
        vh = v[:, g // G, :]
        s = (q[:, g, :] @ kh.T) / math.sqrt(D)                # [M, N]
        s = np.where(allowed, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, g, :] = p @ vh
    return out


def attention_bruteforce(q, k, v, allowed):
    """The same quantity written out with scalar loops (tiny shapes only)."""
    M, nq, D = q.shape
    N, nkv, _ = k.shape
    G = nq // nkv
    out = np.zeros((M, nq, D))
    for i in range(M):
        for g in range(nq):
            hk = g // G
            keys = [j for j in range(N) if allowed[i, j]]
            scores = []
            for j in keys:
                acc = 0.0
                for c in range(D):
                    acc += float(q[i, g, c]) * float(k[j, hk, c])
                scores.append(acc / math.sqrt(D))
            mx = max(scores)
            w = [math.exp(s - mx) for s in scores]
            tot = sum(w)
            for c in range(D):
                acc = 0.0
                for jj, j in enumerate(keys):
                    acc += w[jj] * float(v[j, hk, c])
                out[i, g, c] = acc / tot
    return out


def euler(velocity, x0: np.ndarray, timesteps, dtype=np.float64) -> np.ndarray:
    """Fixed-step explicit Euler integration of dx/dt = velocity(x, t) along the
    caller's schedule t_0 .. t_K, evaluating the velocity at the left end of
    each step: x_{k+1} = x_k + (t_{k+1} - t_k) * velocity(x_k, t_k).

    The paper's policy refines an action latent over several steps (Section
    "Embodied Task Formulation", "From Observation to Action") and its pi0.5
    configuration takes ten Euler steps (paragraph "Graph replay")."""
    x = np.array(x0, dtype=dtype)
    ts = [float(t) for t in timesteps]
    for k in range(len(ts) - 1):
        x = x + dtype(ts[k + 1] - ts[k]) * velocity(x, ts[k])
    return x
