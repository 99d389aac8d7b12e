"""Pins that tie the oracle to facts outside itself (CPU only).

Each test checks the oracle against a closed form, a hand-computed value, an
independent definition (complex multiplication for RoPE, a scalar triple loop
for attention, torch's dtype casts for the storage formats), or an invariant
that the method's definition forces.  The composed pi0 / pi0.5 / DiT networks
have no worked example in the paper; they are pinned only through the
invariants below (padding, batch independence, permutation equivariance,
block-mask independence of the state token, the zero-readout closed form).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import expert as oexp
from oracle import numerics as onum
import workloads as wl


# ----------------------------------------------------------------------------
# storage formats
# ----------------------------------------------------------------------------

def test_bf16_rounding_matches_torch():
    g = np.random.default_rng(0)
    x = np.concatenate([g.standard_normal(100000).astype(np.float32) * 10 ** g.uniform(-8, 8, 100000).astype(np.float32),
                        np.float32([0.0, -0.0, 1.0, 1.00390625, 1.005859375, 3.0e38, -1e-40])])
    ours = wl.bf16_bits_from_f32(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_bf16_decode_matches_torch():
    bits = np.arange(65536, dtype=np.uint16)
    ours = onum.decode_bf16(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])


def test_e4m3fn_table_matches_torch_all_codes():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert nan.sum() == 2 and nan[0x7F] and nan[0xFF]
    assert np.array_equal(np.isnan(onum.E4M3FN_TABLE), nan)
    assert np.array_equal(onum.E4M3FN_TABLE[~nan], ref[~nan])
    # hand facts of the format: max normal 448, min subnormal 2^-9, min normal 2^-6
    assert onum.E4M3FN_TABLE[0x7E] == 448.0
    assert onum.E4M3FN_TABLE[0x01] == 2.0 ** -9
    assert onum.E4M3FN_TABLE[0x08] == 2.0 ** -6
    assert onum.E4M3FN_TABLE[0x80] == 0.0 and math.copysign(1, onum.E4M3FN_TABLE[0x80]) < 0


def test_e4m3fn_encode_matches_torch_in_range():
    g = np.random.default_rng(1)
    vals = np.concatenate([g.uniform(-448, 448, 200000), g.standard_normal(100000) * 1e-2,
                           onum.E4M3FN_TABLE[np.isfinite(onum.E4M3FN_TABLE)]])
    # midpoints between neighbouring codes exercise ties-to-even
    pos = np.sort(np.unique(onum.E4M3FN_TABLE[np.isfinite(onum.E4M3FN_TABLE) & (onum.E4M3FN_TABLE >= 0)]))
    mids = (pos[1:] + pos[:-1]) / 2
    vals = np.concatenate([vals, mids, -mids]).astype(np.float32)
    ours = wl.e4m3fn_encode(vals)
    ref = torch.from_numpy(vals).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    # both signed zeros decode to zero; compare decoded values
    assert np.array_equal(onum.E4M3FN_TABLE[ours], onum.E4M3FN_TABLE[ref])


def test_e4m3fn_encode_saturates():
    assert onum.E4M3FN_TABLE[wl.e4m3fn_encode(np.array([1e6, -500.0, 449.0]))].tolist() == [448.0, -448.0, 448.0]


# OCP Microscaling Formats spec, FP4 E2M1 element values for codes 0..7
# (the sign is bit 3): 0, 0.5, 1, 1.5, 2, 3, 4, 6.
OCP_E2M1_POSITIVE = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]


def test_e2m1_table_matches_the_ocp_values():
    assert onum.E2M1_TABLE[:8].tolist() == OCP_E2M1_POSITIVE
    assert onum.E2M1_TABLE[8:].tolist() == [-v for v in OCP_E2M1_POSITIVE]
    assert math.copysign(1, onum.E2M1_TABLE[8]) < 0


def test_e2m1_encode_round_trip_and_ties_to_even():
    codes = np.arange(16, dtype=np.uint8)
    back = wl.e2m1_encode(onum.E2M1_TABLE[codes])
    assert np.array_equal(onum.E2M1_TABLE[back], onum.E2M1_TABLE[codes])
    # midpoints between neighbours round to the neighbour with an even mantissa bit
    pos = np.array(OCP_E2M1_POSITIVE)
    mids = (pos[1:] + pos[:-1]) / 2          # 0.25 0.75 1.25 1.75 2.5 3.5 5
    want = [0.0, 1.0, 1.0, 2.0, 2.0, 4.0, 4.0]
    assert onum.E2M1_TABLE[wl.e2m1_encode(mids)].tolist() == want
    assert onum.E2M1_TABLE[wl.e2m1_encode(-mids)].tolist() == [-v for v in want]
    # everywhere else: the nearest grid value
    v = np.random.default_rng(3).uniform(-6, 6, 100000)
    got = onum.E2M1_TABLE[wl.e2m1_encode(v)]
    grid = np.concatenate([-pos[::-1], pos])
    nearest = np.abs(v[:, None] - grid[None, :]).min(axis=1)
    assert np.allclose(np.abs(got - v), nearest, rtol=0, atol=1e-12)


def test_fp4_quantizer_groups_scales_and_packing():
    g = np.random.default_rng(4)
    w = (g.standard_normal((96, 10)) * 0.02).astype(np.float32)
    w[32:64, 3] = 0.0                        # an all-zero group
    w[0, 7] = 0.75                            # amax exactly 6 * 2^-3
    packed, scale = wl.quantize_fp4_groups(w)
    assert packed.shape == (96, 5) and scale.shape == (3, 10)
    # scales are powers of two, the smallest with amax <= 6 * scale
    amax = np.abs(w.reshape(3, 32, 10)).max(axis=1)
    assert np.all(np.frexp(scale)[0] == 0.5)
    assert np.all(amax <= 6 * scale)
    assert np.all((amax > 3 * scale) | (amax == 0))
    assert scale[1, 3] == 1.0 and scale[0, 7] == 0.125
    # unpacking: low nibble is the even column
    codes = np.empty((96, 10), np.uint8)
    codes[:, 0::2] = packed & 15
    codes[:, 1::2] = packed >> 4
    dec = onum.decode_fp4(packed, scale)
    assert np.array_equal(dec, onum.E2M1_TABLE[codes] * np.repeat(scale, 32, axis=0))
    # round to nearest: the error is at most half a quantum of the code's binade
    r = w / np.repeat(scale, 32, axis=0)
    q = np.where(np.abs(r) < 2, 0.5, np.where(np.abs(r) < 4, 1.0, 2.0))
    assert np.all(np.abs(dec - w) <= q / 2 * np.repeat(scale, 32, axis=0) + 1e-12)


def test_fp4_decode_hand_example():
    # two rows x four columns; row 0 codes [1, 15, 7, 8], row 1 codes [4, 0, 11, 6]
    packed = np.array([[0xF1, 0x87], [0x04, 0x6B]], dtype=np.uint8)
    scale = np.array([[0.5, 2.0, 1.0, 0.25]], dtype=np.float32)
    packed = np.repeat(packed, 16, axis=0)    # one 32-row group
    dec = onum.decode_fp4(packed, scale)
    assert dec[0].tolist() == [0.5 * 0.5, -6.0 * 2.0, 6.0 * 1.0, -0.0 * 0.25]
    assert dec[16].tolist() == [2.0 * 0.5, 0.0 * 2.0, -1.5 * 1.0, 4.0 * 0.25]


def test_fp8_quantizer_scale_and_error():
    g = np.random.default_rng(2)
    w = (g.standard_normal((64, 48)) * 0.02).astype(np.float32)
    w[:, 5] = 0.0
    codes, scale = wl.quantize_fp8_per_column(w)
    assert scale[5] == 1.0
    deq = onum.decode_fp8(codes, scale)
    col_amax = np.abs(w).max(axis=0)
    # the column maximum maps to code 448 exactly; the relative RTN error is <= 2^-4
    assert np.allclose(np.abs(deq).max(axis=0)[col_amax > 0], col_amax[col_amax > 0], rtol=1e-6)
    err = np.abs(deq - w)
    assert np.all(err <= np.maximum(np.abs(w) * 2.0 ** -4, 2.0 ** -10 * scale[None, :]) + 1e-12)


# ----------------------------------------------------------------------------
# Euler integration (closed forms)
# ----------------------------------------------------------------------------

def test_euler_constant_field():
    x0 = np.array([[0.5, -2.0]])
    c = np.array([[3.0, 1.0]])
    out = onum.euler(lambda x, t: c, x0, wl.default_timesteps(10))
    assert np.allclose(out, x0 - c, atol=1e-12)          # t_K - t_0 = -1


def test_euler_linear_field_is_euler_not_exact():
    x0 = np.array([2.0])
    out = onum.euler(lambda x, t: x, x0, wl.default_timesteps(4))
    assert out[0] == pytest.approx(2.0 * 0.31640625, abs=1e-15)       # (1 - 1/4)^4
    assert abs(out[0] - 2.0 * math.exp(-1)) > 0.1                     # not the exact ODE flow


def test_euler_time_dependent_field_left_endpoint():
    # v = a + b t, uniform 1 -> 0, K=4: left Riemann sum gives -a - 0.625 b
    out = onum.euler(lambda x, t: np.array([1.0 + 2.0 * t]), np.array([0.0]), wl.default_timesteps(4))
    assert out[0] == pytest.approx(-1.0 - 2.0 * 0.625, abs=1e-15)


# ----------------------------------------------------------------------------
# scalar operations
# ----------------------------------------------------------------------------

def test_gelu_tanh_values():
    assert onum.gelu_tanh(np.array(0.0)) == 0.0
    assert onum.gelu_tanh(np.array(1.0)) == pytest.approx(0.8411919906082768, abs=1e-13)
    assert onum.gelu_tanh(np.array(-1.0)) == pytest.approx(-0.15880800939172324, abs=1e-13)
    # the tanh form, not the erf form (0.8413447460685429)
    assert abs(onum.gelu_tanh(np.array(1.0)) - 0.8413447460685429) > 1e-4


def test_swish_values():
    assert onum.swish(np.array(0.0)) == 0.0
    assert onum.swish(np.array(1.0)) == pytest.approx(0.7310585786300049, abs=1e-14)
    assert onum.swish(np.array(-30.0)) == pytest.approx(0.0, abs=1e-11)


def test_rms_normalize_constant_row():
    for c in (3.0, -0.5, 1e-4):
        h = np.full((1, 8), c)
        eps = 1e-6
        assert np.allclose(onum.rms_normalize(h, eps), np.sign(c) * abs(c) / math.sqrt(c * c + eps), atol=1e-14)
    h = np.array([[3.0, 4.0]])        # mean square 12.5
    assert np.allclose(onum.rms_normalize(h, 0.0), h / math.sqrt(12.5))


def test_layer_normalize_values():
    h = np.array([[1.0, 2.0, 3.0, 4.0]])
    # mean 2.5, variance 1.25
    assert np.allclose(onum.layer_normalize(h, 0.0), (h - 2.5) / math.sqrt(1.25), atol=1e-15)


def test_sinusoid_values():
    tau0 = onum.sinusoid(0.0, 8, 4e-3, 4.0)
    assert np.array_equal(tau0, [0, 0, 0, 0, 1, 1, 1, 1])
    tau1 = onum.sinusoid(1.0, 8, 4e-3, 4.0)
    # periods 4e-3, 4e-2, 4e-1, 4: t=1 is 250, 25 and 2.5 turns for the first three
    assert np.allclose(tau1[:3], 0.0, atol=1e-12)
    assert np.allclose(tau1[4:7], [1.0, 1.0, -1.0], atol=1e-12)
    assert tau1[3] == pytest.approx(1.0, abs=1e-15)     # sin(2 pi / 4)
    assert tau1[7] == pytest.approx(0.0, abs=1e-15)     # cos(2 pi / 4)


def test_rope_is_complex_rotation():
    g = np.random.default_rng(3)
    D, base = 16, 10000.0
    x = g.standard_normal((5, 3, D))
    pos = np.array([0, 1, 7, 100, 12345])
    ours = onum.rope(x, pos, base)
    z = x[..., :D // 2] + 1j * x[..., D // 2:]
    theta = pos[:, None, None] * base ** (-np.arange(D // 2) * 2.0 / D)[None, None, :]
    zr = z * np.exp(1j * theta)
    assert np.allclose(ours, np.concatenate([zr.real, zr.imag], axis=-1), atol=1e-12)
    assert np.array_equal(ours[0], x[0])                                   # position 0
    assert np.allclose(np.linalg.norm(ours, axis=-1), np.linalg.norm(x, axis=-1))


def test_rope_relative_positions():
    g = np.random.default_rng(4)
    q, k = g.standard_normal((1, 32)), g.standard_normal((1, 32))
    s = [(onum.rope(q, np.array([p]), 1e4) @ onum.rope(k, np.array([p - 5]), 1e4).T).item() for p in (5, 17, 900)]
    assert np.allclose(s, s[0], atol=1e-10)


# ----------------------------------------------------------------------------
# attention
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("nq,nkv", [(2, 1), (4, 2), (3, 3)])
def test_attention_vectorised_equals_bruteforce(nq, nkv):
    g = np.random.default_rng(5 + nq)
    M, N, D = 3, 8, 4
    q, k, v = g.standard_normal((M, nq, D)), g.standard_normal((N, nkv, D)), g.standard_normal((N, nkv, D))
    allowed = g.random((M, N)) < 0.6
    allowed[:, 0] = True
    assert np.allclose(onum.attention(q, k, v, allowed), onum.attention_bruteforce(q, k, v, allowed),
                       atol=1e-13, rtol=0)


def test_attention_uniform_scores_average_allowed_rows():
    g = np.random.default_rng(6)
    v = g.standard_normal((6, 1, 4))
    allowed = np.array([[1, 0, 1, 1, 0, 0], [0, 0, 0, 0, 1, 0]], dtype=bool)
    out = onum.attention(np.zeros((2, 2, 4)), g.standard_normal((6, 1, 4)), v, allowed)
    assert np.allclose(out[0, 1], v[[0, 2, 3], 0].mean(axis=0), atol=1e-14)
    assert np.allclose(out[1, 0], v[4, 0], atol=1e-15)          # a single allowed key


def test_attention_scale_is_inverse_sqrt_dh():
    # two keys, scores differ by exactly sqrt(D) before scaling -> weights e^1 : 1
    D = 16
    q = np.zeros((1, 1, D)); q[0, 0, 0] = 1.0
    k = np.zeros((2, 1, D)); k[0, 0, 0] = math.sqrt(D)
    v = np.zeros((2, 1, D)); v[0, 0, 1] = 1.0
    out = onum.attention(q, k, v, np.ones((1, 2), bool))
    assert out[0, 0, 1] == pytest.approx(math.e / (math.e + 1), abs=1e-14)


# ----------------------------------------------------------------------------
# composed network: invariants and closed forms
# ----------------------------------------------------------------------------

def _small(variant, **kw):
    base = dict(n_layers=2, d_model=64, n_q_heads=4, n_kv_heads=1, head_dim=16, d_mlp=128,
                horizon=5, action_dim=3, n_steps=3, prefix_cap=12, prefix_min=9, prefix_max=12, batch=3,
                weight_dtype="f32", kv_dtype="f32", init_std=0.2)
    if variant == "pi0":
        base.update(state_token=True, rope=True)
    elif variant == "pi05":
        base.update(state_token=False, rope=True)
    else:
        base.update(n_q_heads=4, n_kv_heads=4, state_token=True, rope=False, d_feat=48, time_dim=32)
    base.update(kw)
    base.setdefault("time_dim", base["d_model"])
    return wl.ExpertConfig(name=f"small_{variant}", cfg_id=90, variant=variant, **base)


def _run(cfg, case=None, **kw):
    case = case or wl.make_case(cfg, seed=11)
    return case, oracle.denoise(cfg, case.weights, case.prefix, case.prefix_len, case.noise,
                                case.timesteps, case.state, **kw)


@pytest.mark.parametrize("variant", ["pi0", "pi05", "dit"])
def test_zero_readout_gives_noise_minus_bias(variant):
    cfg = _small(variant)
    A = cfg.action_dim
    out_b = np.array([[0.3, -1.25, 2.0]])
    w = wl.make_weights(cfg, 11, overrides={"out_w": np.zeros((cfg.d_model, A)), "out_b": out_b})
    case = wl.make_case(cfg, seed=11, weights=w)
    _, out = _run(cfg, case)
    assert np.allclose(out, case.noise - out_b[None], atol=1e-12)


@pytest.mark.parametrize("variant", ["pi0", "pi05", "dit"])
def test_padding_rows_never_read(variant):
    cfg = _small(variant)
    plen = wl.make_prefix_lengths(cfg, 11)
    assert plen.min() < cfg.prefix_cap
    case = wl.make_case(cfg, seed=11)
    _, ref = _run(cfg, case)
    case.prefix = wl.make_prefix(cfg, case.prefix_len, 11, pad_value=float("nan"))
    _, out = _run(cfg, case)
    assert np.isfinite(out).all() and np.array_equal(out, ref)


@pytest.mark.parametrize("variant", ["pi0", "pi05", "dit"])
def test_requests_are_independent(variant):
    cfg = _small(variant)
    case, ref = _run(cfg)
    case.noise = case.noise.copy()
    case.noise[1] += 5.0
    case.prefix = case.prefix.copy()
    if variant == "dit":
        case.prefix[2] *= -1.0
    else:
        case.prefix[:, :, 2] *= -1.0
    _, out = _run(cfg, case)
    assert np.array_equal(out[0], ref[0])
    assert not np.allclose(out[1], ref[1]) and not np.allclose(out[2], ref[2])


def test_subset_slots_match_full_batch():
    cfg = _small("pi0")
    case, ref = _run(cfg)
    pre = wl.make_prefix(cfg, case.prefix_len, 11, requests=[2])
    out = oracle.denoise(cfg, case.weights, pre, case.prefix_len[2:3], case.noise[2:3], case.timesteps,
                         case.state[2:3], slots=[0])
    assert np.array_equal(out[0], ref[2])


def test_permutation_equivariance_without_positions():
    # tiny fp32 shape: no RoPE, no state token -> action tokens are exchangeable
    cfg = wl.CONFIGS["tiny_fp32"].replace(n_layers=1, d_model=64, head_dim=16, d_mlp=128, time_dim=64)
    case, ref = _run(cfg)
    perm = np.random.default_rng(7).permutation(cfg.horizon)
    case.noise = case.noise[:, perm]
    _, out = _run(cfg, case)
    assert np.allclose(out, ref[:, perm], atol=1e-12, rtol=0)


def test_positions_break_equivariance_when_rope_on():
    cfg = _small("pi05", batch=1, prefix_min=12)
    case, ref = _run(cfg)
    perm = np.array([1, 0, 2, 3, 4])
    case.noise = case.noise[:, perm]
    _, out = _run(cfg, case)
    assert not np.allclose(out, ref[:, perm], atol=1e-6)


def test_state_token_stream_ignores_actions_and_time():
    """Block mask: the state token sees only the prefix and itself, so its
    hidden state at every layer is the same whatever the noise and the time;
    action tokens do depend on both."""
    cfg = _small("pi0", batch=1, prefix_min=12)
    case = wl.make_case(cfg, seed=11)
    W = oexp.DecodedWeights(case.weights)
    P = int(case.prefix_len[0])
    seen = []
    orig = oexp._trunk

    def spy(cfg_, W_, h, P_, kv_rows, norm_fn):
        out = orig(cfg_, W_, h, P_, kv_rows, norm_fn)
        seen.append(out.copy())
        return out

    kv = lambda l: oexp._prefix_rows(cfg, case.prefix.astype(np.float64), 0, P, l)
    oexp._trunk = spy
    try:
        for x, t in ((case.noise[0], 1.0), (case.noise[0] * -3.0 + 1.0, 0.3)):
            oexp.velocity_pi0(cfg, W, np.asarray(x, np.float64), t, kv, P, case.state[0].astype(np.float64))
    finally:
        oexp._trunk = orig
    assert np.array_equal(seen[0][0], seen[1][0])
    assert not np.allclose(seen[0][1:], seen[1][1:])


def test_one_hot_value_probe_counts_allowed_keys():
    """With W_q = 0 every allowed key gets the same weight, so a one-hot value
    row e_j reads back 1 / (number of allowed keys) in coordinate j."""
    cfg = _small("pi0", n_layers=1, batch=1, prefix_min=12)
    d, D = cfg.d_model, cfg.head_dim
    case = wl.make_case(cfg, seed=11)
    W = oexp.DecodedWeights(case.weights)
    W.w["layers.0.wq"] = np.zeros_like(W["layers.0.wq"])
    W.w["layers.0.wv"] = np.zeros_like(W["layers.0.wv"])
    P = 7
    pre = np.zeros((1, 2, 1, cfg.prefix_cap, D))
    for j in range(P):
        pre[0, 1, 0, j, j] = 1.0
    captured = {}
    orig = onum.attention

    def spy(q, k, v, allowed):
        out = orig(q, k, v, allowed)
        captured["o"] = out
        return out

    oexp.attention = spy
    try:
        oexp.velocity_pi0(cfg, W, case.noise[0].astype(np.float64), 1.0,
                          lambda l: oexp._prefix_rows(cfg, pre, 0, P, l), P, case.state[0].astype(np.float64))
    finally:
        oexp.attention = orig
    o = captured["o"]
    # state token: prefix (7) + itself; action tokens: prefix + state + 5 actions
    assert np.allclose(o[0, :, :P], 1.0 / (P + 1), atol=1e-15)
    assert np.allclose(o[1:, :, :P], 1.0 / (P + 1 + cfg.horizon), atol=1e-15)
    assert np.allclose(o[:, :, P:], 0.0)


# ----------------------------------------------------------------------------
# wiring probe: structured weights whose output follows from pinned parts
# ----------------------------------------------------------------------------

def _wiring_probe_case(P=6):
    """One pi0 layer, one Euler step, with weights chosen so that the output is
    a hand-derivable function of pinned pieces (attention weights 1/N, a
    permutation W_o, RMSNorm):
      in_w = 0, time_w2 = 0   -> every action token embeds to time_b2 = beta
      state_w = 0             -> the state token embeds to state_b = sigma
      wq = 0, wv = 0          -> uniform attention, suffix values 0
      prefix V row j = e_j    -> head output = (1/N_i) sum_{j<P} e_j
      W_o = permutation Pi    -> h1 = e + o Pi
      w_gate = 0              -> the MLP adds gelu(0) * up = 0
    """
    cfg = _small("pi0", n_layers=1, n_steps=1, batch=1, prefix_min=12, prefix_max=12)
    d, D, nq, H = cfg.d_model, cfg.head_dim, cfg.n_q_heads, cfg.horizon
    assert nq * D == d
    g = np.random.default_rng(12)
    perm = g.permutation(d)
    Pi = np.zeros((d, d)); Pi[np.arange(d), perm] = 1.0
    beta = g.standard_normal((1, d)).astype(np.float32).astype(np.float64)
    sigma = g.standard_normal((1, d)).astype(np.float32).astype(np.float64)
    ov = {"in_w": np.zeros((cfg.action_dim, d)), "time_w2": np.zeros((d, d)), "time_b2": beta,
          "state_w": np.zeros((cfg.action_dim, d)), "state_b": sigma,
          "layers.0.wq": np.zeros((d, d)), "layers.0.wv": np.zeros((d, D)), "layers.0.wo": Pi,
          "layers.0.w_gate": np.zeros((d, cfg.d_mlp))}
    case = wl.make_case(cfg, seed=11, weights=wl.make_weights(cfg, 11, overrides=ov))
    case.prefix_len = np.array([P], np.int32)
    pre = np.zeros((1, 2, 1, cfg.prefix_cap, D), np.float32)
    pre[0, 0, 0, :P] = g.standard_normal((P, D))
    pre[0, 1, 0, np.arange(P), np.arange(P)] = 1.0
    case.prefix = pre
    # expected output, assembled from pinned parts
    W = oexp.DecodedWeights(case.weights)
    e = np.concatenate([sigma, np.repeat(beta, H, axis=0)])
    n_allowed = np.array([P + 1] + [P + 1 + H] * H, dtype=np.float64)
    head = np.zeros((H + 1, D)); head[:, :P] = 1.0 / n_allowed[:, None]
    o = np.tile(head, (1, nq))
    h1 = e + o @ Pi
    v = onum.rms_normalize(h1, cfg.rms_eps)[1:] * (1.0 + W.vec("final_norm")) @ W["out_w"] + W.vec("out_b")
    expected = case.noise[0] + (case.timesteps[1] - case.timesteps[0]) * v
    return cfg, case, expected


def test_wiring_probe_matches_hand_derivation():
    cfg, case, expected = _wiring_probe_case()
    _, out = _run(cfg, case)
    assert np.allclose(out[0], expected, atol=1e-12, rtol=0)


class _Planted(oexp.DecodedWeights):
    """Decoded weights that hand back a planted mistake for one name."""

    def __init__(self, stored, name, fn):
        super().__init__(stored)
        self.w[name] = fn(self.w[name])


@pytest.mark.parametrize("mistake", ["transposed_wo", "readout_first_rows", "dropped_attn_residual"])
def test_wiring_probe_catches_planted_mistakes(mistake, monkeypatch):
    """Plant a plausible mistake in the oracle (on the CPU) and check the probe
    sees it."""
    cfg, case, expected = _wiring_probe_case()
    kw = {}
    if mistake == "transposed_wo":
        kw["decoded"] = _Planted(case.weights, "layers.0.wo", lambda w: w.T.copy())
    elif mistake == "readout_first_rows":
        # read the first H suffix rows instead of the last H
        src = oexp._trunk

        def trunk_shift(cfg_, W, h, P, kv, nf):
            out = src(cfg_, W, h, P, kv, nf)
            return np.concatenate([out[:1], out[:-1]])
        monkeypatch.setattr(oexp, "_trunk", trunk_shift)
    else:
        src = oexp._trunk

        def no_resid(cfg_, W, h, P, kv, nf):
            W.w["layers.0.wo"] = np.zeros_like(W["layers.0.wo"])
            return src(cfg_, W, h, P, kv, nf)
        monkeypatch.setattr(oexp, "_trunk", no_resid)
    out = oracle.denoise(cfg, case.weights, case.prefix, case.prefix_len, case.noise, case.timesteps,
                         case.state, **kw)
    assert not np.allclose(out[0], expected, atol=1e-6)


def test_single_precision_timing_mode_tracks_float64():
    """The float32 mode (a CPU timing baseline only) runs the same steps: it
    returns float32 and stays within float32 rounding of the reference."""
    cfg = wl.CONFIGS["tiny_fp32"]
    case = wl.make_case(cfg, seed=1)
    ref = oracle.denoise(cfg, case.weights, case.prefix, case.prefix_len, case.noise, case.timesteps, case.state)
    got = oracle.denoise(cfg, case.weights, case.prefix, case.prefix_len, case.noise, case.timesteps, case.state,
                         dtype=np.float32)
    assert got.dtype == np.float32 and ref.dtype == np.float64
    assert np.abs(got - ref).max() < 1e-5
