"""Wiring probes for the oracle's composed networks (CPU only).

The paper prints no worked example of the expert, so the composed pi0 / pi0.5
/ DiT velocity networks are pinned here by structured weights: each probe
sets weights so that one Euler step's output follows by hand from parts that
are pinned elsewhere (RMSNorm, LayerNorm, GELU, swish, the sinusoid, RoPE as a
complex rotation, attention against a scalar triple loop).  The hand
derivation uses a simplification the structure allows (identical tokens,
uniform attention weights, the relative-position property of RoPE, zeroed
gates, block sums in place of a concatenation), not the oracle's own code
path.

Each probe is paired with plausible mistakes planted in a copy of the oracle's
source text (run on the CPU); every planted mistake must move the output away
from the hand derivation.  The readings probed are the ones the paper leaves
open (pre-norm sites, GeGLU gate/up roles, RoPE on both queries and keys at
positions prefix_len + i, the pi0 time-MLP input order, the pi0.5 condition
and adaRMS scale/shift order, the DiT adaLN chunk order and final
modulation).
"""
import math
import pathlib
import types

import numpy as np
import pytest

import oracle
from oracle import expert as oexp
from oracle import numerics as onum
import workloads as wl

_SRC = pathlib.Path(oexp.__file__).read_text()


def _mutant(edits):
    """A copy of oracle/expert.py with textual edits applied (each anchor must
    occur exactly once, so a drifting source fails loudly here)."""
    src = _SRC
    for old, new in edits:
        assert src.count(old) == 1, f"mutation anchor not found exactly once: {old!r}"
        src = src.replace(old, new)
    mod = types.ModuleType("oracle._mutant")
    mod.__package__ = "oracle"
    mod.__file__ = oexp.__file__
    exec(compile(src, oexp.__file__ + " (mutant)", "exec"), mod.__dict__)
    return mod


def _cfg(variant, **kw):
    base = dict(n_layers=1, d_model=64, n_q_heads=4, n_kv_heads=1, head_dim=16, d_mlp=128,
                horizon=5, action_dim=3, n_steps=1, prefix_cap=12, prefix_min=12, prefix_max=12,
                batch=1, weight_dtype="f32", kv_dtype="f32", init_std=0.2)
    if variant == "pi0":
        base.update(state_token=True, rope=True)
    elif variant == "pi05":
        base.update(state_token=False, rope=True)
    else:
        base.update(n_layers=2, n_q_heads=4, n_kv_heads=4, state_token=True, rope=False, d_feat=48,
                    time_dim=32)
    base.update(kw)
    base.setdefault("time_dim", base["d_model"])
    return wl.ExpertConfig(name=f"probe_{variant}", cfg_id=91, variant=variant, **base)


def _vec(g, n, scale=1.0, offset=0.0):
    """A float32-exact row vector [1][n]."""
    return (offset + scale * g.standard_normal((1, n))).astype(np.float32).astype(np.float64)


def _f32(x):
    return np.asarray(x, np.float32).astype(np.float64)


def _run(mod, cfg, case):
    return mod.denoise(cfg, case.weights, case.prefix, case.prefix_len, case.noise, case.timesteps,
                       case.state)


def _euler_one(case, v):
    """x_1 = x_0 + (t_1 - t_0) v for the single request (one Euler step)."""
    dt = float(case.timesteps[1]) - float(case.timesteps[0])
    return case.noise[0].astype(np.float64) + dt * v


def _rms_readout(cfg, W, h, scale, shift=0.0):
    off = 1 if cfg.state_token else 0
    n = onum.rms_normalize(h, cfg.rms_eps)[off:] * (1.0 + scale) + shift
    return n @ W["out_w"] + W.vec("out_b")


def _permutation(g, d):
    Pi = np.zeros((d, d))
    Pi[np.arange(d), g.permutation(d)] = 1.0
    return Pi


def _check(probe, mistakes, name):
    cfg, case, expected = probe()
    out = _run(oexp, cfg, case)
    if name is None:
        assert np.allclose(out[0], expected, atol=1e-12, rtol=0)
        return
    bad = _run(_mutant(mistakes[name]), cfg, case)
    assert not np.allclose(bad[0], expected, atol=1e-6), f"planted mistake '{name}' went unseen"


# ----------------------------------------------------------------------------
# pi0: GeGLU gate/up roles and the MLP norm site
# ----------------------------------------------------------------------------

def _probe_pi0_mlp():
    """Attention off (W_o = 0); embeddings constant (in_w = time_w2 = state_w
    = 0); W_gate = a S, W_up = b S, W_down = S^T with S = [I | 0], so the block
    adds gelu(a n) * (b n) to h with n = RMSNorm(h) (1 + w_mlp)."""
    cfg = _cfg("pi0")
    d, F, A = cfg.d_model, cfg.d_mlp, cfg.action_dim
    g = np.random.default_rng(21)
    beta, sigma = _vec(g, d, 3.0), _vec(g, d, 0.5)
    a_g, b_u = 1.5, -0.75
    S = np.zeros((d, F)); S[np.arange(d), np.arange(d)] = 1.0
    ov = {"in_w": np.zeros((A, d)), "time_w2": np.zeros((d, d)), "time_b2": beta,
          "state_w": np.zeros((A, d)), "state_b": sigma, "layers.0.wo": np.zeros((d, d)),
          "layers.0.w_gate": a_g * S, "layers.0.w_up": b_u * S, "layers.0.w_down": S.T}
    case = wl.make_case(cfg, seed=3, weights=wl.make_weights(cfg, 3, overrides=ov))
    W = oexp.DecodedWeights(case.weights)
    h0 = np.concatenate([sigma, np.repeat(beta, cfg.horizon, axis=0)])
    n = onum.rms_normalize(h0, cfg.rms_eps) * (1.0 + W.vec("layers.0.mlp_norm"))
    h1 = h0 + onum.gelu_tanh(a_g * n) * (b_u * n)
    return cfg, case, _euler_one(case, _rms_readout(cfg, W, h1, W.vec("final_norm")))


_PI0_MLP_MISTAKES = {
    "geglu_gate_up_swapped": [(
        'h = h + (gelu_tanh(n @ W[p + "w_gate"]) * (n @ W[p + "w_up"])) @ W[p + "w_down"]',
        'h = h + (gelu_tanh(n @ W[p + "w_up"]) * (n @ W[p + "w_gate"])) @ W[p + "w_down"]')],
    "mlp_norm_skipped": [('n = norm_fn(("mlp", l), h)', 'n = h')],
    "mlp_residual_dropped": [(
        'h = h + (gelu_tanh(n @ W[p + "w_gate"]) * (n @ W[p + "w_up"])) @ W[p + "w_down"]',
        'h = (gelu_tanh(n @ W[p + "w_gate"]) * (n @ W[p + "w_up"])) @ W[p + "w_down"]')],
}


@pytest.mark.parametrize("name", [None, *_PI0_MLP_MISTAKES])
def test_pi0_mlp_probe(name):
    _check(_probe_pi0_mlp, _PI0_MLP_MISTAKES, name)


# ----------------------------------------------------------------------------
# pi0: the pre-attention norm site and the value path
# ----------------------------------------------------------------------------

def _probe_pi0_attn_norm(P=7):
    """W_q = 0 makes every allowed key weigh the same; prefix V rows are e_j;
    W_v = c [I; 0] makes the suffix values c n_j[:D] with n = RMSNorm(h)
    (1 + w_attn); W_o = a permutation; the MLP adds gelu(0) * up = 0.  Head
    output of token i = (sum_{j<P} e_j + sum of allowed suffix values) / N_i
    with the block mask's N_i (state: P + 1; actions: P + 1 + H)."""
    cfg = _cfg("pi0")
    d, D, nq, H, A = cfg.d_model, cfg.head_dim, cfg.n_q_heads, cfg.horizon, cfg.action_dim
    g = np.random.default_rng(22)
    beta, sigma = _vec(g, d, 3.0), _vec(g, d, 0.5)
    c = 1.75
    Wv = np.zeros((d, D)); Wv[np.arange(D), np.arange(D)] = c
    Pi = _permutation(g, d)
    ov = {"in_w": np.zeros((A, d)), "time_w2": np.zeros((d, d)), "time_b2": beta,
          "state_w": np.zeros((A, d)), "state_b": sigma, "layers.0.wq": np.zeros((d, nq * D)),
          "layers.0.wv": Wv, "layers.0.wo": Pi, "layers.0.w_gate": np.zeros((d, cfg.d_mlp))}
    case = wl.make_case(cfg, seed=4, weights=wl.make_weights(cfg, 4, overrides=ov))
    case.prefix_len = np.array([P], np.int32)
    pre = np.zeros((1, 2, 1, cfg.prefix_cap, D), np.float32)
    pre[0, 0, 0, :P] = g.standard_normal((P, D))
    pre[0, 1, 0, np.arange(P), np.arange(P)] = 1.0
    case.prefix = pre
    W = oexp.DecodedWeights(case.weights)
    h0 = np.concatenate([sigma, np.repeat(beta, H, axis=0)])
    n = onum.rms_normalize(h0, cfg.rms_eps) * (1.0 + W.vec("layers.0.attn_norm"))
    vals = n @ W["layers.0.wv"]                       # [M, D]
    ones = np.zeros(D); ones[:P] = 1.0
    o_state = (ones + vals[0]) / (P + 1)
    o_act = (ones + vals[0] + H * vals[1]) / (P + 1 + H)
    o = np.tile(np.vstack([o_state, np.repeat(o_act[None], H, axis=0)]), (1, nq))
    h1 = h0 + o @ Pi
    return cfg, case, _euler_one(case, _rms_readout(cfg, W, h1, W.vec("final_norm")))


_PI0_ATTN_MISTAKES = {
    "attn_norm_skipped": [('n = norm_fn(("attn", l), h)', 'n = h')],
    "attn_norm_uses_mlp_gain": [('n = norm_fn(("attn", l), h)', 'n = norm_fn(("mlp", l), h)')],
    "attn_residual_dropped": [('h = h + o.reshape(M, nq * D) @ W[p + "wo"]',
                               'h = o.reshape(M, nq * D) @ W[p + "wo"]')],
}


@pytest.mark.parametrize("name", [None, *_PI0_ATTN_MISTAKES])
def test_pi0_attention_norm_probe(name):
    _check(_probe_pi0_attn_norm, _PI0_ATTN_MISTAKES, name)


# ----------------------------------------------------------------------------
# RoPE on queries and keys, positions prefix_len + i
# ----------------------------------------------------------------------------

def _probe_rope(P=6):
    """No state token; every action token embeds to the same row, so before
    rotation all queries (one head pattern repeated over the heads), keys and
    values are the same vectors q, k, v.  Scores of token i: against prefix
    key p, rope(q, P + i) . K_p / sqrt(D); against suffix token j, by the
    relative-position property, rope(q, i - j) . k / sqrt(D).  Prefix values
    are e_p, so head output i = (sum_p w_ip e_p + (sum_j w_ij) v)."""
    cfg = _cfg("pi0", state_token=False)
    d, D, nq, H, A = cfg.d_model, cfg.head_dim, cfg.n_q_heads, cfg.horizon, cfg.action_dim
    g = np.random.default_rng(23)
    beta = _vec(g, d, 2.0)
    Wq1 = _f32(g.standard_normal((d, D)) * 0.6)
    Wk1 = _f32(g.standard_normal((d, D)) * 0.6)
    Wv1 = _f32(g.standard_normal((d, D)) * 0.3)
    Pi = _permutation(g, d)
    ov = {"in_w": np.zeros((A, d)), "time_w2": np.zeros((d, d)), "time_b2": beta,
          "layers.0.wq": np.tile(Wq1, (1, nq)), "layers.0.wk": Wk1, "layers.0.wv": Wv1,
          "layers.0.wo": Pi, "layers.0.w_gate": np.zeros((d, cfg.d_mlp))}
    case = wl.make_case(cfg, seed=5, weights=wl.make_weights(cfg, 5, overrides=ov))
    case.prefix_len = np.array([P], np.int32)
    pre = np.zeros((1, 2, 1, cfg.prefix_cap, D), np.float32)
    Kp = _f32(g.standard_normal((P, D)))
    pre[0, 0, 0, :P] = Kp
    pre[0, 1, 0, np.arange(P), np.arange(P)] = 1.0
    case.prefix = pre
    W = oexp.DecodedWeights(case.weights)
    n = onum.rms_normalize(beta, cfg.rms_eps) * (1.0 + W.vec("layers.0.attn_norm"))
    q, k, v = (n @ Wq1)[0], (n @ Wk1)[0], (n @ Wv1)[0]
    rows = []
    for i in range(H):
        s_pre = onum.rope(q[None], np.array([P + i]), cfg.rope_base)[0] @ Kp.T / math.sqrt(D)
        s_suf = np.array([onum.rope(q[None], np.array([i - j]), cfg.rope_base)[0] @ k
                          for j in range(H)]) / math.sqrt(D)
        mx = max(s_pre.max(), s_suf.max())
        w_pre, w_suf = np.exp(s_pre - mx), np.exp(s_suf - mx)
        o = np.zeros(D)
        o[:P] += w_pre
        o += w_suf.sum() * v
        rows.append(o / (w_pre.sum() + w_suf.sum()))
    h1 = np.repeat(beta, H, axis=0) + np.tile(np.array(rows), (1, nq)) @ Pi
    return cfg, case, _euler_one(case, _rms_readout(cfg, W, h1, W.vec("final_norm")))


_ROPE_MISTAKES = {
    "rope_dropped_on_keys": [("k = rope(k, pos, cfg.rope_base)", "k = k")],
    "rope_dropped_on_queries": [("q = rope(q, pos, cfg.rope_base)", "q = q")],
    "positions_without_prefix_offset": [("pos = P + np.arange(M)", "pos = np.arange(M)")],
}


@pytest.mark.parametrize("name", [None, *_ROPE_MISTAKES])
def test_rope_probe(name):
    _check(_probe_rope, _ROPE_MISTAKES, name)


# ----------------------------------------------------------------------------
# pi0: the time MLP's input order [W_in x + b_in ; tau(t)]
# ----------------------------------------------------------------------------

def _probe_pi0_time_mlp():
    """The trunk adds nothing (W_o = 0, W_gate = 0), so the output reads the
    embedding e = [W_s s + b_s ; u_j] back through the final norm.  The first
    time-MLP layer is written as two row blocks of W_1 acting on the action
    embedding (rows 0..d-1) and on tau(t) (rows d..), with time_dim = d so
    that a swapped concatenation still type-checks."""
    cfg = _cfg("pi0")
    d = cfg.d_model
    assert cfg.time_dim == d
    ov = {"layers.0.wo": np.zeros((d, d)), "layers.0.w_gate": np.zeros((d, cfg.d_mlp))}
    case = wl.make_case(cfg, seed=6, weights=wl.make_weights(cfg, 6, overrides=ov))
    W = oexp.DecodedWeights(case.weights)
    x = case.noise[0].astype(np.float64)
    t0 = float(case.timesteps[0])
    a = x @ W["in_w"] + W.vec("in_b")
    tau = onum.sinusoid(t0, cfg.time_dim, cfg.sin_min_period, cfg.sin_max_period)
    W1 = W["time_w1"]
    z = a @ W1[:d] + (tau @ W1[d:])[None, :] + W.vec("time_b1")
    u = onum.swish(z) @ W["time_w2"] + W.vec("time_b2")
    s_emb = case.state[0].astype(np.float64) @ W["state_w"] + W.vec("state_b")
    h = np.concatenate([s_emb[None, :], u])
    return cfg, case, _euler_one(case, _rms_readout(cfg, W, h, W.vec("final_norm")))


_TIME_MISTAKES = {
    "time_concat_order_swapped": [(
        "z = np.concatenate([a, np.broadcast_to(tau, (a.shape[0], cfg.time_dim))], axis=1)",
        "z = np.concatenate([np.broadcast_to(tau, (a.shape[0], cfg.time_dim)), a], axis=1)")],
    "time_mlp_swish_dropped": [(
        'u = swish(z @ W["time_w1"] + W.vec("time_b1")) @ W["time_w2"] + W.vec("time_b2")',
        'u = (z @ W["time_w1"] + W.vec("time_b1")) @ W["time_w2"] + W.vec("time_b2")')],
}


@pytest.mark.parametrize("name", [None, *_TIME_MISTAKES])
def test_pi0_time_mlp_probe(name):
    _check(_probe_pi0_time_mlp, _TIME_MISTAKES, name)


# ----------------------------------------------------------------------------
# pi0.5: adaRMS scale/shift order and the timestep condition
# ----------------------------------------------------------------------------

def _probe_pi05_adarms():
    """Modulation weights zero, so every adaRMS site uses its bias split as
    [scale; shift]; the trunk adds nothing; the final site's planted scale and
    shift differ, so the output is (RMSNorm(e) (1 + scale) + shift) W_out +
    b_out with e = W_in x + b_in."""
    cfg = _cfg("pi05")
    d = cfg.d_model
    g = np.random.default_rng(25)
    sc_f, sh_f = _vec(g, d, 0.3, 0.5), _vec(g, d, 2.0)
    ov = {"layers.0.attn_mod_w": np.zeros((d, 2 * d)), "layers.0.mlp_mod_w": np.zeros((d, 2 * d)),
          "final_mod_w": np.zeros((d, 2 * d)), "final_mod_b": np.concatenate([sc_f, sh_f], axis=1),
          "layers.0.wo": np.zeros((d, d)), "layers.0.w_gate": np.zeros((d, cfg.d_mlp))}
    case = wl.make_case(cfg, seed=7, weights=wl.make_weights(cfg, 7, overrides=ov))
    W = oexp.DecodedWeights(case.weights)
    e = case.noise[0].astype(np.float64) @ W["in_w"] + W.vec("in_b")
    return cfg, case, _euler_one(case, _rms_readout(cfg, W, e, sc_f, sh_f))


def _probe_pi05_condition():
    """The final site's shift reads the condition directly (final_mod_w =
    [0 | I]) and cond_w2 = I, so c = swish(swish(tau W_c1 + b_c1) + b_c2) and
    the output is (RMSNorm(e) (1 + b_scale) + c + b_shift) W_out + b_out."""
    cfg = _cfg("pi05")
    d = cfg.d_model
    g = np.random.default_rng(26)
    fm = np.zeros((d, 2 * d)); fm[np.arange(d), d + np.arange(d)] = 1.0
    ov = {"layers.0.attn_mod_w": np.zeros((d, 2 * d)), "layers.0.mlp_mod_w": np.zeros((d, 2 * d)),
          "final_mod_w": fm, "cond_w2": np.eye(d), "cond_b1": _vec(g, d), "cond_b2": _vec(g, d),
          "layers.0.wo": np.zeros((d, d)), "layers.0.w_gate": np.zeros((d, cfg.d_mlp))}
    case = wl.make_case(cfg, seed=8, weights=wl.make_weights(cfg, 8, overrides=ov))
    W = oexp.DecodedWeights(case.weights)
    tau = onum.sinusoid(float(case.timesteps[0]), cfg.time_dim, cfg.sin_min_period, cfg.sin_max_period)
    c = onum.swish(onum.swish(tau @ W["cond_w1"] + W.vec("cond_b1")) + W.vec("cond_b2"))
    fb = W.vec("final_mod_b")
    e = case.noise[0].astype(np.float64) @ W["in_w"] + W.vec("in_b")
    return cfg, case, _euler_one(case, _rms_readout(cfg, W, e, fb[:d], c + fb[d:]))


_PI05_MOD_MISTAKES = {
    "adarms_scale_shift_swapped": [("scale, shift = mod[:d], mod[d:]", "shift, scale = mod[:d], mod[d:]")],
    "adarms_gain_without_one": [("rms_normalize(h, cfg.rms_eps) * (1.0 + scale) + shift",
                                 "rms_normalize(h, cfg.rms_eps) * scale + shift")],
}

_PI05_COND_MISTAKES = {
    "condition_outer_swish_dropped": [(
        'return swish(swish(tau @ W["cond_w1"] + W.vec("cond_b1")) @ W["cond_w2"] + W.vec("cond_b2"))',
        'return swish(tau @ W["cond_w1"] + W.vec("cond_b1")) @ W["cond_w2"] + W.vec("cond_b2")')],
    "condition_inner_swish_dropped": [(
        'return swish(swish(tau @ W["cond_w1"] + W.vec("cond_b1")) @ W["cond_w2"] + W.vec("cond_b2"))',
        'return swish((tau @ W["cond_w1"] + W.vec("cond_b1")) @ W["cond_w2"] + W.vec("cond_b2"))')],
}


@pytest.mark.parametrize("name", [None, *_PI05_MOD_MISTAKES])
def test_pi05_adarms_probe(name):
    _check(_probe_pi05_adarms, _PI05_MOD_MISTAKES, name)


@pytest.mark.parametrize("name", [None, *_PI05_COND_MISTAKES])
def test_pi05_condition_probe(name):
    _check(_probe_pi05_condition, _PI05_COND_MISTAKES, name)


# ----------------------------------------------------------------------------
# DiT: final modulation, condition, adaLN chunk order, cross/self alternation
# ----------------------------------------------------------------------------

def _dit_base(g, ada_b, cond_w2_eye=False, final_w=None, final_b=None):
    cfg = _cfg("dit")
    d, L = cfg.d_model, cfg.n_layers
    ov = {"final_ada_w": final_w if final_w is not None else np.zeros((d, 2 * d)),
          "final_ada_b": final_b}
    for l in range(L):
        ov[f"layers.{l}.ada_w"] = np.zeros((d, 6 * d))
        ov[f"layers.{l}.ada_b"] = ada_b[l]
    if cond_w2_eye:
        ov["cond_w2"] = np.eye(d)
    return cfg, ov


def _dit_embedding(cfg, W, case):
    x = case.noise[0].astype(np.float64)
    act = x @ W["in_w"] + W.vec("in_b") + W["pos_emb"]
    s_emb = case.state[0].astype(np.float64) @ W["state_w"] + W.vec("state_b")
    return np.concatenate([s_emb[None, :], act])


def _ln_readout(cfg, W, h, scale, shift):
    n = onum.layer_normalize(h, cfg.rms_eps)[1:] * (1.0 + scale) + shift
    return n @ W["out_w"] + W.vec("out_b")


def _probe_dit_final():
    """Every gate zero (adaLN weights zero, biases with zero gate chunks), so
    the blocks add nothing; final_ada_w = [I | 0] and cond_w2 = I, so the
    final shift is SiLU(c) + b_shift with c = SiLU(tau W_c1 + b_c1) + b_c2,
    and the scale is b_scale."""
    cfg = _cfg("dit")
    d = cfg.d_model
    g = np.random.default_rng(27)
    ada_b = []
    for _ in range(cfg.n_layers):
        ch = [_vec(g, d) for _ in range(6)]
        ch[2] = np.zeros((1, d)); ch[5] = np.zeros((1, d))
        ada_b.append(np.concatenate(ch, axis=1))
    fw = np.zeros((d, 2 * d)); fw[np.arange(d), np.arange(d)] = 1.0
    fb = np.concatenate([_vec(g, d, 1.0), _vec(g, d, 0.3, 0.4)], axis=1)
    cfg, ov = _dit_base(g, ada_b, cond_w2_eye=True, final_w=fw, final_b=fb)
    case = wl.make_case(cfg, seed=9, weights=wl.make_weights(cfg, 9, overrides=ov))
    W = oexp.DecodedWeights(case.weights)
    tau = onum.sinusoid(float(case.timesteps[0]), cfg.time_dim, cfg.sin_min_period, cfg.sin_max_period)
    c = onum.swish(tau @ W["cond_w1"] + W.vec("cond_b1")) + W.vec("cond_b2")
    b = W.vec("final_ada_b")
    h = _dit_embedding(cfg, W, case)
    return cfg, case, _euler_one(case, _ln_readout(cfg, W, h, b[d:], onum.swish(c) + b[:d]))


def _probe_dit_blocks(P=5):
    """Gates on for attention only (g2 = 0), W_q = 0 in both blocks so every
    key weighs the same: block 0 (cross) adds g1 * (mean of the projected
    features) W_o; block 1 (self) adds g1' * (mean over the 17 tokens of
    (LN(h) (1 + sc1') + sh1') W_v) W_o.  Final modulation from its bias."""
    cfg = _cfg("dit")
    d, nq, D = cfg.d_model, cfg.n_q_heads, cfg.head_dim
    g = np.random.default_rng(28)
    ada_b = []
    for _ in range(cfg.n_layers):
        sh1, sc1, g1 = _vec(g, d, 1.0), _vec(g, d, 0.5, 0.3), _vec(g, d, 1.0, 0.5)
        sh2, sc2 = _vec(g, d), _vec(g, d)
        ada_b.append(np.concatenate([sh1, sc1, g1, sh2, sc2, np.zeros((1, d))], axis=1))
    fb = np.concatenate([_vec(g, d, 1.0), _vec(g, d, 0.3, 0.4)], axis=1)
    cfg, ov = _dit_base(g, ada_b, final_b=fb)
    for l in range(cfg.n_layers):
        ov[f"layers.{l}.wq"] = np.zeros((d, nq * D))
    case = wl.make_case(cfg, seed=10, weights=wl.make_weights(cfg, 10, overrides=ov))
    case.prefix_len = np.array([P], np.int32)
    W = oexp.DecodedWeights(case.weights)
    feats = onum.decode_bf16(case.prefix)[0, :P] if case.prefix.dtype == np.uint16 else \
        case.prefix[0, :P].astype(np.float64)
    h = _dit_embedding(cfg, W, case)
    ab0, ab1 = W.vec("layers.0.ada_b"), W.vec("layers.1.ada_b")
    o0 = feats.mean(axis=0) @ W["layers.0.wv"]
    h = h + ab0[2 * d:3 * d] * (o0 @ W["layers.0.wo"])[None, :]
    xh = onum.layer_normalize(h, cfg.rms_eps) * (1.0 + ab1[d:2 * d]) + ab1[:d]
    o1 = xh.mean(axis=0) @ W["layers.1.wv"]
    h = h + ab1[2 * d:3 * d] * (o1 @ W["layers.1.wo"])[None, :]
    b = W.vec("final_ada_b")
    return cfg, case, _euler_one(case, _ln_readout(cfg, W, h, b[d:], b[:d]))


_DIT_FINAL_MISTAKES = {
    "dit_final_shift_scale_swapped": [("shf, scf = fin[:d], fin[d:]", "scf, shf = fin[:d], fin[d:]")],
    "dit_condition_silu_missing": [("sc = swish(c)", "sc = c")],
}

_DIT_BLOCK_MISTAKES = {
    "dit_adaln_chunk_order": [("sh1, sc1, g1, sh2, sc2, g2 = (ada[i * d:(i + 1) * d] for i in range(6))",
                               "sc1, sh1, g1, sc2, sh2, g2 = (ada[i * d:(i + 1) * d] for i in range(6))")],
    "dit_gates_swapped": [("sh1, sc1, g1, sh2, sc2, g2 = (ada[i * d:(i + 1) * d] for i in range(6))",
                           "sh1, sc1, g2, sh2, sc2, g1 = (ada[i * d:(i + 1) * d] for i in range(6))")],
    "dit_self_attention_on_raw_h": [("src = feats if l % 2 == 0 else xh", "src = feats if l % 2 == 0 else h")],
}


@pytest.mark.parametrize("name", [None, *_DIT_FINAL_MISTAKES])
def test_dit_final_modulation_probe(name):
    _check(_probe_dit_final, _DIT_FINAL_MISTAKES, name)


@pytest.mark.parametrize("name", [None, *_DIT_BLOCK_MISTAKES])
def test_dit_block_probe(name):
    _check(_probe_dit_blocks, _DIT_BLOCK_MISTAKES, name)


def test_mutant_loader_reproduces_the_oracle():
    """The mutant loader itself: with no edits it gives the oracle's output."""
    cfg, case, _ = _probe_rope()
    assert np.array_equal(_run(_mutant([]), cfg, case), _run(oexp, cfg, case))
