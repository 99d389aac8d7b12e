"""Pins for the prefix-LM oracle (oracle/prefix_lm.py), CPU only.

The paper prints no worked example of the language prefix, so the oracle is
tied to facts outside itself:
  * a hand derivation on structured weights (uniform attention, MLP off)
    whose layer-1 keys follow from pinned parts only (RMSNorm, the matmuls
    written out here), with mistakes planted in a copy of the oracle's
    source that must each move the result;
  * agreement, layer by layer, with the expert trunk's own K/V when the
    expert runs the same weights over the same tokens as its suffix with an
    empty prefix (that trunk is pinned by the wiring probes);
  * properties of a bidirectional prefix block: a later token changes an
    earlier token's layer-1 K/V (a causal mask would not), layer-0 K/V are
    per-token, permutation equivariance without positions (broken with
    RoPE), padding never read, requests independent.
"""
import pathlib
import types

import numpy as np
import pytest

import oracle
from oracle import expert as oexp
from oracle import prefix_lm as opre
from oracle.numerics import rms_normalize
import workloads as wl

_SRC = pathlib.Path(opre.__file__).read_text()


def _mutant(edits):
    """A copy of oracle/prefix_lm.py with textual edits applied (each anchor
    must occur exactly once)."""
    src = _SRC
    for old, new in edits:
        assert src.count(old) == 1, f"mutation anchor not found exactly once: {old!r}"
        src = src.replace(old, new)
    mod = types.ModuleType("oracle._prefill_mutant")
    mod.__package__ = "oracle"
    mod.__file__ = opre.__file__
    exec(compile(src, opre.__file__ + " (mutant)", "exec"), mod.__dict__)
    return mod


def _cfg(**kw):
    base = dict(name="probe_plm", cfg_id=92, variant="prefix_lm", n_layers=2, d_model=64, n_q_heads=4,
                n_kv_heads=1, head_dim=16, d_mlp=128, horizon=0, action_dim=0, n_steps=0, prefix_cap=12,
                prefix_min=12, prefix_max=12, batch=1, state_token=False, rope=True, weight_dtype="f32",
                kv_dtype="f32", time_dim=0, init_std=0.2)
    base.update(kw)
    return wl.ExpertConfig(**base)


def _case(cfg, seed=0, batch=None, overrides=None):
    w = wl.make_weights(cfg, seed, overrides=overrides)
    return wl.make_prefill_case(cfg, seed, batch=batch, weights=w)


def _f64(t):
    return np.asarray(t.data, np.float32).astype(np.float64)


# ---------------------------------------------------------------------------
# Hand derivation on structured weights
# ---------------------------------------------------------------------------

def _probe_case(n=9, cap=12):
    """W_q = 0 in layer 0 (every valid key weighs the same), W_gate = 0 (GeGLU
    output zero), no RoPE, a ragged prefix (n of cap rows valid)."""
    cfg = _cfg(rope=False, prefix_cap=cap, prefix_min=n, prefix_max=n)
    d, qd = cfg.d_model, cfg.n_q_heads * cfg.head_dim
    ov = {"layers.0.wq": np.zeros((d, qd), np.float32), "layers.0.w_gate": np.zeros((d, cfg.d_mlp), np.float32)}
    return cfg, _case(cfg, seed=3, overrides=ov)


def _hand_layer1_keys(cfg, case):
    """Layer-1 keys from the structure: every query of layer 0 averages the
    values of the n valid tokens, so every head outputs that mean value
    vector; the MLP adds nothing; x1 = x0 + [mean v, ..., mean v] W_o."""
    n = int(case.prefix_len[0])
    w = case.weights
    x0 = case.embeds[0, :n].astype(np.float64)
    a0 = rms_normalize(x0, cfg.rms_eps) * (1.0 + _f64(w["layers.0.attn_norm"])[0])
    v0 = a0 @ _f64(w["layers.0.wv"])                                  # [n, D] (one kv head)
    vbar = v0.mean(axis=0)
    o = np.tile(vbar, cfg.n_q_heads)                                  # every query head
    x1 = x0 + (o @ _f64(w["layers.0.wo"]))[None, :]
    a1 = rms_normalize(x1, cfg.rms_eps) * (1.0 + _f64(w["layers.1.attn_norm"])[0])
    return a1 @ _f64(w["layers.1.wk"]), a1 @ _f64(w["layers.1.wv"])


_PROBE_MISTAKES = {
    "residual_dropped": [("h = h + o.reshape(n, nq * D) @ W(p + \"wo\")", "h = o.reshape(n, nq * D) @ W(p + \"wo\")")],
    "attn_norm_gain_without_one": [("* (1.0 + W(p + \"attn_norm\")[0])", "* W(p + \"attn_norm\")[0]")],
    "causal_mask": [("allowed = np.ones((n, n), dtype=bool)", "allowed = np.tril(np.ones((n, n), dtype=bool))")],
    "keys_from_queries_projection": [("k = (a @ W(p + \"wk\")).reshape(n, nkv, D)",
                                      "k = (a @ W(p + \"wv\")).reshape(n, nkv, D)")],
    "padding_rows_attended": [("out[:, :, b, :n] = prefill_request(cfg, weights, np.asarray(embeds[b, :n]), L, dtype)",
                               "out[:, :, b, :n] = prefill_request(cfg, weights, np.asarray(embeds[b]), L, dtype)[:, :, :n]")],
}


@pytest.mark.parametrize("name", [None, *_PROBE_MISTAKES])
def test_uniform_attention_probe(name):
    cfg, case = _probe_case()
    mod = opre if name is None else _mutant(_PROBE_MISTAKES[name])
    kv = mod.prefill(cfg, case.weights, case.embeds, case.prefix_len)
    k1, v1 = _hand_layer1_keys(cfg, case)
    n = int(case.prefix_len[0])
    err = max(np.abs(kv[1, 0, 0, :n] - k1).max(), np.abs(kv[1, 1, 0, :n] - v1).max())
    if name is None:
        assert err < 1e-12, err
        assert not kv[:, :, 0, n:].any(), "padding rows must be zero"
    else:
        assert err > 1e-6, f"planted mistake {name} not detected ({err})"


def test_mlp_probe():
    """W_q = 0 and W_o = 0 in layer 0 (attention adds nothing): x1 = x0 +
    GeGLU(n0) W_down, written out here with the tanh GELU (pinned)."""
    cfg = _cfg(rope=False)
    d, qd = cfg.d_model, cfg.n_q_heads * cfg.head_dim
    case = _case(cfg, seed=5, overrides={"layers.0.wq": np.zeros((d, qd), np.float32),
                                         "layers.0.wo": np.zeros((qd, d), np.float32)})
    w = case.weights
    x0 = case.embeds[0].astype(np.float64)
    m = rms_normalize(x0, cfg.rms_eps) * (1.0 + _f64(w["layers.0.mlp_norm"])[0])
    gate, up = m @ _f64(w["layers.0.w_gate"]), m @ _f64(w["layers.0.w_up"])
    gelu = 0.5 * gate * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (gate + 0.044715 * gate ** 3)))
    x1 = x0 + (gelu * up) @ _f64(w["layers.0.w_down"])
    a1 = rms_normalize(x1, cfg.rms_eps) * (1.0 + _f64(w["layers.1.attn_norm"])[0])
    kv = oracle.prefill(cfg, case.weights, case.embeds, case.prefix_len)
    assert np.abs(kv[1, 0, 0] - a1 @ _f64(w["layers.1.wk"])).max() < 1e-12
    swapped = _mutant([("(gelu_tanh(m @ W(p + \"w_gate\")) * (m @ W(p + \"w_up\")))",
                        "(gelu_tanh(m @ W(p + \"w_up\")) * (m @ W(p + \"w_gate\")))")])
    kv2 = swapped.prefill(cfg, case.weights, case.embeds, case.prefix_len)
    assert np.abs(kv2[1, 0, 0] - a1 @ _f64(w["layers.1.wk"])).max() > 1e-6


# ---------------------------------------------------------------------------
# Agreement with the expert trunk
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("rope", [True, False])
def test_matches_expert_trunk_over_the_same_tokens(rope, monkeypatch):
    """An expert whose suffix is the prefix tokens themselves, with an empty
    prefix and no state token, computes at every layer the K/V that the
    prefix LM must return (same weights, positions 0.., all-to-all mask)."""
    cfg = _cfg(rope=rope, n_layers=3)
    case = _case(cfg, seed=7)
    kv = oracle.prefill(cfg, case.weights, case.embeds, case.prefix_len)
    # the expert's trunk also runs the last block's MLP: give it zero weights
    d, qd, F = cfg.d_model, cfg.n_q_heads * cfg.head_dim, cfg.d_mlp
    wts = dict(case.weights)
    last = f"layers.{cfg.n_layers - 1}."
    for nm, shape in (("wo", (qd, d)), ("mlp_norm", (1, d)), ("w_gate", (d, F)), ("w_up", (d, F)),
                      ("w_down", (F, d))):
        wts[last + nm] = wl.StoredTensor("f32", np.zeros(shape, np.float32))
    ecfg = cfg.replace(variant="pi0", horizon=cfg.prefix_cap, prefix_cap=0, prefix_min=0, prefix_max=0)
    seen = []
    real = oexp.attention

    def spy(q, k, v, allowed):
        seen.append((k.copy(), v.copy()))
        return real(q, k, v, allowed)

    monkeypatch.setattr(oexp, "attention", spy)
    W = oexp.DecodedWeights(wts)

    def norm_fn(site, h):
        kind, l = site
        return rms_normalize(h, cfg.rms_eps) * (1.0 + W.vec(f"layers.{l}.{kind}_norm"))

    D, nkv = cfg.head_dim, cfg.n_kv_heads
    empty = lambda l: (np.zeros((0, nkv, D)), np.zeros((0, nkv, D)))
    oexp._trunk(ecfg, W, case.embeds[0].astype(np.float64), 0, empty, norm_fn)
    assert len(seen) == cfg.n_layers
    for l, (k, v) in enumerate(seen):
        assert np.abs(kv[l, 0, 0] - k.reshape(k.shape[0], -1)).max() < 1e-12
        assert np.abs(kv[l, 1, 0] - v.reshape(v.shape[0], -1)).max() < 1e-12


# ---------------------------------------------------------------------------
# Properties of the bidirectional prefix block
# ---------------------------------------------------------------------------

def test_later_token_changes_earlier_tokens_deeper_layers_only():
    cfg = _cfg()
    case = _case(cfg, seed=11)
    kv = oracle.prefill(cfg, case.weights, case.embeds, case.prefix_len)
    emb = case.embeds.copy()
    emb[0, -1] += 1.0                       # the last token only
    kv2 = oracle.prefill(cfg, case.weights, emb, case.prefix_len)
    # layer 0: per token (no mixing before the first attention)
    assert np.array_equal(kv[0, :, 0, :-1], kv2[0, :, 0, :-1])
    assert not np.array_equal(kv[0, :, 0, -1], kv2[0, :, 0, -1])
    # layer 1: the first token sees the last one (bidirectional block)
    assert np.abs(kv[1, :, 0, 0] - kv2[1, :, 0, 0]).max() > 1e-6


def test_permutation_equivariance_without_positions_and_broken_with_rope():
    for rope, equivariant in ((False, True), (True, False)):
        cfg = _cfg(rope=rope)
        case = _case(cfg, seed=13)
        perm = np.random.default_rng(0).permutation(cfg.prefix_cap)
        kv = oracle.prefill(cfg, case.weights, case.embeds, case.prefix_len)
        kvp = oracle.prefill(cfg, case.weights, case.embeds[:, perm], case.prefix_len)
        err = np.abs(kvp[1] - kv[1][:, :, perm]).max()
        assert (err < 1e-12) if equivariant else (err > 1e-6), (rope, err)


def test_padding_never_read_and_requests_independent():
    cfg = _cfg(prefix_cap=16, prefix_min=5, prefix_max=16, batch=4)
    case = _case(cfg, seed=17)
    kv = oracle.prefill(cfg, case.weights, case.embeds, case.prefix_len)
    emb = case.embeds.copy()
    for b, n in enumerate(case.prefix_len):
        emb[b, n:] = np.nan
    kvn = oracle.prefill(cfg, case.weights, emb, case.prefix_len)
    assert np.array_equal(kv, kvn)
    for b, n in enumerate(case.prefix_len):
        assert not kv[:, :, b, n:].any()
    # a request alone gives its slice of the batch result
    one = oracle.prefill(cfg, case.weights, case.embeds[2:3], case.prefix_len[2:3])
    assert np.array_equal(one[:, :, 0], kv[:, :, 2])


def test_empty_prefix_gives_zeros():
    cfg = _cfg()
    case = _case(cfg, seed=19)
    kv = oracle.prefill(cfg, case.weights, case.embeds, np.array([0], np.int32))
    assert kv.shape == (cfg.n_layers, 2, 1, cfg.prefix_cap, cfg.n_kv_heads * cfg.head_dim)
    assert not kv.any()


def test_layer_limit_is_a_prefix_of_the_full_result():
    cfg = _cfg(n_layers=3)
    case = _case(cfg, seed=23)
    full = oracle.prefill(cfg, case.weights, case.embeds, case.prefix_len)
    part = oracle.prefill(cfg, case.weights, case.embeds, case.prefix_len, n_layers=2)
    assert np.array_equal(full[:2], part)
