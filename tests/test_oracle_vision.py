"""Pins for the vision-tower oracle (oracle/vision.py), CPU only.

The paper prints no worked example of the vision tower, so the oracle is tied
to facts outside itself:
  * the whole tower, on small shapes, against PyTorch's own pre-norm
    transformer encoder layer (nn.TransformerEncoderLayer with norm_first,
    nn.MultiheadAttention inside, LayerNorm and a tanh-GELU MLP), composed
    with a linear patch embedding, a final LayerNorm and a linear projector,
    all in float64: a library implementation of the same definition;
  * mistakes planted in a copy of the oracle's source (a dropped bias, the
    plain gain instead of 1 + w, no position embedding, a causal mask,
    swapped key/value weights, heads split the wrong way) each move the result
    off that library value;
  * properties: images and requests are independent, the patches of an image
    are permutation-equivariant together with their position embeddings, and
    fewer blocks is a prefix of the computation.
"""
import pathlib
import types

import numpy as np
import pytest

import oracle
from oracle import vision as ovis
import workloads as wl

torch = pytest.importorskip("torch")

_SRC = pathlib.Path(ovis.__file__).read_text()


def _cfg(**kw):
    base = dict(name="probe_vit", cfg_id=93, variant="vision", n_layers=2, d_model=64, n_q_heads=4,
                n_kv_heads=4, head_dim=16, d_mlp=128, horizon=0, action_dim=0, n_steps=0, prefix_cap=24,
                prefix_min=24, prefix_max=24, batch=2, state_token=False, rope=False, weight_dtype="f32",
                kv_dtype="f32", time_dim=0, init_std=0.2, n_images=2, n_patches=12, patch_dim=48, d_out=32)
    base.update(kw)
    return wl.ExpertConfig(**base)


def _mutant(edits):
    """A copy of oracle/vision.py with textual edits applied (each anchor must
    occur exactly once)."""
    src = _SRC
    for old, new in edits:
        assert src.count(old) == 1, f"mutation anchor not found exactly once: {old!r}"
        src = src.replace(old, new)
    mod = types.ModuleType("oracle._vision_mutant")
    mod.__package__ = "oracle"
    mod.__file__ = ovis.__file__
    exec(compile(src, ovis.__file__ + " (mutant)", "exec"), mod.__dict__)
    return mod


def _torch_tower(cfg, weights, patches):
    """The tower built from torch.nn modules: [B][I][N][patch_dim] -> [B][I*N][d_out]."""
    import torch.nn as nn
    import torch.nn.functional as F

    def T(name):
        return torch.from_numpy(oracle.decode_stored(weights[name]).astype(np.float64))

    d, eps = cfg.d_model, cfg.rms_eps
    layers = []
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        m = nn.TransformerEncoderLayer(d, cfg.n_q_heads, dim_feedforward=cfg.d_mlp, dropout=0.0,
                                       activation=lambda z: F.gelu(z, approximate="tanh"), layer_norm_eps=eps,
                                       batch_first=True, norm_first=True, dtype=torch.float64)
        with torch.no_grad():
            # nn.Linear keeps [out][in]; the stored matrices are [in][out]
            m.self_attn.in_proj_weight.copy_(torch.cat([T(p + "wq").T, T(p + "wk").T, T(p + "wv").T]))
            m.self_attn.in_proj_bias.copy_(torch.cat([T(p + "bq")[0], T(p + "bk")[0], T(p + "bv")[0]]))
            m.self_attn.out_proj.weight.copy_(T(p + "wo").T)
            m.self_attn.out_proj.bias.copy_(T(p + "bo")[0])
            m.linear1.weight.copy_(T(p + "mlp_w1").T)
            m.linear1.bias.copy_(T(p + "mlp_b1")[0])
            m.linear2.weight.copy_(T(p + "mlp_w2").T)
            m.linear2.bias.copy_(T(p + "mlp_b2")[0])
            m.norm1.weight.copy_(1.0 + T(p + "ln1_w")[0])
            m.norm1.bias.copy_(T(p + "ln1_b")[0])
            m.norm2.weight.copy_(1.0 + T(p + "ln2_w")[0])
            m.norm2.bias.copy_(T(p + "ln2_b")[0])
        layers.append(m.eval())
    B, I, N, _ = patches.shape
    x = torch.from_numpy(patches.astype(np.float64)).reshape(B * I, N, -1)
    with torch.no_grad():
        h = x @ T("patch_w") + T("patch_b")[0] + T("pos_emb")
        for m in layers:
            h = m(h)
        z = F.layer_norm(h, (d,), 1.0 + T("post_ln_w")[0], T("post_ln_b")[0], eps)
        y = z @ T("proj_w") + T("proj_b")[0]
    return y.reshape(B, I * N, cfg.d_out).numpy()


def _case(cfg, seed=0):
    return wl.make_vision_case(cfg, seed)


def _rel(a, b):
    return float(np.abs(a - b).max() / max(1e-30, np.abs(b).max()))


def test_matches_torch_encoder_layers():
    cfg = _cfg()
    case = _case(cfg, 5)
    got = oracle.encode_images(cfg, case.weights, case.patches)
    ref = _torch_tower(cfg, case.weights, case.patches)
    assert got.shape == (cfg.batch, cfg.n_images * cfg.n_patches, cfg.d_out)
    assert _rel(got, ref) < 1e-12, _rel(got, ref)


def test_matches_torch_with_bf16_weights_and_one_head():
    # stored bf16 weights are decoded exactly; one head of the full width
    cfg = _cfg(weight_dtype="bf16", n_q_heads=1, n_kv_heads=1, head_dim=64, n_layers=1)
    case = _case(cfg, 6)
    assert _rel(oracle.encode_images(cfg, case.weights, case.patches),
                _torch_tower(cfg, case.weights, case.patches)) < 1e-12


MUTANTS = {
    "q bias dropped": [('+ W.vec(p + "bq")', "")],
    "gain w instead of 1 + w": [("* (1.0 + W.vec(wname))", "* W.vec(wname)")],
    "norm bias dropped": [("+ W.vec(bname)\n", "\n")],
    "no position embedding": [('+ W("pos_emb")[:n]', "")],
    "causal mask": [("everyone = np.ones((n, n), dtype=bool)", "everyone = np.tril(np.ones((n, n), dtype=bool))")],
    "key and value weights swapped": [('(a @ W(p + "wk")', '(a @ W(p + "wTMP")'), ('(a @ W(p + "wv")', '(a @ W(p + "wk")'),
                                      ('(a @ W(p + "wTMP")', '(a @ W(p + "wv")')],
    "heads split head-minor": [(".reshape(n, H, D)\n        k", ".reshape(n, D, H).transpose(0, 2, 1)\n        k")],
    "MLP bias inside the GELU dropped": [('+ W.vec(p + "mlp_b1")', "")],
    "post-norm skipped": [('z = _layer_norm(W, h, "post_ln_w", "post_ln_b", eps)', "z = h")],
    "residual of the attention dropped": [('h = h + o @ W(p + "wo")', 'h = o @ W(p + "wo")')],
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name):
    cfg = _cfg()
    case = _case(cfg, 7)
    ref = _torch_tower(cfg, case.weights, case.patches)
    assert _rel(oracle.encode_images(cfg, case.weights, case.patches), ref) < 1e-12
    mod = _mutant(MUTANTS[name])
    bad = mod.encode_images(cfg, case.weights, case.patches)
    assert _rel(bad, ref) > 1e-3, f"planted mistake '{name}' not caught ({_rel(bad, ref):.2e})"


def test_images_and_requests_are_independent():
    cfg = _cfg()
    case = _case(cfg, 8)
    a = oracle.encode_images(cfg, case.weights, case.patches)
    p = case.patches.copy()
    p[0, 1] += 1.0          # request 0, image 1
    p[1] *= -1.0            # every image of request 1
    b = oracle.encode_images(cfg, case.weights, p)
    N = cfg.n_patches
    assert np.array_equal(a[0, :N], b[0, :N])
    assert not np.allclose(a[0, N:], b[0, N:])
    assert not np.allclose(a[1], b[1])


def test_patches_permute_with_their_position_embeddings():
    cfg = _cfg()
    case = _case(cfg, 9)
    perm = np.random.default_rng(0).permutation(cfg.n_patches)
    a = oracle.encode_images(cfg, case.weights, case.patches)
    w = dict(case.weights)
    pos = np.asarray(w["pos_emb"].data)
    w["pos_emb"] = wl.StoredTensor("f32", np.ascontiguousarray(pos[perm]))
    b = oracle.encode_images(cfg, w, case.patches[:, :, perm])
    N = cfg.n_patches
    for i in range(cfg.n_images):
        np.testing.assert_allclose(b[:, i * N:(i + 1) * N], a[:, i * N + perm], rtol=0, atol=1e-12)
    # the patches alone, position embeddings left in place: a different result
    c = oracle.encode_images(cfg, case.weights, case.patches[:, :, perm])
    assert not np.allclose(c[:, :N], a[:, perm], atol=1e-6)


def test_fewer_blocks_is_a_prefix_of_the_computation():
    cfg = _cfg(n_layers=3)
    case = _case(cfg, 10)
    two = oracle.encode_images(cfg, case.weights, case.patches, n_layers=2)
    ref = oracle.encode_images(cfg.replace(n_layers=2), case.weights, case.patches)
    assert np.array_equal(two, ref)
