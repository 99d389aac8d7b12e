"""GPU invariants of the denoising path (through the C ABI): properties the
method forces at any size, checked bit-exactly where the arithmetic allows."""
import os

import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_helpers import compare, run_gpu, small_cfg, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _px():
    import paper_2608_03682_amd as px
    return px


def test_prefix_buffer_is_read_only_and_calls_are_deterministic():
    cfg = small_cfg("pi0", batch=3)
    print("[case] prefix read-only / determinism", flush=True)
    case = wl.make_case(cfg, seed=5)
    ex = _px().Expert(cfg, case.weights)
    dev = to_device(case)
    before = dev[0].clone()
    a = run_gpu(ex, case, dev)
    b = run_gpu(ex, case, dev)
    assert torch.equal(dev[0], before)
    assert np.array_equal(a, b)


def test_graph_replay_equals_eager_launches():
    cfg = small_cfg("pi05", batch=2)
    print("[case] graph vs eager", flush=True)
    case = wl.make_case(cfg, seed=6)
    ex = _px().Expert(cfg, case.weights)
    dev = to_device(case)
    g = run_gpu(ex, case, dev)
    os.environ["PHYAI_NO_GRAPH"] = "1"
    try:
        e = run_gpu(ex, case, dev)
    finally:
        del os.environ["PHYAI_NO_GRAPH"]
    assert np.array_equal(g, e)


@pytest.mark.parametrize("variant", ["pi0", "dit"])
def test_nan_padding_never_read(variant):
    cfg = small_cfg(variant, batch=3)
    print(f"[case] NaN padding {variant}", flush=True)
    case = wl.make_case(cfg, seed=7)
    assert case.prefix_len.min() < cfg.prefix_cap
    ex = _px().Expert(cfg, case.weights)
    ref = run_gpu(ex, case)
    case.prefix = wl.make_prefix(cfg, case.prefix_len, 7, pad_value=float("nan"))
    out = run_gpu(ex, case)
    assert np.isfinite(out).all()
    assert np.array_equal(out, ref)


def test_requests_are_bit_independent():
    cfg = small_cfg("pi0", batch=7)        # 357 rows: the tiled GEMM path
    print("[case] batch independence", flush=True)
    case = wl.make_case(cfg, seed=8)
    ex = _px().Expert(cfg, case.weights)
    ref = run_gpu(ex, case)
    case.noise = case.noise.copy()
    case.noise[1:] = -case.noise[1:]
    case.prefix = case.prefix.copy()
    case.prefix[:, :, 2:] = case.prefix[:, :, :1]
    case.state = case.state.copy()
    case.state[3] += 1.0
    out = run_gpu(ex, case)
    assert np.array_equal(out[0], ref[0])
    assert not np.allclose(out[1], ref[1])


def test_schedule_change_rebuilds_tables():
    cfg = small_cfg("pi05", batch=1)
    print("[case] non-uniform schedule", flush=True)
    case = wl.make_case(cfg, seed=9)
    ex = _px().Expert(cfg, case.weights)
    default = run_gpu(ex, case)
    case.timesteps = np.array([1.0, 0.9, 0.5, 0.0], dtype=np.float32)
    got = run_gpu(ex, case)
    ref = oracle.denoise(cfg, case.weights, case.prefix, case.prefix_len, case.noise, case.timesteps, case.state)
    compare("pi05 non-uniform schedule", got, ref, cfg)
    case.timesteps = wl.default_timesteps(cfg.n_steps)
    assert np.array_equal(run_gpu(ex, case), default)


def test_output_may_alias_noise():
    cfg = small_cfg("pi0", batch=2)
    case = wl.make_case(cfg, seed=10)
    ex = _px().Expert(cfg, case.weights)
    prefix, noise, state = to_device(case)
    ref = run_gpu(ex, case, (prefix, noise.clone(), state))
    ex.denoise(prefix, case.prefix_len, noise, case.timesteps, state, out=noise)
    torch.cuda.synchronize()
    assert np.array_equal(noise.cpu().numpy().astype(np.float64), ref)


@pytest.mark.parametrize("variant", ["pi0", "pi05", "dit"])
def test_zero_readout_closed_form(variant):
    """W_out = 0 makes v = b_out at every step, so x_K = x_0 - b_out exactly up
    to the fp32 Euler sums."""
    cfg = small_cfg(variant, batch=2)
    out_b = np.linspace(-1.0, 1.0, cfg.action_dim, dtype=np.float32)[None]
    w = wl.make_weights(cfg, 11, overrides={"out_w": np.zeros((cfg.d_model, cfg.action_dim)), "out_b": out_b})
    case = wl.make_case(cfg, seed=11, weights=w)
    ex = _px().Expert(cfg, case.weights)
    got = run_gpu(ex, case)
    b = oracle.decode_bf16(case.weights["out_b"].data)[0]
    assert np.allclose(got, case.noise - b[None, None, :], atol=1e-6, rtol=1e-6)


def test_one_hot_value_probe_is_bit_exact():
    """Embeddings 0, W_q = 0 (uniform scores), suffix V = 0, prefix V row j =
    e_j, W_o = identity, MLP off.  After one layer the residual stream of
    token i holds bf16(1/N_i) in the first prefix_len coordinates of every
    head and 0 elsewhere, N_i = keys token i may see: prefix_len + 1 for the
    state token, prefix_len + H + 1 for actions.  Checks the block mask and the
    key indexing bit for bit, for prefix lengths ending mid-tile."""
    cfg = small_cfg("pi0", n_layers=1, n_steps=1, batch=3, prefix_cap=64, prefix_min=5, prefix_max=64)
    d, D, nq, H, M = cfg.d_model, cfg.head_dim, cfg.n_q_heads, cfg.horizon, cfg.tokens
    z = lambda r, c: np.zeros((r, c))
    ov = {"in_w": z(cfg.action_dim, d), "in_b": z(1, d), "time_w2": z(d, d), "time_b2": z(1, d),
          "state_w": z(cfg.action_dim, d), "state_b": z(1, d), "layers.0.wq": z(d, nq * D),
          "layers.0.wv": z(d, D), "layers.0.wo": np.eye(nq * D, d), "layers.0.w_gate": z(d, cfg.d_mlp)}
    case = wl.make_case(cfg, seed=12, weights=wl.make_weights(cfg, 12, overrides=ov))
    case.prefix_len = np.array([5, 37, 64], dtype=np.int32)
    pre = np.zeros((1, 2, cfg.batch, cfg.prefix_cap, D), dtype=np.float32)
    pre[0, 0] = np.random.default_rng(0).standard_normal(pre[0, 0].shape)
    for b, P in enumerate(case.prefix_len):
        pre[0, 1, b, np.arange(P), np.arange(P)] = 1.0
    case.prefix = wl.bf16_bits_from_f32(pre)
    ex = _px().Expert(cfg, case.weights)
    dev = to_device(case)
    run_gpu(ex, case, dev)
    h = ex.debug_hidden(cfg.batch).cpu().numpy()
    for b, P in enumerate(case.prefix_len):
        for i in range(M):
            n_allowed = P + 1 if i == 0 else P + M
            want = np.zeros(D, dtype=np.float32)
            want[:P] = oracle.decode_bf16(wl.bf16_bits_from_f32(np.float32([1.0 / n_allowed])))[0]
            row = h[b * M + i]
            for g in range(nq):
                assert np.array_equal(row[g * D:(g + 1) * D], want), (b, i, g)


def test_invalid_arguments_leave_output_untouched():
    px = _px()
    cfg = small_cfg("pi0", batch=2)
    case = wl.make_case(cfg, seed=13)
    ex = px.Expert(cfg, case.weights)
    prefix, noise, state = to_device(case)
    out = torch.full_like(noise, 7.0)
    bad_len = case.prefix_len.copy()
    bad_len[1] = cfg.prefix_cap + 1
    with pytest.raises(px.PhyaiError, match="prefix_len"):
        ex.denoise(prefix, bad_len, noise, case.timesteps, state, out=out)
    with pytest.raises(px.PhyaiError, match="state"):
        ex.denoise(prefix, case.prefix_len, noise, case.timesteps, None, out=out)
    with pytest.raises(px.PhyaiError, match="n_steps"):
        ex.denoise(prefix, case.prefix_len, noise, wl.default_timesteps(cfg.n_steps + 1), state, out=out)
    with pytest.raises(px.PhyaiError, match="non-finite"):
        ex.denoise(prefix, case.prefix_len, noise, np.float32([1.0, np.nan, 0.5, 0.0]), state, out=out)
    # a contiguous view 4 bytes past a 16-byte boundary
    shifted = torch.empty(noise.numel() + 1, dtype=noise.dtype, device=noise.device)[1:].view(noise.shape)
    shifted.copy_(noise)
    with pytest.raises(px.PhyaiError, match="16-byte aligned"):
        ex.denoise(prefix, case.prefix_len, shifted, case.timesteps, state, out=out)
    with pytest.raises(px.PhyaiError, match="16-byte aligned"):
        ex.denoise(prefix, case.prefix_len, noise, case.timesteps, state, out=shifted)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())


def test_permutation_equivariance_tiny_fp32_config():
    """Without positional terms (the tiny fp32 workload has no RoPE and no
    state token) the action tokens are exchangeable: permuting the noise rows
    permutes the output rows the same way.  Only the order of the attention
    sums over the suffix keys changes, so the two runs agree to float32
    rounding; the oracle checks the unpermuted run to the parity bar."""
    cfg = wl.CONFIGS["tiny_fp32"]
    assert not cfg.rope and not cfg.state_token
    print("[case] permutation equivariance tiny_fp32", flush=True)
    case = wl.make_case(cfg, seed=9)
    ex = _px().Expert(cfg, case.weights)
    ref = run_gpu(ex, case)
    compare("tiny_fp32 seed 9", ref, oracle.denoise(cfg, case.weights, case.prefix, case.prefix_len, case.noise,
                                                    case.timesteps, case.state), cfg)
    for seed in (1, 2):
        perm = np.random.default_rng(seed).permutation(cfg.horizon)
        case.noise = case.noise.copy()
        noise0 = case.noise.copy()
        case.noise = noise0[:, perm]
        out = run_gpu(ex, case)
        case.noise = noise0
        err = np.abs(out - ref[:, perm]).max()
        print(f"[parity] permuted run vs permuted reference: max_abs={err:.3e}", flush=True)
        assert err <= 1e-5 * max(1.0, float(np.sqrt(np.mean(ref ** 2))))
    ex.close()
