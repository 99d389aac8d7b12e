"""The allocation-free entry point, phyai_denoise_static, against phyai_denoise
(through the C ABI): same inputs, same kernels, so the outputs must agree bit
for bit; the oracle checks the first call to the parity bar as well.  Two
calls in a row, the second with a smaller batch, so that the second reads a
static scratch array the first has left full."""
import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_helpers import compare, small_cfg, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _px():
    import paper_2608_03682_amd as px
    return px


def _both(ex, case):
    prefix, noise, state = to_device(case)
    ref = ex.denoise(prefix, case.prefix_len, noise, case.timesteps, state)
    out = torch.full_like(noise, float("nan"))
    ex.denoise(prefix, case.prefix_len, noise, case.timesteps, state, out=out, static=True)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64), ref.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("variant", ["pi0", "pi05"])
def test_static_entry_point_matches_graph_entry_point(variant):
    cfg = small_cfg(variant, batch=3)
    print(f"[case] static entry point {variant}: batch 3 then batch 1", flush=True)
    case = wl.make_case(cfg, seed=31)
    ex = _px().Expert(cfg, case.weights)
    got, ref = _both(ex, case)
    assert np.array_equal(got, ref)
    orc = oracle.denoise(cfg, case.weights, case.prefix, case.prefix_len, case.noise, case.timesteps, case.state)
    compare(f"static {variant} batch 3", got, orc, cfg)
    small = wl.make_case(cfg, seed=32, batch=1, weights=case.weights)
    got1, ref1 = _both(ex, small)
    assert np.array_equal(got1, ref1)
    # the graph path is untouched by the static calls
    again, _ = _both(ex, case)
    assert np.array_equal(again, ref)
    ex.close()


def test_static_entry_point_full_batch1_workload():
    """The pi0-shaped batch-1 workload in the bench's launch configuration
    (14 key splits merged by the output projection, split-K residual GEMMs)."""
    cfg = wl.CONFIGS["pi0_bf16_b1"]
    print("[case] static entry point, pi0 batch-1 workload", flush=True)
    case = wl.make_case(cfg, seed=33)
    ex = _px().Expert(cfg, case.weights)
    got, ref = _both(ex, case)
    assert np.array_equal(got, ref)
    ex.close()


def test_static_entry_point_rejects_oversized_scratch():
    """A call whose key-split partials exceed the 32 MiB array is refused
    before anything is enqueued: 255 requests of one 128-row attention block
    each, two key splits over 307 keys (five key tiles, enough to split),
    head_dim 256 (about 34 MB of partials)."""
    px = _px()
    cfg = small_cfg("pi0", batch=255, n_layers=1, d_model=512, n_q_heads=2, head_dim=256, d_mlp=512,
                    prefix_cap=256, prefix_min=256, prefix_max=256)
    print("[case] static entry point oversized scratch", flush=True)
    case = wl.make_case(cfg, seed=34)
    ex = px.Expert(cfg, case.weights)
    prefix, noise, state = to_device(case)
    out = torch.full_like(noise, 7.0)
    with pytest.raises(px.PhyaiError, match="static limit"):
        ex.denoise(prefix, case.prefix_len, noise, case.timesteps, state, out=out, static=True)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    ex.close()
