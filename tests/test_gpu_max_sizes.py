"""The largest batches the library accepts (512 requests, 512 images), on
small shapes, through the C ABI: every output finite, sampled requests (the
first, one in the middle, the last) against the oracle on each path's own
bar, and one request past the limit refused at load.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_helpers import compare, run_gpu, small_cfg

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

MAX = 512
SAMPLE = (0, MAX // 2 - 1, MAX - 1)


def _px():
    import paper_2608_03682_amd as px
    return px


def test_expert_at_the_batch_limit():
    px = _px()
    cfg = small_cfg("pi0", batch=MAX, n_steps=2)
    print(f"[case] expert pi0 batch {MAX}", flush=True)
    case = wl.make_case(cfg, seed=61)
    ex = px.Expert(cfg, case.weights)
    got = run_gpu(ex, case)
    ex.close()
    assert np.isfinite(got).all()
    idx = list(SAMPLE)
    ref = oracle.denoise(cfg, case.weights, case.prefix, case.prefix_len[idx], case.noise[idx], case.timesteps,
                         case.state[idx], slots=idx)
    compare(f"expert batch {MAX} requests {idx}", got[idx], ref, cfg)
    with pytest.raises(px.PhyaiError, match="max_batch"):
        px.Expert(cfg.replace(batch=MAX + 1), case.weights)


def test_prefix_lm_at_the_batch_limit():
    px = _px()
    from test_gpu_prefill import check_kv, plm_cfg
    cfg = plm_cfg(batch=MAX, prefix_cap=40, prefix_min=1, prefix_max=40)
    print(f"[case] prefix LM batch {MAX}", flush=True)
    case = wl.make_prefill_case(cfg, seed=63)
    m = px.PrefixLM(cfg, case.weights, max_batch=MAX)
    kv = m.prefill(torch.from_numpy(case.embeds).cuda(), case.prefix_len)
    torch.cuda.synchronize()
    got = oracle.decode_bf16(kv.cpu().numpy().view(np.uint16)).astype(np.float64)
    m.close()
    assert np.isfinite(got).all()
    idx = list(SAMPLE)
    ref = oracle.prefill(cfg, case.weights, case.embeds[idx], case.prefix_len[idx])
    check_kv(f"prefix LM batch {MAX} requests {idx}", cfg, got[:, :, idx], ref, case.prefix_len[idx])


def test_vision_at_the_image_limit():
    px = _px()
    from test_gpu_vision import check_tokens, vit_cfg
    cfg = vit_cfg(batch=MAX // 2, n_images=2)
    print(f"[case] vision {MAX // 2} requests x 2 images", flush=True)
    case = wl.make_vision_case(cfg, seed=65)
    m = px.VisionTower(cfg, case.weights)
    tok = m.encode(torch.from_numpy(case.patches).cuda())
    torch.cuda.synchronize()
    got = tok.cpu().numpy().astype(np.float64)
    m.close()
    assert np.isfinite(got).all()
    idx = [0, cfg.batch // 2, cfg.batch - 1]
    ref = oracle.encode_images(cfg, case.weights, case.patches[idx])
    check_tokens(f"vision {MAX} images, requests {idx}", cfg, got[idx], ref)
    with pytest.raises(px.PhyaiError, match="max_batch"):
        px.VisionTower(cfg.replace(batch=cfg.batch + 1), case.weights)
