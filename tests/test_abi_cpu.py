"""Host-only checks of the C ABI library: it loads, exports every symbol the
header declares, reports its version and rejects bad arguments without a
GPU (validation happens before any device work)."""
import ctypes
import os
import re

import pytest

import paper_2608_03682_amd as px

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "phyai.h")).read()
    return sorted(set(re.findall(r"\b(phyai_[a-z0-9_]+)\s*\(", src)))


def test_library_is_built():
    assert os.path.exists(px.LIB_PATH), "run __graft_entry__.build() first"


def test_exports_every_declared_symbol():
    L = px.lib()
    names = _declared()
    assert set(names) == set(px.EXPORTS)
    for n in names:
        assert hasattr(L, n), n


def test_version():
    assert px.version() == 100


def test_null_arguments_are_rejected():
    L = px.lib()
    h = ctypes.c_void_p()
    assert L.phyai_load_expert(None, None, 0, None, ctypes.byref(h)) == px.PHYAI_EINVAL
    assert b"NULL" in L.phyai_last_error()
    assert L.phyai_denoise(None, None, None, None, None, 1, 1, None, None, None) == px.PHYAI_EINVAL
    assert L.phyai_prepare(None, 1, 1, None) == px.PHYAI_EINVAL
    assert L.phyai_fp8_to_bf16(None, None, -1, None) == px.PHYAI_EINVAL
    L.phyai_free_expert(None)


@pytest.mark.parametrize("field,value,needle", [
    ("head_dim", 96, b"head_dim"),
    ("d_model", 100, b"d_model"),
    ("d_model", 320, b"multiple of 256"),       # the row kernels take whole 256-column groups
    ("action_dim", 65, b"action_dim"),
    ("max_batch", 513, b"max_batch"),
    ("n_kv_heads", 3, b"multiple"),
])
def test_bad_config_rejected_before_device_work(field, value, needle):
    import workloads as wl
    cfg = px.make_config(wl.CONFIGS["pi0_bf16_b1"])
    setattr(cfg, field, value)
    h = ctypes.c_void_p()
    rc = px.lib().phyai_load_expert(ctypes.byref(cfg), None, 0, None, ctypes.byref(h))
    assert rc == px.PHYAI_EINVAL and not h.value
    assert needle in px.lib().phyai_last_error()


def test_missing_tensor_rejected():
    import workloads as wl
    cfg = px.make_config(wl.CONFIGS["tiny_fp32"])
    h = ctypes.c_void_p()
    rc = px.lib().phyai_load_expert(ctypes.byref(cfg), (px.Tensor * 1)(), 0, None, ctypes.byref(h))
    assert rc == px.PHYAI_EINVAL
    assert b"missing tensor 'in_w'" in px.lib().phyai_last_error()


def test_prefix_lm_rejections_before_device_work():
    """The prefix-LM variant: its own config rules and tensor list, and the
    prefill entry point's NULL handling (no GPU needed)."""
    import workloads as wl
    L = px.lib()
    assert L.phyai_prefill(None, None, None, None, 1, None) == px.PHYAI_EINVAL
    assert b"NULL" in L.phyai_last_error()
    base = wl.CONFIGS["plm_tiny_fp32"]
    h = ctypes.c_void_p()
    cfg = px.make_config(base, max_steps=0)
    cfg.state_token = 1
    assert L.phyai_load_expert(ctypes.byref(cfg), None, 0, None, ctypes.byref(h)) == px.PHYAI_EINVAL
    assert b"no state token" in L.phyai_last_error()
    cfg = px.make_config(base, max_steps=0)
    cfg.prefix_cap = 0
    assert L.phyai_load_expert(ctypes.byref(cfg), None, 0, None, ctypes.byref(h)) == px.PHYAI_EINVAL
    assert b"prefix_cap >= 1" in L.phyai_last_error()
    # horizon, action_dim, steps and timestep fields are not required
    cfg = px.make_config(base, max_steps=0)
    rc = L.phyai_load_expert(ctypes.byref(cfg), (px.Tensor * 1)(), 0, None, ctypes.byref(h))
    assert rc == px.PHYAI_EINVAL and not h.value
    assert b"missing tensor 'layers.0.attn_norm'" in L.phyai_last_error()


def test_vision_rejections_before_device_work():
    """The vision variant: its own config rules and tensor list, and the
    encode entry point's NULL handling (no GPU needed)."""
    import workloads as wl
    L = px.lib()
    assert L.phyai_encode_images(None, None, None, 768, 1, None) == px.PHYAI_EINVAL
    assert b"NULL" in L.phyai_last_error()
    base = wl.CONFIGS["vit_siglip_bf16_b1"]
    h = ctypes.c_void_p()
    for field, value, needle in [("patch_dim", 100, b"patch_dim"), ("d_out", 48, b"d_out"),
                                 ("n_kv_heads", 4, b"one key/value head per query head"),
                                 ("rope", 1, b"no RoPE"), ("n_images", 0, b"n_images >= 1"),
                                 ("max_batch", 200, b"max_batch * n_images")]:
        cfg = px.make_config(base, max_steps=0)
        setattr(cfg, field, value)
        assert L.phyai_load_expert(ctypes.byref(cfg), None, 0, None, ctypes.byref(h)) == px.PHYAI_EINVAL, field
        assert needle in L.phyai_last_error(), (field, L.phyai_last_error())
    cfg = px.make_config(base, max_steps=0)
    rc = L.phyai_load_expert(ctypes.byref(cfg), (px.Tensor * 1)(), 0, None, ctypes.byref(h))
    assert rc == px.PHYAI_EINVAL and not h.value
    assert b"missing tensor 'patch_w'" in L.phyai_last_error()
