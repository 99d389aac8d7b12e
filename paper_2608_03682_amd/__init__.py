"""Python binding of the gfx950 action-expert library (``libphyai.so``).

Argument marshalling only: every step of the denoising loop runs in the HIP
kernels behind the C ABI declared in ``include/phyai.h``.  PyTorch supplies
device memory and streams.  Importing this package never falls back to a CPU
path: if the library is missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libphyai.so")

PHYAI_OK, PHYAI_EINVAL, PHYAI_ENOMEM, PHYAI_EHIP, PHYAI_EUNSUPPORTED = 0, -1, -2, -3, -4
_VARIANT = {"pi0": 0, "pi05": 1, "dit": 2, "prefix_lm": 3, "vision": 4}
_DTYPE = {"f32": 0, "bf16": 1, "fp8": 2, "fp4": 3}

# Every symbol include/phyai.h declares.
EXPORTS = ("phyai_load_expert", "phyai_denoise", "phyai_denoise_static", "phyai_prepare", "phyai_debug_hidden",
           "phyai_profile_stage", "phyai_fp8_to_bf16", "phyai_free_expert", "phyai_last_error",
           "phyai_version", "phyai_prefill", "phyai_encode_images")
STAGES = {"norm1": 0, "qkv": 1, "attn": 2, "oproj": 3, "norm2": 4, "mlp_up": 5, "mlp_down": 6}


class PhyaiError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"phyai error {code}: {msg}")
        self.code = code


class Config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "variant", "n_layers", "d_model", "n_q_heads", "n_kv_heads", "head_dim", "d_mlp", "horizon",
        "action_dim", "max_steps", "prefix_cap", "max_batch", "state_token", "rope", "weight_dtype",
        "kv_dtype", "d_feat", "time_dim")] + [(n, ctypes.c_float) for n in (
        "rms_eps", "sin_min_period", "sin_max_period", "rope_base")] + [(n, ctypes.c_int32) for n in (
        "n_images", "n_patches", "patch_dim", "d_out")]


class Tensor(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("dtype", ctypes.c_int32), ("rows", ctypes.c_int32),
                ("cols", ctypes.c_int32), ("data", ctypes.c_void_p), ("scale", ctypes.c_void_p)]


_lib_handle = None


def lib() -> ctypes.CDLL:
    """Load libphyai.so (raises if it is missing: there is no fallback)."""
    global _lib_handle
    if _lib_handle is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing; build it with `python -m paper_2608_03682_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.phyai_load_expert.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(Tensor), i32, vp,
                                        ctypes.POINTER(vp)]
        L.phyai_denoise.argtypes = [vp, vp, vp, vp, vp, i32, i32, vp, vp, vp]
        L.phyai_denoise_static.argtypes = [vp, vp, vp, vp, vp, i32, i32, vp, vp, vp]
        L.phyai_prepare.argtypes = [vp, i32, i32, vp]
        L.phyai_debug_hidden.argtypes = [vp, vp, i32, vp]
        L.phyai_fp8_to_bf16.argtypes = [vp, vp, i64, vp]
        L.phyai_profile_stage.argtypes = [vp, i32, i32, vp]
        L.phyai_prefill.argtypes = [vp, vp, vp, vp, i32, vp]
        L.phyai_encode_images.argtypes = [vp, vp, vp, i32, i32, vp]
        L.phyai_free_expert.argtypes = [vp]
        L.phyai_free_expert.restype = None
        L.phyai_last_error.restype = ctypes.c_char_p
        for f in ("phyai_load_expert", "phyai_denoise", "phyai_denoise_static", "phyai_prepare", "phyai_debug_hidden",
                  "phyai_profile_stage", "phyai_fp8_to_bf16", "phyai_version", "phyai_prefill",
                  "phyai_encode_images"):
            getattr(L, f).restype = ctypes.c_int
        _lib_handle = L
    return _lib_handle


def _check(rc: int):
    if rc != PHYAI_OK:
        raise PhyaiError(rc, lib().phyai_last_error().decode())


def _stream(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous device tensor")
    return t.data_ptr()


def make_config(cfg, max_batch: Optional[int] = None, max_steps: Optional[int] = None) -> Config:
    """Fill the C config from any object with the workload fields."""
    return Config(
        variant=_VARIANT[cfg.variant], n_layers=cfg.n_layers, d_model=cfg.d_model,
        n_q_heads=cfg.n_q_heads, n_kv_heads=cfg.n_kv_heads, head_dim=cfg.head_dim, d_mlp=cfg.d_mlp,
        horizon=cfg.horizon, action_dim=cfg.action_dim,
        max_steps=max_steps if max_steps is not None else cfg.n_steps,
        prefix_cap=cfg.prefix_cap, max_batch=max_batch if max_batch is not None else cfg.batch,
        state_token=int(cfg.state_token), rope=int(cfg.rope), weight_dtype=_DTYPE[cfg.weight_dtype],
        kv_dtype=_DTYPE[cfg.kv_dtype], d_feat=cfg.d_feat, time_dim=cfg.time_dim,
        rms_eps=cfg.rms_eps, sin_min_period=cfg.sin_min_period, sin_max_period=cfg.sin_max_period,
        rope_base=cfg.rope_base, n_images=getattr(cfg, "n_images", 0), n_patches=getattr(cfg, "n_patches", 0),
        patch_dim=getattr(cfg, "patch_dim", 0), d_out=getattr(cfg, "d_out", 0))


def _tensor_array(weights: Dict[str, object]):
    """The C tensor list of a weight dict (and the host arrays it points into)."""
    keep = []
    arr = (Tensor * len(weights))()
    for i, (name, t) in enumerate(weights.items()):
        data = np.ascontiguousarray(t.data)
        keep.append(data)
        sc = None
        if t.scale is not None:
            sc = np.ascontiguousarray(t.scale, dtype=np.float32)
            keep.append(sc)
        nm = name.encode()
        keep.append(nm)
        # fp4 data holds two codes per byte: the logical width is twice its columns
        cols = data.shape[1] * (2 if t.dtype == "fp4" else 1)
        arr[i] = Tensor(nm, _DTYPE[t.dtype], data.shape[0], cols, data.ctypes.data,
                        None if sc is None else sc.ctypes.data)
    return arr, keep


class Expert:
    """One loaded expert (owns its device weights, buffers and graphs)."""

    def __init__(self, cfg, weights: Dict[str, object], max_batch: Optional[int] = None,
                 max_steps: Optional[int] = None, stream=None):
        self.cfg = cfg
        c = make_config(cfg, max_batch, max_steps)
        arr, keep = _tensor_array(weights)
        h = ctypes.c_void_p()
        _check(lib().phyai_load_expert(ctypes.byref(c), arr, len(weights), _stream(stream), ctypes.byref(h)))
        del keep
        self._h = h

    def prepare(self, batch: int, n_steps: int, stream=None):
        _check(lib().phyai_prepare(self._h, batch, n_steps, _stream(stream)))

    def denoise(self, prefix, prefix_len, noise, timesteps, state=None, out=None, stream=None,
                static: bool = False):
        """prefix, noise, state, out: device tensors; prefix_len, timesteps: host arrays.
        static=True calls phyai_denoise_static (allocates nothing; `out` must then be given)."""
        plen = np.ascontiguousarray(prefix_len, dtype=np.int32)
        ts = np.ascontiguousarray(timesteps, dtype=np.float32)
        B = int(noise.shape[0])
        if plen.shape[0] < B:
            raise ValueError("prefix_len shorter than the batch")
        if out is None:
            if static:
                raise ValueError("the allocation-free entry point needs a caller-provided `out`")
            import torch
            out = torch.empty_like(noise)
        fn = lib().phyai_denoise_static if static else lib().phyai_denoise
        _check(fn(self._h, _ptr(prefix), plen.ctypes.data, _ptr(noise), ts.ctypes.data,
                  len(ts) - 1, B, _ptr(state), _ptr(out), _stream(stream)))
        return out

    def debug_hidden(self, batch: int, stream=None):
        import torch
        c = self.cfg
        M = c.horizon + (1 if c.state_token else 0)
        dst = torch.empty((batch * M, c.d_model), dtype=torch.float32, device="cuda")
        _check(lib().phyai_debug_hidden(self._h, _ptr(dst), batch, _stream(stream)))
        return dst

    def profile_stage(self, stage: str, reps: int, stream=None):
        """Enqueue `reps` passes over all layers of one block stage (for timing)."""
        _check(lib().phyai_profile_stage(self._h, STAGES[stage], reps, _stream(stream)))

    def close(self):
        if getattr(self, "_h", None):
            lib().phyai_free_expert(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class PrefixLM:
    """One loaded prefix LM (variant ``prefix_lm``): prefix token embeddings in,
    the prefix K/V cache an expert reads out (``phyai_prefill``)."""

    def __init__(self, cfg, weights: Dict[str, object], max_batch: Optional[int] = None, stream=None):
        if cfg.variant != "prefix_lm":
            raise ValueError("PrefixLM needs a prefix_lm config")
        self.cfg = cfg
        c = make_config(cfg, max_batch, 0)
        arr, keep = _tensor_array(weights)
        h = ctypes.c_void_p()
        _check(lib().phyai_load_expert(ctypes.byref(c), arr, len(weights), _stream(stream), ctypes.byref(h)))
        del keep
        self._h = h

    def prefill(self, embeds, prefix_len, out=None, stream=None):
        """embeds: device float32 [B][prefix_cap][d]; prefix_len: host array.
        Returns (or fills) the device K/V cache [L][2][B][prefix_cap][n_kv*d_h]
        (bf16 bit patterns as int16, or float32 on the fp32 path)."""
        c = self.cfg
        plen = np.ascontiguousarray(prefix_len, dtype=np.int32)
        B = int(embeds.shape[0])
        if plen.shape[0] < B:
            raise ValueError("prefix_len shorter than the batch")
        if out is None:
            import torch
            dt = torch.float32 if c.kv_dtype == "f32" else torch.int16
            out = torch.empty((c.n_layers, 2, B, c.prefix_cap, c.n_kv_heads * c.head_dim), dtype=dt,
                              device=embeds.device)
        _check(lib().phyai_prefill(self._h, _ptr(embeds), plen.ctypes.data, _ptr(out), B, _stream(stream)))
        return out

    def profile_stage(self, stage: str, reps: int, stream=None):
        """Enqueue `reps` passes over the layers of one block stage (timing aid;
        needs a previous prefill)."""
        _check(lib().phyai_profile_stage(self._h, STAGES[stage], reps, _stream(stream)))

    def close(self):
        if getattr(self, "_h", None):
            lib().phyai_free_expert(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class VisionTower:
    """One loaded vision tower (variant ``vision``): image patches in, the
    image tokens that open the prefix out (``phyai_encode_images``)."""

    def __init__(self, cfg, weights: Dict[str, object], max_batch: Optional[int] = None, stream=None):
        if cfg.variant != "vision":
            raise ValueError("VisionTower needs a vision config")
        self.cfg = cfg
        c = make_config(cfg, max_batch, 0)
        arr, keep = _tensor_array(weights)
        h = ctypes.c_void_p()
        _check(lib().phyai_load_expert(ctypes.byref(c), arr, len(weights), _stream(stream), ctypes.byref(h)))
        del keep
        self._h = h

    def encode(self, patches, out=None, out_rows: Optional[int] = None, stream=None):
        """patches: device float32 [B][n_images][n_patches][patch_dim].  Returns
        (or fills rows 0 .. n_images*n_patches-1 of each request's slab of)
        the device float32 tokens [B][out_rows][d_out]; out_rows defaults to
        out's second dimension, or n_images*n_patches for a new buffer."""
        c = self.cfg
        B = int(patches.shape[0])
        n_tok = c.n_images * c.n_patches
        if out is None:
            import torch
            out = torch.empty((B, out_rows or n_tok, c.d_out), dtype=torch.float32, device=patches.device)
        rows = out_rows if out_rows is not None else int(out.shape[1])
        _check(lib().phyai_encode_images(self._h, _ptr(patches), _ptr(out), rows, B, _stream(stream)))
        return out

    def profile_stage(self, stage: str, reps: int, stream=None):
        """Enqueue `reps` passes over the blocks of one stage (timing aid; needs
        a previous encode)."""
        _check(lib().phyai_profile_stage(self._h, STAGES[stage], reps, _stream(stream)))

    def close(self):
        if getattr(self, "_h", None):
            lib().phyai_free_expert(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def fp8_to_bf16(codes, stream=None):
    """Decode device uint8 e4m3fn codes to bf16 bit patterns (device int16)."""
    import torch
    out = torch.empty(codes.shape, dtype=torch.int16, device=codes.device)
    _check(lib().phyai_fp8_to_bf16(_ptr(codes), _ptr(out), codes.numel(), _stream(stream)))
    return out


def version() -> int:
    return lib().phyai_version()
