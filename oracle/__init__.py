"""Oracle for the action-expert denoising loop, the prefix K/V producer and
the vision tower before it (float64 NumPy).

TEST INFRASTRUCTURE ONLY: a plain, slow, obviously correct CPU reference.
Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's
``cpu_baseline`` leg may import it.  It shares no code with the HIP library
and never calls it.  Pins that tie it to facts outside itself live in
``tests/test_oracle_pins.py``.  The composed networks are pinned only by
invariants and special cases (no worked numerical example exists in the
paper), which is stated there.
"""
from .expert import (DecodedWeights, denoise, pi05_condition, velocity_dit, velocity_pi0,
                     velocity_pi05)
from .prefix_lm import prefill, prefill_request
from .vision import encode_images
from .numerics import (E2M1_TABLE, E4M3FN_TABLE, attention, attention_bruteforce, decode_bf16,
                       decode_fp4, decode_fp8, decode_stored, euler, gelu_tanh, layer_normalize, rms_normalize, rope,
                       sinusoid, swish)

__all__ = [
    "DecodedWeights", "denoise", "pi05_condition", "velocity_dit", "velocity_pi0", "velocity_pi05",
    "E2M1_TABLE", "E4M3FN_TABLE", "attention", "attention_bruteforce", "decode_bf16", "decode_fp4",
    "decode_fp8",
    "decode_stored", "euler", "gelu_tanh", "layer_normalize", "rms_normalize", "rope", "sinusoid",
    "swish", "prefill", "prefill_request", "encode_images",
]
