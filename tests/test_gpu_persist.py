"""The persistent batch-1 loop (one cooperative launch for all K steps of one
pi0 request; opt-in with PHYAI_PERSIST=1) against the oracle, through the C
ABI, and against the default graph path on the same inputs.  Shapes span head_dim 64 and 256,
widths 256 and 1024, with and without the state token and RoPE, and prefix
lengths at the edges of the 64-key tiles."""
import dataclasses
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


def _oracle(cfg, case):
    return oracle.denoise(cfg, case.weights, case.prefix, case.prefix_len, case.noise, case.timesteps,
                          case.state)


def _persist(ex, case, dev=None):
    os.environ["PHYAI_PERSIST"] = "1"
    try:
        return run_gpu(ex, case, dev)
    finally:
        del os.environ["PHYAI_PERSIST"]


SHAPES = [
    ("d256_dh64", dict()),
    ("d256_dh256", dict(head_dim=256, n_q_heads=1)),
    ("d512_dh128", dict(d_model=512, head_dim=128, n_q_heads=4, d_mlp=1024)),
    ("d1024_dh256", dict(d_model=1024, head_dim=256, n_q_heads=4, d_mlp=2048, n_layers=3)),
    ("no_state_no_rope", dict(state_token=False, rope=False)),
    ("no_state_rope", dict(state_token=False)),
    ("two_steps_h16", dict(n_steps=2, horizon=16)),
    # 37 steps run as launches of 16, 16 and 5 steps
    ("k37_three_launches", dict(n_steps=37)),
]


@pytest.mark.parametrize("name,kw", SHAPES)
def test_persist_matches_oracle_and_graph(name, kw):
    cfg = small_cfg("pi0", batch=1, **kw)
    print(f"[case] persistent {name} {kw}", flush=True)
    case = wl.make_case(cfg, seed=41)
    ex = _px().Expert(cfg, case.weights)
    dev = to_device(case)
    got = _persist(ex, case, dev)
    ref = _oracle(cfg, case)
    compare(f"persistent {name}", got, ref, cfg)
    graph = run_gpu(ex, case, dev)
    compare(f"graph {name}", graph, ref, cfg)
    again = _persist(ex, case, dev)
    assert np.array_equal(again, got), "persistent path is not deterministic"
    ex.close()


@pytest.mark.parametrize("plen", [0, 1, 13, 63, 64, 65, 100])
def test_persist_edge_prefix_lengths(plen):
    """Prefix lengths at the edges of the 64-key tiles (with 51 suffix keys the
    key range ends mid-tile), the empty prefix and the full capacity."""
    cfg = small_cfg("pi0", batch=1)
    print(f"[case] persistent prefix {plen}", flush=True)
    case = wl.make_case(cfg, seed=42)
    pl = np.array([plen], np.int32)
    case = dataclasses.replace(case, prefix_len=pl, prefix=wl.make_prefix(cfg, pl, 42))
    ex = _px().Expert(cfg, case.weights)
    compare(f"persistent prefix {plen}", _persist(ex, case), _oracle(cfg, case), cfg)
    ex.close()


def test_persist_schedule_change_and_fewer_steps():
    """A non-uniform schedule and a call with fewer steps than the handle's
    maximum run through the same persistent launch."""
    cfg = small_cfg("pi0", batch=1, n_steps=4)
    print("[case] persistent schedule", flush=True)
    case = wl.make_case(cfg, seed=43)
    ex = _px().Expert(cfg, case.weights)
    for ts in (np.float32([1.0, 0.8, 0.3, 0.1, 0.0]), np.float32([1.0, 0.5, 0.0])):
        c2 = dataclasses.replace(case, timesteps=ts)
        compare(f"persistent schedule {list(ts)}", _persist(ex, c2), _oracle(cfg, c2), cfg)
    ex.close()
