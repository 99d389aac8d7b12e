"""Writes c5_expected.npz: the oracle's final actions (float64) for all 64
requests of the cloud-rollout batch (pi0 shape, fp8 weights, ragged prefixes,
seed 0), so that the GPU test can compare every request without running the
oracle for minutes.  Calls only the oracle and the seeded input generators.

    python tests/golden/make_c5_expected.py [--workers N]
"""
import argparse
import os
import sys
from concurrent.futures import ProcessPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

CONFIG, SEED = "pi0_fp8_b64", 0


def _run(requests):
    import oracle
    import workloads as wl
    cfg = wl.CONFIGS[CONFIG]
    case = wl.make_case(cfg, seed=SEED)
    W = oracle.DecodedWeights(case.weights)
    pl = case.prefix_len
    out = {}
    for b in requests:
        pre = wl.make_prefix(cfg, pl, SEED, requests=[b])
        out[b] = oracle.denoise(cfg, case.weights, pre, pl[[b]], case.noise[[b]], case.timesteps,
                                case.state[[b]], decoded=W, slots=[0])[0]
        print(f"request {b} done", flush=True)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workers", type=int, default=2)
    args = ap.parse_args()
    import workloads as wl
    B = wl.CONFIGS[CONFIG].batch
    chunks = [list(range(i, B, args.workers)) for i in range(args.workers)]
    res = {}
    with ProcessPoolExecutor(args.workers) as ex:
        for part in ex.map(_run, chunks):
            res.update(part)
    x = np.stack([res[b] for b in range(B)]).astype(np.float64)
    np.savez_compressed(os.path.join(HERE, "c5_expected.npz"), actions=x, config=CONFIG, seed=SEED)
    print("wrote", x.shape)


if __name__ == "__main__":
    main()
