"""Write the oracle's result for the full-size ResNet-20 runs (batch 128,
4 stages at the Table 1 PPV (7,13,19), staleness [3,2,1,0], 50 steps, lr 0.01,
momentum 0.9) to tests/golden/.  Calls only the oracle and the seeded input
generator; never the GPU path.

    python tests/golden/make_golden.py [fp32|bf16 ...]

Stored: the parameter update W^(50) - W^(0) (float32; W^(0) is regenerated
from the seed), the 50 losses and the version table.
"""
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from paper_1912_12675_amd import synth  # noqa: E402


def make(mode):
    wl = synth.resnet20_workload(bf16=(mode == "bf16"))
    T = wl.steps
    p0 = synth.init_params(wl)
    xs, ys = synth.batches(wl, T)
    t0 = time.time()
    out = O.train(wl.ops, wl.in_shape, wl.stage_end, p0, xs, ys, wl.staleness(T), wl.lr, wl.momentum,
                  wl.weight_decay, wl.nesterov, bf16=wl.bf16)
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), f"resnet20_b128_50steps_{mode}.npz")
    np.savez_compressed(path, delta=(out["params"] - p0.astype(np.float64)).astype(np.float32),
                        losses=out["losses"], versions=out["versions"])
    print(f"{mode}: {time.time() - t0:.0f} s, final loss {out['losses'][-1]:.6f} -> {path}", flush=True)


if __name__ == "__main__":
    for m in (sys.argv[1:] or ["fp32", "bf16"]):
        make(m)
