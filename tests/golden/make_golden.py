"""Writes tests/golden/tiny_alif2.json from the oracle alone.

The paper prints no worked numeric example, so the stored values are the
oracle's own output on a tiny two-layer ALIF network (B=2, 3 inputs, 5
neurons per layer, 3 adaptive, 3 classes, T=12, fp32 forward).  They pin the
oracle against accidental change; the autograd, finite-difference and
closed-form checks in test_oracle_pins.py pin it against the mathematics.
Run: python tests/golden/make_golden.py
"""
import json
import math
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2501_11407_amd import synth  # noqa: E402

SHAPE = synth.EpropShape(batch=2, n_in=3, n_rec=5, n_out=3, T=12, n_layers=2, recurrent=1,
                         n_adaptive=3, kappa=synth.f32(math.exp(-1 / 7)),
                         rho=synth.f32(math.exp(-1 / 50)))
SEED = 2501
INPUT_SCALE = 12.0
OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_alif2.json")


def compute():
    wl = synth.make_workload(SHAPE, SEED, input_scale=INPUT_SCALE)
    for w in wl.W:
        w *= 4.0
    r = oracle.run(SHAPE, wl.W, wl.Wout, wl.x, wl.labels, fwd_fp32=True)
    return wl, r


if __name__ == "__main__":
    wl, r = compute()
    doc = {"shape": {k: getattr(SHAPE, k) for k in ("batch", "n_in", "n_rec", "n_out", "T", "n_layers",
                                                    "recurrent", "n_adaptive", "alpha", "rho", "kappa",
                                                    "thr", "beta", "gamma")},
           "seed": SEED, "input_scale": INPUT_SCALE, "weight_scale": 4.0,
           "spike_words": r.spikes.reshape(-1).tolist(),
           "dW": [d.tolist() for d in r.dW], "dWout": [d.tolist() for d in r.dWout], "loss": r.loss}
    with open(OUT, "w") as f:
        json.dump(doc, f, indent=0)
    print(OUT)
