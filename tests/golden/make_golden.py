"""Write tests/golden/tiny_cnn_ags_k4.json from the float64 oracle.

The fixture freezes what the oracle computes for the tiny CNN layout
(K = 4 fp32 replicas, seed 0, AGS mode, refresh every step, the default
hyperparameters lr 0.1, momentum 0.9, weight decay 5e-4, delta 0.5,
eps 1e-8) over three steps: every per-layer statistic, the global record
and 64 sampled elements of w and m after each step.  It calls only the
oracle and the seeded input generator.  Re-run it only for a change of the
oracle's arithmetic that the paper justifies.
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from oracle import OracleAGS  # noqa: E402
from paper_2603_18112_amd import layouts, synth  # noqa: E402

OUT = os.path.join(HERE, "tiny_cnn_ags_k4.json")
HYPER = dict(lr=0.1, momentum=0.9, weight_decay=5e-4, delta=0.5, eps=1e-8, refresh_every=1,
             small_replica=0)


def sample_index(lay):
    idx = []
    for o, n, _ in lay.table():
        idx += [o, o + n // 2, o + n - 1]
    extra = np.linspace(0, lay.n_params - 1, 64 - len(idx)).astype(int)
    flat = np.concatenate([np.arange(o, o + n) for o, n, _ in lay.table()])
    idx += [int(flat[i]) for i in extra]
    return sorted(set(idx))


def generate():
    lay = layouts.get_layout("tiny_cnn")
    w0 = synth.init_weights(lay, 0)
    o = OracleAGS(lay.table(), lay.n_flat, 4, w0, **HYPER)
    idx = sample_index(lay)
    steps = []
    for t in range(3):
        st, gl = o.step(synth.replica_grads(lay, 4, t, 0))
        steps.append({"layer": {k: [float(x) for x in v] for k, v in st.items()},
                      "global": gl,
                      "w": [float(o.w[i]) for i in idx],
                      "m": [float(o.m[i]) for i in idx]})
    return {"layout": "tiny_cnn", "K": 4, "seed": 0, "grad_dtype": "f32", "mode": "ags",
            "hyper": HYPER, "index": idx, "steps": steps}


if __name__ == "__main__":
    with open(OUT, "w") as f:
        json.dump(generate(), f, indent=1)
    print(OUT)
