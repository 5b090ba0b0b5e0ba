"""Write the stored expected values of the full-size parity tests.

Calls only the fp64 oracle (and the seeded input generator that feeds it): for each benchmark
workload, the oracle scores a few sampled candidates of the full batch (Eq. (score), section
4.1: z = w_r . RMSNorm(h) + b_r and P(+) = sigmoid(z)). The GPU test runs the library on the
whole batch, in the launch configuration the benchmark times, and compares those candidates.

    python tests/golden/make_golden.py [workload ...]
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import synth  # noqa: E402
from oracle import inputs as oin  # noqa: E402
from oracle import kvprm_oracle as ko  # noqa: E402

SAMPLES = {
    "b7_bf16": [0, 7, 15],
    "ragged_32k": [0, 1, 5],
    "beam_prefix": [0, 33, 63],
    "large_fp8": [0, 9],
}


def make(name):
    w = synth.make_workload(name)
    cand = SAMPLES[name]
    t0 = time.time()
    ro = oin.readout_from_synth(w.shape, w.seed, layer_cache=1)
    cache = oin.cache_from_synth(w, page_cache=64)
    z, p = ko.verify_pass(w.shape, ro, cache, [w.lengths[b] for b in cand],
                          [w.page_table[b] for b in cand])
    out = {
        "workload": name,
        "seed": w.seed,
        "batch": w.batch,
        "candidates": cand,
        "lengths": [w.lengths[b] for b in cand],
        "z": [float(v) for v in z],
        "p": [float(v) for v in p],
        "source": "fp64 oracle (oracle/kvprm_oracle.py verify_pass), Eq. (score) of section 4.1",
        "oracle_seconds": round(time.time() - t0, 1),
    }
    path = os.path.join(HERE, f"{name}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(f"{name}: z={out['z']} in {out['oracle_seconds']} s -> {path}", flush=True)


if __name__ == "__main__":
    for name in (sys.argv[1:] or list(SAMPLES)):
        make(name)
