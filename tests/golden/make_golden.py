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

# sampled candidates of each batch: the first, the longest and the shortest cached sequence among
# them (ragged: 2 is the longest at 31832 tokens and fills the most chunk slots, 1 the shortest;
# beam: 2 the longest suffix, 0 the shortest; large fp8: 0 the longest, 14 the shortest at 8834;
# fixed 32k: every candidate holds 32768 tokens, so the first and the last)
SAMPLES = {
    "b7_bf16": [0, 7, 15],
    "ragged_32k": [0, 1, 2, 5],
    "fixed_32k": [0, 7],
    "beam_prefix": [0, 2, 33, 63],
    "large_fp8": [0, 9, 14],
}


# workloads scored with the unmerged adapter of this rank on every projection (the verify
# token runs theta + scale * B A; kvprm_score_lora on the GPU): file <workload>_lora<rank>.json
LORA_SAMPLES = {
    "ragged_32k": ([0, 5], 256),
}


def make(name, lora_rank=0):
    w = synth.make_workload(name)
    cand = LORA_SAMPLES[name][0] if lora_rank else SAMPLES[name]
    t0 = time.time()
    ro = oin.readout_from_synth(w.shape, w.seed, layer_cache=1)
    if lora_rank:
        ro = ko.readout_with_adapter(ro, oin.lora_from_synth(w.shape, w.seed, lora_rank,
                                                             layer_cache=1),
                                     synth.lora_scale(lora_rank))
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
        "fp8_scale": w.fp8_scale if w.shape.kv_dtype == "fp8" else None,
        "oracle_seconds": round(time.time() - t0, 1),
    }
    if lora_rank:
        out["lora_rank"] = lora_rank
        out["lora_targets"] = list(synth.LORA_PROJECTIONS)
        out["source"] += "; adapter theta + scale * B A on the verify token (readout_with_adapter)"
    path = os.path.join(HERE, f"{name}_lora{lora_rank}.json" if lora_rank else f"{name}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(f"{name}: z={out['z']} in {out['oracle_seconds']} s -> {path}", flush=True)


if __name__ == "__main__":
    # names: a workload (stored values of the base readout) or <workload>_lora (with the adapter)
    for name in (sys.argv[1:] or list(SAMPLES) + [f"{n}_lora" for n in LORA_SAMPLES]):
        if name.endswith("_lora"):
            base = name[: -len("_lora")]
            make(base, LORA_SAMPLES[base][1])
        else:
            make(name)
