"""Full-size parity: each benchmark workload at its real shape and batch, scored by the library
in the launch configuration the benchmark times; sampled candidates are compared with fp64
oracle values stored in tests/golden/ (written by tests/golden/make_golden.py, which calls only
the oracle). Bar for bf16 weights: max |dP(+)| <= 2e-3; the logit z is checked as well."""
import json
import os
import sys

import numpy as np
import pytest
import torch

import synth
from synth.device import DeviceWorkload

from gpu_common import run_score

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
WORKLOADS = ["b7_bf16", "ragged_32k", "fixed_32k", "beam_prefix", "large_fp8"]


@pytest.mark.parametrize("name", WORKLOADS)
def test_full_size_against_stored_oracle(name):
    path = os.path.join(GOLDEN, f"{name}.json")
    if not os.path.exists(path):
        pytest.skip(f"no stored oracle values for {name} (run tests/golden/make_golden.py {name})")
    ref = json.load(open(path))
    w = synth.make_workload(name)
    assert w.seed == ref["seed"] and w.batch == ref["batch"]
    assert [w.lengths[b] for b in ref["candidates"]] == ref["lengths"]
    print(f"case: full size {name} B={w.batch} layers={w.shape.num_layers}", flush=True)
    sys.stdout.flush()
    dw = DeviceWorkload(w, nan_unused_pages=True)
    try:
        p, z = run_score(dw)
    finally:
        del dw
        torch.cuda.empty_cache()
    assert np.all(np.isfinite(p)) and np.all((p >= 0) & (p <= 1))
    cand = ref["candidates"]
    dp = np.max(np.abs(p[cand] - np.array(ref["p"])))
    dz = np.max(np.abs(z[cand] - np.array(ref["z"])))
    print(f"  max|dP| = {dp:.3e}  max|dz| = {dz:.3e}", flush=True)
    assert dp <= 2e-3
    assert dz <= 2e-2


def test_full_size_adapter_against_stored_oracle():
    """The ragged 32k batch with the unmerged rank-256 adapter on every projection
    (kvprm_score_lora, as the benchmark's adapter line runs it), sampled candidates against
    stored fp64 oracle values."""
    from gpu_common import run_score_lora
    path = os.path.join(GOLDEN, "ragged_32k_lora256.json")
    if not os.path.exists(path):
        pytest.skip("no stored oracle values (run tests/golden/make_golden.py ragged_32k_lora)")
    ref = json.load(open(path))
    w = synth.make_workload(ref["workload"])
    assert w.seed == ref["seed"] and w.batch == ref["batch"]
    assert [w.lengths[b] for b in ref["candidates"]] == ref["lengths"]
    print(f"case: full size {ref['workload']} with a rank-{ref['lora_rank']} adapter", flush=True)
    dw = DeviceWorkload(w, nan_unused_pages=True)
    dw.add_lora(ref["lora_rank"], tuple(ref["lora_targets"]))
    try:
        p, z = run_score_lora(dw)
    finally:
        del dw
        torch.cuda.empty_cache()
    cand = ref["candidates"]
    dp = np.max(np.abs(p[cand] - np.array(ref["p"])))
    dz = np.max(np.abs(z[cand] - np.array(ref["z"])))
    print(f"  max|dP| = {dp:.3e}  max|dz| = {dz:.3e}", flush=True)
    assert np.all(np.isfinite(p)) and np.all((p >= 0) & (p <= 1))
    assert dp <= 2e-3
    assert dz <= 2e-2
