"""Seeded random configurations scored on the GPU and by the fp64 oracle (section 4.1, Eq.
(score); the options and the KV Steering gradient further down): model shapes within what the library accepts (hidden and FFN sizes, 1 to 16 query
heads per kv-head, d_h 64 or 128), the three dtype pairs, batch sizes from 1 to 24, lengths that
include 0, 1 and every page edge, and shared-prefix groups, all drawn from one generator per
case. Bars as in the fixed parity tests: |dP(+)| <= 1e-5 and |dz| <= 4e-5 with fp32 weights and
cache, 2e-3 and 2e-2 with bf16 weights."""
import sys

import numpy as np
import pytest

import synth
from oracle import inputs as oin
from synth.device import DeviceWorkload

from gpu_common import run_score
from test_gpu_depth import _depth_parity
from test_gpu_lora import _lora_parity
from test_gpu_steer import _grad_case

pytestmark = pytest.mark.gpu

CASES = 24
EDGE_LENGTHS = (0, 1, 15, 16, 17, 31, 32, 33)


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _draw(case: int):
    rng = np.random.default_rng(7000 + case)
    d = int(rng.choice([64, 128]))
    wdt = "f32" if rng.random() < 0.25 else "bf16"
    kvdt = "f32" if wdt == "f32" else str(rng.choice(["bf16", "fp8"]))
    nkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.choice([1, 2, 4, 7, 8, 16]))
    H = 64 * int(rng.integers(2, 9))
    F = 64 * int(rng.integers(4, 17))
    shape = synth.ModelShape(2, H, nkv * g, nkv, d, F, weight_dtype=wdt, kv_dtype=kvdt)
    B = int(rng.integers(1, 9 if wdt == "f32" else 25))
    groups = None
    if wdt == "bf16" and B >= 2 and rng.random() < 0.35:
        ng = int(rng.integers(1, min(3, B) + 1))
        cuts = sorted(rng.choice(np.arange(1, B), size=ng - 1, replace=False).tolist()) if ng > 1 else []
        starts = [0] + [int(c) for c in cuts] + [B]
        prefix = [16 * int(rng.integers(0, 41)) for _ in range(ng)]
        lengths = []
        for gi in range(ng):
            for _ in range(starts[gi + 1] - starts[gi]):
                lengths.append(prefix[gi] + int(rng.integers(0, 301)))
        groups = (starts, prefix)
    else:
        lengths = [int(rng.choice(EDGE_LENGTHS)) if rng.random() < 0.4 else int(rng.integers(0, 701))
                   for _ in range(B)]
    return shape, lengths, groups


@pytest.mark.parametrize("case", range(CASES))
def test_random_configuration(case):
    shape, lengths, groups = _draw(case)
    _say(f"case {case}: H={shape.hidden} heads={shape.num_q_heads}/{shape.num_kv_heads} "
         f"d_h={shape.head_dim} F={shape.ffn_dim} {shape.weight_dtype}/{shape.kv_dtype} "
         f"B={len(lengths)} lengths={lengths} groups={groups}")
    w = synth.make_workload("custom", shape=shape, lengths=lengths, seed=7100 + case, groups=groups)
    p, z = run_score(DeviceWorkload(w, nan_unused_pages=True))
    zr, pr = oin.score_workload(w)
    dp, dz = float(np.max(np.abs(p - pr))), float(np.max(np.abs(z - zr)))
    _say(f"  max|dP| = {dp:.3e}  max|dz| = {dz:.3e}")
    assert np.all(np.isfinite(p)) and np.all(np.isfinite(z))
    tol_p, tol_z = (1e-5, 4e-5) if shape.weight_dtype == "f32" else (2e-3, 2e-2)
    assert dp <= tol_p and dz <= tol_z


GRAD_CASES = 8


def _draw_grad(case: int):
    rng = np.random.default_rng(7500 + case)
    d = int(rng.choice([64, 128]))
    nkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.choice([1, 2, 4, 7, 8, 16]))
    H = 64 * int(rng.integers(2, 9))
    F = 64 * int(rng.integers(4, 17))
    shape = synth.ModelShape(2, H, nkv * g, nkv, d, F)
    B = int(rng.integers(1, 5))
    lengths = [int(rng.choice(EDGE_LENGTHS)) if rng.random() < 0.4 else int(rng.integers(0, 401))
               for _ in range(B)]
    return shape, lengths


@pytest.mark.parametrize("case", range(GRAD_CASES))
def test_random_cache_gradient(case):
    """The KV Steering gradient (appendix, KV Steering algorithm) element by element against
    the oracle's reverse mode on seeded random shapes (bf16 weights and cache, 1-4 candidates):
    the transposed products over hidden, FFN and n_q d_h inputs of every size the library takes."""
    shape, lengths = _draw_grad(case)
    _say(f"grad case {case}: H={shape.hidden} heads={shape.num_q_heads}/{shape.num_kv_heads} "
         f"d_h={shape.head_dim} F={shape.ffn_dim} B={len(lengths)} lengths={lengths}")
    w = synth.make_workload("custom", shape=shape, lengths=lengths, seed=7600 + case)
    _grad_case(w)


OPTION_CASES = 10


def _draw_options(case: int):
    rng = np.random.default_rng(7800 + case)
    d = int(rng.choice([64, 128]))
    nkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.choice([1, 2, 4, 7, 8]))
    H = 64 * int(rng.integers(2, 9))
    F = 64 * int(rng.integers(4, 17))
    kvdt = str(rng.choice(["bf16", "fp8"]))
    shape = synth.ModelShape(2, H, nkv * g, nkv, d, F, kv_dtype=kvdt)
    depth = int(rng.choice([d_ for d_ in (1, 2, 3, 4) if d_ * g <= 16]))
    B = int(rng.integers(1, min(24, 64 // depth) + 1))
    rank = int(rng.choice([0, 32, 64, 128, 256])) if depth > 1 else int(rng.choice([32, 64, 128, 256]))
    targets = synth.LORA_PROJECTIONS
    if depth == 1:
        k = int(rng.integers(1, len(targets) + 1))
        targets = tuple(sorted(rng.choice(targets, size=k, replace=False).tolist(),
                               key=synth.LORA_PROJECTIONS.index))
    groups = None
    if B >= 2 and rng.random() < 0.3:
        cut = int(rng.integers(1, B))
        prefix = [16 * int(rng.integers(0, 31)), 16 * int(rng.integers(0, 31))]
        lengths = [prefix[0 if i < cut else 1] + int(rng.integers(0, 301)) for i in range(B)]
        groups = ([0, cut, B], prefix)
    else:
        lengths = [int(rng.choice(EDGE_LENGTHS)) if rng.random() < 0.4 else int(rng.integers(0, 601))
                   for _ in range(B)]
    return shape, lengths, groups, depth, rank, targets


@pytest.mark.parametrize("case", range(OPTION_CASES))
def test_random_readout_options(case):
    """The options of the readout on seeded random configurations: the depth-k readout (1-4
    verify tokens per candidate, with or without an adapter on every projection) and unmerged
    adapters of rank 32-256 on random subsets of the projections, with shared-prefix groups
    sometimes, each against the oracle at the bf16 bars."""
    shape, lengths, groups, depth, rank, targets = _draw_options(case)
    _say(f"options case {case}: H={shape.hidden} heads={shape.num_q_heads}/{shape.num_kv_heads} "
         f"d_h={shape.head_dim} F={shape.ffn_dim} kv={shape.kv_dtype} B={len(lengths)} "
         f"depth={depth} rank={rank} targets={targets} groups={groups} lengths={lengths}")
    w = synth.make_workload("custom", shape=shape, lengths=lengths, seed=7900 + case, groups=groups)
    if depth == 1:
        _lora_parity(w, rank, targets)
    else:
        _depth_parity(w, depth, lora_rank=rank)
