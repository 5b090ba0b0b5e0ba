"""GPU parity of the depth-k readout (kvprm_score_ex, k verify tokens per candidate, causal
among themselves, score at the last one) against the fp64 oracle (verify_pass_depth).
Bar: the bf16 one, max |dP(+)| <= 2e-3 and max |dz| <= 2e-2."""
import dataclasses
import sys

import numpy as np
import pytest

import synth
from oracle import inputs as oin
from synth.device import DeviceWorkload

from gpu_common import run_score, run_score_ex

pytestmark = pytest.mark.gpu

G2 = synth.ModelShape(2, 256, 4, 2, 64, 1024)                    # 2 q-heads per kv-head
G4_FP8 = synth.ModelShape(2, 512, 8, 2, 128, 1024, kv_dtype="fp8")  # 4 per kv-head, e4m3 cache


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _depth_parity(w, depth, lora_rank=0, with_hint=True):
    dw = DeviceWorkload(w, nan_unused_pages=True)
    if lora_rank:
        dw.add_lora(lora_rank)
    p, z = run_score_ex(dw, depth, lora=bool(lora_rank), with_hint=with_hint)
    zr, pr = oin.score_workload(w, depth=depth, lora_rank=lora_rank)
    z1, _ = oin.score_workload(w, lora_rank=lora_rank)
    dp, dz = np.max(np.abs(p - pr)), np.max(np.abs(z - zr))
    _say(f"  max|dP| = {dp:.3e}  max|dz| = {dz:.3e}  depth moves z by {np.max(np.abs(zr - z1)):.3f}")
    assert np.all(np.isfinite(p)) and np.all(np.isfinite(z))
    assert dp <= 2e-3 and dz <= 2e-2
    return p, z


@pytest.mark.parametrize("depth,B", [(2, 5), (4, 7), (8, 8)])
def test_depth_parity_small_shape(depth, B):
    _say(f"case: depth {depth}, g = 2, B = {B}, ragged lengths incl. 0")
    lengths = [0, 1, 16, 17, 300, 1025, 64, 700][:B]
    w = synth.make_workload("custom", shape=G2, lengths=lengths, seed=301 + depth)
    _depth_parity(w, depth)


def test_depth_2_on_the_7b_shape():
    """g = 7: 14 query columns per kv-head; B x depth = 10 rows (two operand column tiles)."""
    _say("case: depth 2, 7B shape, 2 layers")
    shape = dataclasses.replace(synth.B7, num_layers=2)
    w = synth.make_workload("custom", shape=shape, lengths=[4096, 0, 17, 1200, 2049], seed=310)
    _depth_parity(w, 2)


def test_depth_4_fp8_cache():
    _say("case: depth 4, g = 4 (16 columns), e4m3 cache")
    w = synth.make_workload("custom", shape=G4_FP8, lengths=[900, 33, 0, 512], seed=311)
    _depth_parity(w, 4)


@pytest.mark.parametrize("with_hint", [True, False])
def test_depth_3_with_shared_prefixes(with_hint):
    """Beam groups share prefix pages; with the hint the shared-prefix kernel reads them once
    for every verify token of every member."""
    _say(f"case: depth 3, shared prefixes, hint {with_hint}")
    lengths = [700, 650, 900, 40, 520, 530, 600, 513, 1000, 17]
    w = synth.make_workload("custom", shape=G2, lengths=lengths, seed=312,
                            groups=([0, 3, 4, 8, 10], [512, 0, 512, 0]))
    _depth_parity(w, 3, with_hint=with_hint)


def test_depth_2_with_the_adapter():
    _say("case: depth 2 with a rank-64 adapter on every projection")
    w = synth.make_workload("custom", shape=G2, lengths=[400, 0, 129, 777], seed=313)
    _depth_parity(w, 2, lora_rank=64)


def test_depth_1_options_equal_the_plain_call_bitwise():
    _say("case: kvprm_score_ex depth 1 vs kvprm_score")
    shape = dataclasses.replace(synth.B7, num_layers=2)
    w = synth.make_workload("custom", shape=shape, lengths=[333, 0, 4000], seed=314)
    dw = DeviceWorkload(w)
    a = run_score(dw)
    b = run_score_ex(dw, 1)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
