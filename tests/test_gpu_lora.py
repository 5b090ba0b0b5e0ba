"""GPU parity of the unmerged low-rank adapter readout (kvprm_score_lora) against the fp64
oracle, which applies the adapter as the merged matrix W + scale * B A on the verify token
(section 4.1, Eq. (score)). Bar: the bf16 one, max |dP(+)| <= 2e-3 and max |dz| <= 2e-2."""
import dataclasses
import sys

import numpy as np
import pytest
import torch

import synth
from oracle import inputs as oin
from synth.device import DeviceWorkload

from gpu_common import run_score, run_score_lora

pytestmark = pytest.mark.gpu

SMALL = synth.ModelShape(2, 256, 4, 2, 64, 1024)  # bf16 weights and cache


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _lora_parity(w, rank, targets=synth.LORA_PROJECTIONS, tol_p=2e-3, tol_z=2e-2):
    dw = DeviceWorkload(w, nan_unused_pages=True)
    dw.add_lora(rank, targets)
    p, z = run_score_lora(dw)
    zr, pr = oin.score_workload(w, lora_rank=rank, lora_targets=targets)
    zb, _ = oin.score_workload(w)
    dp, dz = np.max(np.abs(p - pr)), np.max(np.abs(z - zr))
    _say(f"  max|dP| = {dp:.3e}  max|dz| = {dz:.3e}  adapter moves z by "
         f"{np.max(np.abs(zr - zb)):.3f}")
    assert np.all(np.isfinite(p)) and np.all(np.isfinite(z))
    assert dp <= tol_p and dz <= tol_z
    return dw, p, z


@pytest.mark.parametrize("rank", [32, 256])
def test_lora_parity_small_shape(rank):
    _say(f"case: adapter rank {rank}, small bf16 shape, ragged lengths incl. 0")
    w = synth.make_workload("custom", shape=SMALL, lengths=[0, 1, 17, 300, 1025], seed=201)
    _lora_parity(w, rank)


def test_lora_parity_7b_two_layers():
    _say("case: adapter rank 256 on every projection, 7B shape, 2 layers")
    shape = dataclasses.replace(synth.B7, num_layers=2)
    w = synth.make_workload("custom", shape=shape, lengths=[4096, 0, 17, 1200], seed=202)
    _lora_parity(w, 256)


@pytest.mark.parametrize("targets,B", [(("q", "v", "down"), 17), (("o", "up"), 9),
                                       (("k", "gate"), 40)])
def test_lora_parity_target_subsets(targets, B):
    """Adapters on some projections only, with two to six operand column tiles."""
    _say(f"case: adapter on {targets}, B={B}")
    lengths = [(53 * i * i + 7 * i) % 600 for i in range(B)]
    w = synth.make_workload("custom", shape=SMALL, lengths=lengths, seed=203 + B)
    _lora_parity(w, 64, targets)


def test_lora_rank_512_batch_64():
    _say("case: adapter rank 512, B=64")
    lengths = [(29 * i) % 400 for i in range(64)]
    w = synth.make_workload("custom", shape=SMALL, lengths=lengths, seed=210)
    _lora_parity(w, 512)


def test_lora_with_zero_b_is_the_base_pass_bitwise():
    """B = 0 adds exact zeros to every projection: kvprm_score_lora equals kvprm_score bit for
    bit, and repeated calls are bitwise identical."""
    _say("case: adapter with B = 0 vs base pass")
    shape = dataclasses.replace(synth.B7, num_layers=2)
    w = synth.make_workload("custom", shape=shape, lengths=[500, 33, 0], seed=211)
    dw = DeviceWorkload(w)
    dw.add_lora(64)
    for d in dw.lora_layers:
        for name, t in d.items():
            if name.startswith("lora_b_"):
                t.zero_()
    torch.cuda.synchronize()
    p0, z0 = run_score(dw)
    p1, z1 = run_score_lora(dw)
    p2, z2 = run_score_lora(dw)
    assert np.array_equal(z0, z1) and np.array_equal(p0, p1)
    assert np.array_equal(z1, z2)
