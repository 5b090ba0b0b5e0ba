"""The scoring pass inside a captured HIP graph: kvprm_score enqueues kernels only (no
allocation, no host synchronisation, no memset nodes), so a caller can capture one call and
replay it. Each replay, with the program's own eager work and synchronisations between the
replays, must give the eager result bit for bit (the kernels are deterministic)."""
import sys

import numpy as np
import pytest
import torch

import synth
from synth.device import DeviceWorkload

from gpu_common import kv

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("shape_name,lengths", [
    ("7b_2layers", [900, 17, 0, 3000, 64]),
    ("tiny_fp32", [100, 513, 7]),
])
def test_score_replayed_from_a_graph_matches_eager(shape_name, lengths):
    _say(f"case: graph replay, {shape_name}")
    import dataclasses
    shape = (dataclasses.replace(synth.B7, num_layers=2) if shape_name == "7b_2layers"
             else synth.TINY)
    w = synth.make_workload("custom", shape=shape, lengths=lengths, seed=501)
    dw = DeviceWorkload(w)
    m = kv()
    h = m.kvprm_create(dw.desc(m))
    try:
        batch = dw.batch(m)
        n = m.kvprm_workspace_size(h, batch)
        ws = torch.empty(max(n, 256), dtype=torch.uint8, device="cuda")
        scores = torch.full((w.batch,), float("nan"), device="cuda")
        logits = torch.full((w.batch,), float("nan"), device="cuda")
        cache, ro = dw.cache(m), dw.readout(m)

        def call():
            m.kvprm_score(h, cache, batch, ro, ws.data_ptr(), n, scores.data_ptr(),
                          logits.data_ptr(), torch.cuda.current_stream().cuda_stream)

        call()
        torch.cuda.synchronize()
        want_p, want_z = scores.clone(), logits.clone()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):  # warm-up on the capture stream, outside the capture
            call()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            call()
        junk = torch.randn(1 << 20, device="cuda")
        for r in range(3):
            scores.fill_(float("nan"))
            logits.fill_(float("nan"))
            junk.mul_(1.0001).add_(0.5)  # eager work between replays
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(scores, want_p), r
            assert torch.equal(logits, want_z), r
        del g
    finally:
        m.kvprm_destroy(h)
