"""One handle, several calls in flight: the handle holds only the model description, so calls
with distinct workspaces may overlap, on different streams or from different host threads. Each
must give, bit for bit, what the same call gives alone (the kernels are deterministic)."""
import dataclasses
import sys
import threading

import pytest
import torch

import synth
from synth.device import DeviceWorkload

from gpu_common import kv

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


class _Call:
    """One workload's call on a shared handle: its own workspace, scores and logits."""

    def __init__(self, m, h, dw):
        self.m, self.h, self.dw = m, h, dw
        self.batch = dw.batch(m)
        self.n = m.kvprm_workspace_size(h, self.batch)
        self.ws = torch.empty(max(self.n, 256), dtype=torch.uint8, device="cuda")
        self.scores = torch.full((dw.w.batch,), float("nan"), device="cuda")
        self.logits = torch.full((dw.w.batch,), float("nan"), device="cuda")
        self.cache, self.ro = dw.cache(m), dw.readout(m)

    def run(self, stream):
        self.m.kvprm_score(self.h, self.cache, self.batch, self.ro, self.ws.data_ptr(), self.n,
                           self.scores.data_ptr(), self.logits.data_ptr(), stream.cuda_stream)


def _workloads():
    shape = dataclasses.replace(synth.B7, num_layers=2)
    return [synth.make_workload("custom", shape=shape, lengths=lens, seed=seed)
            for lens, seed in (([900, 17, 0, 3000, 64], 601), ([2049, 5], 602),
                               ([33, 4100, 1, 700, 1500, 16, 0, 250, 12], 603))]


def test_calls_overlapping_on_two_streams():
    _say("case: three calls on one handle, overlapping on two streams")
    m = kv()
    dws = [DeviceWorkload(w) for w in _workloads()]
    h = m.kvprm_create(dws[0].desc(m))
    try:
        calls = [_Call(m, h, dw) for dw in dws]
        alone = []
        for c in calls:  # each call by itself
            c.run(torch.cuda.current_stream())
            torch.cuda.synchronize()
            alone.append((c.scores.clone(), c.logits.clone()))
        s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()  # default priority
        for rep in range(3):
            for c in calls:
                c.scores.fill_(float("nan"))
                c.logits.fill_(float("nan"))
            torch.cuda.synchronize()
            calls[0].run(s1)
            calls[1].run(s2)
            calls[2].run(s1 if rep % 2 else s2)
            torch.cuda.synchronize()
            for i, c in enumerate(calls):
                assert torch.equal(c.scores, alone[i][0]), (rep, i)
                assert torch.equal(c.logits, alone[i][1]), (rep, i)
    finally:
        m.kvprm_destroy(h)


def test_calls_from_two_host_threads():
    _say("case: two host threads calling one handle, each on its own stream")
    m = kv()
    dws = [DeviceWorkload(w) for w in _workloads()[:2]]
    h = m.kvprm_create(dws[0].desc(m))
    try:
        calls = [_Call(m, h, dw) for dw in dws]
        alone = []
        for c in calls:
            c.run(torch.cuda.current_stream())
            torch.cuda.synchronize()
            alone.append((c.scores.clone(), c.logits.clone()))
        errors = []

        def worker(c, want):
            try:
                st = torch.cuda.Stream()
                for _ in range(5):
                    with torch.cuda.stream(st):
                        c.scores.fill_(float("nan"))
                    c.run(st)
                    st.synchronize()
                    if not (torch.equal(c.scores, want[0]) and torch.equal(c.logits, want[1])):
                        errors.append("mismatch")
            except Exception as e:  # surfaced in the main thread
                errors.append(repr(e))

        threads = [threading.Thread(target=worker, args=(c, a)) for c, a in zip(calls, alone)]
        for t in threads:
            t.start()
        for t in threads:
            t.join(timeout=120)
        assert not any(t.is_alive() for t in threads)
        assert not errors, errors
    finally:
        m.kvprm_destroy(h)
