"""kvprm_score_static (the allocation-free scoring entry point: its workspace is the library's
static device array) against kvprm_score with a caller workspace, through the C ABI: two calls
in a row on one GPU, the second with a smaller batch, each equal to kvprm_score bit for bit (same
kernels, same plan), and a batch above the static size refused before anything is enqueued."""
import dataclasses
import sys

import numpy as np
import pytest
import torch

import synth
from synth.device import DeviceWorkload

from gpu_common import kv, run_score

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _static_scores(dw: DeviceWorkload):
    m = kv()
    h = m.kvprm_create(dw.desc(m))
    try:
        B = dw.w.batch
        scores = torch.full((B,), float("nan"), dtype=torch.float32, device="cuda")
        logits = torch.full((B,), float("nan"), dtype=torch.float32, device="cuda")
        st = torch.cuda.current_stream()
        m.kvprm_score_static(h, dw.cache(m), dw.batch(m), dw.readout(m), scores.data_ptr(),
                             logits.data_ptr(), st.cuda_stream)
        st.synchronize()
        return scores.cpu().numpy().astype(np.float64), logits.cpu().numpy().astype(np.float64)
    finally:
        m.kvprm_destroy(h)


def test_static_workspace_equals_caller_workspace_twice_then_smaller():
    shape = dataclasses.replace(synth.B7, num_layers=2)
    big = synth.make_workload("custom", shape=shape, lengths=[32768, 0, 17, 20001, 4096, 31000, 1, 9999],
                              seed=5150)
    small = synth.make_workload("custom", shape=shape, lengths=[300, 16, 2049], seed=5151)
    for w in (big, small):
        _say(f"case: static workspace, B={w.batch} lengths={w.lengths}")
        dw = DeviceWorkload(w, nan_unused_pages=True)
        p_s, z_s = _static_scores(dw)
        p_r, z_r = run_score(dw)
        _say(f"  P static {np.round(p_s, 5)}; max|dP| vs caller workspace {np.max(np.abs(p_s - p_r)):.2e}")
        assert np.all(np.isfinite(p_s)) and np.all(np.isfinite(z_s))
        assert np.array_equal(p_s, p_r) and np.array_equal(z_s, z_r)
        del dw
        torch.cuda.empty_cache()


def test_static_workspace_more_than_16_rows():
    """More than 16 candidates: the output and down projections run as split-K products whose
    slice partials live in the workspace; two calls in a row, the second with fewer rows."""
    shape = dataclasses.replace(synth.B7, num_layers=2)
    for B, seed in ((40, 5152), (20, 5153)):
        lengths = [(53 * i * i + 7 * i) % 1500 for i in range(B)]
        w = synth.make_workload("custom", shape=shape, lengths=lengths, seed=seed)
        _say(f"case: static workspace, B={w.batch} (split-K output/down)")
        dw = DeviceWorkload(w, nan_unused_pages=True)
        p_s, z_s = _static_scores(dw)
        p_r, z_r = run_score(dw)
        _say(f"  max|dP| vs caller workspace {np.max(np.abs(p_s - p_r)):.2e}")
        assert np.all(np.isfinite(p_s)) and np.all(np.isfinite(z_s))
        assert np.array_equal(p_s, p_r) and np.array_equal(z_s, z_r)
        del dw
        torch.cuda.empty_cache()


def test_static_workspace_fp32_tiny_and_refusal():
    w = synth.make_workload("tiny_fp32")
    _say(f"case: static workspace tiny fp32 B={w.batch}")
    dw = DeviceWorkload(w, nan_unused_pages=True)
    p_s, z_s = _static_scores(dw)
    p_r, z_r = run_score(dw)
    assert np.array_equal(p_s, p_r) and np.array_equal(z_s, z_r)
    m = kv()
    # a batch whose workspace exceeds the static array: refused on the host
    h = m.kvprm_create(m.make_desc(28, 3584, 28, 4, 128, 18944))
    try:
        b = m.make_batch(64, dw.page_table.data_ptr(), 2048, dw.lengths.data_ptr())
        assert m.kvprm_workspace_size(h, b) > m.STATIC_WORKSPACE_BYTES
        with pytest.raises(m.KvprmError) as e:
            m.kvprm_score_static(h, dw.cache(m), b, dw.readout(m), 0, 0, 0)
        assert e.value.status == m.KVPRM_E_WORKSPACE
    finally:
        m.kvprm_destroy(h)
