"""Invariants of the scoring pass on the GPU (section 4.1, Eq. (score)): a candidate's P(+)
depends on the keys and values its page-table row names, in row order, and on nothing else.

* Physical placement: moving every page of the pool to another physical slot (pools, fp8
  scales and page-table entries permuted together) leaves every score and logit bit for bit
  unchanged, with and without a shared-prefix group; unused pages hold NaN throughout.
* The same for the KV Steering gradient (appendix, KV Steering algorithm), which is written per
  physical page: after the move it equals the first gradient moved the same way, bit for bit.
* Candidate independence: each candidate scored alone (a batch of one, same pools and row)
  equals its score inside the batch up to the summation order of the attention chunks, which
  the plan sizes from the batch.
"""
import dataclasses
import sys

import numpy as np
import pytest
import torch

import synth
from synth.device import DeviceWorkload

from gpu_common import kv, run_score

pytestmark = pytest.mark.gpu

SHAPE = dataclasses.replace(synth.B7, num_layers=2)


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _moved(t: torch.Tensor, perm: torch.Tensor, layers: int, per_page: int) -> torch.Tensor:
    """t ([layers][pages ...] in page-major order) with page p moved to slot perm[p]."""
    raw = t.view(torch.uint8).view(layers, perm.numel(), -1)
    assert raw.shape[2] == per_page
    out = torch.empty_like(raw)
    out[:, perm] = raw
    return out.view(-1).view(t.dtype).view(t.shape)


def _permute_pages(dw: DeviceWorkload, seed: int) -> torch.Tensor:
    """Move physical page p to slot perm[p] in both pools (and the fp8 scales), and rewrite
    the page table to match; returns perm."""
    s, P = dw.w.shape, dw.w.num_pages
    perm = torch.from_numpy(np.random.default_rng(seed).permutation(P)).to(dw.device)
    tile = s.num_kv_heads * s.tile_elems * dw.k_pool.element_size()
    dw.k_pool = _moved(dw.k_pool, perm, s.num_layers, tile)
    dw.v_pool = _moved(dw.v_pool, perm, s.num_layers, tile)
    if dw.k_scale is not None:
        dw.k_scale = _moved(dw.k_scale, perm, s.num_layers, s.num_kv_heads * 4)
        dw.v_scale = _moved(dw.v_scale, perm, s.num_layers, s.num_kv_heads * 4)
    pt = dw.page_table
    dw.page_table = torch.where(pt >= 0, perm[pt.clamp(min=0).long()].to(torch.int32), pt)
    assert not torch.equal(dw.page_table, pt)
    return perm


def _cache_gradient(dw: DeviceWorkload):
    m = kv()
    h = m.kvprm_create(dw.desc(m))
    try:
        batch = dw.batch(m)
        n = m.kvprm_workspace_size_grad(h, batch)
        ws = torch.empty(n, dtype=torch.uint8, device="cuda")
        scores = torch.full((dw.w.batch,), float("nan"), device="cuda")
        gk = torch.zeros(dw.k_pool.shape, dtype=torch.float32, device="cuda")
        gv = torch.zeros(dw.v_pool.shape, dtype=torch.float32, device="cuda")
        m.kvprm_score_grad(h, dw.cache(m), batch, dw.readout(m), ws.data_ptr(), n,
                           scores.data_ptr(), gk.data_ptr(), gv.data_ptr(),
                           torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
    finally:
        m.kvprm_destroy(h)
    return scores.cpu().numpy(), gk, gv


@pytest.mark.parametrize("kv_dtype,groups", [("bf16", False), ("fp8", False), ("bf16", True)])
def test_physical_page_placement_is_bitwise_invisible(kv_dtype, groups):
    shape = dataclasses.replace(SHAPE, kv_dtype=kv_dtype)
    if groups:  # two groups sharing 40 and 7 prefix pages, one candidate on its own
        lengths, g = [640 + 5, 640 + 300, 640, 112 + 77, 112 + 1, 900], ([0, 3, 5, 6], [640, 112, 0])
    else:
        lengths, g = [4100, 0, 17, 1, 2049, 33, 700, 3000], None
    _say(f"case: page placement {kv_dtype} groups={g} lengths={lengths}")
    w = synth.make_workload("custom", shape=shape, lengths=lengths, seed=8100, groups=g)
    dw = DeviceWorkload(w, nan_unused_pages=True)
    p0, z0 = run_score(dw)
    _permute_pages(dw, seed=8101)
    p1, z1 = run_score(dw)
    _say(f"  P(+) = {np.round(p0, 5)}; max|dz| after the move = {np.max(np.abs(z1 - z0)):.3e}")
    assert np.all(np.isfinite(p0)) and np.all(np.isfinite(z0))
    assert np.array_equal(p0, p1) and np.array_equal(z0, z1)


def test_candidate_scored_alone_matches_the_batch():
    lengths = [3000, 0, 129, 2048, 16, 1500]
    _say(f"case: candidates alone vs in the batch, lengths={lengths}")
    w = synth.make_workload("custom", shape=SHAPE, lengths=lengths, seed=8200)
    dw = DeviceWorkload(w, nan_unused_pages=True)
    p, z = run_score(dw)
    pt_full, len_full, w_full = dw.page_table, dw.lengths, dw.w
    try:
        for b in range(len(lengths)):
            dw.w = dataclasses.replace(w_full, lengths=[lengths[b]], page_table=[w_full.page_table[b]],
                                       group_start=[], group_prefix_len=[])
            dw.page_table = pt_full[b:b + 1].contiguous()
            dw.lengths = len_full[b:b + 1].contiguous()
            pb, zb = run_score(dw)
            _say(f"  candidate {b}: P(+) {pb[0]:.6f} alone, {p[b]:.6f} in the batch, "
                 f"|dz| = {abs(zb[0] - z[b]):.2e}")
            assert np.isfinite(zb[0])
            assert abs(pb[0] - p[b]) <= 1e-5 and abs(zb[0] - z[b]) <= 5e-5
    finally:
        dw.page_table, dw.lengths, dw.w = pt_full, len_full, w_full


def test_cache_gradient_moves_with_the_pages():
    lengths = [3000, 17, 0, 1100, 64]
    _say(f"case: cache gradient under a page move, lengths={lengths}")
    w = synth.make_workload("custom", shape=SHAPE, lengths=lengths, seed=8300)
    dw = DeviceWorkload(w, nan_unused_pages=True)
    p0, gk0, gv0 = _cache_gradient(dw)
    perm = _permute_pages(dw, seed=8301)
    p1, gk1, gv1 = _cache_gradient(dw)
    s = w.shape
    per_page = s.num_kv_heads * s.tile_elems * 4
    assert np.all(np.isfinite(p0)) and np.array_equal(p0, p1)
    assert torch.count_nonzero(gk0) > 0 and torch.count_nonzero(gv0) > 0
    assert torch.equal(_moved(gk0, perm, s.num_layers, per_page), gk1)
    assert torch.equal(_moved(gv0, perm, s.num_layers, per_page), gv1)
    _say(f"  P(+) = {np.round(p0, 5)}; gradients moved with their pages, bit for bit")
