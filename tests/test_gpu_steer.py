"""GPU parity of the cache gradients (kvprm_score_grad) and of KV Steering (kvprm_steer)
against the fp64 oracle (oracle.kv_steering: torch float64 reverse-mode differentiation of the
verify pass, pinned by finite differences; steps rounded to bf16 like the pools).

Bars: gradients element by element within 1e-3 of the largest gradient magnitude (fp32
arithmetic on the same bf16 inputs); zero gradient on slots past L_b; after steering, P(+)
within 2e-3 of the oracle's, the stored values within two bf16 ulps of the oracle's (a step
can round either way when the fp32 and fp64 gradients straddle a rounding boundary), and pages
no candidate reads unchanged bit for bit."""
import dataclasses
import sys

import numpy as np
import pytest
import torch

import synth
from oracle import inputs as oin
from oracle import kv_steering as ksr
from oracle import kvprm_oracle as ko
from synth.device import DeviceWorkload

from gpu_common import kv

pytestmark = pytest.mark.gpu

SMALL = synth.ModelShape(2, 256, 4, 2, 64, 1024)


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _dense_from_pools(w, kpool, vpool):
    """Per candidate [N_L][n_kv][L][d] float64 from device pools (any float dtype)."""
    s = w.shape
    kp = kpool.float().cpu().numpy().astype(np.float64).reshape(s.num_layers, w.num_pages,
                                                               s.num_kv_heads, s.tile_elems)
    vp = vpool.float().cpu().numpy().astype(np.float64).reshape(s.num_layers, w.num_pages,
                                                               s.num_kv_heads, s.tile_elems)
    K, V = [], []
    for b, L in enumerate(w.lengths):
        kb = np.zeros((s.num_layers, s.num_kv_heads, L, s.head_dim))
        vb = np.zeros_like(kb)
        for l in range(s.num_layers):
            for i in range(-(-L // s.page_size)):
                pg = w.page_table[b][i]
                n = min(s.page_size, L - i * s.page_size)
                for j in range(s.num_kv_heads):
                    kt = ko.k_tile_to_tokens(kp[l, pg, j], s.page_size, s.head_dim, 2)
                    vt = ko.v_tile_to_tokens(vp[l, pg, j], s.page_size, s.head_dim, 2)
                    kb[l, j, i * s.page_size: i * s.page_size + n] = kt[:n]
                    vb[l, j, i * s.page_size: i * s.page_size + n] = vt[:n]
        K.append(kb), V.append(vb)
    return K, V


def _tail_slots_zero(w, gpool, which):
    """Gradient entries of slots at or beyond L_b in each candidate's last page are zero."""
    s = w.shape
    g = gpool.cpu().numpy().reshape(s.num_layers, w.num_pages, s.num_kv_heads, s.tile_elems)
    for b, L in enumerate(w.lengths):
        if L % s.page_size == 0 or L == 0:
            continue
        pg = w.page_table[b][L // s.page_size]
        for l in range(s.num_layers):
            for j in range(s.num_kv_heads):
                to_tokens = ko.k_tile_to_tokens if which == "k" else ko.v_tile_to_tokens
                t = to_tokens(g[l, pg, j], s.page_size, s.head_dim, 2)
                assert np.all(t[L % s.page_size:] == 0)


def _grad_case(w):
    dw = DeviceWorkload(w, nan_unused_pages=True)
    m = kv()
    h = m.kvprm_create(dw.desc(m))
    try:
        batch = dw.batch(m)
        n = m.kvprm_workspace_size_grad(h, batch)
        ws = torch.empty(n, dtype=torch.uint8, device="cuda")
        scores = torch.full((w.batch,), float("nan"), device="cuda")
        gk = torch.zeros(dw.k_pool.shape, dtype=torch.float32, device="cuda")
        gv = torch.zeros(dw.v_pool.shape, dtype=torch.float32, device="cuda")
        m.kvprm_score_grad(h, dw.cache(m), batch, dw.readout(m), ws.data_ptr(), n,
                           scores.data_ptr(), gk.data_ptr(), gv.data_ptr(),
                           torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
    finally:
        m.kvprm_destroy(h)
    ro = oin.readout_from_synth(w.shape, w.seed, layer_cache=64)
    cache = oin.cache_from_synth(w)
    K, V = ksr.dense_cache(cache, w.shape, w.lengths, w.page_table)
    ref = ksr.loss_and_grads(w.shape, ro, K, V, w.lengths)
    GK, GV = _dense_from_pools(w, gk, gv)
    p = scores.cpu().numpy()
    for b in range(w.batch):
        loss, z, dK, dV = ref[b]
        assert abs(p[b] - ko.sigmoid(np.array([z]))[0]) < 2e-3
        if w.lengths[b] == 0:
            continue
        big = max(np.max(np.abs(dK)), np.max(np.abs(dV)))
        ek, ev = np.max(np.abs(GK[b] - dK)), np.max(np.abs(GV[b] - dV))
        _say(f"  candidate {b}: L={w.lengths[b]} max|dK err| {ek:.2e} max|dV err| {ev:.2e} "
             f"(max |grad| {big:.2e})")
        assert ek <= 1e-3 * big and ev <= 1e-3 * big
    _tail_slots_zero(w, gk, "k")
    _tail_slots_zero(w, gv, "v")


def test_cache_gradient_small_shape():
    _say("case: cache gradient, small bf16 shape, ragged lengths incl. 0 and partial pages")
    w = synth.make_workload("custom", shape=SMALL, lengths=[37, 0, 300, 16], seed=401)
    _grad_case(w)


def test_cache_gradient_7b_two_layers():
    _say("case: cache gradient, 7B shape, 2 layers")
    shape = dataclasses.replace(synth.B7, num_layers=2)
    w = synth.make_workload("custom", shape=shape, lengths=[700, 17], seed=402)
    _grad_case(w)


def test_kv_steering_matches_the_oracle():
    _say("case: KV steering, 3 steps, small bf16 shape")
    w = synth.make_workload("custom", shape=SMALL, lengths=[150, 33, 64], seed=403)
    dw = DeviceWorkload(w)
    k0, v0 = dw.k_pool.clone(), dw.v_pool.clone()
    eta, steps = 0.5, 3
    m = kv()
    h = m.kvprm_create(dw.desc(m))
    try:
        batch = dw.batch(m)
        n = m.kvprm_workspace_size_grad(h, batch)
        ws = torch.empty(n, dtype=torch.uint8, device="cuda")
        before = torch.full((w.batch,), float("nan"), device="cuda")
        after = torch.full((w.batch,), float("nan"), device="cuda")
        m.kvprm_steer(h, dw.cache(m), batch, dw.readout(m), eta, steps, ws.data_ptr(), n,
                      before.data_ptr(), after.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
    finally:
        m.kvprm_destroy(h)
    ro = oin.readout_from_synth(w.shape, w.seed, layer_cache=64)
    K, V = ksr.dense_cache(oin.cache_from_synth(w), w.shape, w.lengths, w.page_table)
    K2, V2, losses = ksr.steer(w.shape, ro, K, V, w.lengths, eta, steps, "bf16")
    pb, pa = before.cpu().numpy(), after.cpu().numpy()
    p_ref0 = np.exp(-np.array(losses[0]))
    p_ref1 = np.exp(-np.array(losses[-1]))
    _say(f"  P before {pb} (oracle {p_ref0}), after {pa} (oracle {p_ref1})")
    assert np.max(np.abs(pb - p_ref0)) < 2e-3 and np.max(np.abs(pa - p_ref1)) < 2e-3
    assert np.all(pa > pb)
    GK, GV = _dense_from_pools(w, dw.k_pool.view(torch.bfloat16), dw.v_pool.view(torch.bfloat16))
    for b in range(w.batch):
        for got, want, start in ((GK[b], K2[b], K[b]), (GV[b], V2[b], V[b])):
            ulp = np.abs(want) * 2.0 ** -7 + 1e-30
            assert np.all(np.abs(got - want) <= 2 * ulp + 1e-6)
            moved = np.mean(got != start)
            assert moved > 0.01  # the step changes the cache
    # pages no candidate reads are untouched
    used = set(w.used_pages())
    s = w.shape
    tile = s.num_kv_heads * s.tile_elems
    for pool, orig in ((dw.k_pool, k0), (dw.v_pool, v0)):
        a = pool.view(s.num_layers, w.num_pages, tile)
        o = orig.view(s.num_layers, w.num_pages, tile)
        for pg in range(w.num_pages):
            if pg not in used:
                assert torch.equal(a[:, pg], o[:, pg])
