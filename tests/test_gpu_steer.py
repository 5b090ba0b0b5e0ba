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


def test_cache_gradient_7b_long_multi_chunk():
    """Long caches against the oracle: 8192 tokens (32 chunks of the backward's 16-page
    chunks) and 3001 (a partial last page), 7B shape, 2 layers."""
    _say("case: cache gradient, 7B shape, 2 layers, L = 8192 and 3001")
    shape = dataclasses.replace(synth.B7, num_layers=2)
    w = synth.make_workload("custom", shape=shape, lengths=[8192, 3001], seed=405)
    _grad_case(w)


@pytest.mark.parametrize("head_dim", [64, 128])
def test_cache_gradient_sixteen_heads_per_kv_head(head_dim):
    """g = 16 (the most q-heads per kv-head the kernels take): every column of the matrix-core
    products is a head."""
    _say(f"case: cache gradient, 16 q-heads over 1 kv-head, d_h = {head_dim}")
    shape = synth.ModelShape(2, 512, 16, 1, head_dim, 1024)
    w = synth.make_workload("custom", shape=shape, lengths=[333, 16, 1], seed=404 + head_dim)
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


def test_kv_steering_7b_two_layers_matches_the_oracle():
    """Two steering steps at the 7B shape (2 layers, 4096 and 999 cached tokens) with the step
    size of the benchmark: the stored caches within 2 bf16 spacings of the oracle's steps, P(+)
    before and after within 2e-3 of the oracle's."""
    _say("case: KV steering, 2 steps, 7B shape, 2 layers")
    shape = dataclasses.replace(synth.B7, num_layers=2)
    w = synth.make_workload("custom", shape=shape, lengths=[4096, 999], seed=406)
    dw = DeviceWorkload(w)
    eta, steps = 20.0, 2
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
    GK, GV = _dense_from_pools(w, dw.k_pool.view(torch.bfloat16), dw.v_pool.view(torch.bfloat16))
    for b in range(w.batch):
        for got, want in ((GK[b], K2[b]), (GV[b], V2[b])):
            ulp = np.abs(want) * 2.0 ** -7 + 1e-30
            assert np.all(np.abs(got - want) <= 2 * ulp + 1e-6)


# ---------------------------------------------------------------------------------------------
# Full size (the ragged 32k batch: 28 layers of the 7B shape, 8 candidates, 216k cached tokens).
# The fp64 oracle cannot differentiate this size in memory, so the gradient is checked against
# what holds at any size: central differences of the scores themselves (kvprm_score, whose
# full-size values are checked against the stored oracle values elsewhere), and the steering
# step against the gradient it is built from.

def _bf16_spacing(x: torch.Tensor) -> torch.Tensor:
    """Spacing of bf16 numbers in the binade of |x| (x holds bf16 values, float32): x +- it are
    both bf16 numbers (just below a power of two the spacing halves, so the step down stays
    representable). Zero where x is zero."""
    _, e = torch.frexp(x)  # x = m 2^e, 0.5 <= |m| < 1: 8 significant bits -> spacing 2^(e-8)
    sp = torch.pow(2.0, (e - 8).to(torch.float32))
    return torch.where(x == 0, torch.zeros_like(x), sp)


def _page_owner(w) -> torch.Tensor:
    owner = np.full(w.num_pages, -1, dtype=np.int64)
    for b, L in enumerate(w.lengths):
        for i in range(-(-L // w.shape.page_size)):
            owner[w.page_table[b][i]] = b
    return torch.from_numpy(owner).cuda()


def _softplus_neg(z: np.ndarray) -> np.ndarray:
    return np.logaddexp(0.0, -np.asarray(z, dtype=np.float64))  # -log sigmoid(z)


@pytest.fixture(scope="module")
def full_size():
    _say("setup: ragged 32k workload on the device, cache gradient by kvprm_score_grad")
    w = synth.make_workload("ragged_32k")
    dw = DeviceWorkload(w)
    m = kv()
    h = m.kvprm_create(dw.desc(m))
    batch = dw.batch(m)
    n = m.kvprm_workspace_size_grad(h, batch)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    scores = torch.full((w.batch,), float("nan"), device="cuda")
    gk = torch.zeros(dw.k_pool.shape, dtype=torch.float32, device="cuda")
    gv = torch.zeros(dw.v_pool.shape, dtype=torch.float32, device="cuda")
    m.kvprm_score_grad(h, dw.cache(m), batch, dw.readout(m), ws.data_ptr(), n, scores.data_ptr(),
                       gk.data_ptr(), gv.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    state = dict(w=w, dw=dw, m=m, h=h, batch=batch, ws=ws, n=n, gk=gk, gv=gv,
                 p=scores.cpu().numpy().astype(np.float64), owner=_page_owner(w))
    yield state
    m.kvprm_destroy(h)


def _logits(st) -> np.ndarray:
    m, dw, w = st["m"], st["dw"], st["w"]
    nbytes = m.kvprm_workspace_size(st["h"], st["batch"])
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda")
    scores = torch.full((w.batch,), float("nan"), device="cuda")
    logits = torch.full((w.batch,), float("nan"), device="cuda")
    m.kvprm_score(st["h"], dw.cache(m), st["batch"], dw.readout(m), ws.data_ptr(), nbytes,
                  scores.data_ptr(), logits.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return logits.cpu().numpy().astype(np.float64)


def test_full_size_gradient_matches_central_differences(full_size):
    """For each candidate, a perturbation d of one bf16 spacing against the gradient's sign on a
    seeded random subset of its cached elements (sized so that g.d is about -0.02): the central
    difference (loss(kv + d) - loss(kv - d)) / 2 of the scoring pass equals g.d within 2%.
    A wrong sign, a missing term or a misplaced element anywhere in the 28 layers' backward
    moves g.d away from the scores' own change."""
    st = full_size
    w, dw, owner = st["w"], st["dw"], st["owner"]
    s = w.shape
    B, P = w.batch, w.num_pages
    _say("case: full-size gradient vs central differences of kvprm_score (ragged 32k)")
    z0 = _logits(st)
    assert np.allclose(1.0 / (1.0 + np.exp(-z0)), st["p"], atol=1e-6)
    # first pass: sum over each candidate's elements of |g| * spacing
    mass = torch.zeros(B, dtype=torch.float64, device="cuda")
    valid = owner >= 0
    oidx = owner.clamp(min=0)
    for pool, grad in ((dw.k_pool, st["gk"]), (dw.v_pool, st["gv"])):
        for l in range(s.num_layers):
            x = pool[l].view(P, -1).float()
            g = grad[l].view(P, -1)
            per_page = (g.abs() * _bf16_spacing(x)).sum(dim=1, dtype=torch.float64)
            mass.index_add_(0, oidx[valid], per_page[valid])
    target = 0.02
    frac = torch.clamp(target / mass, max=1.0)
    frac_page = torch.where(valid, frac[oidx], torch.zeros_like(frac[oidx])).float()
    gen = torch.Generator(device="cuda").manual_seed(20260)
    pred = torch.zeros(B, dtype=torch.float64, device="cuda")
    plus, minus = [], []
    for pool, grad in ((dw.k_pool, st["gk"]), (dw.v_pool, st["gv"])):
        pp, mm = torch.empty_like(pool), torch.empty_like(pool)
        for l in range(s.num_layers):
            x = pool[l].view(P, -1).float()
            g = grad[l].view(P, -1)
            pick = torch.rand(x.shape, generator=gen, device="cuda") < frac_page[:, None]
            d = torch.where(pick & (g != 0), -torch.sign(g) * _bf16_spacing(x),
                            torch.zeros_like(x))
            pred.index_add_(0, oidx[valid], (g.double() * d.double()).sum(dim=1)[valid])
            xp, xm = x + d, x - d
            pp[l].view(P, -1).copy_(xp.to(torch.bfloat16))
            mm[l].view(P, -1).copy_(xm.to(torch.bfloat16))
            assert torch.equal(pp[l].view(P, -1).float(), xp)  # exactly representable
            assert torch.equal(mm[l].view(P, -1).float(), xm)
        plus.append(pp), minus.append(mm)
    k0, v0 = dw.k_pool.clone(), dw.v_pool.clone()
    try:
        dw.k_pool.copy_(plus[0]), dw.v_pool.copy_(plus[1])
        zp = _logits(st)
        dw.k_pool.copy_(minus[0]), dw.v_pool.copy_(minus[1])
        zm = _logits(st)
    finally:
        dw.k_pool.copy_(k0), dw.v_pool.copy_(v0)
    cd = (_softplus_neg(zp) - _softplus_neg(zm)) / 2
    pr = pred.cpu().numpy()
    for b in range(B):
        _say(f"  candidate {b}: L={w.lengths[b]} g.d {pr[b]:+.6e} central difference {cd[b]:+.6e}"
             f" (rel {abs(cd[b] - pr[b]) / abs(pr[b]):.2e})")
    assert np.all(pr < -0.01)
    assert np.all(np.abs(cd - pr) <= 0.02 * np.abs(pr) + 2e-5)


def test_full_size_steering_step(full_size):
    """kvprm_steer at full size, one step: every stored key and value of every candidate equals
    round_bf16(kv - eta g) with g from kvprm_score_grad (within one bf16 spacing: a value can
    land on either side of a rounding boundary), pages no candidate reads are untouched bit for bit, and P(+) rises
    for every candidate. Runs last on the module's workload: it rewrites the cache."""
    st = full_size
    w, dw, m, owner = st["w"], st["dw"], st["m"], st["owner"]
    s = w.shape
    P = w.num_pages
    _say("case: full-size steering step (ragged 32k)")
    gn2 = torch.zeros(w.batch, dtype=torch.float64, device="cuda")
    valid = owner >= 0
    for grad in (st["gk"], st["gv"]):
        for l in range(s.num_layers):
            gn2.index_add_(0, owner[valid],
                           (grad[l].view(P, -1).double() ** 2).sum(dim=1)[valid])
    eta = float(0.05 / gn2.max().item())  # a first-order decrease of up to 0.05 in the loss
    k0, v0 = dw.k_pool.clone(), dw.v_pool.clone()
    before = torch.full((w.batch,), float("nan"), device="cuda")
    after = torch.full((w.batch,), float("nan"), device="cuda")
    m.kvprm_steer(st["h"], dw.cache(m), st["batch"], dw.readout(m), eta, 1, st["ws"].data_ptr(),
                  st["n"], before.data_ptr(), after.data_ptr(),
                  torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    pb, pa = before.cpu().numpy(), after.cpu().numpy()
    _say(f"  eta {eta:.4e}; P before {pb}; after {pa}")
    assert np.allclose(pb, st["p"], atol=1e-6)
    assert np.all(pa > pb)
    moved_total = 0
    eta32 = float(np.float32(eta))  # the step the library applies (fp32)
    for pool, orig, grad in ((dw.k_pool, k0, st["gk"]), (dw.v_pool, v0, st["gv"])):
        for l in range(s.num_layers):
            x = orig[l].view(P, -1).float()
            got = pool[l].view(P, -1).float()
            # x - eta g exactly (float64), rounded to float32 and then to bf16: where x and
            # eta g nearly cancel, rounding eta g first would move the result by many bf16 steps
            want = (x.double() - eta32 * grad[l].view(P, -1).double()).float()
            want = want.to(torch.bfloat16).float()
            off = (got - want).abs()
            assert bool((off <= _bf16_spacing(want) + 1e-30).all()), f"layer {l}"
            assert float((off > 0).float().mean()) < 1e-3
            assert torch.equal(pool[l].view(P, -1)[~valid], orig[l].view(P, -1)[~valid])
            moved_total += int((got != x).sum())
    _say(f"  elements changed: {moved_total}")
    assert moved_total > 0
