"""GPU parity of libkvprm against the fp64 oracle on identical seeded inputs.

Tolerances: fp32 weights and cache, max |dP(+)| <= 1e-5; bf16 weights (bf16 or fp8 cache),
max |dP(+)| <= 2e-3. The logit z is also checked, so that a saturated sigmoid cannot hide an
error. The attention step alone is compared element by element.
"""
import sys

import numpy as np
import pytest
import torch

import synth
from oracle import inputs as oin
from oracle import kv_steering as ksr
from oracle import kvprm_oracle as ko
from synth.device import DeviceWorkload

from gpu_common import host_activations, kv, run_attention, run_score

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def test_device_generator_matches_host_bits():
    _say("case: device generator vs host")
    n = 1 << 20
    for dt, tdt in ((synth.DT_F32, torch.float32), (synth.DT_BF16, torch.bfloat16),
                    (synth.DT_F64, torch.float64)):
        t = torch.empty(n, dtype=tdt, device="cuda")
        synth.device_normal(t.data_ptr(), n, 17, 5, 1000, 0.5, 0.25, dt, 0)
        torch.cuda.synchronize()
        host = synth.host_normal(n, 17, 5, 1000, 0.5, 0.25, dt)
        dev = t.cpu()
        if dt == synth.DT_BF16:
            dev = dev.view(torch.int16).numpy().view(np.uint16)
        else:
            dev = dev.numpy()
        assert np.array_equal(dev.view(np.uint8), host.view(np.uint8))
    T, nt = 2048, 333
    for mode in ("pow2", "amax"):
        codes = torch.empty(nt * T, dtype=torch.uint8, device="cuda")
        scales = torch.empty(nt, dtype=torch.float32, device="cuda")
        synth.device_fp8_tiles(codes.data_ptr(), scales.data_ptr(), nt, T, 9, 3, 50, 0,
                               scale=mode)
        torch.cuda.synchronize()
        hc, hs = synth.host_fp8_tiles(nt, T, 9, 3, 50, scale=mode)
        assert np.array_equal(codes.cpu().numpy(), hc)
        assert np.array_equal(scales.cpu().numpy(), hs)


ATTN_CASES = [
    # name, lengths (incl. empty, one token, page edges, ragged tails), K scale; fp8 caches have
    # per-tile scales amax / 448 (not powers of two) unless the name ends in _pow2
    ("tiny_fp32", [512, 0, 1, 15, 16, 17, 700, 1025], 1.0),
    ("b7_bf16", [4096, 0, 1, 17, 5000, 9000], 1.0),
    ("b7_bf16_spiky", [3000, 33, 16], 30.0),
    ("fp8", [2049, 0, 31, 8192], 1.0),
    # 16 q-heads per kv-head
    ("g16_bf16", [1000, 0, 17, 4100], 1.0),
    ("g16_fp8", [33, 2500], 1.0),
    # batches large enough for 32-page and 64-page attention chunks (the plan picks the chunk
    # from batch x max_pages)
    ("b7_bf16", [16384, 300, 17, 9000, 0, 12000], 1.0),
    ("b7_bf16", [32768, 1, 20000, 33, 5000, 31000], 1.0),
    ("fp8", [32768, 16, 17000, 4000, 29999, 2], 1.0),
    ("fp8_pow2", [2049, 0, 31, 8192], 1.0),
    ("fp8", [3000, 33, 16], 30.0),
]


def _shape(name):
    import dataclasses
    if name == "tiny_fp32":
        return synth.TINY
    if name.startswith("b7"):
        return dataclasses.replace(synth.B7, num_layers=2)
    if name in ("fp8", "fp8_pow2"):
        return dataclasses.replace(synth.LARGE_FP8, num_layers=2)
    if name == "g16_bf16":
        return synth.ModelShape(2, 1024, 16, 1, 64, 2048)
    if name == "g16_fp8":
        return synth.ModelShape(2, 2048, 32, 2, 128, 2048, kv_dtype="fp8")
    raise KeyError(name)


@pytest.mark.parametrize("name,lengths,k_std", ATTN_CASES)
def test_attention_parity(name, lengths, k_std):
    _say(f"case: attention {name} lengths={lengths}")
    shape = _shape(name)
    w = synth.make_workload("custom", shape=shape, lengths=lengths, seed=4242, k_std=k_std,
                            fp8_scale="pow2" if name.endswith("_pow2") else "amax")
    dw = DeviceWorkload(w, nan_unused_pages=True, fill_weights=False)
    q, ks, vs = host_activations(w, 0xABC, scale=1.0)
    layer = 1
    o = run_attention(dw, layer, q, ks, vs)
    cache = oin.cache_from_synth(w)
    ref = ko.attention_layer(shape, cache, layer, w.lengths, w.page_table, q.astype(np.float64),
                             ks.astype(np.float64), vs.astype(np.float64))
    assert np.all(np.isfinite(o))
    err = np.max(np.abs(o - ref))
    scale = max(1.0, float(np.max(np.abs(ref))))
    _say(f"  max|do| = {err:.3e} (max|o| = {np.max(np.abs(ref)):.3e})")
    assert err <= 2e-5 * scale


@pytest.mark.parametrize("name", ["b7_bf16", "fp8"])
def test_attention_sink_key(name):
    """A key the query points straight at (an attention sink): every q-head of kv-head j of a
    candidate is a multiple of one cached key of that head, so its score stands ~30 above the
    rest and the softmax is one-hot to fp32 precision. Sinks at token 0, mid-cache (not on a
    page or chunk boundary) and at the last token of a partial page; the other kv-heads keep
    random queries."""
    import dataclasses
    _say(f"case: attention sink key {name}")
    shape = _shape(name)
    lengths = [4100, 20000, 3001]
    sinks = [0, 12345, 3000]
    w = synth.make_workload("custom", shape=shape, lengths=lengths, seed=4747)
    dw = DeviceWorkload(w, nan_unused_pages=True, fill_weights=False)
    q, ks, vs = host_activations(w, 0xABE, scale=1.0)
    layer = 1
    cache = oin.cache_from_synth(w)
    K, _ = ksr.dense_cache(cache, shape, w.lengths, w.page_table)
    g = shape.num_q_heads // shape.num_kv_heads
    for b, t in enumerate(sinks):
        j = b % shape.num_kv_heads
        key = K[b][layer][j][t]
        alpha = 4.0 * np.sqrt(shape.head_dim) / float(np.dot(key, key)) * np.sqrt(shape.head_dim)
        q[b, j * g:(j + 1) * g] = (alpha * key).astype(np.float32)
    o = run_attention(dw, layer, q, ks, vs)
    ref = ko.attention_layer(shape, cache, layer, w.lengths, w.page_table, q.astype(np.float64),
                             ks.astype(np.float64), vs.astype(np.float64))
    assert np.all(np.isfinite(o))
    err = np.max(np.abs(o - ref))
    scale = max(1.0, float(np.max(np.abs(ref))))
    _say(f"  max|do| = {err:.3e} (max|o| = {np.max(np.abs(ref)):.3e})")
    assert err <= 2e-5 * scale
    # the sink heads' outputs are the sink's value row (to the softmax's rounding)
    _, V = ksr.dense_cache(cache, shape, w.lengths, w.page_table)
    for b, t in enumerate(sinks):
        j = b % shape.num_kv_heads
        for h in range(j * g, (j + 1) * g):
            assert np.max(np.abs(ref[b, h] - V[b][layer][j][t])) < 1e-6 * max(1.0, np.max(np.abs(V[b][layer][j][t])))


@pytest.mark.parametrize("name,lengths", [("b7_bf16", [32768, 1, 20000, 33, 5000, 31000]),
                                          ("fp8", [9000, 0, 17000])])
def test_attention_partials_match_the_attention_step(name, lengths):
    """kvprm_attention_partials writes exactly what the chunk kernels of kvprm_attention write
    into the workspace (same bytes from the same starting contents) and nothing else: bytes
    past the workspace size and the query stay untouched."""
    _say(f"case: attention partials {name} lengths={lengths}")
    w = synth.make_workload("custom", shape=_shape(name), lengths=lengths, seed=4343)
    dw = DeviceWorkload(w, nan_unused_pages=True, fill_weights=False)
    q, ks, vs = host_activations(w, 0xABD, scale=1.0)
    m = kv()
    h = m.kvprm_create(dw.desc(m))
    try:
        batch = dw.batch(m)
        n = m.kvprm_workspace_size(h, batch)
        guard = 4096
        qd, kd, vd = (torch.from_numpy(a).cuda() for a in (q, ks, vs))
        q0 = qd.clone()
        st = torch.cuda.current_stream().cuda_stream
        ws1 = torch.full((n + guard,), 0x5A, dtype=torch.uint8, device="cuda")
        ws2 = ws1.clone()
        m.kvprm_attention_partials(h, dw.cache(m), batch, 1, qd.data_ptr(), ws1.data_ptr(), n, st)
        o = torch.empty_like(qd)
        m.kvprm_attention(h, dw.cache(m), batch, 1, qd.data_ptr(), kd.data_ptr(), vd.data_ptr(),
                          ws2.data_ptr(), n, o.data_ptr(), st)
        torch.cuda.synchronize()
        assert torch.equal(ws1[n:], torch.full((guard,), 0x5A, dtype=torch.uint8, device="cuda"))
        assert torch.equal(ws1, ws2)
        assert torch.equal(qd, q0)
    finally:
        m.kvprm_destroy(h)


# Shared-prefix attention: groups whose prefix ends inside a chunk, on a chunk edge, on the
# first page; a member whose length equals the prefix; a one-member group without a prefix;
# a group with more (member, head) columns than one shared-prefix block holds.
def _prefix_groups(pl_pages=(40, 0, 96, 1), sizes=(5, 1, 40, 4)):
    starts = [0]
    for n in sizes:
        starts.append(starts[-1] + n)
    pl = [p * 16 for p in pl_pages]
    lens = []
    for gi, n in enumerate(sizes):
        for i in range(n):
            extra = [0, 60, 460, 1360, 1][i] if gi == 0 else (i * 37) % 900 + (i == 1)
            lens.append(max(pl[gi] + extra, 16 if gi == 3 else 0) + (300 if gi == 1 else 0))
    return starts, pl, lens


def _prefix_shape(name):
    import dataclasses
    if name == "bf16_d128":
        return dataclasses.replace(synth.B7, num_layers=2)
    if name == "fp8_d128":
        return dataclasses.replace(synth.LARGE_FP8, num_layers=2)
    if name == "bf16_d64":
        return synth.ModelShape(2, 1024, 16, 4, 64, 2048)
    if name == "fp8_d64":
        return synth.ModelShape(2, 1024, 16, 4, 64, 2048, kv_dtype="fp8")
    raise KeyError(name)


@pytest.mark.parametrize("name", ["bf16_d128", "fp8_d128", "bf16_d64", "fp8_d64"])
def test_attention_shared_prefix(name):
    shape = _prefix_shape(name)
    starts, pl, lens = _prefix_groups()
    _say(f"case: shared-prefix attention {name} groups={starts} prefix={pl} B={len(lens)}")
    w = synth.make_workload("custom", shape=shape, lengths=lens, seed=4343, groups=(starts, pl))
    dw = DeviceWorkload(w, nan_unused_pages=True, fill_weights=False)
    q, ks, vs = host_activations(w, 0xBCD, scale=1.0)
    layer = 1
    o_hint = run_attention(dw, layer, q, ks, vs, with_hint=True)
    o_none = run_attention(dw, layer, q, ks, vs, with_hint=False)
    cache = oin.cache_from_synth(w)
    ref = ko.attention_layer(shape, cache, layer, w.lengths, w.page_table, q.astype(np.float64),
                             ks.astype(np.float64), vs.astype(np.float64))
    assert np.all(np.isfinite(o_hint))
    scale = max(1.0, float(np.max(np.abs(ref))))
    e_hint, e_none = np.max(np.abs(o_hint - ref)), np.max(np.abs(o_none - ref))
    _say(f"  max|do| hint {e_hint:.3e}, no hint {e_none:.3e}")
    assert e_hint <= 2e-5 * scale and e_none <= 2e-5 * scale


def test_score_shared_prefix_bf16():
    import dataclasses
    shape = dataclasses.replace(synth.B7, num_layers=2)
    starts, pl, lens = _prefix_groups(pl_pages=(64, 0, 33), sizes=(3, 1, 20))
    _say(f"case: shared-prefix score groups={starts} prefix={pl}")
    w = synth.make_workload("custom", shape=shape, lengths=lens, seed=4344, groups=(starts, pl))
    p, z = _parity(w, 2e-3, 2e-2, with_hint=True)
    p2, z2 = run_score(DeviceWorkload(w, nan_unused_pages=True), with_hint=False)
    _say(f"  hint vs no hint: max|dz| = {np.max(np.abs(z - z2)):.3e}")
    assert np.max(np.abs(z - z2)) <= 1e-3


def _parity(w, tol_p, tol_z, **kw):
    dw = DeviceWorkload(w, nan_unused_pages=True)
    p, z = run_score(dw, **kw)
    zr, pr = oin.score_workload(w)
    dp, dz = np.max(np.abs(p - pr)), np.max(np.abs(z - zr))
    _say(f"  max|dP| = {dp:.3e}  max|dz| = {dz:.3e}  P = {np.round(p, 4)}")
    assert np.all(np.isfinite(p)) and np.all(np.isfinite(z))
    assert dp <= tol_p and dz <= tol_z
    return p, z


def test_score_parity_tiny_fp32():
    _say("case: score tiny_fp32 (B=4, L=512)")
    _parity(synth.make_workload("tiny_fp32"), 1e-5, 4e-5)


def test_score_parity_tiny_ragged_and_empty():
    _say("case: score tiny ragged lengths incl. 0")
    w = synth.make_workload("custom", shape=synth.TINY, lengths=[0, 1, 15, 16, 17, 511, 2000],
                            seed=77)
    _parity(w, 1e-5, 4e-5)


def test_score_parity_tiny_spiky_keys():
    _say("case: score tiny, K scaled x30 (peaked softmax)")
    w = synth.make_workload("custom", shape=synth.TINY, lengths=[300, 64, 129], seed=78,
                            k_std=30.0)
    _parity(w, 1e-5, 4e-5)


@pytest.mark.parametrize("kv_dtype,fp8_scale", [("bf16", None), ("fp8", "amax"), ("fp8", "pow2")])
def test_score_parity_two_layers_cache_dtypes(kv_dtype, fp8_scale):
    """Whole scoring pass over bf16 and e4m3 caches (scales amax / 448, or powers of two)."""
    _say(f"case: score 7B shape, 2 layers, {kv_dtype} cache {fp8_scale or ''}")
    import dataclasses
    shape = dataclasses.replace(synth.B7, num_layers=2, kv_dtype=kv_dtype)
    w = synth.make_workload("custom", shape=shape, lengths=[4100, 0, 17, 3001, 1200], seed=85,
                            fp8_scale=fp8_scale or "amax")
    _parity(w, 2e-3, 2e-2)


def test_score_long_peaked_softmax_moves_z():
    """L ~ 32k over 2 layers of the 7B shape with K scaled x30: one cached key dominates each
    head's softmax, so the attention output is an O(1) cached value row and the cache moves z by
    more than 1 (against the same model with an empty cache): a wrong page, chunk or merge at
    long L would show far above the |dz| bar, which is held at 2e-2 here too."""
    import dataclasses
    shape = dataclasses.replace(synth.B7, num_layers=2)
    lens = [32768, 30001, 16385]
    _say(f"case: score long peaked softmax lengths={lens}")
    w = synth.make_workload("custom", shape=shape, lengths=lens, seed=4601, k_std=30.0)
    p, z = _parity(w, 2e-3, 2e-2)
    z_empty, _ = oin.score_workload(
        synth.make_workload("custom", shape=shape, lengths=[0] * len(lens), seed=4601))
    zr, _ = oin.score_workload(w)
    _say(f"  oracle z {np.round(zr, 4)}; with an empty cache {np.round(z_empty, 4)}")
    assert np.max(np.abs(zr - z_empty)) > 1.0
    assert np.ptp(zr) > 0.5


def test_score_parity_7b_two_layers_bf16():
    _say("case: score 7B shape, 2 layers, bf16, ragged")
    import dataclasses
    shape = dataclasses.replace(synth.B7, num_layers=2)
    w = synth.make_workload("custom", shape=shape, lengths=[4096, 0, 17, 3001, 1200], seed=79)
    _parity(w, 2e-3, 2e-2)


@pytest.mark.parametrize("B", [9, 17, 40, 64])
def test_score_parity_batch_sizes_bf16(B):
    """One, two, four, six and eight operand column tiles (per-wave and shared-operand kernels)."""
    _say(f"case: score 7B shape, 2 layers, bf16, B={B}")
    import dataclasses
    shape = dataclasses.replace(synth.B7, num_layers=2)
    lengths = [(37 * i * i + 11 * i) % 700 for i in range(B)]
    w = synth.make_workload("custom", shape=shape, lengths=lengths, seed=90 + B)
    _parity(w, 2e-3, 2e-2)


def test_score_deterministic_and_batch_zero():
    _say("case: determinism + B=0")
    w = synth.make_workload("custom", shape=synth.TINY, lengths=[100, 513, 7], seed=80)
    dw = DeviceWorkload(w)
    a = run_score(dw)
    b = run_score(dw)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    m = kv()
    h = m.kvprm_create(dw.desc(m))
    try:
        empty = m.make_batch(0, 0, 1, 0)
        assert m.kvprm_workspace_size(h, empty) == 0
        m.kvprm_score(h, dw.cache(m), empty, dw.readout(m), 0, 0, 0, 0, 0)
    finally:
        m.kvprm_destroy(h)


def test_cache_and_weights_unchanged():
    _say("case: inputs are read-only")
    w = synth.make_workload("custom", shape=synth.TINY, lengths=[100, 37], seed=81)
    dw = DeviceWorkload(w)
    kc, vc = dw.k_pool.clone(), dw.v_pool.clone()
    wq = dw.layers[0]["wq"].clone()
    run_score(dw)
    assert torch.equal(kc, dw.k_pool) and torch.equal(vc, dw.v_pool)
    assert torch.equal(wq, dw.layers[0]["wq"])


def test_pack_weight_roundtrip():
    _say("case: kvprm_pack_weight")
    rows, K = 4608, 3584
    raw = synth.host_normal(rows * K, 5, 77, 0, 0.0, 0.02, synth.DT_BF16)
    src = torch.from_numpy(raw.view(np.int16)).cuda()
    dst = torch.empty_like(src)
    kv().kvprm_pack_weight(src.data_ptr(), dst.data_ptr(), rows, K,
                           torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    back = ko.unpack_tiled(dst.cpu().numpy().view(np.uint16), rows, K)
    assert np.array_equal(back, raw.reshape(rows, K))


def test_debug_mode_rejects_out_of_range_page_ids():
    _say("case: KVPRM_DEBUG page-table check")
    import os
    w = synth.make_workload("custom", shape=synth.TINY, lengths=[100, 37, 0], seed=82)
    dw = DeviceWorkload(w)
    m = kv()
    old = os.environ.get("KVPRM_DEBUG")
    os.environ["KVPRM_DEBUG"] = "1"
    try:
        h = m.kvprm_create(dw.desc(m))
    finally:
        if old is None:
            del os.environ["KVPRM_DEBUG"]
        else:
            os.environ["KVPRM_DEBUG"] = old
    try:
        batch = dw.batch(m)
        n = m.kvprm_workspace_size(h, batch)
        ws = torch.empty(max(n, 256), dtype=torch.uint8, device="cuda")
        scores = torch.empty(w.batch, dtype=torch.float32, device="cuda")
        st = torch.cuda.current_stream().cuda_stream
        # valid call in debug mode: same scores as without it
        m.kvprm_score(h, dw.cache(m), batch, dw.readout(m), ws.data_ptr(), n, scores.data_ptr(), 0,
                      st)
        torch.cuda.synchronize()
        ref, _ = run_score(dw)
        assert np.array_equal(scores.cpu().numpy().astype(np.float64), ref)
        # the library is told the pool is one page smaller; a row naming that (allocated) page
        # must be rejected on the host, before anything is enqueued
        cache = m.make_cache(dw.k_pool.data_ptr(), dw.v_pool.data_ptr(), w.num_pages - 1)
        bad = dw.page_table.clone()
        bad[1, 0] = w.num_pages - 1
        bb = m.make_batch(w.batch, bad.data_ptr(), w.max_pages, dw.lengths.data_ptr(), w.lengths)
        with pytest.raises(m.KvprmError) as e:
            m.kvprm_score(h, cache, bb, dw.readout(m), ws.data_ptr(), n, scores.data_ptr(), 0, st)
        assert e.value.status == m.KVPRM_E_INVALID and "page_table" in m.kvprm_last_error()
    finally:
        m.kvprm_destroy(h)


@pytest.mark.parametrize("name,lengths", [("b7_bf16", [32768, 1, 20000, 33, 5000, 31000]),
                                          ("b7_bf16", [4096, 0, 17, 3001, 1200]),
                                          ("fp8", [9000, 0, 17000, 31])])
def test_score_without_host_lengths(name, lengths):
    """lengths_host = NULL: the attention chunk grid is sized from max_pages (every chunk any
    device length could need) and the chunk length from batch x max_pages; the scores match the
    oracle as with the host lengths (the two differ only in summation order)."""
    _say(f"case: score without lengths_host {name} lengths={lengths}")
    w = synth.make_workload("custom", shape=_shape(name), lengths=lengths, seed=4545)
    dw = DeviceWorkload(w, nan_unused_pages=True)
    p0, z0 = run_score(dw, lengths_host=False)
    p1, z1 = run_score(dw)
    zr, pr = oin.score_workload(w)
    _say(f"  no host lengths: max|dP| = {np.max(np.abs(p0 - pr)):.3e} max|dz| = "
         f"{np.max(np.abs(z0 - zr)):.3e}; with: max|dz| = {np.max(np.abs(z1 - zr)):.3e}")
    assert np.all(np.isfinite(p0)) and np.all(np.isfinite(z0))
    assert np.max(np.abs(p0 - pr)) <= 2e-3 and np.max(np.abs(z0 - zr)) <= 2e-2
    assert np.max(np.abs(z0 - z1)) <= 1e-3


def _debug_handle(m, desc):
    import os
    old = os.environ.get("KVPRM_DEBUG")
    os.environ["KVPRM_DEBUG"] = "1"
    try:
        return m.kvprm_create(desc)
    finally:
        if old is None:
            del os.environ["KVPRM_DEBUG"]
        else:
            os.environ["KVPRM_DEBUG"] = old


def test_debug_mode_rejects_stale_host_lengths():
    _say("case: KVPRM_DEBUG lengths_host check")
    w = synth.make_workload("custom", shape=synth.TINY, lengths=[100, 37, 0], seed=83)
    dw = DeviceWorkload(w)
    m = kv()
    h = _debug_handle(m, dw.desc(m))
    try:
        n = m.kvprm_workspace_size(h, dw.batch(m))
        ws = torch.empty(max(n, 256), dtype=torch.uint8, device="cuda")
        scores = torch.empty(w.batch, dtype=torch.float32, device="cuda")
        st = torch.cuda.current_stream().cuda_stream
        stale = m.make_batch(w.batch, dw.page_table.data_ptr(), w.max_pages, dw.lengths.data_ptr(),
                             [100, 36, 0])
        with pytest.raises(m.KvprmError) as e:
            m.kvprm_score(h, dw.cache(m), stale, dw.readout(m), ws.data_ptr(), n,
                          scores.data_ptr(), 0, st)
        assert e.value.status == m.KVPRM_E_INVALID and "lengths_host" in m.kvprm_last_error()
        # without the mirror the same call is valid
        m.kvprm_score(h, dw.cache(m), dw.batch(m, lengths_host=False), dw.readout(m),
                      ws.data_ptr(), n, scores.data_ptr(), 0, st)
        torch.cuda.synchronize()
        assert np.all(np.isfinite(scores.cpu().numpy()))
    finally:
        m.kvprm_destroy(h)


def test_debug_mode_rejects_shared_pages_in_steering():
    """kvprm_score_grad / kvprm_steer write per-page results: a physical page read by two
    candidates is refused in the debug mode before anything is enqueued (the cache unchanged)."""
    _say("case: KVPRM_DEBUG shared pages in steering")
    shape = synth.ModelShape(2, 1024, 16, 4, 64, 2048)
    w = synth.make_workload("custom", shape=shape, lengths=[64, 40], seed=84)
    dw = DeviceWorkload(w)
    m = kv()
    h = _debug_handle(m, dw.desc(m))
    try:
        shared = dw.page_table.clone()
        shared[1, 0] = shared[0, 1]
        b = m.make_batch(w.batch, shared.data_ptr(), w.max_pages, dw.lengths.data_ptr(), w.lengths)
        n = m.kvprm_workspace_size_grad(h, b)
        ws = torch.empty(n, dtype=torch.uint8, device="cuda")
        p0 = torch.empty(w.batch, dtype=torch.float32, device="cuda")
        p1 = torch.empty_like(p0)
        kc, vc = dw.k_pool.clone(), dw.v_pool.clone()
        st = torch.cuda.current_stream().cuda_stream
        with pytest.raises(m.KvprmError) as e:
            m.kvprm_steer(h, dw.cache(m), b, dw.readout(m), 1.0, 1, ws.data_ptr(), n,
                          p0.data_ptr(), p1.data_ptr(), st)
        assert e.value.status == m.KVPRM_E_INVALID and "read by candidates" in m.kvprm_last_error()
        torch.cuda.synchronize()
        assert torch.equal(kc, dw.k_pool) and torch.equal(vc, dw.v_pool)
    finally:
        m.kvprm_destroy(h)


@pytest.mark.parametrize("nwords", [4, 4 * 1000003, 16 << 20])
def test_stream_read_touches_every_word_once(nwords):
    """The streaming-read diagnostic XORs every 32-bit word of the buffer into its sink: the
    result equals the host's XOR of the buffer, so every word was read exactly once (a word read
    twice or skipped changes the XOR unless it is zero, which the seeded values rule out), and a
    second call restores the sink."""
    _say(f"case: stream read, {nwords} words")
    g = np.random.default_rng(77 + nwords)
    host = g.integers(1, 2**32, size=nwords, dtype=np.uint64).astype(np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).cuda()
    x = int(np.bitwise_xor.reduce(host))
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    kv().kvprm_stream_read(buf.data_ptr(), nwords * 4, sink.data_ptr(), st)
    torch.cuda.synchronize()
    assert int(sink.cpu().numpy().view(np.uint32)[0]) == x
    kv().kvprm_stream_read(buf.data_ptr(), nwords * 4, sink.data_ptr(), st)
    torch.cuda.synchronize()
    assert int(sink.cpu().numpy().view(np.uint32)[0]) == 0
