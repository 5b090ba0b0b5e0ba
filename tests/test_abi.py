"""C ABI of libkvprm on the CPU: the library loads, exports every declared entry point, and
rejects bad arguments with the documented status before touching the GPU."""
import ctypes
import os
import re

import pytest

import paper_2607_09153_amd as kv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "kvprm.h")).read()
    return sorted(set(re.findall(r"\b(kvprm_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = _declared()
    assert set(names) == set(kv.EXPORTED)
    lib = ctypes.CDLL(kv.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def _desc(**over):
    d = dict(num_layers=2, hidden=256, num_q_heads=4, num_kv_heads=2, head_dim=64, ffn_dim=1024,
             weight_dtype="f32", kv_dtype="f32")
    d.update(over)
    return kv.make_desc(**d)


@pytest.mark.parametrize("over,status", [
    (dict(head_dim=96), kv.KVPRM_E_UNSUPPORTED),
    (dict(page_size=32), kv.KVPRM_E_UNSUPPORTED),
    (dict(num_q_heads=5), kv.KVPRM_E_INVALID),
    (dict(hidden=0), kv.KVPRM_E_INVALID),
    (dict(hidden=250), kv.KVPRM_E_UNSUPPORTED),
    (dict(weight_dtype="f32", kv_dtype="bf16"), kv.KVPRM_E_UNSUPPORTED),
    (dict(weight_dtype="bf16", kv_dtype="f32"), kv.KVPRM_E_UNSUPPORTED),
    (dict(num_q_heads=34, num_kv_heads=2), kv.KVPRM_E_UNSUPPORTED),
])
def test_create_rejects(over, status):
    with pytest.raises(kv.KvprmError) as e:
        kv.kvprm_create(_desc(**over))
    assert e.value.status == status
    assert kv.kvprm_last_error()


def test_create_accepts_supported_shapes():
    for over in ({}, dict(weight_dtype="bf16", kv_dtype="bf16", head_dim=128, num_q_heads=28,
                          num_kv_heads=4, hidden=3584, ffn_dim=18944),
                 dict(weight_dtype="bf16", kv_dtype="fp8", head_dim=128)):
        h = kv.kvprm_create(_desc(**over))
        kv.kvprm_destroy(h)
    kv.kvprm_destroy(None)


FAKE = 0x10000  # never dereferenced: validation fails before anything is enqueued


def _cache(**o):
    c = dict(k_ptr=FAKE, v_ptr=FAKE, num_pages=4)
    c.update(o)
    return kv.make_cache(**c)


def _weights(nl=2, null_layer=None):
    layers = []
    for l in range(nl):
        d = {n: FAKE for n, _ in kv.LayerWeights._fields_}
        if l == null_layer:
            d["w_up"] = 0
        layers.append(d)
    return kv.make_readout(layers, FAKE, FAKE, FAKE)


def _score(h, batch, cache=None, weights=None, ws=FAKE, ws_bytes=1 << 40, scores=FAKE):
    kv.kvprm_score(h, cache or _cache(), batch, weights or _weights(), ws, ws_bytes, scores, 0, 0)


@pytest.fixture
def handle():
    h = kv.kvprm_create(_desc())
    yield h
    kv.kvprm_destroy(h)


def test_score_validation_errors(handle):
    h = handle
    ok_batch = kv.make_batch(2, FAKE, 4, FAKE, [10, 64])
    cases = [
        (kv.make_batch(-1, FAKE, 4, FAKE), {}, kv.KVPRM_E_INVALID),
        (kv.make_batch(2, 0, 4, FAKE), {}, kv.KVPRM_E_INVALID),
        (kv.make_batch(2, FAKE, 0, FAKE), {}, kv.KVPRM_E_INVALID),
        (kv.make_batch(2, FAKE, 4, FAKE, [10, 65]), {}, kv.KVPRM_E_INVALID),
        (kv.make_batch(2, FAKE, 4, FAKE, [10, -1]), {}, kv.KVPRM_E_INVALID),
        (kv.make_batch(300, FAKE, 4, FAKE), {}, kv.KVPRM_E_UNSUPPORTED),
        (kv.make_batch(2, FAKE, 4, FAKE, [32, 40], [0, 1], [16]), {}, kv.KVPRM_E_INVALID),
        (kv.make_batch(2, FAKE, 4, FAKE, [32, 40], [0, 2], [8]), {}, kv.KVPRM_E_INVALID),
        (kv.make_batch(2, FAKE, 4, FAKE, [16, 40], [0, 2], [32]), {}, kv.KVPRM_E_INVALID),
        (kv.make_batch(2, FAKE, 4, FAKE, None, [0, 2], [16]), {}, kv.KVPRM_E_INVALID),
        (kv.make_batch(2, FAKE, 4, FAKE, [32, 40], [0, 1, 1, 2], [16, 0, 16]), {},
         kv.KVPRM_E_INVALID),
        (ok_batch, dict(cache=_cache(k_ptr=0)), kv.KVPRM_E_INVALID),
        (ok_batch, dict(cache=_cache(num_pages=0)), kv.KVPRM_E_INVALID),
        (ok_batch, dict(weights=_weights(null_layer=1)), kv.KVPRM_E_INVALID),
        (ok_batch, dict(scores=0), kv.KVPRM_E_INVALID),
        (ok_batch, dict(ws=0), kv.KVPRM_E_WORKSPACE),
        (ok_batch, dict(ws_bytes=1000), kv.KVPRM_E_WORKSPACE),
        (ok_batch, dict(ws=FAKE + 8), kv.KVPRM_E_WORKSPACE),
    ]
    for batch, kw, status in cases:
        with pytest.raises(kv.KvprmError) as e:
            _score(h, batch, **kw)
        assert e.value.status == status, (kw, kv.kvprm_last_error())


def test_fp8_cache_needs_scales():
    h = kv.kvprm_create(_desc(weight_dtype="bf16", kv_dtype="fp8"))
    try:
        with pytest.raises(kv.KvprmError) as e:
            _score(h, kv.make_batch(1, FAKE, 4, FAKE), cache=_cache())
        assert e.value.status == kv.KVPRM_E_INVALID and "scale" in kv.kvprm_last_error()
    finally:
        kv.kvprm_destroy(h)


def test_batch_zero_is_noop_and_workspace_sizes(handle):
    _score(handle, kv.make_batch(0, 0, 1, 0), ws=0, ws_bytes=0, scores=0)
    assert kv.kvprm_workspace_size(handle, kv.make_batch(0, 0, 1, 0)) == 0
    a = kv.kvprm_workspace_size(handle, kv.make_batch(4, FAKE, 32, FAKE))
    b = kv.kvprm_workspace_size(handle, kv.make_batch(4, FAKE, 64, FAKE))
    c = kv.kvprm_workspace_size(handle, kv.make_batch(8, FAKE, 64, FAKE))
    assert 0 < a <= b < c


def test_attention_validation(handle):
    batch = kv.make_batch(1, FAKE, 4, FAKE)
    with pytest.raises(kv.KvprmError) as e:
        kv.kvprm_attention(handle, _cache(), batch, 2, FAKE, FAKE, FAKE, FAKE, 1 << 40, FAKE)
    assert e.value.status == kv.KVPRM_E_INVALID
    with pytest.raises(kv.KvprmError) as e:
        kv.kvprm_attention(handle, _cache(), batch, 0, 0, FAKE, FAKE, FAKE, 1 << 40, FAKE)
    assert e.value.status == kv.KVPRM_E_INVALID


def test_attention_partials_validation(handle):
    batch = kv.make_batch(1, FAKE, 4, FAKE)
    cases = [dict(layer=2), dict(q=0), dict(ws=0), dict(ws_bytes=16), dict(cache=_cache(k_ptr=0))]
    for c in cases:
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_attention_partials(handle, c.get("cache", _cache()), batch, c.get("layer", 0),
                                        c.get("q", FAKE), c.get("ws", FAKE),
                                        c.get("ws_bytes", 1 << 40))
        assert e.value.status in (kv.KVPRM_E_INVALID, kv.KVPRM_E_WORKSPACE), c
    kv.kvprm_attention_partials(handle, _cache(), kv.make_batch(0, 0, 1, 0), 0, FAKE, FAKE, 0)


def test_pack_weight_validation():
    for args in [(0, FAKE, 16, 32), (FAKE, 0, 16, 32), (FAKE, FAKE * 4, 15, 32),
                 (FAKE, FAKE * 4, 16, 48), (FAKE, FAKE * 4, 0, 32), (FAKE, FAKE + 64, 16, 32),
                 (FAKE + 8, FAKE * 4, 16, 32)]:
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_pack_weight(*args)
        assert e.value.status == kv.KVPRM_E_INVALID


def test_stream_read_validation():
    for args in [(0, 1024, FAKE), (FAKE, 1024, 0), (FAKE, 0, FAKE), (FAKE, 1000, FAKE),
                 (FAKE + 8, 1024, FAKE), (FAKE, 1024, FAKE + 2)]:
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_stream_read(*args)
        assert e.value.status == kv.KVPRM_E_INVALID


def _lora(nl=2, rank=32, scale=1.0, drop=None, half=None):
    layers = []
    for l in range(nl):
        d = {p: (FAKE, FAKE) for p in kv.LORA_PROJECTIONS}
        if drop:
            del d[drop]
        if half and l == 1:
            d[half] = (FAKE, 0)
        layers.append(d)
    return kv.make_lora(layers, rank, scale)


def test_score_lora_validation():
    """Adapters need bf16 weights; the rank must be a multiple of 32 in [32, 512]; a factor
    pair is both set or both null; the workspace covers the adapter slots."""
    hf = kv.kvprm_create(_desc())
    try:
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_workspace_size_lora(hf, kv.make_batch(1, FAKE, 4, FAKE), 32)
        assert e.value.status == kv.KVPRM_E_UNSUPPORTED
    finally:
        kv.kvprm_destroy(hf)
    h = kv.kvprm_create(_desc(weight_dtype="bf16", kv_dtype="bf16"))
    try:
        batch = kv.make_batch(2, FAKE, 4, FAKE, [10, 64])
        base = kv.kvprm_workspace_size(h, batch)
        n = kv.kvprm_workspace_size_lora(h, batch, 64)
        assert n > base
        assert kv.kvprm_workspace_size_lora(h, batch, 512) > n
        assert kv.kvprm_workspace_size_lora(h, kv.make_batch(0, FAKE, 4, FAKE), 64) == 0
        cases = [
            (dict(lora=_lora(rank=48)), kv.KVPRM_E_INVALID),
            (dict(lora=_lora(rank=0)), kv.KVPRM_E_INVALID),
            (dict(lora=_lora(rank=544)), kv.KVPRM_E_INVALID),
            (dict(lora=_lora(half="up")), kv.KVPRM_E_INVALID),
            (dict(lora=_lora(scale=float("nan"))), kv.KVPRM_E_INVALID),
            (dict(ws_bytes=base), kv.KVPRM_E_WORKSPACE),
            (dict(weights=_weights(null_layer=0)), kv.KVPRM_E_INVALID),
            (dict(scores=0), kv.KVPRM_E_INVALID),
        ]
        for kw, status in cases:
            args = dict(lora=_lora(rank=64), ws_bytes=n, weights=_weights(), scores=FAKE)
            args.update(kw)
            with pytest.raises(kv.KvprmError) as e:
                kv.kvprm_score_lora(h, _cache(), batch, args["weights"], args["lora"], FAKE,
                                    args["ws_bytes"], args["scores"])
            assert e.value.status == status, (kw, kv.kvprm_last_error())
        # B = 0: nothing to check or enqueue
        kv.kvprm_score_lora(h, _cache(), kv.make_batch(0, FAKE, 4, FAKE), _weights(),
                            _lora(drop="q"), 0, 0, FAKE)
    finally:
        kv.kvprm_destroy(h)


def test_score_ex_validation():
    """Depth-k readout: depth >= 1; depth > 1 needs bf16 weights, depth x g <= 16 and
    batch x depth <= 64; the workspace grows with the rows; options NULL is kvprm_score."""
    hf = kv.kvprm_create(_desc())  # fp32 weights, g = 2
    try:
        batch = kv.make_batch(2, FAKE, 4, FAKE, [10, 64])
        assert (kv.kvprm_workspace_size_ex(hf, batch, None) ==
                kv.kvprm_workspace_size(hf, batch))
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_workspace_size_ex(hf, batch, kv.make_options(depth=2))
        assert e.value.status == kv.KVPRM_E_UNSUPPORTED
    finally:
        kv.kvprm_destroy(hf)
    h = kv.kvprm_create(_desc(weight_dtype="bf16", kv_dtype="bf16"))  # g = 2
    try:
        batch = kv.make_batch(2, FAKE, 4, FAKE, [10, 64])
        n1 = kv.kvprm_workspace_size_ex(h, batch, kv.make_options(depth=1))
        n8 = kv.kvprm_workspace_size_ex(h, batch, kv.make_options(depth=8))
        assert n8 > n1 == kv.kvprm_workspace_size(h, batch)
        nl = kv.kvprm_workspace_size_ex(h, batch, kv.make_options(_lora(rank=64), depth=4))
        assert nl > kv.kvprm_workspace_size_ex(h, batch, kv.make_options(depth=4))
        cases = [
            (kv.make_options(depth=0), batch, kv.KVPRM_E_INVALID),
            (kv.make_options(depth=9), batch, kv.KVPRM_E_UNSUPPORTED),  # 9 x 2 > 16 columns
            (kv.make_options(depth=8), kv.make_batch(9, FAKE, 4, FAKE), kv.KVPRM_E_UNSUPPORTED),
            (kv.make_options(_lora(rank=40), depth=2), batch, kv.KVPRM_E_INVALID),
        ]
        for opt, bt, status in cases:
            with pytest.raises(kv.KvprmError) as e:
                kv.kvprm_score_ex(h, _cache(), bt, _weights(), opt, FAKE, 1 << 40, FAKE)
            assert e.value.status == status, kv.kvprm_last_error()
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_score_ex(h, _cache(), batch, _weights(), kv.make_options(depth=8), FAKE, n1,
                              FAKE)
        assert e.value.status == kv.KVPRM_E_WORKSPACE
    finally:
        kv.kvprm_destroy(h)


def test_grad_and_steer_validation():
    """Cache gradients need bf16 weights and cache, at most 8 candidates and no shared pages."""
    hf = kv.kvprm_create(_desc())
    try:
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_workspace_size_grad(hf, kv.make_batch(1, FAKE, 4, FAKE))
        assert e.value.status == kv.KVPRM_E_UNSUPPORTED
    finally:
        kv.kvprm_destroy(hf)
    h8 = kv.kvprm_create(_desc(weight_dtype="bf16", kv_dtype="fp8"))
    try:
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_workspace_size_grad(h8, kv.make_batch(1, FAKE, 4, FAKE))
        assert e.value.status == kv.KVPRM_E_UNSUPPORTED
    finally:
        kv.kvprm_destroy(h8)
    hw = kv.kvprm_create(_desc(weight_dtype="bf16", kv_dtype="bf16", hidden=16448))
    try:  # the RMSNorm backward holds a candidate's hidden vector in one block's registers
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_workspace_size_grad(hw, kv.make_batch(1, FAKE, 4, FAKE))
        assert e.value.status == kv.KVPRM_E_UNSUPPORTED
    finally:
        kv.kvprm_destroy(hw)
    h = kv.kvprm_create(_desc(weight_dtype="bf16", kv_dtype="bf16"))
    try:
        batch = kv.make_batch(2, FAKE, 4, FAKE, [10, 64])
        n = kv.kvprm_workspace_size_grad(h, batch)
        assert n > kv.kvprm_workspace_size(h, batch)
        cases = [
            (kv.make_batch(9, FAKE, 4, FAKE), {}, kv.KVPRM_E_UNSUPPORTED),
            (kv.make_batch(2, FAKE, 4, FAKE, [32, 40], [0, 2], [16]), {}, kv.KVPRM_E_INVALID),
            (batch, dict(ws_bytes=n - 1), kv.KVPRM_E_WORKSPACE),
            (batch, dict(steps=0), kv.KVPRM_E_INVALID),
            (batch, dict(after=0), kv.KVPRM_E_INVALID),
        ]
        for bt, kw, status in cases:
            with pytest.raises(kv.KvprmError) as e:
                kv.kvprm_steer(h, _cache(), bt, _weights(), 0.1, kw.get("steps", 2), FAKE,
                               kw.get("ws_bytes", n), FAKE, kw.get("after", FAKE))
            assert e.value.status == status, kv.kvprm_last_error()
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_score_grad(h, _cache(), batch, _weights(), FAKE, n, FAKE, 0, FAKE)
        assert e.value.status == kv.KVPRM_E_INVALID
    finally:
        kv.kvprm_destroy(h)


def test_score_static_validates_on_the_host():
    """kvprm_score_static: B = 0 is a no-op; a batch whose workspace exceeds the static array is
    refused with KVPRM_E_WORKSPACE, and bad arguments with their status, before the device is
    touched."""
    h = kv.kvprm_create(_desc(weight_dtype="bf16", kv_dtype="bf16", head_dim=128, num_q_heads=28,
                              num_kv_heads=4, hidden=3584, ffn_dim=18944, num_layers=28))
    try:
        kv.kvprm_score_static(h, _cache(), kv.make_batch(0, 0, 1, 0), _weights(28), FAKE)
        big = kv.make_batch(64, FAKE, 1152, FAKE)
        assert kv.kvprm_workspace_size(h, big) > kv.STATIC_WORKSPACE_BYTES
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_score_static(h, _cache(), big, _weights(28), FAKE)
        assert e.value.status == kv.KVPRM_E_WORKSPACE and "static" in kv.kvprm_last_error()
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_score_static(h, _cache(), kv.make_batch(2, 0, 4, FAKE), _weights(28), FAKE)
        assert e.value.status == kv.KVPRM_E_INVALID
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_score_static(None, _cache(), big, _weights(28), FAKE)
        assert e.value.status == kv.KVPRM_E_INVALID
    finally:
        kv.kvprm_destroy(h)


def test_pack_kv_validates_on_the_host():
    kv.kvprm_pack_kv(0, 0, 0, 128, "bf16", kv.KVPRM_KEYS)  # nothing to do
    for args, status in [((FAKE, FAKE + (1 << 30), 4, 96, "bf16", kv.KVPRM_KEYS), kv.KVPRM_E_UNSUPPORTED),
                         ((FAKE, FAKE + 4096, 4, 128, "bf16", kv.KVPRM_VALUES), kv.KVPRM_E_INVALID),
                         ((FAKE + 8, FAKE + (1 << 30), 4, 128, "fp8", kv.KVPRM_KEYS), kv.KVPRM_E_INVALID),
                         ((FAKE, 0, 4, 64, "f32", kv.KVPRM_KEYS), kv.KVPRM_E_INVALID),
                         ((FAKE, FAKE + (1 << 30), 4, 64, "f32", 2), kv.KVPRM_E_INVALID),
                         ((FAKE, FAKE + (1 << 30), -1, 64, "f32", kv.KVPRM_KEYS), kv.KVPRM_E_INVALID)]:
        with pytest.raises(kv.KvprmError) as e:
            kv.kvprm_pack_kv(*args)
        assert e.value.status == status, args
