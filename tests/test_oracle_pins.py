"""Pins of the fp64 oracle against closed forms, invariants, library routines and brute
force (CPU only). Each test names the property it fixes; together they are chosen so that a
dropped term, a wrong sign or index, or a transposed operand in the oracle fails one of them.
"""
import math

import numpy as np
import pytest
import scipy.special
import torch

import synth
from oracle import kvprm_oracle as ko
from oracle import inputs

RNG = np.random.default_rng(1234)


# ------------------------------------------------------------------------ number formats


def test_e4m3_all_256_codes_against_torch():
    codes = np.arange(256, dtype=np.uint8)
    ours = ko.e4m3fn_to_f64(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert nan.sum() == 2  # 0x7F and 0xFF
    assert np.array_equal(ours[~nan], ref[~nan])
    assert ours[0x7E] == 448.0 and ours[0x01] == 2.0 ** -9 and ours[0x08] == 2.0 ** -6


def test_bf16_decode_against_torch():
    bits = np.arange(0, 65536, 7, dtype=np.uint32).astype(np.uint16)
    ours = ko.bf16_bits_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    fin = np.isfinite(ref)
    assert np.array_equal(ours[fin], ref[fin])


# ------------------------------------------------------------------------ attention


def test_attention_one_key_returns_its_value():
    for d in (4, 64, 128):
        q, k, v = RNG.normal(size=d) * 5, RNG.normal(size=(1, d)), RNG.normal(size=(1, d))
        assert np.allclose(ko.attention(q, k, v), v[0], rtol=0, atol=1e-14)


def test_attention_identical_keys_give_mean_of_values():
    d, n = 64, 37
    q = RNG.normal(size=d)
    K = np.tile(RNG.normal(size=d), (n, 1))
    V = RNG.normal(size=(n, d))
    assert np.allclose(ko.attention(q, K, V), V.mean(axis=0), rtol=0, atol=1e-14)
    # a zero query sees equal logits for any keys
    assert np.allclose(ko.attention(np.zeros(d), RNG.normal(size=(n, d)), V), V.mean(axis=0),
                       rtol=0, atol=1e-14)


def test_attention_two_keys_closed_form():
    """Keys along q with q.k1 - q.k2 = delta: weight of key 1 is sigmoid(delta / sqrt(d))."""
    d = 16
    q = RNG.normal(size=d)
    qq = q @ q
    a, b = 3.0, -1.5
    K = np.stack([a * q / qq, b * q / qq])
    V = RNG.normal(size=(2, d))
    w1 = scipy.special.expit((a - b) / math.sqrt(d))
    assert np.allclose(ko.attention(q, K, V), w1 * V[0] + (1 - w1) * V[1], rtol=0, atol=1e-14)


def test_attention_brute_force_against_torch_sdpa():
    d, n = 64, 300
    q = RNG.normal(size=d) * 2
    K, V = RNG.normal(size=(n, d)), RNG.normal(size=(n, d))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None, None, None, :], torch.from_numpy(K)[None, None],
        torch.from_numpy(V)[None, None]).numpy()[0, 0, 0]
    assert np.allclose(ko.attention(q, K, V), ref, rtol=0, atol=1e-13)


def test_attention_invariances():
    d, n = 32, 50
    q = RNG.normal(size=d)
    K, V = RNG.normal(size=(n, d)), RNG.normal(size=(n, d))
    o = ko.attention(q, K, V)
    perm = RNG.permutation(n)
    assert np.allclose(ko.attention(q, K[perm], V[perm]), o, rtol=0, atol=1e-14)
    # adding one vector w to every key shifts all logits by q.w / sqrt(d): no effect
    w = RNG.normal(size=d) * 10
    assert np.allclose(ko.attention(q, K + w, V), o, rtol=0, atol=1e-13)
    # huge logits stay finite (max subtraction)
    o2 = ko.attention(q * 1e4, K, V)
    assert np.all(np.isfinite(o2))
    s = K @ q
    assert np.allclose(o2, V[np.argmax(s)], atol=1e-12)


# ------------------------------------------------------------------------ rotary, norms, FFN


def test_rope_position_zero_is_identity_and_norm_preserving():
    y = RNG.normal(size=(3, 64))
    assert np.array_equal(ko.rope(y, 0, 1e6), y)
    r = ko.rope(y, 12345, 1e6)
    assert np.allclose(np.linalg.norm(r, axis=1), np.linalg.norm(y, axis=1), atol=1e-12)


def test_rope_relative_position():
    q, k = RNG.normal(size=(1, 128)), RNG.normal(size=(1, 128))
    for m, n, c in [(5, 3, 100), (30000, 17, 2345), (0, 4096, 7)]:
        a = ko.rope(q, m, 1e6) @ ko.rope(k, n, 1e6).T
        b = ko.rope(q, m + c, 1e6) @ ko.rope(k, n + c, 1e6).T
        assert np.allclose(a, b, rtol=0, atol=1e-10)


def test_rope_basis_vectors_closed_form():
    """e_i rotates in the (i, i + d/2) plane by pos * theta^(-2i/d)."""
    d, th, pos = 8, 1e6, 7
    for i in range(d // 2):
        e = np.zeros((1, d))
        e[0, i] = 1.0
        r = ko.rope(e, pos, th)[0]
        ang = pos * th ** (-2 * i / d)
        expect = np.zeros(d)
        expect[i], expect[i + d // 2] = math.cos(ang), math.sin(ang)
        assert np.allclose(r, expect, atol=1e-15)


def test_rope_matches_transformers_rotate_half():
    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb
    d, th = 64, 1e6
    pos = np.array([0, 1, 7, 300, 511])
    q = RNG.normal(size=(1, 2, len(pos), d))
    inv = 1.0 / th ** (np.arange(0, d, 2) / d)
    emb = np.concatenate([np.outer(pos, inv)] * 2, axis=-1)
    cos, sin = torch.from_numpy(np.cos(emb))[None], torch.from_numpy(np.sin(emb))[None]
    ref, _ = apply_rotary_pos_emb(torch.from_numpy(q), torch.from_numpy(q), cos, sin)
    for t, p in enumerate(pos):
        assert np.allclose(ko.rope(q[0, :, t], int(p), th), ref.numpy()[0, :, t], atol=1e-13)


def test_rmsnorm_scale_invariance_and_unit_rms():
    x = RNG.normal(size=(4, 256)) * 3
    g = np.ones(256)
    a = ko.rms_norm(x, g, 0.0)
    assert np.allclose(ko.rms_norm(x * 7.5, g, 0.0), a, atol=1e-14)
    assert np.allclose(np.mean(a * a, axis=1), 1.0, atol=1e-14)
    gam = RNG.normal(size=256)
    assert np.allclose(ko.rms_norm(x, gam, 0.0), a * gam, atol=1e-14)
    # eps enters under the root: x = c * ones gives c / sqrt(c^2 + eps)
    c, eps = 1e-3, 1e-6
    assert np.allclose(ko.rms_norm(np.full(8, c), np.ones(8), eps), c / math.sqrt(c * c + eps))


def test_swiglu_closed_form_and_orientation():
    # scalar case: w_d * silu(w_g u) * (w_u u), silu(a) = a * sigmoid(a)
    u, wg, wu, wd = 0.7, 1.3, -0.4, 2.0
    a = wg * u
    expect = wd * a * scipy.special.expit(a) * (wu * u)
    got = ko.swiglu_ffn(np.array([u]), np.array([[wg]]), np.array([[wu]]), np.array([[wd]]))
    assert np.allclose(got, expect, atol=1e-15)
    # matrix case against torch's silu with [out, in] weights (nn.Linear convention)
    H, F = 6, 10
    U = RNG.normal(size=H)
    Wg, Wu, Wd = RNG.normal(size=(F, H)), RNG.normal(size=(F, H)), RNG.normal(size=(H, F))
    t = lambda m: torch.from_numpy(m)
    ref = torch.nn.functional.linear(
        torch.nn.functional.silu(torch.nn.functional.linear(t(U), t(Wg))) *
        torch.nn.functional.linear(t(U), t(Wu)), t(Wd)).numpy()
    assert np.allclose(ko.swiglu_ffn(U, Wg, Wu, Wd), ref, atol=1e-13)


def test_two_logit_softmax_equals_sigmoid_head():
    zm = RNG.normal(size=1000) * 10
    zp = RNG.normal(size=1000) * 10
    ref = scipy.special.softmax(np.stack([zm, zp], axis=1), axis=1)[:, 1]
    assert np.allclose(ko.judgment_probability(zm, zp), ref, rtol=0, atol=1e-15)
    assert np.allclose(ko.sigmoid(zp - zm), ref, rtol=0, atol=1e-15)
    big = np.array([-800.0, -40.0, 0.0, 40.0, 800.0])
    assert np.allclose(ko.sigmoid(big), scipy.special.expit(big), rtol=1e-15, atol=0)


# ------------------------------------------------------------------------ cache layout


def test_cache_tile_layouts():
    ps, d = 16, 128
    tok = np.arange(ps * d).reshape(ps, d)  # value = slot * d + dim
    for eb in (4, 2, 1):
        x = 16 // eb
        stored = np.empty(ps * d, dtype=np.int64)
        for s in range(ps):
            for m in range(d):
                stored[((m // x) * ps + s) * x + m % x] = tok[s, m]
        assert np.array_equal(ko.k_tile_to_tokens(stored, ps, d, eb), tok)
    for eb in (4, 2, 1):
        r = 16 // eb // 4
        stored_v = np.empty(ps * d, dtype=np.int64)
        for s in range(ps):
            for m in range(d):
                idx = ((((m // (16 * r)) * 4 + s // 4) * 16 + m % 16) * r + (m // 16) % r) * 4 + s % 4
                stored_v[idx] = tok[s, m]
        assert np.array_equal(ko.v_tile_to_tokens(stored_v, ps, d, eb), tok)


# ------------------------------------------------------------------------ model-level pins

TINY = synth.TINY


def _tiny_small(layers=2, **kw):
    return synth.ModelShape(layers, 64, 4, 2, 16, 96, weight_dtype="f32", kv_dtype="f32", **kw)


def _dense_cache(K, V, ps):
    """Paged cache over dense per-candidate K/V ([B][n_kv... as [L][n_kv][n][d]]), pages
    laid out in logical order, physical ids given by page tables built here."""
    B = len(K)
    tiles = {}
    page_table = []
    nxt = 0
    for b in range(B):
        NL, nkv, n, d = K[b].shape
        npg = -(-n // ps)
        row = []
        for i in range(npg):
            phys = 1000 + 3 * nxt  # arbitrary physical ids
            nxt += 1
            row.append(phys)
            for l in range(NL):
                kt = np.full((nkv, ps, d), np.nan)
                vt = np.full((nkv, ps, d), np.nan)
                cnt = min(ps, n - i * ps)
                kt[:, :cnt] = K[b][l][:, i * ps: i * ps + cnt]
                vt[:, :cnt] = V[b][l][:, i * ps: i * ps + cnt]
                tiles[(l, "k", phys)] = kt
                tiles[(l, "v", phys)] = vt
        page_table.append(row)
    return ko.PagedCache(lambda l, w, p: tiles[(l, w, p)]), page_table


def _readout(shape, seed):
    return inputs.readout_from_synth(shape, seed, layer_cache=64)


def _embed(shape, seed, vocab=1000):
    return synth.host_normal(vocab * shape.hidden, seed, synth.stream_id(synth.GLOBAL,
                             synth.G_EMBED_TABLE)).reshape(vocab, shape.hidden)


@pytest.mark.parametrize("mixed", [False, True])
def test_verify_pass_equals_causal_reencode(mixed):
    """Re-encode equivalence: the verify pass over the cache a causal forward wrote equals
    that forward's last position; with mixed=True the verify token alone uses other weights
    (adapter on for the verify token only)."""
    shape = _tiny_small()
    seed = 77
    base = _readout(shape, seed)
    ver = _readout(shape, seed + synth.ADAPTER_SEED_OFFSET) if mixed else base
    E = _embed(shape, seed)
    Ks, Vs, zs, hs, lens = [], [], [], [], []
    for b, n in enumerate([40, 16, 1, 23]):
        toks = synth.token_ids(seed + b, n)
        z, p, h, K, V = ko.reencode(shape, base.layer, ver.layer, E, toks, ver.verify_embed,
                                    ver.final_norm, ver.reward_w)
        Ks.append(K), Vs.append(V), zs.append(z), hs.append(h), lens.append(n)
    cache, pt = _dense_cache(Ks, Vs, shape.page_size)
    z2, p2, h2 = ko.verify_pass(shape, ver, cache, lens, pt, return_hidden=True)
    assert np.allclose(z2, zs, rtol=0, atol=1e-12)
    assert np.allclose(h2, np.stack(hs), rtol=0, atol=1e-12)
    assert np.allclose(p2, ko.sigmoid(np.array(zs)), rtol=0, atol=1e-12)


@pytest.mark.parametrize("mixed", [False, True])
def test_tiny_reencode_mode_at_full_length(mixed):
    """The tiny workload's re-encode mode at its own size (2 layers, H = 256, 4/2 heads, d_h 64,
    FFN 1024, fp32): four sequences of 512 token ids from the 1000-word vocabulary, verify id
    999, written causally (section 5.1, the Text-PRM re-encode of [x; v]); the verify pass over
    the cache that pass wrote equals its last position. mixed: the verify token alone runs
    other weights (adapter on the verify token only, section 4.1)."""
    shape = synth.TINY
    lens = [512] * 4
    r = inputs.reencode_batch(shape, 1000, lens, mixed=mixed)
    cache, pt = _dense_cache(r["K"], r["V"], shape.page_size)
    ver = r["verify"]
    ro = ko.Readout(ver.layer, r["verify_embed"], ver.final_norm, ver.reward_w, ver.reward_b)
    z2, p2 = ko.verify_pass(shape, ro, cache, lens, pt)
    assert np.allclose(z2, r["z"], rtol=0, atol=1e-12)
    assert np.allclose(p2, r["p"], rtol=0, atol=1e-12)
    assert np.ptp(r["z"]) > 1e-3  # the four sequences score differently


def test_empty_cache_is_one_token_forward():
    shape = _tiny_small()
    ro = _readout(shape, 5)
    E = _embed(shape, 5)
    z, p, h, _, _ = ko.reencode(shape, ro.layer, ro.layer, E, [], ro.verify_embed, ro.final_norm,
                                ro.reward_w)
    cache = ko.PagedCache(lambda l, w, pg: (_ for _ in ()).throw(AssertionError("read")))
    z2, p2 = ko.verify_pass(shape, ro, cache, [0], [[-1]])
    assert abs(z2[0] - z) < 1e-14


def test_gqa_equals_mha_with_replicated_kv_heads():
    """n_kv = 2, g = 2 equals n_kv = 4 (MHA) with each kv-head's projection rows and cache
    replicated for its g query heads."""
    shape = _tiny_small(layers=1)
    ro = _readout(shape, 9)
    d, nkv, g = shape.head_dim, shape.num_kv_heads, shape.group
    W = ro.layer(0)
    rep = lambda M: np.concatenate([M[(j // g) * d:(j // g + 1) * d] for j in range(nkv * g)])
    Wm = ko.LayerWeights(W.attn_norm, W.wq, rep(W.wk), rep(W.wv), W.wo, W.ffn_norm, W.w_gate,
                         W.w_up, W.w_down)
    mha = synth.ModelShape(1, 64, 4, 4, 16, 96, weight_dtype="f32", kv_dtype="f32")
    ro_m = ko.Readout(lambda l: Wm, ro.verify_embed, ro.final_norm, ro.reward_w)
    n = 37
    K = RNG.normal(size=(1, nkv, n, d))
    V = RNG.normal(size=(1, nkv, n, d))
    c1, pt1 = _dense_cache([K], [V], 16)
    c2, pt2 = _dense_cache([np.repeat(K, g, axis=1)], [np.repeat(V, g, axis=1)], 16)
    z1, _ = ko.verify_pass(shape, ro, c1, [n], pt1)
    z2, _ = ko.verify_pass(mha, ro_m, c2, [n], pt2)
    assert abs(z1[0] - z2[0]) < 1e-13


def test_page_permutation_nan_slots_and_candidate_independence():
    w = synth.make_workload("custom", shape=_tiny_small(), lengths=[0, 1, 15, 16, 17, 70],
                            seed=31)
    ro = _readout(w.shape, w.seed)
    base = inputs.cache_from_synth(w)
    ps = w.shape.page_size

    # NaN in every slot at or beyond each candidate's length, and in every unused page
    valid = {}
    for b, row in enumerate(w.page_table):
        L = w.lengths[b]
        for i in range(-(-L // ps)):
            valid[row[i]] = min(ps, L - i * ps)

    def poisoned(l, which, page):
        t = base.tiles(l, which, page).copy() if page in valid else np.full(
            (w.shape.num_kv_heads, ps, w.shape.head_dim), np.nan)
        if page in valid:
            t[:, valid[page]:] = np.nan
        return t

    z, p = ko.verify_pass(w.shape, ro, base, w.lengths, w.page_table)
    z_nan, _ = ko.verify_pass(w.shape, ro, ko.PagedCache(poisoned), w.lengths, w.page_table)
    assert np.all(np.isfinite(z_nan)) and np.array_equal(z, z_nan)

    # relabel physical pages
    perm = {pg: 5000 + 7 * i for i, pg in enumerate(sorted(valid))}
    inv = {v: k for k, v in perm.items()}
    relab = ko.PagedCache(lambda l, wh, pg: base.tiles(l, wh, inv[pg]))
    pt2 = [[perm.get(x, -1) for x in row] for row in w.page_table]
    z2, _ = ko.verify_pass(w.shape, ro, relab, w.lengths, pt2)
    assert np.array_equal(z, z2)

    # one candidate alone scores the same as inside the batch
    for b in (0, 3, 5):
        zb, _ = ko.verify_pass(w.shape, ro, base, [w.lengths[b]], [w.page_table[b]])
        assert abs(zb[0] - z[b]) < 1e-14  # BLAS blocking may differ with batch width


def test_cached_length_changes_the_score():
    """The cache is really read: dropping the last cached token changes z."""
    w = synth.make_workload("custom", shape=_tiny_small(), lengths=[33, 32], seed=4)
    ro = _readout(w.shape, w.seed)
    c = inputs.cache_from_synth(w)
    z, _ = ko.verify_pass(w.shape, ro, c, w.lengths, w.page_table)
    z2, _ = ko.verify_pass(w.shape, ro, c, [32], [w.page_table[0]])
    assert abs(z[0] - z2[0]) > 1e-6


# ------------------------------------------------------------------------ library decoder


def _hf_model(shape, ro, E):
    from transformers import LlamaConfig, LlamaForCausalLM
    cfg = LlamaConfig(hidden_size=shape.hidden, intermediate_size=shape.ffn_dim,
                      num_hidden_layers=shape.num_layers, num_attention_heads=shape.num_q_heads,
                      num_key_value_heads=shape.num_kv_heads, head_dim=shape.head_dim,
                      rms_norm_eps=shape.rms_eps, rope_theta=shape.rope_theta,
                      vocab_size=E.shape[0], attention_bias=False, mlp_bias=False,
                      tie_word_embeddings=False)
    cfg._attn_implementation = "eager"
    m = LlamaForCausalLM(cfg).to(torch.float64).eval()
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(E))
        for l, layer in enumerate(m.model.layers):
            W = ro.layer(l)
            layer.input_layernorm.weight.copy_(t(W.attn_norm))
            layer.self_attn.q_proj.weight.copy_(t(W.wq))
            layer.self_attn.k_proj.weight.copy_(t(W.wk))
            layer.self_attn.v_proj.weight.copy_(t(W.wv))
            layer.self_attn.o_proj.weight.copy_(t(W.wo))
            layer.post_attention_layernorm.weight.copy_(t(W.ffn_norm))
            layer.mlp.gate_proj.weight.copy_(t(W.w_gate))
            layer.mlp.up_proj.weight.copy_(t(W.w_up))
            layer.mlp.down_proj.weight.copy_(t(W.w_down))
        m.model.norm.weight.copy_(t(ro.final_norm))
        # two judgment rows: "+" = reward vector, "-" = zero
        m.lm_head.weight.zero_()
        m.lm_head.weight[1].copy_(t(ro.reward_w))
    return m


@pytest.mark.parametrize("mixed", [False, True])
def test_verify_pass_against_transformers_llama_with_kv_cache(mixed):
    """A library decoder (transformers' Llama block: pre-norm RMSNorm, rotate-half rotary,
    grouped-query attention, SwiGLU) encodes the trajectory with base weights, then runs the
    verify token against its own KV cache with the verify weights. The oracle's verify pass
    over that same cache must agree. The library computes norms, rotary angles and softmax in
    fp32, hence the 1e-5 tolerance."""
    shape = synth.ModelShape(2, 256, 4, 2, 64, 1024, weight_dtype="f32", kv_dtype="f32")
    seed = 1000
    base = _readout(shape, seed)
    ver = _readout(shape, seed + synth.ADAPTER_SEED_OFFSET) if mixed else base
    E = _embed(shape, seed).copy()
    vid = 999
    E_v = E.copy()
    E_v[vid] = ver.verify_embed
    mb = _hf_model(shape, base, E)
    mv = _hf_model(shape, ver, E_v)
    n = 48
    toks = torch.tensor([synth.token_ids(seed, n)])
    with torch.no_grad():
        out = mb(input_ids=toks, use_cache=True)
        pkv = out.past_key_values
        out2 = mv(input_ids=torch.tensor([[vid]]), past_key_values=pkv, use_cache=True,
                  output_hidden_states=True)
    h_ref = out2.hidden_states[-1][0, -1].numpy()
    z_ref = out2.logits[0, -1, 1].item() - out2.logits[0, -1, 0].item()
    # the cache the library wrote during the prefix pass: [layers][n_kv][n][d] after rotation
    Ks = np.stack([pkv.layers[l].keys[0, :, :n].numpy() for l in range(shape.num_layers)])
    Vs = np.stack([pkv.layers[l].values[0, :, :n].numpy() for l in range(shape.num_layers)])
    cache, pt = _dense_cache([Ks], [Vs], shape.page_size)
    z, p, h = ko.verify_pass(shape, ver, cache, [n], pt, return_hidden=True)
    assert np.max(np.abs(h[0] - h_ref)) < 1e-5
    assert abs(z[0] - z_ref) < 1e-5
    # and the full causal re-encode of [x; v] in the library equals the oracle's re-encode
    if not mixed:
        with torch.no_grad():
            full = mv(input_ids=torch.cat([toks, torch.tensor([[vid]])], dim=1),
                      output_hidden_states=True)
        zr, _, hr, _, _ = ko.reencode(shape, base.layer, base.layer, E, toks[0].tolist(),
                                      base.verify_embed, base.final_norm, base.reward_w)
        assert np.max(np.abs(hr - full.hidden_states[-1][0, -1].numpy())) < 1e-5


def test_packed_weight_layout():
    """Block kb * (rows/16) + t, group l, element i holds W[16 t + l % 16][32 kb + 8 (l // 16) + i]."""
    rows, K = 48, 96
    W = np.arange(rows * K).reshape(rows, K)
    stored = np.empty(rows * K, dtype=np.int64)
    for r in range(rows):
        for k in range(K):
            t, kb = r // 16, k // 32
            l = (r % 16) + 16 * ((k % 32) // 8)
            stored[((kb * (rows // 16) + t) * 64 + l) * 8 + k % 8] = W[r, k]
    assert np.array_equal(ko.unpack_tiled(stored, rows, K), W)


def test_split_lse_merge_equals_one_pass_softmax():
    """Any chunking of the keys, merged by log-sum-exp with the verify token's own key as a
    last one-element chunk, gives the one-pass attention of the oracle (the identity the
    split-L kernels rely on)."""
    d, n = 64, 333
    q = RNG.normal(size=d) * 3
    K, V = RNG.normal(size=(n + 1, d)), RNG.normal(size=(n + 1, d))
    ref = ko.attention(q, K, V)
    for cuts in ([0, n], [0, 16, 32, 300, n], sorted(set([0, n] + list(RNG.integers(1, n, 7))))):
        parts = []
        for a, b in zip(cuts[:-1], cuts[1:]):
            s = K[a:b] @ q / np.sqrt(d)
            m = s.max()
            e = np.exp(s - m)
            parts.append((m, e.sum(), e @ V[a:b]))
        s_self = K[n] @ q / np.sqrt(d)
        M = max([p[0] for p in parts] + [s_self])
        num = sum(np.exp(m - M) * acc for m, _, acc in parts) + np.exp(s_self - M) * V[n]
        den = sum(np.exp(m - M) * l for m, l, _ in parts) + np.exp(s_self - M)
        assert np.allclose(num / den, ref, rtol=0, atol=1e-13)


# ---------------------------------------------------------------------------------------------
# low-rank adapter of the verify token (Eq. (score): f_{theta + dtheta})


def _adapter(shape, seed, rank, targets=synth.LORA_PROJECTIONS):
    return inputs.lora_from_synth(shape, seed, rank, targets, layer_cache=64)


def _random_cache(shape, lengths, seed):
    """Paged cache of random K/V for the listed lengths (NaN past each length)."""
    rng = np.random.default_rng(seed)
    Ks = [rng.normal(size=(shape.num_layers, shape.num_kv_heads, n, shape.head_dim)) for n in lengths]
    Vs = [rng.normal(size=(shape.num_layers, shape.num_kv_heads, n, shape.head_dim)) for n in lengths]
    return _dense_cache(Ks, Vs, shape.page_size)


def test_adapter_with_zero_b_is_the_base_readout():
    """B = 0 leaves every projection unchanged: the adapted pass equals the base pass exactly."""
    shape = _tiny_small()
    base = _readout(shape, 31)
    fac = _adapter(shape, 31, 32)
    zero_b = lambda l: {p: (A, np.zeros_like(B)) for p, (A, B) in fac(l).items()}
    ro = ko.readout_with_adapter(base, zero_b, synth.lora_scale(32))
    cache, pt = _random_cache(shape, [37, 0, 16], 3)
    z0, _ = ko.verify_pass(shape, base, cache, [37, 0, 16], pt)
    z1, _ = ko.verify_pass(shape, ro, cache, [37, 0, 16], pt)
    assert np.array_equal(z0, z1)


@pytest.mark.parametrize("proj", synth.LORA_PROJECTIONS)
def test_rank_one_adapter_moves_one_weight(proj):
    """A = e_i^T (a row selector), B = c e_j: the update scale * B A is scale * c at entry
    (j, i) of the projection alone, so the adapted pass equals the base pass with that one
    weight changed (pins the product order B A, its orientation and the scale)."""
    shape = _tiny_small()
    base = _readout(shape, 41)
    W0 = base.layer(1)
    f = ko.LORA_FIELDS[proj]
    out, inn = getattr(W0, f).shape
    i, j, c, scale = inn - 3, out // 2 + 1, 0.75, 0.125
    A = np.zeros((1, inn))
    A[0, i] = 1.0
    B = np.zeros((out, 1))
    B[j, 0] = c
    ro = ko.readout_with_adapter(base, lambda l: {proj: (A, B)} if l == 1 else {}, scale)
    edited = {k: getattr(W0, k) for k in ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm",
                                           "w_gate", "w_up", "w_down")}
    M = edited[f].copy()
    M[j, i] += scale * c
    edited[f] = M
    W1 = ko.LayerWeights(**edited)
    ref = ko.Readout(lambda l: W1 if l == 1 else base.layer(l), base.verify_embed,
                     base.final_norm, base.reward_w)
    cache, pt = _random_cache(shape, [29, 5], 4)
    z_ad, _ = ko.verify_pass(shape, ro, cache, [29, 5], pt)
    z_ref, _ = ko.verify_pass(shape, ref, cache, [29, 5], pt)
    z_base, _ = ko.verify_pass(shape, base, cache, [29, 5], pt)
    assert np.allclose(z_ad, z_ref, rtol=0, atol=1e-14)
    assert np.max(np.abs(z_ad - z_base)) > 1e-6  # the edited weight matters


def test_adapter_rank_split_is_additive():
    """An adapter of rank r equals its two halves applied one after the other
    (B A = B_1 A_1 + B_2 A_2 for A = [A_1; A_2], B = [B_1 B_2])."""
    shape = _tiny_small(layers=1)
    base = _readout(shape, 51)
    fac = _adapter(shape, 51, 64)(0)
    h1 = {p: (A[:32], B[:, :32]) for p, (A, B) in fac.items()}
    h2 = {p: (A[32:], B[:, 32:]) for p, (A, B) in fac.items()}
    W = base.layer(0)
    full = ko.lora_adapted(W, fac, 0.5)
    two = ko.lora_adapted(ko.lora_adapted(W, h1, 0.5), h2, 0.5)
    for f in ko.LORA_FIELDS.values():
        assert np.allclose(getattr(full, f), getattr(two, f), rtol=0, atol=1e-14)


@pytest.mark.parametrize("targets", [synth.LORA_PROJECTIONS, ("q", "v", "down")])
def test_adapter_on_the_verify_token_only_equals_reencode(targets):
    """The cache comes from the base model (adapter disabled during generation) and only the
    verify token runs theta + dtheta: the verify pass with the adapter equals a causal
    re-encode whose last position alone uses the adapted weights."""
    shape = _tiny_small()
    seed = 61
    base = _readout(shape, seed)
    ro = ko.readout_with_adapter(base, _adapter(shape, seed, 32, targets), synth.lora_scale(32))
    E = _embed(shape, seed)
    Ks, Vs, zs, lens = [], [], [], []
    for b, n in enumerate([33, 16, 0]):
        toks = synth.token_ids(seed + b, n)
        z, p, h, K, V = ko.reencode(shape, base.layer, ro.layer, E, toks, ro.verify_embed,
                                    ro.final_norm, ro.reward_w)
        Ks.append(K), Vs.append(V), zs.append(z), lens.append(n)
    cache, pt = _dense_cache(Ks, Vs, shape.page_size)
    z2, _ = ko.verify_pass(shape, ro, cache, lens, pt)
    assert np.allclose(z2, zs, rtol=0, atol=1e-12)
    z_base, _ = ko.verify_pass(shape, base, cache, lens, pt)
    assert np.max(np.abs(z2 - z_base)) > 1e-3  # the adapter changes the score


# ---------------------------------------------------------------------------------------------
# depth-k readout (k verify tokens, causal among themselves, score at the last one)


def test_depth_one_is_the_verify_pass():
    shape = _tiny_small()
    ro = _readout(shape, 71)
    cache, pt = _random_cache(shape, [40, 0, 17], 5)
    z1, _ = ko.verify_pass(shape, ro, cache, [40, 0, 17], pt)
    zk, _ = ko.verify_pass_depth(shape, ro, cache, [40, 0, 17], pt, 1)
    assert np.allclose(z1, zk, rtol=0, atol=1e-13)


@pytest.mark.parametrize("depth,mixed", [(2, False), (3, True), (5, True)])
def test_depth_k_equals_causal_reencode(depth, mixed):
    """The depth-k pass over the cache a causal forward wrote equals that forward continued
    over k verify tokens (the verify tokens using the adapted weights when mixed), read at the
    last position."""
    shape = _tiny_small()
    seed = 81
    base = _readout(shape, seed)
    ver = (ko.readout_with_adapter(base, _adapter(shape, seed, 32), synth.lora_scale(32))
           if mixed else base)
    E = _embed(shape, seed)
    Ks, Vs, zs, lens = [], [], [], []
    for b, n in enumerate([21, 16, 0]):
        toks = synth.token_ids(seed + b, n)
        z, p, h, K, V = ko.reencode(shape, base.layer, ver.layer, E, toks, ver.verify_embed,
                                    ver.final_norm, ver.reward_w, n_verify=depth)
        Ks.append(K), Vs.append(V), zs.append(z), lens.append(n)
    cache, pt = _dense_cache(Ks, Vs, shape.page_size)
    zk, _ = ko.verify_pass_depth(shape, ver, cache, lens, pt, depth)
    assert np.allclose(zk, zs, rtol=0, atol=1e-12)
    z1, _ = ko.verify_pass(shape, ver, cache, lens, pt)
    assert np.max(np.abs(zk - z1)) > 1e-3  # more verify tokens change the score


def test_depth_k_against_transformers_llama_with_kv_cache():
    """transformers' Llama decoder encodes the trajectory, then runs k verify tokens at once
    against its own cache (causal among themselves); the oracle's depth-k pass over that cache
    agrees at the last position."""
    shape = synth.ModelShape(2, 256, 4, 2, 64, 1024, weight_dtype="f32", kv_dtype="f32")
    seed = 1000
    ro = _readout(shape, seed)
    E = _embed(shape, seed).copy()
    vid = 999
    E[vid] = ro.verify_embed
    m = _hf_model(shape, ro, E)
    n, depth = 40, 3
    toks = torch.tensor([synth.token_ids(seed, n)])
    with torch.no_grad():
        out = m(input_ids=toks, use_cache=True)
        pkv = out.past_key_values
        Ks = np.stack([pkv.layers[l].keys[0, :, :n].numpy() for l in range(shape.num_layers)])
        Vs = np.stack([pkv.layers[l].values[0, :, :n].numpy() for l in range(shape.num_layers)])
        out2 = m(input_ids=torch.tensor([[vid] * depth]), past_key_values=pkv, use_cache=True)
    z_ref = out2.logits[0, -1, 1].item() - out2.logits[0, -1, 0].item()
    cache, pt = _dense_cache([Ks], [Vs], shape.page_size)
    z, _ = ko.verify_pass_depth(shape, ro, cache, [n], pt, depth)
    assert abs(z[0] - z_ref) < 1e-5


# ---------------------------------------------------------------------------------------------
# KV steering: the gradient of -log P(+) with respect to the cache (appendix algorithm)

from oracle import kv_steering as ks  # noqa: E402


def _dense_random(shape, lengths, seed):
    rng = np.random.default_rng(seed)
    K = [rng.normal(size=(shape.num_layers, shape.num_kv_heads, n, shape.head_dim)) for n in lengths]
    V = [rng.normal(size=(shape.num_layers, shape.num_kv_heads, n, shape.head_dim)) for n in lengths]
    return K, V


def test_steering_forward_equals_the_verify_pass():
    """The torch float64 forward that is differentiated is the oracle's verify pass."""
    shape = _tiny_small()
    ro = _readout(shape, 91)
    lengths = [37, 0, 16]
    K, V = _dense_random(shape, lengths, 7)
    cache, pt = _dense_cache(K, V, shape.page_size)
    z_ref, _ = ko.verify_pass(shape, ro, cache, lengths, pt)
    res = ks.loss_and_grads(shape, ro, K, V, lengths)
    for b in range(len(lengths)):
        assert abs(res[b][1] - z_ref[b]) < 1e-12
        assert abs(res[b][0] - (-math.log(ko.sigmoid(np.array([z_ref[b]]))[0]))) < 1e-12


def test_steering_gradient_matches_finite_differences():
    """d(-log P(+))/d(K, V) at sampled cache entries (every layer, keys and values, first and
    last positions) against central differences of the loss."""
    shape = _tiny_small()
    ro = _readout(shape, 92)
    lengths = [29]
    K, V = _dense_random(shape, lengths, 8)
    (_, _, dK, dV), = ks.loss_and_grads(shape, ro, K, V, lengths)
    rng = np.random.default_rng(3)
    hstep = 1e-6
    for which, G in (("k", dK), ("v", dV)):
        for _ in range(12):
            l = int(rng.integers(shape.num_layers))
            j = int(rng.integers(shape.num_kv_heads))
            t = int(rng.choice([0, lengths[0] - 1, int(rng.integers(lengths[0]))]))
            m = int(rng.integers(shape.head_dim))
            vals = []
            for sgn in (1.0, -1.0):
                Kp = [torch.tensor(K[0][i]) for i in range(shape.num_layers)]
                Vp = [torch.tensor(V[0][i]) for i in range(shape.num_layers)]
                T = Kp if which == "k" else Vp
                T[l] = T[l].clone()
                T[l][j, t, m] += sgn * hstep
                vals.append(float(ks.candidate_loss(shape, ro, Kp, Vp, lengths[0])[0]))
            fd = (vals[0] - vals[1]) / (2 * hstep)
            assert abs(fd - G[l, j, t, m]) <= 1e-7 + 1e-5 * abs(G[l, j, t, m]), (which, l, j, t, m)


def test_steering_steps_lower_the_loss_and_round_to_storage():
    shape = _tiny_small()
    ro = _readout(shape, 93)
    lengths = [40, 17]
    K, V = _dense_random(shape, lengths, 9)
    K = [ks.round_to_storage(k, "bf16") for k in K]
    V = [ks.round_to_storage(v, "bf16") for v in V]
    K2, V2, losses = ks.steer(shape, ro, K, V, lengths, eta=0.5, steps=3, store_dtype="bf16")
    for b in range(len(lengths)):
        assert losses[-1][b] < losses[0][b]
    # stored values stay bf16: rounding them again changes nothing, and equals torch's bf16
    assert np.array_equal(ks.round_to_storage(K2[0], "bf16"), K2[0])
    x = np.random.default_rng(4).normal(size=10000) * 3
    ref = torch.tensor(x, dtype=torch.float64).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ks.round_to_storage(x, "bf16"), ref)
