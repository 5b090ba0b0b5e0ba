"""Pins of the oracle's attention step over a paged cache (kvprm_oracle.attention_layer) and of
its dense-cache reader (kv_steering.dense_cache), on the CPU.

attention_layer is the checker of every element-wise GPU attention case, so it is pinned here
against references that share nothing with it: torch's scaled_dot_product_attention in float64
over token-major ground truth (kv-heads repeated g times for the query heads, the verify token's
own key and value appended), i.e. the appendix's head softmax(q^T K / sqrt(d_k)) V applied to
one query against L cached positions (section 4.1, Eq. (cost_kv)); and the last position of a
causal re-encode (section 5.1), whose own layout of keys is contiguous, not paged. The caches
are scattered over shuffled physical pages with NaN in every slot and page that is not part of
a candidate's sequence. Mutants of the oracle with one planted mistake each (query head h
reading kv-head h % n_kv instead of h // g; the self key dropped; the page walk shifted by one
page; one token short) must fail the same checks.
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import inputs
from oracle import kv_steering as ks
from oracle import kvprm_oracle as ko

PS = 16


def _token_major(rng, L_list, nkv, d, layers=1, k_scale=1.0):
    """Ground truth per candidate: K, V [layers][n_kv][L][d] float64."""
    K = [rng.normal(size=(layers, nkv, L, d)) * k_scale for L in L_list]
    V = [rng.normal(size=(layers, nkv, L, d)) for L in L_list]
    return K, V


def _scatter(K, V, L_list, nkv, d, layers, rng, extra_pages=7):
    """Paged cache over shuffled physical ids: logical page i of candidate b lives at a random
    physical page; slots past L_b and pages no candidate uses hold NaN."""
    npg = [-(-L // PS) for L in L_list]
    total = sum(npg) + extra_pages
    perm = rng.permutation(total)
    tiles = {}
    for l in range(layers):
        for p in range(total):
            for w in "kv":
                tiles[(l, w, p)] = np.full((nkv, PS, d), np.nan)
    table, nxt = [], 0
    for b, L in enumerate(L_list):
        row = []
        for i in range(npg[b]):
            phys = int(perm[nxt])
            nxt += 1
            row.append(phys)
            cnt = min(PS, L - i * PS)
            for l in range(layers):
                tiles[(l, "k", phys)][:, :cnt] = K[b][l][:, i * PS: i * PS + cnt]
                tiles[(l, "v", phys)][:, :cnt] = V[b][l][:, i * PS: i * PS + cnt]
        table.append(row + [-1] * 3)
    nan_tile = np.full((nkv, PS, d), np.nan)  # what a read outside the pool would see
    return ko.PagedCache(lambda l, w, p: tiles.get((l, w, p), nan_tile)), table


def _sdpa_reference(K, V, L_list, q, k_self, v_self, layer, g):
    """torch SDPA (float64, math path on the CPU), one query per head: the keys are the
    candidate's cached keys then its own key; kv-head j serves query heads j g .. j g + g - 1."""
    out = []
    for b, L in enumerate(L_list):
        Kc = torch.from_numpy(K[b][layer])  # [n_kv][L][d]
        Vc = torch.from_numpy(V[b][layer])
        ksf = torch.from_numpy(np.asarray(k_self[b], dtype=np.float64))[:, None, :]
        vsf = torch.from_numpy(np.asarray(v_self[b], dtype=np.float64))[:, None, :]
        Kf = torch.cat([Kc, ksf], dim=1).repeat_interleave(g, dim=0)  # [n_q][L+1][d]
        Vf = torch.cat([Vc, vsf], dim=1).repeat_interleave(g, dim=0)
        qb = torch.from_numpy(np.asarray(q[b], dtype=np.float64))[:, None, :]  # [n_q][1][d]
        o = torch.nn.functional.scaled_dot_product_attention(qb, Kf, Vf)
        out.append(o[:, 0, :].numpy())
    return np.stack(out)


# ---- mutants: the oracle's attention step with one planted mistake each ----------------------


def _mutant(kind):
    def fn(shape, cache, layer, lengths, page_table, q, k_self, v_self):
        B = len(lengths)
        nq, nkv, d, ps = shape.num_q_heads, shape.num_kv_heads, shape.head_dim, shape.page_size
        g = nq // nkv
        o = np.empty((B, nq, d))
        for b in range(B):
            L = int(lengths[b])
            pages = page_table[b]
            if kind == "page_shift":
                pages = list(pages[1:]) + [pages[0]]
            Lr = L - 1 if kind == "short" and L > 0 else L
            Kc = cache.sequence(layer, "k", pages, Lr, ps)
            Vc = cache.sequence(layer, "v", pages, Lr, ps)
            for h in range(nq):
                j = h % nkv if kind == "head_map" else h // g
                parts_k = [] if Kc is None else [Kc[j]]
                parts_v = [] if Vc is None else [Vc[j]]
                if kind != "no_self":
                    parts_k.append(k_self[b][j][None, :])
                    parts_v.append(v_self[b][j][None, :])
                if not parts_k:
                    o[b, h] = np.nan
                    continue
                o[b, h] = ko.attention(np.asarray(q[b][h], dtype=np.float64),
                                       np.concatenate(parts_k), np.concatenate(parts_v))
        return o
    return fn


SHAPE = synth.ModelShape(1, 64, 6, 2, 16, 96, weight_dtype="f32", kv_dtype="f32")  # g = 3


def _case(seed, L_list, k_scale=1.0, shape=SHAPE):
    rng = np.random.default_rng(seed)
    nq, nkv, d = shape.num_q_heads, shape.num_kv_heads, shape.head_dim
    K, V = _token_major(rng, L_list, nkv, d, k_scale=k_scale)
    cache, table = _scatter(K, V, L_list, nkv, d, 1, rng)
    B = len(L_list)
    q = rng.normal(size=(B, nq, d)) * (2.0 if k_scale > 1 else 1.0)
    k_self = rng.normal(size=(B, nkv, d))
    v_self = rng.normal(size=(B, nkv, d))
    ref = _sdpa_reference(K, V, L_list, q, k_self, v_self, 0, nq // nkv)
    return cache, table, q, k_self, v_self, ref


def _err(fn, seed, L_list, k_scale=1.0):
    cache, table, q, k_self, v_self, ref = _case(seed, L_list, k_scale)
    o = fn(SHAPE, cache, 0, L_list, table, q, k_self, v_self)
    if not np.all(np.isfinite(o)):
        return math.inf
    return float(np.max(np.abs(o - ref)))


CASES = [
    (11, [0, 1, 15, 16, 17, 40, 63, 64, 65, 130]),  # empty, one token, every page edge
    (12, [200, 3, 97]),
    (13, [50, 0, 33]),
]


@pytest.mark.parametrize("seed,lengths", CASES)
def test_attention_layer_equals_torch_sdpa_over_paged_ragged_cache(seed, lengths):
    assert _err(ko.attention_layer, seed, lengths) <= 1e-13


def test_attention_layer_peaked_softmax_equals_torch_sdpa():
    """K scaled x30: the softmax puts almost all weight on one key (the GPU tests use this
    variant), still equal to the library routine."""
    assert _err(ko.attention_layer, 14, [300, 1, 47], k_scale=30.0) <= 1e-12


@pytest.mark.parametrize("kind", ["head_map", "no_self", "page_shift", "short"])
def test_planted_mistakes_fail_the_attention_pins(kind):
    """Every mutant fails at least one of the cases the real oracle passes (non-finite output
    from a NaN slot, or a difference far above the rounding level)."""
    errs = [_err(_mutant(kind), s, L) for s, L in CASES]
    assert max(errs) > 1e-6, (kind, errs)


def test_unmutated_copy_passes():
    """The mutant scaffold without a planted mistake is the oracle (so the failures above come
    from the mistakes alone)."""
    for s, L in CASES:
        assert _err(_mutant("none"), s, L) <= 1e-13


def test_attention_layer_with_empty_cache_returns_own_value():
    """L = 0: the verify token attends only to itself, so every head of kv-head j returns
    v_self[j] exactly; the page table is never read."""
    rng = np.random.default_rng(3)
    q = rng.normal(size=(1, 6, 16))
    k_self = rng.normal(size=(1, 2, 16))
    v_self = rng.normal(size=(1, 2, 16))
    cache = ko.PagedCache(lambda l, w, p: (_ for _ in ()).throw(AssertionError("read")))
    o = ko.attention_layer(SHAPE, cache, 0, [0], [[-1]], q, k_self, v_self)
    for h in range(6):
        assert np.array_equal(o[0, h], v_self[0, h // 3])


def test_attention_layer_equals_the_causal_reencode_last_position():
    """A one-layer tiny model: the re-encode of [x; v] (contiguous causal attention over
    positions 0..n) and the verify pass assembled from attention_layer over the cache the
    re-encode wrote (scattered into shuffled pages), the verify token's own q, k, v, then the
    output projection, FFN and head, give the same logit."""
    shape = synth.ModelShape(1, 64, 4, 2, 16, 96, weight_dtype="f32", kv_dtype="f32")
    seed = 21
    ro = inputs.readout_from_synth(shape, seed, layer_cache=4)
    E = synth.host_normal(1000 * shape.hidden, seed, synth.stream_id(synth.GLOBAL,
                          synth.G_EMBED_TABLE)).reshape(1000, shape.hidden)
    rng = np.random.default_rng(5)
    for n in (0, 1, 16, 45):
        toks = synth.token_ids(seed + n, n)
        z_re, _, _, Kc, Vc = ko.reencode(shape, ro.layer, ro.layer, E, toks, ro.verify_embed,
                                         ro.final_norm, ro.reward_w)
        W = ro.layer(0)
        x = np.asarray(ro.verify_embed, dtype=np.float64)
        u = ko.rms_norm(x, W.attn_norm, shape.rms_eps)
        q = ko.rope((W.wq @ u).reshape(4, 16), n, shape.rope_theta)
        k = ko.rope((W.wk @ u).reshape(2, 16), n, shape.rope_theta)
        v = (W.wv @ u).reshape(2, 16)
        cache, table = _scatter([Kc], [Vc], [n], 2, 16, 1, rng)
        o = ko.attention_layer(shape, cache, 0, [n], table, q[None], k[None], v[None])[0]
        x = x + W.wo @ o.reshape(-1)
        x = x + ko.swiglu_ffn(ko.rms_norm(x, W.ffn_norm, shape.rms_eps), W.w_gate, W.w_up,
                              W.w_down)
        z = ko.rms_norm(x, ro.final_norm, shape.rms_eps) @ ro.reward_w
        assert abs(z - z_re) <= 1e-12, (n, z, z_re)


# ---- dense_cache (the steering tests' reader of the paged pools) ----------------------------


@pytest.mark.parametrize("lengths", [[0, 1, 15, 16, 17, 40], [33], [0]])
def test_dense_cache_returns_the_token_major_truth(lengths):
    """dense_cache reads every candidate's keys and values of every layer through the page
    table into [N_L][n_kv][L_b][d_h]: exactly the ground truth scattered into shuffled pages
    with NaN around it (an off-by-one page or token would show NaN or other values)."""
    shape = synth.ModelShape(3, 64, 4, 2, 16, 96, weight_dtype="f32", kv_dtype="f32")
    rng = np.random.default_rng(len(lengths) * 7 + sum(lengths))
    K, V = _token_major(rng, lengths, 2, 16, layers=3)
    cache, table = _scatter(K, V, lengths, 2, 16, 3, rng)
    Kd, Vd = ks.dense_cache(cache, shape, lengths, table)
    assert len(Kd) == len(lengths) == len(Vd)
    for b, L in enumerate(lengths):
        assert Kd[b].shape == (3, 2, L, 16) and Vd[b].shape == (3, 2, L, 16)
        assert np.array_equal(Kd[b], K[b]) and np.array_equal(Vd[b], V[b])


def test_dense_cache_reads_the_synthetic_pools_in_stored_layout():
    """On a synthetic workload (values from the generator, tiles in the stored K and V layouts),
    dense_cache agrees with the tile decoders applied page by page by hand."""
    shape = synth.ModelShape(2, 128, 4, 2, 32, 128, weight_dtype="bf16", kv_dtype="bf16")
    w = synth.make_workload("custom", shape=shape, lengths=[37, 0, 16], seed=61)
    cache = inputs.cache_from_synth(w)
    Kd, Vd = ks.dense_cache(cache, shape, w.lengths, w.page_table)
    T = shape.tile_elems
    for b, L in enumerate(w.lengths):
        for l in range(shape.num_layers):
            for which, D in (("k", Kd), ("v", Vd)):
                rows = []
                for i in range(-(-L // PS)):
                    pg = w.page_table[b][i]
                    raw = synth.host_normal(2 * T, w.seed, synth.kv_stream(l, which), pg * 2 * T,
                                            0.0, 1.0, synth.DT_BF16).reshape(2, T)
                    vals = ko.bf16_bits_to_f64(raw)
                    dec = ko.k_tile_to_tokens if which == "k" else ko.v_tile_to_tokens
                    rows.append(np.stack([dec(vals[j], PS, 32, 2) for j in range(2)]))
                want = (np.concatenate(rows, axis=1)[:, :L] if rows else np.zeros((2, 0, 32)))
                assert np.array_equal(D[b][l], want)
