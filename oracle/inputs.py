"""Host-side inputs for the oracle, regenerated from the seeded generator package.

TEST INFRASTRUCTURE ONLY (see kvprm_oracle). Every tensor is produced by
``synth`` on the host from (seed, stream, element index) and decoded exactly to
float64. Nothing here comes from the GPU library.

Weights are generated one layer at a time on demand (with a small cache), and
cache pages one physical page at a time, so that full-size workloads only ever
hold one layer of weights and the pages of the candidates actually scored.
"""
from __future__ import annotations

from functools import lru_cache
from typing import Optional

import numpy as np

import synth
from . import kvprm_oracle as ko

_DT = {"f32": synth.DT_F32, "bf16": synth.DT_BF16, "f64": synth.DT_F64}


def _gen_tensor(name, kind, dims, seed, layer, wdtype, shape):
    """One weight tensor in its storage order, widened; bf16 matrices are stored packed."""
    mean, std = synth.tensor_mean_std(name, dims)
    n = int(np.prod(dims))
    raw = synth.host_normal(n, seed, synth.stream_id(layer, kind), 0, mean, std, _DT[wdtype])
    vals = ko.decode_storage(raw, wdtype)
    if len(dims) == 2 and wdtype == "bf16":
        return ko.unpack_tiled(vals, dims[0], dims[1])
    return vals.reshape(dims)


def readout_from_synth(shape: synth.ModelShape, seed: int, layer_cache: int = 2) -> ko.Readout:
    """Readout weights of a synthetic model (weights in the stored precision, widened)."""
    wdt = shape.weight_dtype

    @lru_cache(maxsize=layer_cache)
    def layer(l: int) -> ko.LayerWeights:
        t = {name: _gen_tensor(name, kind, dims, seed, l, wdt, shape)
             for name, kind, dims in synth.layer_tensors(shape)}
        return ko.LayerWeights(**t)

    g = {name: _gen_tensor(name, kind, dims, seed, synth.GLOBAL, wdt, shape)
         for name, kind, dims in synth.global_tensors(shape)}
    return ko.Readout(layer, g["verify_embed"], g["final_norm"], g["reward_w"], 0.0)


def lora_from_synth(shape: synth.ModelShape, seed: int, rank: int,
                    targets=synth.LORA_PROJECTIONS, layer_cache: int = 2):
    """Adapter factors of a synthetic model: layer -> {projection: (A, B)} in float64, stored
    like the base matrices (packed when bf16)."""
    wdt = shape.weight_dtype

    @lru_cache(maxsize=layer_cache)
    def factors(l: int):
        t = {name: _gen_tensor(name, kind, dims, seed, l, wdt, shape)
             for name, kind, dims in synth.lora_tensors(shape, rank, targets)}
        return {p: (t[f"lora_a_{p}"], t[f"lora_b_{p}"]) for p in targets}

    return factors


def cache_from_synth(w: synth.Workload, nan_pages=(), page_cache: int = 4096) -> ko.PagedCache:
    """Paged pools of a workload, one physical page per call, decoded to float64."""
    s = w.shape
    nkv, ps, d = s.num_kv_heads, s.page_size, s.head_dim
    T = s.tile_elems
    eb = s.kv_elem_bytes

    @lru_cache(maxsize=page_cache)
    def tiles(layer: int, which: str, page: int) -> np.ndarray:
        stream = synth.kv_stream(layer, which)
        std = w.k_std if which == "k" else w.v_std
        if s.kv_dtype == "fp8":
            codes, scales = synth.host_fp8_tiles(nkv, T, w.seed, stream, page * nkv,
                                                 scale=w.fp8_scale)
            vals = ko.e4m3fn_to_f64(codes).reshape(nkv, T) * scales.astype(np.float64)[:, None]
        else:
            raw = synth.host_normal(nkv * T, w.seed, stream, page * nkv * T, 0.0, std,
                                    _DT[s.kv_dtype])
            vals = ko.decode_storage(raw, s.kv_dtype).reshape(nkv, T)
        out = np.empty((nkv, ps, d))
        for j in range(nkv):
            if which == "k":
                out[j] = ko.k_tile_to_tokens(vals[j], ps, d, eb)
            else:
                out[j] = ko.v_tile_to_tokens(vals[j], ps, d, eb)
        return out

    return ko.PagedCache(tiles)


def score_workload(w: synth.Workload, candidates=None, return_hidden: bool = False,
                   lora_rank: int = 0, lora_targets=synth.LORA_PROJECTIONS, depth: int = 1):
    """Oracle scores (z, P(+)) of the listed candidates (default: all) of a workload; with
    lora_rank > 0 the verify token runs the base weights with the synthetic adapter of that
    rank on lora_targets (scale alpha / rank); depth > 1 scores with that many verify tokens
    (the depth-k readout)."""
    cand = list(range(w.batch)) if candidates is None else list(candidates)
    ro = readout_from_synth(w.shape, w.seed)
    if lora_rank > 0:
        ro = ko.readout_with_adapter(ro, lora_from_synth(w.shape, w.seed, lora_rank, lora_targets),
                                     synth.lora_scale(lora_rank))
    cache = cache_from_synth(w)
    lens = [w.lengths[b] for b in cand]
    pt = [w.page_table[b] for b in cand]
    if depth > 1:
        return ko.verify_pass_depth(w.shape, ro, cache, lens, pt, depth,
                                    return_hidden=return_hidden)
    return ko.verify_pass(w.shape, ro, cache, lens, pt, return_hidden=return_hidden)


def embed_table(shape: synth.ModelShape, seed: int, vocab: int = synth.VOCAB) -> np.ndarray:
    """Token embedding table [vocab][H] of a synthetic model, N(0, 1) in the weight storage
    precision, widened to float64."""
    raw = synth.host_normal(vocab * shape.hidden, seed,
                            synth.stream_id(synth.GLOBAL, synth.G_EMBED_TABLE), 0, 0.0, 1.0,
                            _DT[shape.weight_dtype])
    return ko.decode_storage(raw, shape.weight_dtype).reshape(vocab, shape.hidden)


def reencode_batch(shape: synth.ModelShape, seed: int, lengths, mixed: bool = False):
    """The re-encode mode of a workload: candidate b is a sequence of lengths[b] token ids (from
    the seed's token stream, offset b * 4096) followed by the verify token (id VERIFY_ID), run
    causally through the model by kvprm_oracle.reencode. The cached positions use the weights
    of `seed` (adapter off, as during generation); the verify token uses the same weights, or,
    with mixed, those of seed + ADAPTER_SEED_OFFSET (adapter on the verify token only).

    Returns a dict: z, p [B] (the last position's logit and P(+)), K, V (per candidate
    [N_L][n_kv][L_b][d_h] float64: the cache the causal pass wrote, keys after rotation),
    verify_embed (the verify token's embedding row) and the two readouts (base, verify)."""
    base = readout_from_synth(shape, seed, layer_cache=max(2, shape.num_layers))
    ver = (readout_from_synth(shape, seed + synth.ADAPTER_SEED_OFFSET,
                              layer_cache=max(2, shape.num_layers)) if mixed else base)
    E = embed_table(shape, seed)
    ev = E[synth.VERIFY_ID]
    zs, Ks, Vs = [], [], []
    for b, n in enumerate(lengths):
        toks = synth.token_ids(seed, int(n), offset=4096 * b)
        z, _, _, K, V = ko.reencode(shape, base.layer, ver.layer, E, toks, ev, ver.final_norm,
                                    ver.reward_w, ver.reward_b)
        zs.append(z)
        Ks.append(K)
        Vs.append(V)
    z = np.array(zs)
    return {"z": z, "p": ko.sigmoid(z), "K": Ks, "V": Vs, "verify_embed": ev, "base": base,
            "verify": ver}
