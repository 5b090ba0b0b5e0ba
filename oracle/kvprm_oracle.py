"""fp64 CPU oracle for KV-PRM verify-token scoring.

TEST INFRASTRUCTURE ONLY. This module is the plain, slow definition that the
GPU library is checked against. Only the test suite, the smoke check and the
CPU-baseline leg of the benchmark may import it; the product path never does.
It shares no code with the HIP library: its only input source is the seeded
generator package ``synth``.

What it computes (KV-PRM, section 4.1, Eq. (score)): the verify token v is
pushed through the adapter-merged decoder f_{theta+dtheta}, conditioned on the
existing key/value cache (K, V) of the trajectory; the two judgment logits give
P(+) = softmax([z_-, z_+]) taken at the "+" entry. Everything runs in float64
on exactly decoded inputs (fp32, bf16 and e4m3 * scale all convert to float64
without rounding).

Readings where the paper is silent:
  * the decoder block is the standard pre-norm one: RMSNorm -> Q/K/V ->
    rotary -> grouped-query attention -> output projection -> residual;
    RMSNorm -> SwiGLU -> residual; a final RMSNorm; no biases, no q/k norm;
  * q-head h reads kv-head floor(h / g), g = n_q / n_kv;
  * rotary embedding is the rotate-half form with angle pos * theta^(-2i/d);
  * the verify token sits at position L (after L cached tokens at 0..L-1)
    and attends to the L cached keys plus its own key (L + 1 keys in all);
  * the cache holds keys after rotation; values are not rotated;
  * P(+) is the "+" component, i.e. sigmoid(z_+ - z_-), so the head reduces
    to a reward vector w_r = W_out[+] - W_out[-] (and bias b_r) applied to the
    final normalised state.
"""
from __future__ import annotations

import math
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

# ---------------------------------------------------------------------------------------------
# number formats: exact decoding of the stored values


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bfloat16 is the upper half of an IEEE binary32; widening is exact."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):  # NaN payloads widen to NaN
        return u.view(np.float32).astype(np.float64)


def e4m3fn_to_f64(codes: np.ndarray) -> np.ndarray:
    """OCP 8-bit floating point, E4M3FN variant (OCP FP8 specification v1.0).

    sign 1 bit, exponent 4 bits (bias 7), mantissa 3 bits; exponent 0 gives
    subnormals m/8 * 2^-6; exponent 15 with mantissa 7 is NaN; there are no
    infinities, so the largest finite value is 1.75 * 2^8 = 448.
    """
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = c & 0x7
    normal = sign * (1.0 + m / 8.0) * np.power(2.0, (e - 7).astype(np.float64))
    sub = sign * (m / 8.0) * 2.0 ** -6
    out = np.where(e == 0, sub, normal)
    out = np.where((e == 15) & (m == 7), np.nan, out)
    return out


def decode_storage(raw: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f64":
        return np.asarray(raw, dtype=np.float64)
    if dtype == "f32":
        return np.asarray(raw, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return bf16_bits_to_f64(raw)
    if dtype == "fp8":
        return e4m3fn_to_f64(raw)
    raise ValueError(dtype)


# ---------------------------------------------------------------------------------------------
# paged cache layout (the storage contract of the library's cache arguments)
#
# pool[layer][page][kv_head] is a tile of page_size (16) x head_dim values; x = 16 bytes /
# element size values fill 16 bytes, r = x / 4.
#   K tile: [head_dim / x][16 slots][x]: element (slot s, dim m) at ((m / x) * 16 + s) * x + m % x
#   V tile: [head_dim / (16 r)][4][16][r][4]: element (s, m) at
#           ((((m / (16 r)) * 4 + s / 4) * 16 + m % 16) * r + (m / 16) % r) * 4 + s % 4
#   (16 bytes hold 4 consecutive slots of r dimensions 16 apart)


def k_tile_to_tokens(tile: np.ndarray, page_size: int, head_dim: int, elem_bytes: int) -> np.ndarray:
    """Reorder one stored K tile into [slot][dim]."""
    x = 16 // elem_bytes
    return tile.reshape(head_dim // x, page_size, x).transpose(1, 0, 2).reshape(page_size, head_dim)


def v_tile_to_tokens(tile: np.ndarray, page_size: int, head_dim: int, elem_bytes: int) -> np.ndarray:
    """Reorder one stored V tile into [slot][dim]."""
    r = 16 // elem_bytes // 4
    a = tile.reshape(head_dim // (16 * r), 4, 16, r, 4)  # [m // 16r][s // 4][m % 16][(m // 16) % r][s % 4]
    return a.transpose(1, 4, 0, 3, 2).reshape(page_size, head_dim)


# ---------------------------------------------------------------------------------------------
# packed weight layout (the storage contract of bf16 weight matrices)
#
# A matrix W [rows][K] (rows and K multiples of 16 and 32) is stored as 1 KiB blocks, one per
# (32-input block kb, 16-row tile t), block index kb * (rows / 16) + t; inside a block, 64 groups
# of 8 values, group l holding W[16 t + l % 16][32 kb + 8 (l // 16) + i], i = 0..7.


def unpack_tiled(stored: np.ndarray, rows: int, K: int) -> np.ndarray:
    """Reorder packed storage into the row-major matrix [rows][K]."""
    a = np.asarray(stored).reshape(K // 32, rows // 16, 4, 16, 8)  # [kb][t][l//16][l%16][i]
    return a.transpose(1, 3, 0, 2, 4).reshape(rows, K)


# ---------------------------------------------------------------------------------------------
# decoder pieces


def rms_norm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gamma, over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gamma


def rope_angles(pos: int, head_dim: int, theta: float) -> np.ndarray:
    """phi_i = pos * theta^(-2i/d) for i < d/2."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    return float(pos) * np.power(theta, -2.0 * i / head_dim)


def rope(y: np.ndarray, pos: int, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding of every head row of y ([heads, d]) at position pos.

    The pair (y_i, y_{i+d/2}) is rotated by the angle phi_i.
    """
    d = y.shape[-1]
    phi = rope_angles(pos, d, theta)
    c, s = np.cos(phi), np.sin(phi)
    a, b = y[..., : d // 2], y[..., d // 2:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def attention(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """One attention head for one query: softmax(q K^T / sqrt(d_k)) V (appendix, proof of
    the readout-depth theorem, where each head is this linear map of the cache)."""
    d = q.shape[-1]
    s = K @ q / math.sqrt(d)
    m = np.max(s)
    p = np.exp(s - m)
    return (p @ V) / np.sum(p)


def silu(a: np.ndarray) -> np.ndarray:
    return a / (1.0 + np.exp(-a))


def swiglu_ffn(u: np.ndarray, w_gate: np.ndarray, w_up: np.ndarray, w_down: np.ndarray) -> np.ndarray:
    """W_down (silu(W_gate u) * W_up u); u may be a matrix of column vectors."""
    return w_down @ (silu(w_gate @ u) * (w_up @ u))


def sigmoid(z):
    """Numerically stable logistic function."""
    z = np.asarray(z, dtype=np.float64)
    out = np.empty_like(z)
    pos = z >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-z[pos]))
    ez = np.exp(z[~pos])
    out[~pos] = ez / (1.0 + ez)
    return out


def judgment_probability(z_minus, z_plus):
    """Eq. (score): the "+" entry of softmax([z_-, z_+]) (0-based index 1)."""
    zm = np.asarray(z_minus, dtype=np.float64)
    zp = np.asarray(z_plus, dtype=np.float64)
    m = np.maximum(zm, zp)
    ep, em = np.exp(zp - m), np.exp(zm - m)
    return ep / (ep + em)


# ---------------------------------------------------------------------------------------------
# weights and cache access (plain containers filled by oracle.inputs)


class LayerWeights:
    """fp64 weights of one decoder layer; matrices are [out, in]."""

    def __init__(self, attn_norm, wq, wk, wv, wo, ffn_norm, w_gate, w_up, w_down):
        self.attn_norm, self.wq, self.wk, self.wv, self.wo = attn_norm, wq, wk, wv, wo
        self.ffn_norm, self.w_gate, self.w_up, self.w_down = ffn_norm, w_gate, w_up, w_down


class Readout:
    """Everything the verify pass needs besides the cache: per-layer weights (theta + dtheta,
    merged; readout_with_adapter forms them from a base readout and adapter factors), the
    verify-token embedding, the final norm gain, and the reward vector
    w_r = W_out[+] - W_out[-] with bias b_r = b[+] - b[-]."""

    def __init__(self, layer: Callable[[int], LayerWeights], verify_embed, final_norm, reward_w,
                 reward_b: float = 0.0):
        self.layer = layer
        self.verify_embed = verify_embed
        self.final_norm = final_norm
        self.reward_w = reward_w
        self.reward_b = reward_b


# Low-rank adapter (section 4.1, Eq. (score): the verify token runs f_{theta + dtheta}, where
# dtheta is a LoRA adapter of the base model, Hu et al. 2022). A projection W [out, in] with
# factors A [r, in] and B [out, r] and scale alpha / r acts as W + scale * B A on the verify
# token; the cached positions were produced by the base weights alone.

LORA_FIELDS = {"q": "wq", "k": "wk", "v": "wv", "o": "wo", "gate": "w_gate", "up": "w_up",
               "down": "w_down"}
_LAYER_FIELDS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")


def lora_adapted(W: LayerWeights, factors: Dict[str, Tuple[np.ndarray, np.ndarray]],
                 scale: float) -> LayerWeights:
    """The layer's weights with scale * B @ A added to each projection listed in factors
    (projection name -> (A, B))."""
    mats = {f: getattr(W, f) for f in _LAYER_FIELDS}
    for proj, (A, B) in factors.items():
        f = LORA_FIELDS[proj]
        assert A.shape[1] == mats[f].shape[1] and B.shape[0] == mats[f].shape[0]
        assert A.shape[0] == B.shape[1]
        mats[f] = mats[f] + scale * (B @ A)
    return LayerWeights(**mats)


def readout_with_adapter(base: "Readout", layer_factors: Callable[[int], Dict], scale: float):
    """The readout of f_{theta + dtheta}: base weights with each layer's adapter applied."""
    return Readout(lambda l: lora_adapted(base.layer(l), layer_factors(l), scale),
                   base.verify_embed, base.final_norm, base.reward_w, base.reward_b)


class PagedCache:
    """Read access to the paged pools: `tiles(layer, which, page)` returns the decoded
    [n_kv][page_size][head_dim] float64 values of one physical page ('k' or 'v'),
    scale already applied for fp8 pools."""

    def __init__(self, tiles: Callable[[int, str, int], np.ndarray]):
        self.tiles = tiles

    def sequence(self, layer: int, which: str, pages: Sequence[int], length: int,
                 page_size: int) -> np.ndarray:
        """[n_kv][length][head_dim] for one candidate."""
        if length == 0:
            return None
        npg = -(-length // page_size)
        t = [self.tiles(layer, which, int(pages[i])) for i in range(npg)]
        return np.concatenate(t, axis=1)[:, :length, :]


# ---------------------------------------------------------------------------------------------
# Eq. (score): the verify-token pass


def verify_pass(shape, readout: Readout, cache: PagedCache, lengths: Sequence[int],
                page_table, return_hidden: bool = False):
    """Score every candidate b: x <- e_v at position L_b, N_L decoder layers that attend
    over the candidate's cached keys/values plus the token's own, final RMSNorm, reward
    head, sigmoid. Returns (z[B], P(+)[B]) as float64 (and the final normalised states).

    Candidates are independent; the loop over layers is outside so that one layer's
    weights are live at a time.
    """
    B = len(lengths)
    H, nq, nkv, d = shape.hidden, shape.num_q_heads, shape.num_kv_heads, shape.head_dim
    g = nq // nkv
    eps, theta, ps = shape.rms_eps, shape.rope_theta, shape.page_size
    x = np.tile(np.asarray(readout.verify_embed, dtype=np.float64), (B, 1))  # [B, H]
    for l in range(shape.num_layers):
        W = readout.layer(l)
        u = rms_norm(x, W.attn_norm, eps)  # [B, H]
        q_all = (W.wq @ u.T).T.reshape(B, nq, d)
        k_all = (W.wk @ u.T).T.reshape(B, nkv, d)
        v_all = (W.wv @ u.T).T.reshape(B, nkv, d)
        o = np.empty((B, nq, d))
        for b in range(B):
            L = int(lengths[b])
            q = rope(q_all[b], L, theta)
            k_self = rope(k_all[b], L, theta)
            v_self = v_all[b]
            Kc = cache.sequence(l, "k", page_table[b], L, ps)
            Vc = cache.sequence(l, "v", page_table[b], L, ps)
            for h in range(nq):
                j = h // g
                if Kc is None:
                    K, V = k_self[j][None, :], v_self[j][None, :]
                else:
                    K = np.concatenate([Kc[j], k_self[j][None, :]], axis=0)
                    V = np.concatenate([Vc[j], v_self[j][None, :]], axis=0)
                o[b, h] = attention(q[h], K, V)
        x = x + (W.wo @ o.reshape(B, nq * d).T).T
        u2 = rms_norm(x, W.ffn_norm, eps)
        x = x + swiglu_ffn(u2.T, W.w_gate, W.w_up, W.w_down).T
    h_fin = rms_norm(x, readout.final_norm, eps)
    z = h_fin @ readout.reward_w + readout.reward_b
    p = sigmoid(z)
    if return_hidden:
        return z, p, h_fin
    return z, p


def verify_pass_depth(shape, readout: Readout, cache: PagedCache, lengths: Sequence[int],
                      page_table, depth: int, return_hidden: bool = False):
    """Depth-k readout (section 3, definition of the depth-k readout; the k > 1 experiment of
    section 5): `depth` verify tokens are appended after the L_b cached tokens, at positions
    L_b .. L_b + depth - 1, and pass through the readout layers together, token i attending to
    the cached keys and to verify tokens 0..i (causal, as decoding an appended suffix). The
    score is read from the last verify token. depth = 1 is verify_pass."""
    B = len(lengths)
    H, nq, nkv, d = shape.hidden, shape.num_q_heads, shape.num_kv_heads, shape.head_dim
    g = nq // nkv
    eps, theta, ps = shape.rms_eps, shape.rope_theta, shape.page_size
    k = int(depth)
    x = np.tile(np.asarray(readout.verify_embed, dtype=np.float64), (B, k, 1))  # [B, k, H]
    for l in range(shape.num_layers):
        W = readout.layer(l)
        o = np.empty((B, k, nq, d))
        for b in range(B):
            L = int(lengths[b])
            u = rms_norm(x[b], W.attn_norm, eps)  # [k, H]
            q = np.stack([rope((W.wq @ u[i]).reshape(nq, d), L + i, theta) for i in range(k)])
            ks = np.stack([rope((W.wk @ u[i]).reshape(nkv, d), L + i, theta) for i in range(k)])
            vs = np.stack([(W.wv @ u[i]).reshape(nkv, d) for i in range(k)])
            Kc = cache.sequence(l, "k", page_table[b], L, ps)
            Vc = cache.sequence(l, "v", page_table[b], L, ps)
            for i in range(k):
                for h in range(nq):
                    j = h // g
                    Ks, Vs = ks[: i + 1, j], vs[: i + 1, j]
                    K = Ks if Kc is None else np.concatenate([Kc[j], Ks], axis=0)
                    V = Vs if Vc is None else np.concatenate([Vc[j], Vs], axis=0)
                    o[b, i, h] = attention(q[i, h], K, V)
        x = x + np.einsum("oi,bki->bko", W.wo, o.reshape(B, k, nq * d))
        u2 = rms_norm(x, W.ffn_norm, eps)
        a = np.einsum("fi,bki->bkf", W.w_gate, u2)
        c = np.einsum("fi,bki->bkf", W.w_up, u2)
        x = x + np.einsum("of,bkf->bko", W.w_down, silu(a) * c)
    h_fin = rms_norm(x[:, k - 1], readout.final_norm, eps)
    z = h_fin @ readout.reward_w + readout.reward_b
    p = sigmoid(z)
    if return_hidden:
        return z, p, h_fin
    return z, p


def attention_layer(shape, cache: PagedCache, layer: int, lengths, page_table, q, k_self, v_self):
    """Attention step alone for one layer: q [B][n_q][d] (already rotated), k_self/v_self
    [B][n_kv][d]. Returns o [B][n_q][d]."""
    B = len(lengths)
    nq, nkv, d, ps = shape.num_q_heads, shape.num_kv_heads, shape.head_dim, shape.page_size
    g = nq // nkv
    o = np.empty((B, nq, d))
    for b in range(B):
        L = int(lengths[b])
        Kc = cache.sequence(layer, "k", page_table[b], L, ps)
        Vc = cache.sequence(layer, "v", page_table[b], L, ps)
        for h in range(nq):
            j = h // g
            if Kc is None:
                K, V = k_self[b][j][None, :], v_self[b][j][None, :]
            else:
                K = np.concatenate([Kc[j], k_self[b][j][None, :]], axis=0)
                V = np.concatenate([Vc[j], v_self[b][j][None, :]], axis=0)
            o[b, h] = attention(np.asarray(q[b][h], dtype=np.float64), K, V)
    return o


# ---------------------------------------------------------------------------------------------
# Text-PRM: full causal re-encode of [x; v] (section 5.1 baselines; Eq. (1) cost model)


def reencode(shape, layer_base: Callable[[int], LayerWeights],
             layer_verify: Callable[[int], LayerWeights], embed: np.ndarray,
             tokens: Sequence[int], verify_embed: np.ndarray, final_norm, reward_w,
             reward_b: float = 0.0, n_verify: int = 1):
    """Causal forward over n prefix tokens and n_verify verify tokens at positions n ..

    Positions t < n use the base weights (adapter off, as during generation);
    positions >= n use `layer_verify` (adapter on). With both equal and one verify
    token this is the Text-PRM computation on [x; v]. Attention at position t sees
    keys 0..t. The score is read at the last position.

    Returns (z, P(+), h_final, K, V) where K, V are [N_L][n_kv][n][d] float64:
    the cache the generator would have written (keys after rotation).
    """
    n = len(tokens)
    nv = int(n_verify)
    H, nq, nkv, d = shape.hidden, shape.num_q_heads, shape.num_kv_heads, shape.head_dim
    g = nq // nkv
    eps, theta = shape.rms_eps, shape.rope_theta
    X = np.concatenate([embed[np.asarray(tokens, dtype=np.int64)].reshape(n, embed.shape[1]),
                        np.tile(np.asarray(verify_embed, dtype=np.float64), (nv, 1))],
                       axis=0)  # [n + nv, H]
    T = n + nv
    Kcache = np.empty((shape.num_layers, nkv, n, d))
    Vcache = np.empty((shape.num_layers, nkv, n, d))
    for l in range(shape.num_layers):
        Wb, Wv = layer_base(l), layer_verify(l)
        Xn = np.empty_like(X)
        Q = np.empty((T, nq, d))
        K = np.empty((T, nkv, d))
        V = np.empty((T, nkv, d))
        for t in range(T):
            W = Wb if t < n else Wv
            u = rms_norm(X[t], W.attn_norm, eps)
            Q[t] = rope((W.wq @ u).reshape(nq, d), t, theta)
            K[t] = rope((W.wk @ u).reshape(nkv, d), t, theta)
            V[t] = (W.wv @ u).reshape(nkv, d)
        Kcache[l] = K[:n].transpose(1, 0, 2)
        Vcache[l] = V[:n].transpose(1, 0, 2)
        for t in range(T):
            W = Wb if t < n else Wv
            o = np.empty((nq, d))
            for h in range(nq):
                j = h // g
                o[h] = attention(Q[t, h], K[: t + 1, j], V[: t + 1, j])
            xt = X[t] + W.wo @ o.reshape(-1)
            u2 = rms_norm(xt, W.ffn_norm, eps)
            Xn[t] = xt + swiglu_ffn(u2, W.w_gate, W.w_up, W.w_down)
        X = Xn
    h_fin = rms_norm(X[T - 1], final_norm, eps)
    z = float(h_fin @ reward_w + reward_b)
    return z, float(sigmoid(np.array([z]))[0]), h_fin, Kcache, Vcache
