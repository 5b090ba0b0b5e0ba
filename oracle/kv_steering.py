"""KV Steering on the CPU in float64 (appendix, the KV Steering algorithm at an agent handoff).

TEST INFRASTRUCTURE ONLY (see kvprm_oracle): imported by the tests, never by the library.

The score of Eq. (score) is a differentiable function of the cached keys and values. KV
Steering takes T steps kv <- kv - eta * d(-log P(+))/d(kv) on the whole cache of a trajectory
(every layer, every cached position, keys and values), starting from the cache the generator
wrote. Here the loss is written out in torch float64 operations, following the verify pass of
kvprm_oracle step by step (RMSNorm, projections, rotary embedding at position L, grouped-query
attention over the cached keys plus the token's own, SwiGLU FFN, final RMSNorm, reward vector),
and its gradient with respect to the cache comes from torch's reverse-mode differentiation; the
tests pin that gradient against central finite differences of the same loss. After every step
the cache is rounded back to its storage precision (the pools hold bf16 or fp32 values).

Caches are given densely per candidate: K[b], V[b] are float64 arrays [N_L][n_kv][L_b][d_h].
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple

import numpy as np
import torch

from . import kvprm_oracle as ko


def _t(a) -> torch.Tensor:
    return torch.as_tensor(np.asarray(a, dtype=np.float64))


def _rms(x: torch.Tensor, gamma: torch.Tensor, eps: float) -> torch.Tensor:
    return x / torch.sqrt(torch.mean(x * x) + eps) * gamma


def _rope(y: torch.Tensor, pos: int, theta: float) -> torch.Tensor:
    d = y.shape[-1]
    phi = _t(ko.rope_angles(pos, d, theta))
    c, s = torch.cos(phi), torch.sin(phi)
    a, b = y[..., : d // 2], y[..., d // 2:]
    return torch.cat([a * c - b * s, b * c + a * s], dim=-1)


def candidate_loss(shape, readout: ko.Readout, K: Sequence[torch.Tensor],
                   V: Sequence[torch.Tensor], L: int) -> Tuple[torch.Tensor, torch.Tensor]:
    """(-log P(+), z) of one candidate whose per-layer cache tensors are K[l], V[l]
    ([n_kv][L][d_h]); differentiable in K and V."""
    nq, nkv, d = shape.num_q_heads, shape.num_kv_heads, shape.head_dim
    g = nq // nkv
    eps, theta = shape.rms_eps, shape.rope_theta
    x = _t(readout.verify_embed)
    for l in range(shape.num_layers):
        W = readout.layer(l)
        u = _rms(x, _t(W.attn_norm), eps)
        q = _rope((_t(W.wq) @ u).reshape(nq, d), L, theta)
        k = _rope((_t(W.wk) @ u).reshape(nkv, d), L, theta)
        v = (_t(W.wv) @ u).reshape(nkv, d)
        heads = []
        for h in range(nq):
            j = h // g
            Kj = torch.cat([K[l][j], k[j][None]], dim=0)
            Vj = torch.cat([V[l][j], v[j][None]], dim=0)
            p = torch.softmax(Kj @ q[h] / math.sqrt(d), dim=0)
            heads.append(p @ Vj)
        x = x + _t(W.wo) @ torch.cat(heads)
        u2 = _rms(x, _t(W.ffn_norm), eps)
        a = _t(W.w_gate) @ u2
        x = x + _t(W.w_down) @ (a * torch.sigmoid(a) * (_t(W.w_up) @ u2))
    hf = _rms(x, _t(readout.final_norm), eps)
    z = hf @ _t(readout.reward_w) + readout.reward_b
    # -log sigmoid(z), stable for either sign of z
    return torch.nn.functional.softplus(-z), z


def loss_and_grads(shape, readout: ko.Readout, K: Sequence[np.ndarray], V: Sequence[np.ndarray],
                   lengths: Sequence[int]):
    """Per candidate b: (-log P(+)_b, z_b, dK_b, dV_b) with dK_b, dV_b the gradients of
    -log P(+)_b with respect to K[b], V[b] (same shapes). Candidates are independent."""
    out = []
    for b, L in enumerate(lengths):
        Kt = [torch.tensor(K[b][l], dtype=torch.float64, requires_grad=True)
              for l in range(shape.num_layers)]
        Vt = [torch.tensor(V[b][l], dtype=torch.float64, requires_grad=True)
              for l in range(shape.num_layers)]
        loss, z = candidate_loss(shape, readout, Kt, Vt, int(L))
        gk = torch.autograd.grad(loss, Kt + Vt, allow_unused=True)
        dK = np.stack([(gk[l] if gk[l] is not None else torch.zeros_like(Kt[l])).numpy()
                       for l in range(shape.num_layers)])
        dV = np.stack([(gk[shape.num_layers + l] if gk[shape.num_layers + l] is not None
                        else torch.zeros_like(Vt[l])).numpy() for l in range(shape.num_layers)])
        out.append((float(loss.detach()), float(z.detach()), dK, dV))
    return out


def round_to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values to the cache's storage precision (nearest, ties to even), widened
    back to float64."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)
    if dtype == "bf16":
        f = np.asarray(x, dtype=np.float64)
        # exact RNE to bf16 from float64: keep 8 significant bits
        m, e = np.frexp(f)                      # f = m * 2^e, 0.5 <= |m| < 1
        q = np.round(m * 256.0) / 256.0         # numpy rounds halves to even
        return np.ldexp(q, e)
    raise ValueError(dtype)


def steer(shape, readout: ko.Readout, K: Sequence[np.ndarray], V: Sequence[np.ndarray],
          lengths: Sequence[int], eta: float, steps: int, store_dtype: str):
    """The KV Steering loop: `steps` times, kv <- round(kv - eta * grad(-log P(+))) for every
    candidate's cache. Returns (K, V, losses) with losses[t][b] the loss before step t (and a
    final entry after the last step)."""
    K = [np.array(k, dtype=np.float64) for k in K]
    V = [np.array(v, dtype=np.float64) for v in V]
    losses = []
    for _ in range(steps):
        res = loss_and_grads(shape, readout, K, V, lengths)
        losses.append([r[0] for r in res])
        for b, (_, _, dK, dV) in enumerate(res):
            K[b] = round_to_storage(K[b] - eta * dK, store_dtype)
            V[b] = round_to_storage(V[b] - eta * dV, store_dtype)
    losses.append([r[0] for r in loss_and_grads(shape, readout, K, V, lengths)])
    return K, V, losses


def dense_cache(cache: ko.PagedCache, shape, lengths, page_table):
    """Per candidate [N_L][n_kv][L_b][d_h] keys and values read through the page table."""
    K, V = [], []
    for b, L in enumerate(lengths):
        K.append(np.stack([cache.sequence(l, "k", page_table[b], L, shape.page_size)
                           if L else np.zeros((shape.num_kv_heads, 0, shape.head_dim))
                           for l in range(shape.num_layers)]))
        V.append(np.stack([cache.sequence(l, "v", page_table[b], L, shape.page_size)
                           if L else np.zeros((shape.num_kv_heads, 0, shape.head_dim))
                           for l in range(shape.num_layers)]))
    return K, V
