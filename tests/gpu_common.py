"""Shared helpers of the GPU tests: build device inputs, run the library, compare with the
oracle. Only the tests import this module."""
import math

import numpy as np
import torch

import synth
from synth.device import DeviceWorkload


def kv():
    import paper_2607_09153_amd as m
    return m


def run_score(dw: DeviceWorkload, with_hint=True, lengths_host=True, stream=None):
    m = kv()
    h = m.kvprm_create(dw.desc(m))
    try:
        batch = dw.batch(m, with_hint=with_hint, lengths_host=lengths_host)
        n = m.kvprm_workspace_size(h, batch)
        ws = torch.empty(max(n, 256), dtype=torch.uint8, device="cuda")
        B = dw.w.batch
        scores = torch.full((B,), float("nan"), dtype=torch.float32, device="cuda")
        logits = torch.full((B,), float("nan"), dtype=torch.float32, device="cuda")
        st = stream or torch.cuda.current_stream()
        m.kvprm_score(h, dw.cache(m), batch, dw.readout(m), ws.data_ptr(), n, scores.data_ptr(),
                      logits.data_ptr(), st.cuda_stream)
        st.synchronize()
        return scores.cpu().numpy().astype(np.float64), logits.cpu().numpy().astype(np.float64)
    finally:
        m.kvprm_destroy(h)


def host_activations(w: synth.Workload, seed_stream: int, scale: float = 1.0):
    """Seeded q / k_self / v_self for an attention-only check (fp32, host)."""
    s = w.shape
    B = w.batch
    q = synth.host_normal(B * s.num_q_heads * s.head_dim, w.seed, seed_stream, 0, 0.0, scale,
                          synth.DT_F32).reshape(B, s.num_q_heads, s.head_dim)
    ks = synth.host_normal(B * s.num_kv_heads * s.head_dim, w.seed, seed_stream + 1, 0, 0.0, scale,
                           synth.DT_F32).reshape(B, s.num_kv_heads, s.head_dim)
    vs = synth.host_normal(B * s.num_kv_heads * s.head_dim, w.seed, seed_stream + 2, 0, 0.0, 1.0,
                           synth.DT_F32).reshape(B, s.num_kv_heads, s.head_dim)
    return q, ks, vs


def run_attention(dw: DeviceWorkload, layer, q, ks, vs, with_hint=True):
    m = kv()
    h = m.kvprm_create(dw.desc(m))
    try:
        batch = dw.batch(m, with_hint=with_hint)
        n = m.kvprm_workspace_size(h, batch)
        ws = torch.empty(max(n, 256), dtype=torch.uint8, device="cuda")
        qd = torch.from_numpy(q).cuda()
        kd = torch.from_numpy(ks).cuda()
        vd = torch.from_numpy(vs).cuda()
        o = torch.full(q.shape, float("nan"), dtype=torch.float32, device="cuda")
        m.kvprm_attention(h, dw.cache(m), batch, layer, qd.data_ptr(), kd.data_ptr(),
                          vd.data_ptr(), ws.data_ptr(), n, o.data_ptr(),
                          torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        return o.cpu().numpy().astype(np.float64)
    finally:
        m.kvprm_destroy(h)


def run_score_lora(dw: DeviceWorkload, stream=None):
    """kvprm_score_lora with the workload's base weights and its adapter (dw.add_lora)."""
    m = kv()
    h = m.kvprm_create(dw.desc(m))
    try:
        batch = dw.batch(m)
        n = m.kvprm_workspace_size_lora(h, batch, dw.lora_rank)
        ws = torch.empty(max(n, 256), dtype=torch.uint8, device="cuda")
        B = dw.w.batch
        scores = torch.full((B,), float("nan"), dtype=torch.float32, device="cuda")
        logits = torch.full((B,), float("nan"), dtype=torch.float32, device="cuda")
        st = stream or torch.cuda.current_stream()
        m.kvprm_score_lora(h, dw.cache(m), batch, dw.readout(m), dw.lora(m), ws.data_ptr(), n,
                           scores.data_ptr(), logits.data_ptr(), st.cuda_stream)
        st.synchronize()
        return scores.cpu().numpy().astype(np.float64), logits.cpu().numpy().astype(np.float64)
    finally:
        m.kvprm_destroy(h)


def run_score_ex(dw: DeviceWorkload, depth: int = 1, lora: bool = False, with_hint: bool = True,
                 stream=None):
    """kvprm_score_ex with a depth-k readout (and the workload's adapter when lora)."""
    m = kv()
    h = m.kvprm_create(dw.desc(m))
    try:
        batch = dw.batch(m, with_hint=with_hint)
        opt = m.make_options(dw.lora(m) if lora else None, depth)
        n = m.kvprm_workspace_size_ex(h, batch, opt)
        ws = torch.empty(max(n, 256), dtype=torch.uint8, device="cuda")
        B = dw.w.batch
        scores = torch.full((B,), float("nan"), dtype=torch.float32, device="cuda")
        logits = torch.full((B,), float("nan"), dtype=torch.float32, device="cuda")
        st = stream or torch.cuda.current_stream()
        m.kvprm_score_ex(h, dw.cache(m), batch, dw.readout(m), opt, ws.data_ptr(), n,
                         scores.data_ptr(), logits.data_ptr(), st.cuda_stream)
        st.synchronize()
        return scores.cpu().numpy().astype(np.float64), logits.cpu().numpy().astype(np.float64)
    finally:
        m.kvprm_destroy(h)
