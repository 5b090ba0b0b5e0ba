"""Device-resident synthetic workloads: torch tensors in HBM filled by the device generator.

Holds no arithmetic of the scoring method: it allocates the weight tensors, the paged K/V
pools (with fp8 scales), the page table and the lengths of a ``synth.Workload`` and fills
them with ``synth.device_normal`` / ``synth.device_fp8_tiles``, which produce the same bits the
host generator gives the oracle.
"""
from __future__ import annotations

from typing import Dict, List

import torch

import synth

_TORCH_W = {"f32": torch.float32, "bf16": torch.bfloat16}
_TORCH_KV = {"f32": torch.float32, "bf16": torch.bfloat16, "fp8": torch.uint8}
_DT = {"f32": synth.DT_F32, "bf16": synth.DT_BF16}


class DeviceWorkload:
    def __init__(self, w: synth.Workload, device: str = "cuda", nan_unused_pages: bool = False,
                 fill_weights: bool = True):
        self.w = w
        s = w.shape
        self.device = device
        stream = torch.cuda.current_stream().cuda_stream
        wdt = s.weight_dtype
        self.layers: List[Dict[str, torch.Tensor]] = []
        for l in range(s.num_layers):
            d = {}
            for name, kind, dims in synth.layer_tensors(s):
                t = torch.empty(dims, dtype=_TORCH_W[wdt], device=device)
                if fill_weights:
                    mean, std = synth.tensor_mean_std(name, dims)
                    synth.device_normal(t.data_ptr(), t.numel(), w.seed, synth.stream_id(l, kind),
                                        0, mean, std, _DT[wdt], stream)
                d[name] = t
            self.layers.append(d)
        self.globals: Dict[str, torch.Tensor] = {}
        for name, kind, dims in synth.global_tensors(s):
            t = torch.empty(dims, dtype=_TORCH_W[wdt], device=device)
            mean, std = synth.tensor_mean_std(name, dims)
            synth.device_normal(t.data_ptr(), t.numel(), w.seed, synth.stream_id(synth.GLOBAL, kind),
                                0, mean, std, _DT[wdt], stream)
            self.globals[name] = t
        per_layer = synth.kv_pool_elems(s, w.num_pages)
        kvt = _TORCH_KV[s.kv_dtype]
        self.k_pool = torch.empty((s.num_layers, per_layer), dtype=kvt, device=device)
        self.v_pool = torch.empty((s.num_layers, per_layer), dtype=kvt, device=device)
        self.k_scale = self.v_scale = None
        ntiles = w.num_pages * s.num_kv_heads
        if s.kv_dtype == "fp8":
            self.k_scale = torch.empty((s.num_layers, ntiles), dtype=torch.float32, device=device)
            self.v_scale = torch.empty((s.num_layers, ntiles), dtype=torch.float32, device=device)
        for l in range(s.num_layers):
            for which, pool, std in (("k", self.k_pool, w.k_std), ("v", self.v_pool, w.v_std)):
                if s.kv_dtype == "fp8":
                    sc = self.k_scale if which == "k" else self.v_scale
                    synth.device_fp8_tiles(pool[l].data_ptr(), sc[l].data_ptr(), ntiles,
                                           s.tile_elems, w.seed, synth.kv_stream(l, which), 0,
                                           stream, scale=w.fp8_scale)
                else:
                    synth.device_normal(pool[l].data_ptr(), per_layer, w.seed,
                                        synth.kv_stream(l, which), 0, 0.0, std, _DT[s.kv_dtype],
                                        stream)
        if nan_unused_pages:
            self.poison_unused_pages()
        self.page_table = torch.from_numpy(w.page_table_array()).to(device)
        self.lengths = torch.tensor(w.lengths, dtype=torch.int32, device=device)

    def poison_unused_pages(self):
        """Fill every page no candidate references with NaN (e4m3 code 0x7F for fp8)."""
        s = self.w.shape
        used = torch.zeros(self.w.num_pages, dtype=torch.bool)
        used[self.w.used_pages()] = True
        unused = (~used).nonzero().flatten().to(self.device)
        tile = s.num_kv_heads * s.tile_elems
        for pool in (self.k_pool, self.v_pool):
            v = pool.view(s.num_layers, self.w.num_pages, tile)
            if s.kv_dtype == "fp8":
                v[:, unused] = 0x7F
            else:
                v[:, unused] = float("nan")

    def add_lora(self, rank: int, targets=synth.LORA_PROJECTIONS):
        """Adapter factors of every layer (bf16, packed storage like the base matrices; the
        same values the host generator gives the oracle)."""
        s = self.w.shape
        stream = torch.cuda.current_stream().cuda_stream
        self.lora_rank = rank
        self.lora_targets = tuple(targets)
        self.lora_layers: List[Dict[str, torch.Tensor]] = []
        for l in range(s.num_layers):
            d = {}
            for name, kind, dims in synth.lora_tensors(s, rank, targets):
                t = torch.empty(dims, dtype=_TORCH_W[s.weight_dtype], device=self.device)
                mean, std = synth.tensor_mean_std(name, dims)
                synth.device_normal(t.data_ptr(), t.numel(), self.w.seed, synth.stream_id(l, kind),
                                    0, mean, std, _DT[s.weight_dtype], stream)
                d[name] = t
            self.lora_layers.append(d)

    def lora_bytes(self) -> int:
        return sum(t.numel() * t.element_size() for d in self.lora_layers for t in d.values())

    def lora(self, kv):
        layers = [{p: (d[f"lora_a_{p}"].data_ptr(), d[f"lora_b_{p}"].data_ptr())
                   for p in self.lora_targets} for d in self.lora_layers]
        return kv.make_lora(layers, self.lora_rank, synth.lora_scale(self.lora_rank))

    def weight_bytes(self) -> int:
        n = sum(t.numel() * t.element_size() for d in self.layers for t in d.values())
        return n + sum(t.numel() * t.element_size() for t in self.globals.values())

    # ---- structures of the C ABI (the binding module is passed in to keep packages apart)
    def desc(self, kv):
        s = self.w.shape
        return kv.make_desc(s.num_layers, s.hidden, s.num_q_heads, s.num_kv_heads, s.head_dim,
                            s.ffn_dim, s.rope_theta, s.rms_eps, s.weight_dtype, s.kv_dtype,
                            s.page_size)

    def cache(self, kv):
        return kv.make_cache(self.k_pool.data_ptr(), self.v_pool.data_ptr(), self.w.num_pages,
                             self.k_scale.data_ptr() if self.k_scale is not None else 0,
                             self.v_scale.data_ptr() if self.v_scale is not None else 0)

    def batch(self, kv, with_hint: bool = True, lengths_host: bool = True):
        w = self.w
        return kv.make_batch(w.batch, self.page_table.data_ptr(), w.max_pages,
                             self.lengths.data_ptr(), w.lengths if lengths_host else None,
                             w.group_start if with_hint else None,
                             w.group_prefix_len if with_hint else None)

    def readout(self, kv):
        layers = [{k: t.data_ptr() for k, t in d.items()} for d in self.layers]
        g = self.globals
        return kv.make_readout(layers, g["verify_embed"].data_ptr(), g["final_norm"].data_ptr(),
                               g["reward_w"].data_ptr(), 0.0)
