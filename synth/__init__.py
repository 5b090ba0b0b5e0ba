"""Seeded synthetic inputs for KV-PRM verify-token scoring.

This package is the only thing the fp64 oracle and the GPU path share. It
holds no arithmetic of the scoring method: it produces model shapes, the
per-candidate cache lengths, the scattered page tables, and the values of
every weight and cache tensor, addressed by (seed, stream, element index).

Value generation has two implementations of one definition
(``csrc/synth_host.c`` for host memory, ``csrc/synth_device.hip`` for device
memory) that agree bit for bit; see the header of ``synth_host.c``.

Workloads stand in for the paper's generator caches (Qwen3 models on math
reasoning trajectories; section 5.1): only shapes, lengths and value
statistics are reproduced, since neither the datasets nor the weights exist
here. Integer recipes (lengths, page permutations, token ids) use the same
SplitMix64 counter words, evaluated in Python.
"""
from __future__ import annotations

import ctypes
import importlib.util
import math
import os
from dataclasses import dataclass, field
from typing import Tuple, List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
HOST_LIB = os.path.join(_HERE, "libsynth_host.so")
DEVICE_LIB = os.path.join(_HERE, "libsynth_device.so")

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15

# storage dtype codes shared by both generator implementations
DT_F32, DT_BF16, DT_F64 = 0, 1, 2

# stream ids: per-layer tensors are (layer << 8) | kind
K_ATTN_NORM, K_WQ, K_WK, K_WV, K_WO, K_FFN_NORM, K_WGATE, K_WUP, K_WDOWN, K_KPOOL, K_VPOOL = range(11)
# low-rank adapter factors of projection p (LORA_PROJECTIONS order): A at K_LORA + 2p, B at
# K_LORA + 2p + 1
K_LORA = 16
GLOBAL = 0xFFFF
G_VERIFY_EMBED, G_FINAL_NORM, G_REWARD_W, G_EMBED_TABLE = range(4)
RECIPE = 0xFFFE
R_LENGTHS, R_PERM, R_TOKENS, R_SUFFIX = range(4)
ADAPTER_SEED_OFFSET = 0x100000  # weights theta' of the verify token in the mixed re-encode check


def stream_id(layer: int, kind: int) -> int:
    return (layer << 8) | kind


# --------------------------------------------------------------------------------------------
# integer counter words (Python twin of synth_words in synth_host.c)


def _mix(z: int) -> int:
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def key(seed: int, stream: int) -> int:
    return _mix((_mix((seed + GAMMA) & MASK64) + stream * GAMMA) & MASK64)


def word(k: int, n: int) -> int:
    return _mix((k + (n + 1) * GAMMA) & MASK64)


def uniform_int(k: int, n: int, lo: int, hi: int) -> int:
    """Integer in [lo, hi] from word n: lo + floor(u53 * (hi - lo + 1) / 2^53)."""
    u = word(k, n) >> 11
    return lo + (u * (hi - lo + 1)) // (1 << 53)


def permutation(seed: int, stream: int, n: int) -> List[int]:
    """Fisher-Yates shuffle of range(n) driven by counter words."""
    k = key(seed, stream)
    p = list(range(n))
    c = 0
    for i in range(n - 1, 0, -1):
        j = uniform_int(k, c, 0, i)
        c += 1
        p[i], p[j] = p[j], p[i]
    return p


# --------------------------------------------------------------------------------------------
# value generation (ctypes over the two C implementations)

_host = None
_dev = None


def _load_host():
    global _host
    if _host is None:
        if not os.path.exists(HOST_LIB):
            raise RuntimeError(f"{HOST_LIB} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(HOST_LIB)
        lib.synth_fill_normal.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                          ctypes.c_uint64, ctypes.c_int64, ctypes.c_double,
                                          ctypes.c_double, ctypes.c_int]
        lib.synth_fill_normal.restype = None
        lib.synth_fill_fp8_tiles.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                             ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint64,
                                             ctypes.c_int64, ctypes.c_int]
        lib.synth_fill_fp8_tiles.restype = None
        lib.synth_words.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                    ctypes.c_uint64, ctypes.c_int64]
        lib.synth_words.restype = None
        _host = lib
    return _host


def _preload_hip_runtime():
    """Bind the device generator to the HIP runtime torch ships with (when installed), so that a
    process holds one runtime and torch's memory and streams are valid in the generator."""
    spec = importlib.util.find_spec("torch")
    for d in (spec.submodule_search_locations or []) if spec else []:
        rt = os.path.join(d, "lib", "libamdhip64.so")
        if os.path.exists(rt):
            ctypes.CDLL(rt, mode=ctypes.RTLD_GLOBAL)
            return


def _load_dev():
    global _dev
    if _dev is None:
        _preload_hip_runtime()
        if not os.path.exists(DEVICE_LIB):
            raise RuntimeError(f"{DEVICE_LIB} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(DEVICE_LIB)
        lib.synth_dev_fill_normal.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                              ctypes.c_uint64, ctypes.c_int64, ctypes.c_double,
                                              ctypes.c_double, ctypes.c_int, ctypes.c_void_p]
        lib.synth_dev_fill_normal.restype = ctypes.c_int
        lib.synth_dev_fill_fp8_tiles.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                                 ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint64,
                                                 ctypes.c_int64, ctypes.c_int, ctypes.c_void_p]
        lib.synth_dev_fill_fp8_tiles.restype = ctypes.c_int
        _dev = lib
    return _dev


_NP_OF = {DT_F32: np.float32, DT_BF16: np.uint16, DT_F64: np.float64}


def host_normal(n: int, seed: int, stream: int, offset: int = 0, mean: float = 0.0,
                std: float = 1.0, dtype: int = DT_F64) -> np.ndarray:
    """value(offset .. offset+n) in host memory (bf16 returned as raw uint16 bits)."""
    out = np.empty(n, dtype=_NP_OF[dtype])
    if n:
        _load_host().synth_fill_normal(out.ctypes.data, n, seed, stream, offset, mean, std, dtype)
    return out


# fp8 tile scales: powers of two, or amax / 448 (the largest value of a tile at the top of the
# e4m3 range; not a power of two)
FP8_SCALE_MODES = {"pow2": 0, "amax": 1}


def host_fp8_tiles(ntiles: int, tile: int, seed: int, stream: int, tile0: int = 0,
                   scale: str = "pow2"):
    """(codes uint8 [ntiles*tile], scales fp32 [ntiles]) for tiles tile0 .. tile0+ntiles."""
    codes = np.empty(ntiles * tile, dtype=np.uint8)
    scales = np.empty(ntiles, dtype=np.float32)
    if ntiles:
        _load_host().synth_fill_fp8_tiles(codes.ctypes.data, scales.ctypes.data, ntiles, tile,
                                          seed, stream, tile0, FP8_SCALE_MODES[scale])
    return codes, scales


def device_normal(ptr: int, n: int, seed: int, stream: int, offset: int = 0, mean: float = 0.0,
                  std: float = 1.0, dtype: int = DT_F32, hip_stream: int = 0) -> None:
    """Write value(offset .. offset+n) into device memory at ptr (asynchronous on hip_stream)."""
    rc = _load_dev().synth_dev_fill_normal(ptr, n, seed, stream, offset, mean, std, dtype,
                                           hip_stream)
    if rc != 0:
        raise RuntimeError(f"synth_dev_fill_normal failed with hipError {rc}")


def device_fp8_tiles(codes_ptr: int, scales_ptr: int, ntiles: int, tile: int, seed: int,
                     stream: int, tile0: int = 0, hip_stream: int = 0, scale: str = "pow2") -> None:
    rc = _load_dev().synth_dev_fill_fp8_tiles(codes_ptr, scales_ptr, ntiles, tile, seed, stream,
                                              tile0, FP8_SCALE_MODES[scale], hip_stream)
    if rc != 0:
        raise RuntimeError(f"synth_dev_fill_fp8_tiles failed with hipError {rc}")


# --------------------------------------------------------------------------------------------
# workload recipes


@dataclass(frozen=True)
class ModelShape:
    num_layers: int
    hidden: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    ffn_dim: int
    rope_theta: float = 1.0e6
    rms_eps: float = 1.0e-6
    weight_dtype: str = "bf16"  # "f32" | "bf16"
    kv_dtype: str = "bf16"  # "f32" | "bf16" | "fp8"
    page_size: int = 16

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def kv_elem_bytes(self) -> int:
        return {"f32": 4, "bf16": 2, "fp8": 1, "f64": 8}[self.kv_dtype]

    @property
    def w_elem_bytes(self) -> int:
        return {"f32": 4, "bf16": 2}[self.weight_dtype]

    @property
    def tile_elems(self) -> int:
        """Elements of one (page, kv-head) tile of K or V."""
        return self.page_size * self.head_dim


@dataclass
class Workload:
    """One synthetic scoring batch: model shape, value seeds, lengths and page table."""

    name: str
    shape: ModelShape
    seed: int
    lengths: List[int]
    page_table: List[List[int]]  # physical page ids, rows padded with -1 to max_pages
    num_pages: int
    group_start: List[int] = field(default_factory=list)  # prefix-sharing hint (may be empty)
    group_prefix_len: List[int] = field(default_factory=list)
    k_std: float = 1.0  # test variants scale K to make the softmax peaked
    v_std: float = 1.0
    fp8_scale: str = "amax"  # fp8 tile scales: "amax" (amax / 448) or "pow2" (powers of two)

    @property
    def batch(self) -> int:
        return len(self.lengths)

    @property
    def max_pages(self) -> int:
        return max([len(r) for r in self.page_table] + [1])

    def used_pages(self) -> List[int]:
        s = set()
        for b, row in enumerate(self.page_table):
            npg = -(-self.lengths[b] // self.shape.page_size)
            s.update(row[:npg])
        return sorted(s)

    def page_table_array(self) -> np.ndarray:
        mp = self.max_pages
        a = np.full((self.batch, mp), -1, dtype=np.int32)
        for b, row in enumerate(self.page_table):
            a[b, : len(row)] = row
        return a

    def unique_tokens(self) -> int:
        """Cached tokens counted once per physical page slot (shared prefix counted once)."""
        ps = self.shape.page_size
        seen = {}
        for b, row in enumerate(self.page_table):
            L = self.lengths[b]
            for i in range(-(-L // ps)):
                n = min(ps, L - i * ps)
                seen[row[i]] = max(seen.get(row[i], 0), n)
        return sum(seen.values())


# weight stream descriptions: (kind, rows, cols, is_norm_gain)
def layer_tensors(s: ModelShape):
    H, d, nq, nkv, F = s.hidden, s.head_dim, s.num_q_heads, s.num_kv_heads, s.ffn_dim
    return [
        ("attn_norm", K_ATTN_NORM, (H,)),
        ("wq", K_WQ, (nq * d, H)),
        ("wk", K_WK, (nkv * d, H)),
        ("wv", K_WV, (nkv * d, H)),
        ("wo", K_WO, (H, nq * d)),
        ("ffn_norm", K_FFN_NORM, (H,)),
        ("w_gate", K_WGATE, (F, H)),
        ("w_up", K_WUP, (F, H)),
        ("w_down", K_WDOWN, (H, F)),
    ]


def tensor_mean_std(name: str, dims) -> tuple:
    """Value statistics of the synthetic weights.

    Matrices are N(0, std = 1/sqrt(fan_in)) (fan_in = the input width, the
    second dimension of an [out, in] matrix); norm gains are 1 + 0.1 N(0, 1)
    so that a dropped gain is visible; the verify embedding is N(0, 1); the
    reward vector is N(0, 1/sqrt(H)).
    """
    if name in ("attn_norm", "ffn_norm", "final_norm"):
        return 1.0, 0.1
    if name in ("verify_embed", "embed_table"):
        return 0.0, 1.0
    if name == "reward_w":
        return 0.0, 1.0 / math.sqrt(dims[0])
    return 0.0, 1.0 / math.sqrt(dims[1])


# projections that can carry a low-rank adapter, in the order of their stream kinds
LORA_PROJECTIONS = ("q", "k", "v", "o", "gate", "up", "down")
LORA_ALPHA = 32.0  # the adapter's alpha (with rank 256 as in the paper: scale alpha / r = 0.125)


def lora_tensors(s: ModelShape, rank: int, targets: Sequence[str] = LORA_PROJECTIONS):
    """Factors of the low-rank adapters of one layer: for projection p with base matrix
    [out, in], A_p [rank, in] and B_p [out, rank], as (name, kind, dims) like layer_tensors.
    Both factors are N(0, 1/sqrt(fan_in)) (the matrix rule of tensor_mean_std), so the update
    scale * B A has entries of about scale times the base matrix's."""
    H, d, nq, nkv, F = s.hidden, s.head_dim, s.num_q_heads, s.num_kv_heads, s.ffn_dim
    dims = {"q": (nq * d, H), "k": (nkv * d, H), "v": (nkv * d, H), "o": (H, nq * d),
            "gate": (F, H), "up": (F, H), "down": (H, F)}
    out = []
    for i, p in enumerate(LORA_PROJECTIONS):
        if p in targets:
            o_, in_ = dims[p]
            out.append((f"lora_a_{p}", K_LORA + 2 * i, (rank, in_)))
            out.append((f"lora_b_{p}", K_LORA + 2 * i + 1, (o_, rank)))
    return out


def lora_scale(rank: int) -> float:
    return LORA_ALPHA / rank


def global_tensors(s: ModelShape):
    H = s.hidden
    return [
        ("verify_embed", G_VERIFY_EMBED, (H,)),
        ("final_norm", G_FINAL_NORM, (H,)),
        ("reward_w", G_REWARD_W, (H,)),
    ]


def _assign_pages(seed: int, lengths: Sequence[int], ps: int,
                  group_start: Sequence[int] = (), group_prefix_pages: Sequence[int] = ()):
    """Scatter logical pages over a pool 1.25x the unique page count (Fisher-Yates).

    Groups (candidate ranges [group_start[g], group_start[g+1])) share their first
    group_prefix_pages[g] pages; every other page is private. Pages are dealt in order:
    each group's prefix, then its members' private pages."""
    B = len(lengths)
    starts = list(group_start) if group_start else [0, B]
    pref = list(group_prefix_pages) if group_start else [0]
    first = [0] * B
    for gi in range(len(pref)):
        for b in range(starts[gi], starts[gi + 1]):
            first[b] = pref[gi]
    priv = [-(-max(L - first[b] * ps, 0) // ps) for b, L in enumerate(lengths)]
    unique = sum(pref) + sum(priv)
    num_pages = max(1, math.ceil(1.25 * unique))
    perm = permutation(seed, stream_id(RECIPE, R_PERM), num_pages)
    rows = []
    nxt = 0
    for gi in range(len(pref)):
        shared = [perm[nxt + i] for i in range(pref[gi])]
        nxt += pref[gi]
        for b in range(starts[gi], starts[gi + 1]):
            row = list(shared)
            for _ in range(priv[b]):
                row.append(perm[nxt])
                nxt += 1
            rows.append(row)
    mp = max([len(r) for r in rows] + [1])
    rows = [r + [-1] * (mp - len(r)) for r in rows]
    return rows, num_pages


TINY = ModelShape(2, 256, 4, 2, 64, 1024, weight_dtype="f32", kv_dtype="f32")
B7 = ModelShape(28, 3584, 28, 4, 128, 18944)
LARGE_FP8 = ModelShape(64, 8192, 64, 8, 128, 28672, kv_dtype="fp8")


def make_workload(name: str, shape: Optional[ModelShape] = None, batch: Optional[int] = None,
                  lengths: Optional[Sequence[int]] = None, seed: Optional[int] = None,
                  k_std: float = 1.0,
                  groups: Optional[Tuple[Sequence[int], Sequence[int]]] = None,
                  fp8_scale: str = "amax") -> Workload:
    """The five workloads of the benchmark plan, plus custom ones for tests.

    tiny_fp32    B=4, 2 layers, H=256, 4/2 heads, d_h=64, FFN 1024, fp32, L=512 each
    b7_bf16      B=16, 28 layers, H=3584, 28/4 heads, d_h=128, FFN 18944, bf16, L=4096
    ragged_32k   7B shape, B=8, L_b ~ U[16384, 32768]
    beam_prefix  7B shape, B=64, one shared 16384-token prefix + private U[512, 2048]
    large_fp8    B=16, 64 layers, H=8192, 64/8 heads, FFN 28672, bf16 weights,
                 e4m3 K/V with per-(layer, page, kv-head) scales, L_b ~ U[8192, 16384]
    fixed_32k    7B shape, B=8, every L_b = 32768 (the fixed-length point beside ragged_32k)
    custom       any shape with explicit lengths (tests); ``groups`` = (group starts, prefix
                 lengths in tokens, multiples of the page size) makes members share prefix pages

    fp8 caches get per-(layer, page, kv-head) scales amax / 448 by default (``fp8_scale``
    "pow2": the smallest power of two that fits the tile instead).
    """
    presets = {
        "tiny_fp32": (TINY, 1000),
        "b7_bf16": (B7, 1001),
        "ragged_32k": (B7, 1002),
        "beam_prefix": (B7, 1003),
        "large_fp8": (LARGE_FP8, 1004),
        "fixed_32k": (B7, 1005),
    }
    if name in presets:
        shp, sd = presets[name]
        shape = shape or shp
        seed = sd if seed is None else seed
    if shape is None or seed is None:
        raise ValueError(f"unknown workload {name!r} without explicit shape and seed")
    ps = shape.page_size
    klen = key(seed, stream_id(RECIPE, R_LENGTHS))
    groups_start: List[int] = []
    groups_prefix: List[int] = []
    if groups is not None:
        groups_start, groups_prefix = [int(x) for x in groups[0]], [int(x) for x in groups[1]]
    if lengths is not None:
        lens = [int(x) for x in lengths]
    elif name == "tiny_fp32":
        lens = [512] * (batch or 4)
    elif name == "b7_bf16":
        lens = [4096] * (batch or 16)
    elif name == "ragged_32k":
        lens = [uniform_int(klen, i, 16384, 32768) for i in range(batch or 8)]
    elif name == "beam_prefix":
        B = batch or 64
        prefix = 16384
        lens = [prefix + uniform_int(klen, i, 512, 2048) for i in range(B)]
        groups_start, groups_prefix = [0, B], [prefix]
    elif name == "large_fp8":
        lens = [uniform_int(klen, i, 8192, 16384) for i in range(batch or 16)]
    elif name == "fixed_32k":
        lens = [32768] * (batch or 8)
    else:
        raise ValueError(f"workload {name!r} needs explicit lengths")
    if groups_start:
        assert groups_start[0] == 0 and groups_start[-1] == len(lens)
        assert len(groups_prefix) == len(groups_start) - 1
        for gi, pl in enumerate(groups_prefix):
            assert pl % ps == 0
            assert all(lens[b] >= pl for b in range(groups_start[gi], groups_start[gi + 1]))
    rows, num_pages = _assign_pages(seed, lens, ps, groups_start,
                                    [pl // ps for pl in groups_prefix])
    assert fp8_scale in FP8_SCALE_MODES
    return Workload(name, shape, seed, lens, rows, num_pages, groups_start, groups_prefix,
                    k_std=k_std, fp8_scale=fp8_scale)


# Re-encode mode of the tiny workload: token ids from a 1000-word vocabulary, the verify token is
# the last word of it.
VOCAB = 1000
VERIFY_ID = 999


def token_ids(seed: int, n: int, vocab: int = VOCAB, offset: int = 0) -> List[int]:
    """Random token ids in [0, vocab) for the re-encode workload (counter words offset ..
    offset + n - 1 of the seed's token stream)."""
    k = key(seed, stream_id(RECIPE, R_TOKENS))
    return [uniform_int(k, offset + i, 0, vocab - 1) for i in range(n)]


def kv_pool_elems(shape: ModelShape, num_pages: int) -> int:
    """Elements of one layer's K (or V) pool: [num_pages][n_kv][page_size][head_dim]."""
    return num_pages * shape.num_kv_heads * shape.tile_elems


def kv_stream(layer: int, which: str) -> int:
    return stream_id(layer, K_KPOOL if which == "k" else K_VPOOL)
