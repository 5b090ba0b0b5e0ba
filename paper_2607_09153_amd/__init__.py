"""Python binding of libkvprm (KV-PRM verify-token scoring on MI355X).

Argument marshalling only: every step of the scoring pass runs in the HIP kernels of
``libkvprm.so``; this module maps the C structures of ``include/kvprm.h`` onto ctypes and
raises on a non-OK status. Device memory and streams are the caller's (torch tensors and
streams are the usual source; pass their ``data_ptr()`` and ``cuda_stream``).
There is no fallback: if the library is not built, importing the binding raises.
"""
from __future__ import annotations

import ctypes
import importlib.util
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvprm.so")

KVPRM_OK, KVPRM_E_INVALID, KVPRM_E_UNSUPPORTED, KVPRM_E_WORKSPACE, KVPRM_E_HIP, KVPRM_E_INTERNAL = range(6)
KVPRM_F32, KVPRM_BF16, KVPRM_FP8_E4M3 = 0, 1, 2
DTYPE_CODE = {"f32": KVPRM_F32, "bf16": KVPRM_BF16, "fp8": KVPRM_FP8_E4M3}

EXPORTED = ["kvprm_create", "kvprm_destroy", "kvprm_workspace_size", "kvprm_score",
            "kvprm_attention", "kvprm_attention_partials", "kvprm_pack_weight",
            "kvprm_workspace_size_lora", "kvprm_score_lora", "kvprm_workspace_size_ex",
            "kvprm_score_ex", "kvprm_workspace_size_grad", "kvprm_score_grad", "kvprm_steer",
            "kvprm_stream_read", "kvprm_score_static", "kvprm_pack_kv", "kvprm_last_error"]
KVPRM_KEYS, KVPRM_VALUES = 0, 1
STATIC_WORKSPACE_BYTES = 64 << 20  # KVPRM_STATIC_WORKSPACE_BYTES
LORA_PROJECTIONS = ("q", "k", "v", "o", "gate", "up", "down")


class ModelDesc(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float),
                ("weight_dtype", ctypes.c_int), ("kv_dtype", ctypes.c_int),
                ("page_size", ctypes.c_int32)]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")]


class ReadoutWeights(ctypes.Structure):
    _fields_ = [("layers", ctypes.POINTER(LayerWeights)), ("verify_embed", ctypes.c_void_p),
                ("final_norm", ctypes.c_void_p), ("reward_w", ctypes.c_void_p),
                ("reward_b", ctypes.c_float)]


class LoraFactors(ctypes.Structure):
    _fields_ = [("a", ctypes.c_void_p), ("b", ctypes.c_void_p)]


class LayerLora(ctypes.Structure):
    _fields_ = [(n, LoraFactors) for n in LORA_PROJECTIONS]


class Lora(ctypes.Structure):
    _fields_ = [("layers", ctypes.POINTER(LayerLora)), ("rank", ctypes.c_int32),
                ("scale", ctypes.c_float)]


class ScoreOptions(ctypes.Structure):
    _fields_ = [("lora", ctypes.POINTER(Lora)), ("depth", ctypes.c_int32)]


class KVCache(ctypes.Structure):
    _fields_ = [("k_pages", ctypes.c_void_p), ("v_pages", ctypes.c_void_p),
                ("k_scale", ctypes.c_void_p), ("v_scale", ctypes.c_void_p),
                ("num_pages", ctypes.c_int32)]


class Batch(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("page_table", ctypes.c_void_p),
                ("max_pages", ctypes.c_int32), ("lengths", ctypes.c_void_p),
                ("lengths_host", ctypes.POINTER(ctypes.c_int32)),
                ("num_groups", ctypes.c_int32),
                ("group_start_host", ctypes.POINTER(ctypes.c_int32)),
                ("group_prefix_len_host", ctypes.POINTER(ctypes.c_int32))]


class KvprmError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"kvprm status {status}: {msg}")
        self.status = status


def _preload_hip_runtime():
    """One HIP runtime per process: when torch is installed, load the runtime it ships with
    before this library, so that the library binds to that copy (torch's streams and memory
    are then valid here) rather than starting a second runtime beside torch's."""
    spec = importlib.util.find_spec("torch")
    for d in (spec.submodule_search_locations or []) if spec else []:
        rt = os.path.join(d, "lib", "libamdhip64.so")
        if os.path.exists(rt):
            ctypes.CDLL(rt, mode=ctypes.RTLD_GLOBAL)
            return


def _load():
    _preload_hip_runtime()
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built (run __graft_entry__.build()); "
                          "the scoring pass has no non-GPU implementation")
    lib = ctypes.CDLL(LIB_PATH)
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    lib.kvprm_create.argtypes = [ctypes.POINTER(ModelDesc), ctypes.POINTER(vp)]
    lib.kvprm_destroy.argtypes = [vp]
    lib.kvprm_workspace_size.argtypes = [vp, ctypes.POINTER(Batch), ctypes.POINTER(sz)]
    lib.kvprm_score.argtypes = [vp, ctypes.POINTER(KVCache), ctypes.POINTER(Batch),
                                ctypes.POINTER(ReadoutWeights), vp, sz, vp, vp, vp]
    lib.kvprm_attention.argtypes = [vp, ctypes.POINTER(KVCache), ctypes.POINTER(Batch),
                                    ctypes.c_int32, vp, vp, vp, vp, sz, vp, vp]
    lib.kvprm_attention_partials.argtypes = [vp, ctypes.POINTER(KVCache), ctypes.POINTER(Batch),
                                             ctypes.c_int32, vp, vp, sz, vp]
    lib.kvprm_score_static.argtypes = [vp, ctypes.POINTER(KVCache), ctypes.POINTER(Batch),
                                       ctypes.POINTER(ReadoutWeights), vp, vp, vp]
    lib.kvprm_pack_weight.argtypes = [vp, vp, ctypes.c_int64, ctypes.c_int64, vp]
    lib.kvprm_pack_kv.argtypes = [vp, vp, ctypes.c_int64, ctypes.c_int32, ctypes.c_int,
                                  ctypes.c_int, vp]
    lib.kvprm_stream_read.argtypes = [vp, sz, vp, vp]
    lib.kvprm_workspace_size_lora.argtypes = [vp, ctypes.POINTER(Batch), ctypes.c_int32,
                                              ctypes.POINTER(sz)]
    lib.kvprm_score_lora.argtypes = [vp, ctypes.POINTER(KVCache), ctypes.POINTER(Batch),
                                     ctypes.POINTER(ReadoutWeights), ctypes.POINTER(Lora), vp, sz,
                                     vp, vp, vp]
    lib.kvprm_workspace_size_ex.argtypes = [vp, ctypes.POINTER(Batch), ctypes.POINTER(ScoreOptions),
                                            ctypes.POINTER(sz)]
    lib.kvprm_score_ex.argtypes = [vp, ctypes.POINTER(KVCache), ctypes.POINTER(Batch),
                                   ctypes.POINTER(ReadoutWeights), ctypes.POINTER(ScoreOptions),
                                   vp, sz, vp, vp, vp]
    lib.kvprm_workspace_size_grad.argtypes = [vp, ctypes.POINTER(Batch), ctypes.POINTER(sz)]
    lib.kvprm_score_grad.argtypes = [vp, ctypes.POINTER(KVCache), ctypes.POINTER(Batch),
                                     ctypes.POINTER(ReadoutWeights), vp, sz, vp, vp, vp, vp]
    lib.kvprm_steer.argtypes = [vp, ctypes.POINTER(KVCache), ctypes.POINTER(Batch),
                                ctypes.POINTER(ReadoutWeights), ctypes.c_float, ctypes.c_int32, vp,
                                sz, vp, vp, vp]
    for f in ("kvprm_create", "kvprm_destroy", "kvprm_workspace_size", "kvprm_score",
              "kvprm_attention", "kvprm_attention_partials", "kvprm_pack_weight",
              "kvprm_workspace_size_lora", "kvprm_score_lora", "kvprm_workspace_size_ex",
              "kvprm_score_ex", "kvprm_workspace_size_grad", "kvprm_score_grad", "kvprm_steer",
              "kvprm_stream_read", "kvprm_score_static", "kvprm_pack_kv"):
        getattr(lib, f).restype = ctypes.c_int
    lib.kvprm_last_error.argtypes = []
    lib.kvprm_last_error.restype = ctypes.c_char_p
    return lib


lib = _load()


def _check(st: int):
    if st != KVPRM_OK:
        raise KvprmError(st, lib.kvprm_last_error().decode())


def kvprm_last_error() -> str:
    return lib.kvprm_last_error().decode()


def make_desc(num_layers, hidden, num_q_heads, num_kv_heads, head_dim, ffn_dim,
              rope_theta=1.0e6, rms_eps=1.0e-6, weight_dtype="bf16", kv_dtype="bf16",
              page_size=16) -> ModelDesc:
    return ModelDesc(num_layers, hidden, num_q_heads, num_kv_heads, head_dim, ffn_dim,
                     rope_theta, rms_eps, DTYPE_CODE[weight_dtype], DTYPE_CODE[kv_dtype],
                     page_size)


def kvprm_create(desc: ModelDesc) -> int:
    h = ctypes.c_void_p()
    _check(lib.kvprm_create(ctypes.byref(desc), ctypes.byref(h)))
    return h.value


def kvprm_destroy(handle: int) -> None:
    _check(lib.kvprm_destroy(handle))


def make_batch(batch: int, page_table_ptr: int, max_pages: int, lengths_ptr: int,
               lengths_host: Optional[Sequence[int]] = None,
               group_start: Optional[Sequence[int]] = None,
               group_prefix_len: Optional[Sequence[int]] = None) -> Batch:
    """Batch descriptor; host arrays are copied into ctypes buffers kept alive on the struct."""
    b = Batch()
    b.batch, b.page_table, b.max_pages, b.lengths = batch, page_table_ptr, max_pages, lengths_ptr
    keep = []
    if lengths_host is not None:
        arr = (ctypes.c_int32 * len(lengths_host))(*lengths_host)
        keep.append(arr)
        b.lengths_host = ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32))
    if group_start:
        gs = (ctypes.c_int32 * len(group_start))(*group_start)
        gp = (ctypes.c_int32 * len(group_prefix_len))(*group_prefix_len)
        keep += [gs, gp]
        b.num_groups = len(group_prefix_len)
        b.group_start_host = ctypes.cast(gs, ctypes.POINTER(ctypes.c_int32))
        b.group_prefix_len_host = ctypes.cast(gp, ctypes.POINTER(ctypes.c_int32))
    b._keep = keep
    return b


def make_cache(k_ptr: int, v_ptr: int, num_pages: int, k_scale_ptr: int = 0,
               v_scale_ptr: int = 0) -> KVCache:
    return KVCache(k_ptr, v_ptr, k_scale_ptr or None, v_scale_ptr or None, num_pages)


def make_readout(layers: Sequence[dict], verify_embed: int, final_norm: int, reward_w: int,
                 reward_b: float = 0.0) -> ReadoutWeights:
    """layers: per layer a dict of device pointers with the LayerWeights field names."""
    arr = (LayerWeights * len(layers))()
    for i, d in enumerate(layers):
        for name, _ in LayerWeights._fields_:
            setattr(arr[i], name, d[name])
    r = ReadoutWeights(ctypes.cast(arr, ctypes.POINTER(LayerWeights)), verify_embed, final_norm,
                       reward_w, reward_b)
    r._keep = arr
    return r


def make_lora(layers: Sequence[dict], rank: int, scale: float) -> Lora:
    """layers: per layer a dict projection -> (a_ptr, b_ptr) of device pointers; projections
    missing from the dict have no adapter."""
    arr = (LayerLora * len(layers))()
    for i, d in enumerate(layers):
        for p in LORA_PROJECTIONS:
            a, b = d.get(p, (None, None))
            setattr(arr[i], p, LoraFactors(a or None, b or None))
    r = Lora(ctypes.cast(arr, ctypes.POINTER(LayerLora)), rank, scale)
    r._keep = arr
    return r


def kvprm_workspace_size_lora(handle: int, batch: Batch, rank: int) -> int:
    n = ctypes.c_size_t()
    _check(lib.kvprm_workspace_size_lora(handle, ctypes.byref(batch), rank, ctypes.byref(n)))
    return n.value


def kvprm_score_lora(handle: int, cache: KVCache, batch: Batch, base: ReadoutWeights,
                     lora: Lora, workspace_ptr: int, ws_bytes: int, scores_ptr: int,
                     logits_ptr: int = 0, stream: int = 0) -> None:
    _check(lib.kvprm_score_lora(handle, ctypes.byref(cache), ctypes.byref(batch),
                                ctypes.byref(base), ctypes.byref(lora), workspace_ptr, ws_bytes,
                                scores_ptr, logits_ptr or None, stream or None))


def make_options(lora: Optional[Lora] = None, depth: int = 1) -> ScoreOptions:
    o = ScoreOptions(ctypes.pointer(lora) if lora is not None else None, depth)
    o._keep = lora
    return o


def kvprm_workspace_size_ex(handle: int, batch: Batch, options: Optional[ScoreOptions]) -> int:
    n = ctypes.c_size_t()
    _check(lib.kvprm_workspace_size_ex(handle, ctypes.byref(batch),
                                       ctypes.byref(options) if options is not None else None,
                                       ctypes.byref(n)))
    return n.value


def kvprm_score_ex(handle: int, cache: KVCache, batch: Batch, weights: ReadoutWeights,
                   options: Optional[ScoreOptions], workspace_ptr: int, ws_bytes: int,
                   scores_ptr: int, logits_ptr: int = 0, stream: int = 0) -> None:
    _check(lib.kvprm_score_ex(handle, ctypes.byref(cache), ctypes.byref(batch),
                              ctypes.byref(weights),
                              ctypes.byref(options) if options is not None else None,
                              workspace_ptr, ws_bytes, scores_ptr, logits_ptr or None,
                              stream or None))


def kvprm_workspace_size_grad(handle: int, batch: Batch) -> int:
    n = ctypes.c_size_t()
    _check(lib.kvprm_workspace_size_grad(handle, ctypes.byref(batch), ctypes.byref(n)))
    return n.value


def kvprm_score_grad(handle: int, cache: KVCache, batch: Batch, weights: ReadoutWeights,
                     workspace_ptr: int, ws_bytes: int, scores_ptr: int, grad_k_ptr: int,
                     grad_v_ptr: int, stream: int = 0) -> None:
    _check(lib.kvprm_score_grad(handle, ctypes.byref(cache), ctypes.byref(batch),
                                ctypes.byref(weights), workspace_ptr, ws_bytes, scores_ptr,
                                grad_k_ptr, grad_v_ptr, stream or None))


def kvprm_steer(handle: int, cache: KVCache, batch: Batch, weights: ReadoutWeights, eta: float,
                steps: int, workspace_ptr: int, ws_bytes: int, scores_before_ptr: int,
                scores_after_ptr: int, stream: int = 0) -> None:
    _check(lib.kvprm_steer(handle, ctypes.byref(cache), ctypes.byref(batch), ctypes.byref(weights),
                           eta, steps, workspace_ptr, ws_bytes, scores_before_ptr,
                           scores_after_ptr, stream or None))


def kvprm_workspace_size(handle: int, batch: Batch) -> int:
    n = ctypes.c_size_t()
    _check(lib.kvprm_workspace_size(handle, ctypes.byref(batch), ctypes.byref(n)))
    return n.value


def kvprm_score(handle: int, cache: KVCache, batch: Batch, weights: ReadoutWeights,
                workspace_ptr: int, ws_bytes: int, scores_ptr: int, logits_ptr: int = 0,
                stream: int = 0) -> None:
    _check(lib.kvprm_score(handle, ctypes.byref(cache), ctypes.byref(batch), ctypes.byref(weights),
                           workspace_ptr, ws_bytes, scores_ptr, logits_ptr or None, stream or None))


def kvprm_score_static(handle: int, cache: KVCache, batch: Batch, weights: ReadoutWeights,
                       scores_ptr: int, logits_ptr: int = 0, stream: int = 0) -> None:
    _check(lib.kvprm_score_static(handle, ctypes.byref(cache), ctypes.byref(batch),
                                  ctypes.byref(weights), scores_ptr, logits_ptr or None,
                                  stream or None))


def kvprm_stream_read(buf_ptr: int, nbytes: int, sink_ptr: int, stream: int = 0) -> None:
    _check(lib.kvprm_stream_read(buf_ptr, nbytes, sink_ptr, stream or None))


def kvprm_pack_weight(src_ptr: int, dst_ptr: int, rows: int, K: int, stream: int = 0) -> None:
    _check(lib.kvprm_pack_weight(src_ptr, dst_ptr, rows, K, stream or None))


def kvprm_pack_kv(src_ptr: int, dst_ptr: int, num_tiles: int, head_dim: int, dtype: str,
                  part: int, stream: int = 0) -> None:
    """Token-major cache tiles -> the stored K (part = KVPRM_KEYS) or V tile layout."""
    _check(lib.kvprm_pack_kv(src_ptr or None, dst_ptr or None, num_tiles, head_dim,
                             DTYPE_CODE[dtype], part, stream or None))


def kvprm_attention_partials(handle: int, cache: KVCache, batch: Batch, layer: int, q_ptr: int,
                             workspace_ptr: int, ws_bytes: int, stream: int = 0) -> None:
    _check(lib.kvprm_attention_partials(handle, ctypes.byref(cache), ctypes.byref(batch), layer,
                                        q_ptr, workspace_ptr, ws_bytes, stream or None))


def kvprm_attention(handle: int, cache: KVCache, batch: Batch, layer: int, q_ptr: int,
                    k_self_ptr: int, v_self_ptr: int, workspace_ptr: int, ws_bytes: int,
                    o_ptr: int, stream: int = 0) -> None:
    _check(lib.kvprm_attention(handle, ctypes.byref(cache), ctypes.byref(batch), layer, q_ptr,
                               k_self_ptr, v_self_ptr, workspace_ptr, ws_bytes, o_ptr,
                               stream or None))
