"""ctypes binding of the C ABI in include/kl.h (argument marshalling only).

Every function keeps the C name.  Device buffers are passed as integer
addresses (e.g. ``tensor.data_ptr()``), streams as integer handles
(``torch.cuda.current_stream().cuda_stream``).  The library is the in-tree
``libkl.so``; importing this module fails loudly if it has not been built.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkl.so")

KL_OK = 0
KL_ERR_INVALID_ARGUMENT = -1
KL_ERR_UNSUPPORTED = -2
KL_ERR_OUT_OF_MEMORY = -3
KL_ERR_HIP = -4
KL_ERR_DEVICE_FAULT = -5

KL_MODE_PER_LAYER = 0
KL_MODE_LOOPED = 1
KL_MODE_PER_OP = 2
KL_MODE_PER_LAYER_GRAPH = 3
MODES = {"per_layer": KL_MODE_PER_LAYER, "looped": KL_MODE_LOOPED, "per_op": KL_MODE_PER_OP,
         "per_layer_graph": KL_MODE_PER_LAYER_GRAPH}

KL_DEVERR_TOKEN = 1
KL_DEVERR_POSITION = 2
KL_DEVERR_BARRIER = 4

EXPORTED = ["kl_load_model", "kl_model_create", "kl_model_set_layer", "kl_model_set_globals",
            "kl_decode_step", "kl_decode_step_noalloc", "kl_decode_greedy", "kl_kv_cache_bytes",
            "kl_get_device_error",
            "kl_get_info", "kl_set_trace", "kl_read_stream", "kl_free_model", "kl_last_error"]


class kl_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rope_theta", ctypes.c_float),
                ("rms_eps", ctypes.c_float), ("max_batch", ctypes.c_int32),
                ("max_seq", ctypes.c_int32), ("qkv_bias", ctypes.c_int32),
                ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32)]


LAYER_FIELDS = ["attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down"]
BIAS_FIELDS = ["bq", "bk", "bv"]   # only for models with Q/K/V biases
MOE_FIELDS = ["w_router"]          # only for mixtures of experts
PTR_FIELDS = LAYER_FIELDS + BIAS_FIELDS + MOE_FIELDS


class kl_layer_ptrs(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PTR_FIELDS]


class kl_weight_ptrs(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("lm_head", ctypes.c_void_p), ("layers", ctypes.POINTER(kl_layer_ptrs))]


class kl_kv_cache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("batch", ctypes.c_int32),
                ("capacity", ctypes.c_int32)]


class kl_info(ctypes.Structure):
    _fields_ = [("n_workgroups", ctypes.c_int32), ("threads_per_group", ctypes.c_int32),
                ("lds_bytes", ctypes.c_int32), ("attn_chunks_b1", ctypes.c_int32),
                ("mfma_min_batch", ctypes.c_int32),
                ("arena_bytes", ctypes.c_int64), ("scratch_bytes", ctypes.c_int64),
                ("noalloc_scratch_bytes", ctypes.c_int64),
                ("noalloc_scratch_limit", ctypes.c_int64)]


class KlError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"kl status {status}: {message}")
        self.status = status


_lib = None


def lib():
    """The loaded libkl.so (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                          "(the decode step has no fallback path)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    L.kl_load_model.argtypes = [ctypes.POINTER(kl_config), ctypes.POINTER(kl_weight_ptrs), vp,
                                ctypes.POINTER(vp)]
    L.kl_load_model.restype = i32
    L.kl_model_create.argtypes = [ctypes.POINTER(kl_config), ctypes.POINTER(vp)]
    L.kl_model_create.restype = i32
    L.kl_model_set_layer.argtypes = [vp, i32, ctypes.POINTER(kl_layer_ptrs), vp]
    L.kl_model_set_layer.restype = i32
    L.kl_model_set_globals.argtypes = [vp, vp, vp, vp, vp]
    L.kl_model_set_globals.restype = i32
    L.kl_decode_step.argtypes = [vp, vp, vp, i32, ctypes.POINTER(kl_kv_cache), vp, vp, vp, i32]
    L.kl_decode_step.restype = i32
    L.kl_decode_step_noalloc.argtypes = [vp, vp, vp, i32, ctypes.POINTER(kl_kv_cache), vp, vp, vp,
                                         i32]
    L.kl_decode_step_noalloc.restype = i32
    L.kl_decode_greedy.argtypes = [vp, vp, vp, i32, i32, ctypes.POINTER(kl_kv_cache), vp, vp, vp,
                                   i32]
    L.kl_decode_greedy.restype = i32
    L.kl_kv_cache_bytes.argtypes = [ctypes.POINTER(kl_config), i32, i32]
    L.kl_kv_cache_bytes.restype = ctypes.c_size_t
    L.kl_get_device_error.argtypes = [vp, ctypes.POINTER(i32)]
    L.kl_get_device_error.restype = i32
    L.kl_get_info.argtypes = [vp, ctypes.POINTER(kl_info)]
    L.kl_get_info.restype = i32
    L.kl_set_trace.argtypes = [vp, vp, i32]
    L.kl_set_trace.restype = i32
    L.kl_read_stream.argtypes = [vp, ctypes.c_size_t, i32, vp, vp]
    L.kl_read_stream.restype = i32
    L.kl_free_model.argtypes = [vp]
    L.kl_free_model.restype = None
    L.kl_last_error.argtypes = []
    L.kl_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def kl_last_error() -> str:
    return lib().kl_last_error().decode()


def _check(status: int) -> int:
    if status != KL_OK:
        raise KlError(status, kl_last_error())
    return status


def make_config(model: dict, max_batch: int, max_seq: int) -> kl_config:
    return kl_config(model["n_layers"], model["hidden"], model["n_heads"], model["n_kv_heads"],
                     model["head_dim"], model["ffn_dim"], model["vocab"],
                     float(model["rope_theta"]), float(model["rms_eps"]), max_batch, max_seq,
                     1 if model.get("qkv_bias") else 0, int(model.get("n_experts", 0)),
                     int(model.get("top_k", 0)))


def kl_load_model(cfg: kl_config, embed: int, final_norm: int, lm_head: int, layers: list,
                  stream: int = 0) -> int:
    """layers: list of dicts name -> device address.  Returns the state handle."""
    arr = (kl_layer_ptrs * len(layers))()
    for i, lay in enumerate(layers):
        for n in PTR_FIELDS:
            setattr(arr[i], n, lay.get(n))
    w = kl_weight_ptrs(embed, final_norm, lm_head, arr)
    out = ctypes.c_void_p()
    _check(lib().kl_load_model(ctypes.byref(cfg), ctypes.byref(w), stream, ctypes.byref(out)))
    return out.value


def kl_model_create(cfg: kl_config) -> int:
    out = ctypes.c_void_p()
    _check(lib().kl_model_create(ctypes.byref(cfg), ctypes.byref(out)))
    return out.value


def kl_model_set_layer(state: int, layer: int, ptrs: dict, stream: int = 0) -> None:
    lp = kl_layer_ptrs(*[ptrs.get(n) for n in PTR_FIELDS])
    _check(lib().kl_model_set_layer(state, layer, ctypes.byref(lp), stream))


def kl_model_set_globals(state: int, embed: int, final_norm: int, lm_head: int,
                         stream: int = 0) -> None:
    _check(lib().kl_model_set_globals(state, embed, final_norm, lm_head, stream))


def kl_decode_step(state: int, token_ids: int, positions: int, batch: int, k: int, v: int,
                   kv_batch: int, capacity: int, logits_out: int, hidden_out: int | None,
                   stream: int, mode: int) -> None:
    kv = kl_kv_cache(k, v, kv_batch, capacity)
    _check(lib().kl_decode_step(state, token_ids, positions, batch, ctypes.byref(kv), logits_out,
                                hidden_out, stream, mode))


def kl_decode_step_noalloc(state: int, token_ids: int, positions: int, batch: int, k: int,
                           v: int, kv_batch: int, capacity: int, logits_out: int,
                           hidden_out: int | None, stream: int, mode: int) -> None:
    kv = kl_kv_cache(k, v, kv_batch, capacity)
    _check(lib().kl_decode_step_noalloc(state, token_ids, positions, batch, ctypes.byref(kv),
                                        logits_out, hidden_out, stream, mode))


def kl_decode_greedy(state: int, token_ids: int, positions: int, batch: int, n_steps: int,
                     k: int, v: int, kv_batch: int, capacity: int, tokens_out: int,
                     logits_out: int, stream: int, mode: int) -> None:
    kv = kl_kv_cache(k, v, kv_batch, capacity)
    _check(lib().kl_decode_greedy(state, token_ids, positions, batch, n_steps, ctypes.byref(kv),
                                  tokens_out, logits_out, stream, mode))


def kl_kv_cache_bytes(cfg: kl_config, batch: int, capacity: int) -> int:
    return int(lib().kl_kv_cache_bytes(ctypes.byref(cfg), batch, capacity))


def kl_get_device_error(state: int) -> int:
    """Synchronizes; returns the device error word (0 = none) and clears it."""
    code = ctypes.c_int32(0)
    st = lib().kl_get_device_error(state, ctypes.byref(code))
    if st not in (KL_OK, KL_ERR_DEVICE_FAULT):
        _check(st)
    return code.value


def kl_get_info(state: int) -> kl_info:
    info = kl_info()
    _check(lib().kl_get_info(state, ctypes.byref(info)))
    return info


def kl_set_trace(state: int, dev_buffer: int | None, max_phases: int) -> None:
    _check(lib().kl_set_trace(state, dev_buffer, max_phases))


def kl_read_stream(buf: int, nbytes: int, workgroups: int, dev_out: int, stream: int) -> None:
    _check(lib().kl_read_stream(buf, nbytes, workgroups, dev_out, stream))


def kl_free_model(state: int) -> None:
    lib().kl_free_model(state)
