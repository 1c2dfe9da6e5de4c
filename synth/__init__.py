"""Seeded synthetic inputs (weights, KV cache, token ids) for the decode step.

This module holds none of the decode step's arithmetic; it only produces the
numbers both the HIP path and the oracle are fed.  The generator is the
counter-based SplitMix64 / Box-Muller scheme described in ``synth.c``; the
result does not depend on the number of threads used to fill a buffer.

Tensor ids (``stream_id``) used for one model, so that every tensor draws an
independent stream:
  16*l + {0 attn_norm, 1 wq, 2 wk, 3 wv, 4 wo, 5 ffn_norm, 6 w_gate, 7 w_up, 8 w_down}
  then 1_000_000 + {0 embed, 1 final_norm, 2 lm_head}
  then 2_000_000 + 2*(l*batch_stride + b) + {0 K, 1 V} for the KV cache.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB = os.path.join(_HERE, "libsynth.so")
_lib = None

KIND = {"attn_norm": 0, "wq": 1, "wk": 2, "wv": 3, "wo": 4,
        "ffn_norm": 5, "w_gate": 6, "w_up": 7, "w_down": 8}
GLOBAL = {"embed": 0, "final_norm": 1, "lm_head": 2}
BIAS_KIND = {"bq": 9, "bk": 10, "bv": 11}   # models with Q/K/V biases (cfg["qkv_bias"])
MOE_KIND = {"w_router": 12}                 # mixture-of-experts models (cfg["n_experts"] > 1)
WEIGHT_STD = 0.02
NORM_STD = 0.01
BIAS_STD = 0.5     # of the order of the projections themselves, so a dropped bias shows


def build() -> str:
    """Compile libsynth.so in place with gcc (OpenMP for the fill loops)."""
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-o", _LIB + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    lib.syn_normal_bf16.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                    ctypes.c_uint64, ctypes.c_double, ctypes.c_double,
                                    ctypes.c_int]
    lib.syn_normal_bf16.restype = None
    lib.syn_uniform_int32.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                      ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32]
    lib.syn_uniform_int32.restype = None
    lib.syn_uniform_f64.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                    ctypes.c_uint64]
    lib.syn_uniform_f64.restype = None
    lib.syn_word.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64]
    lib.syn_word.restype = ctypes.c_uint64
    _lib = lib
    return lib


def default_threads() -> int:
    n = os.environ.get("OMP_NUM_THREADS")
    try:
        return max(1, int(n)) if n else max(1, min(16, os.cpu_count() or 1))
    except ValueError:
        return 1


def normal_bf16(shape, seed: int, stream_id: int, mean: float = 0.0, std: float = 1.0,
                nthreads: int | None = None, out: np.ndarray | None = None) -> np.ndarray:
    """bf16 bit patterns (numpy uint16) of mean + std * N(0, 1)."""
    lib = _load()
    if out is None:
        out = np.empty(shape, dtype=np.uint16)
    assert out.dtype == np.uint16 and out.flags["C_CONTIGUOUS"]
    lib.syn_normal_bf16(out.ctypes.data, out.size, seed, stream_id, mean, std,
                        nthreads or default_threads())
    return out


def uniform_int32(n: int, seed: int, stream_id: int, lo: int, hi: int) -> np.ndarray:
    lib = _load()
    out = np.empty(n, dtype=np.int32)
    lib.syn_uniform_int32(out.ctypes.data, n, seed, stream_id, lo, hi)
    return out


def uniform_f64(n: int, seed: int, stream_id: int) -> np.ndarray:
    lib = _load()
    out = np.empty(n, dtype=np.float64)
    lib.syn_uniform_f64(out.ctypes.data, n, seed, stream_id)
    return out


def word(seed: int, stream_id: int, i: int) -> int:
    return int(_load().syn_word(seed, stream_id, i))


# --------------------------------------------------------------------------
# Whole-model inputs.  Shapes follow the nn.Linear convention [out][in].
# --------------------------------------------------------------------------

def layer_shapes(cfg) -> dict:
    H, d, nq, nkv, F = cfg["hidden"], cfg["head_dim"], cfg["n_heads"], cfg["n_kv_heads"], cfg["ffn_dim"]
    shapes = {"attn_norm": (H,), "wq": (nq * d, H), "wk": (nkv * d, H), "wv": (nkv * d, H),
              "wo": (H, nq * d), "ffn_norm": (H,), "w_gate": (F, H), "w_up": (F, H),
              "w_down": (H, F)}
    if cfg.get("qkv_bias"):
        shapes.update(bq=(nq * d,), bk=(nkv * d,), bv=(nkv * d,))
    E = cfg.get("n_experts", 0)
    if E > 1:   # E stacked expert matrices, and the router
        shapes.update(w_gate=(E * F, H), w_up=(E * F, H), w_down=(E * H, F), w_router=(E, H))
    return shapes


def layer_names(cfg) -> list:
    """The layer tensors of this model (the biases only where it has them)."""
    return (list(KIND) + (list(BIAS_KIND) if cfg.get("qkv_bias") else []) +
            (list(MOE_KIND) if cfg.get("n_experts", 0) > 1 else []))


def global_shapes(cfg) -> dict:
    return {"embed": (cfg["vocab"], cfg["hidden"]), "final_norm": (cfg["hidden"],),
            "lm_head": (cfg["vocab"], cfg["hidden"])}


def layer_tensor(cfg, seed: int, layer: int, name: str, nthreads=None, out=None) -> np.ndarray:
    shape = layer_shapes(cfg)[name]
    sid = 16 * layer + {**KIND, **BIAS_KIND, **MOE_KIND}[name]
    if name.endswith("norm"):
        return normal_bf16(shape, seed, sid, 1.0, NORM_STD, nthreads, out)
    if name in BIAS_KIND:
        return normal_bf16(shape, seed, sid, 0.0, BIAS_STD, nthreads, out)
    return normal_bf16(shape, seed, sid, 0.0, WEIGHT_STD, nthreads, out)


def global_tensor(cfg, seed: int, name: str, nthreads=None, out=None) -> np.ndarray:
    shape = global_shapes(cfg)[name]
    if name == "lm_head" and cfg.get("tie_embeddings"):
        name = "embed"   # tied: the LM head is the embedding table
    sid = 1_000_000 + GLOBAL[name]
    if name == "final_norm":
        return normal_bf16(shape, seed, sid, 1.0, NORM_STD, nthreads, out)
    return normal_bf16(shape, seed, sid, 0.0, WEIGHT_STD, nthreads, out)


def model_host(cfg, seed: int, nthreads=None) -> dict:
    """All weights of a model as numpy uint16 (bf16 bits)."""
    layers = [{k: layer_tensor(cfg, seed, l, k, nthreads) for k in layer_names(cfg)}
              for l in range(cfg["n_layers"])]
    g = {k: global_tensor(cfg, seed, k, nthreads) for k in GLOBAL if k != "lm_head"}
    # (tied: the very same array)
    g["lm_head"] = g["embed"] if cfg.get("tie_embeddings") else global_tensor(
        cfg, seed, "lm_head", nthreads)
    g["layers"] = layers
    return g


def kv_cache_host(cfg, seed: int, batch: int, capacity: int, filled, nthreads=None):
    """K and V caches [L][batch][n_kv][capacity][head_dim] bf16; slots >= filled[b] are zero."""
    L, nkv, d = cfg["n_layers"], cfg["n_kv_heads"], cfg["head_dim"]
    K = np.zeros((L, batch, nkv, capacity, d), dtype=np.uint16)
    V = np.zeros_like(K)
    tmp = np.empty((nkv, capacity, d), dtype=np.uint16)
    for l in range(L):
        for b in range(batch):
            P = int(filled[b])
            for which, dst in ((0, K), (1, V)):
                normal_bf16(tmp.shape, seed, 2_000_000 + 2 * (l * batch + b) + which,
                            0.0, 1.0, nthreads, tmp)
                dst[l, b, :, :P, :] = tmp[:, :P, :]
    return K, V


def tokens(cfg, seed: int, batch: int) -> np.ndarray:
    return uniform_int32(batch, seed, 3_000_000, 0, cfg["vocab"])
