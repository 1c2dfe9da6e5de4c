"""Python access to the CPU oracle (test infrastructure only).

The oracle is the plain fp64 definition of one decode step (``kl_oracle.c``).
Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use it; the HIP library never imports or links it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kl_oracle.c")
_LIB = os.path.join(_HERE, "libkl_oracle.so")
_lib = None

_u16p = ctypes.POINTER(ctypes.c_uint16)
_f64p = ctypes.POINTER(ctypes.c_double)
_i32p = ctypes.POINTER(ctypes.c_int32)


class KloConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rope_theta", ctypes.c_double),
                ("rms_eps", ctypes.c_double), ("n_experts", ctypes.c_int32),
                ("top_k", ctypes.c_int32)]


LAYER_FIELDS = ["attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down"]
BIAS_FIELDS = ["bq", "bk", "bv"]   # optional (absent: no bias)
MOE_FIELDS = ["w_router"]          # mixture of experts only


class KloLayer(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in LAYER_FIELDS + BIAS_FIELDS + MOE_FIELDS]


def build() -> str:
    """Compile libkl_oracle.so in place (plain C, fp64, optional OpenMP)."""
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11", "-Wall",
           "-o", _LIB + ".tmp", _SRC, "-lm"]
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
    vp, i32, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_double
    lib.klo_bf16_to_f64.argtypes = [ctypes.c_uint16]
    lib.klo_bf16_to_f64.restype = f64
    lib.klo_f64_to_bf16.argtypes = [f64]
    lib.klo_f64_to_bf16.restype = ctypes.c_uint16
    lib.klo_bf16_to_f64_array.argtypes = [vp, vp, ctypes.c_int64]
    lib.klo_f64_to_bf16_array.argtypes = [vp, vp, ctypes.c_int64]
    lib.klo_rmsnorm.argtypes = [i32, vp, vp, f64, vp]
    lib.klo_gemv.argtypes = [i32, i32, vp, vp, vp, i32]
    lib.klo_rope.argtypes = [i32, f64, i32, vp]
    lib.klo_softmax.argtypes = [i32, vp, vp]
    lib.klo_attention.argtypes = [i32, i32, i32, i32, i32, vp, vp, vp, vp]
    lib.klo_swiglu.argtypes = [i32, vp, vp, vp]
    lib.klo_route.argtypes = [i32, i32, vp, vp, vp]
    lib.klo_decode_step.argtypes = [ctypes.POINTER(KloConfig), vp, vp, vp,
                                    ctypes.POINTER(KloLayer), i32, vp, vp, vp, vp, i32, i32,
                                    vp, vp, vp, i32]
    lib.klo_decode_step.restype = i32
    _lib = lib
    return lib


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle buffers must be C-contiguous"
    return a.ctypes.data


# ---- thin wrappers over the C functions (fp64 numpy arrays in and out) ----

def bf16_to_f64(h: np.ndarray) -> np.ndarray:
    h = np.ascontiguousarray(h, dtype=np.uint16)
    out = np.empty(h.shape, dtype=np.float64)
    _load().klo_bf16_to_f64_array(_p(h), _p(out), h.size)
    return out


def f64_to_bf16(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().klo_f64_to_bf16_array(_p(x), _p(out), x.size)
    return out


def rmsnorm(x, gain_bf16, eps):
    x = np.ascontiguousarray(x, dtype=np.float64)
    g = np.ascontiguousarray(gain_bf16, dtype=np.uint16)
    u = np.empty_like(x)
    _load().klo_rmsnorm(x.size, _p(x), _p(g), eps, _p(u))
    return u


def gemv(w_bf16, u, nthreads=1):
    w = np.ascontiguousarray(w_bf16, dtype=np.uint16)
    u = np.ascontiguousarray(u, dtype=np.float64)
    rows, cols = w.shape
    assert u.size == cols
    y = np.empty(rows, dtype=np.float64)
    _load().klo_gemv(rows, cols, _p(w), _p(u), _p(y), nthreads)
    return y


def rope(y, theta, pos):
    y = np.array(y, dtype=np.float64, copy=True)
    _load().klo_rope(y.size, theta, pos, _p(y))
    return y


def softmax(s):
    s = np.ascontiguousarray(s, dtype=np.float64)
    a = np.empty_like(s)
    _load().klo_softmax(s.size, _p(s), _p(a))
    return a


def attention(q, k_seq, v_seq, pos):
    """q: [nq][d] f64; k_seq, v_seq: [nkv][capacity][d] bf16 bits."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k_seq, dtype=np.uint16)
    v = np.ascontiguousarray(v_seq, dtype=np.uint16)
    nq, d = q.shape
    nkv, cap, d2 = k.shape
    assert d == d2 and v.shape == k.shape
    o = np.empty_like(q)
    _load().klo_attention(nq, nkv, d, pos, cap, _p(q), _p(k), _p(v), _p(o))
    return o


def swiglu(gate, up):
    g = np.ascontiguousarray(gate, dtype=np.float64)
    u = np.ascontiguousarray(up, dtype=np.float64)
    m = np.empty_like(g)
    _load().klo_swiglu(g.size, _p(g), _p(u), _p(m))
    return m


def route(logits, top_k):
    """(expert indices, weights) of the top_k largest router logits."""
    x = np.ascontiguousarray(logits, dtype=np.float64)
    idx = np.empty(top_k, dtype=np.int32)
    w = np.empty(top_k, dtype=np.float64)
    _load().klo_route(x.size, top_k, _p(x), _p(idx), _p(w))
    return idx, w


def config_struct(cfg: dict) -> KloConfig:
    return KloConfig(cfg["n_layers"], cfg["hidden"], cfg["n_heads"], cfg["n_kv_heads"],
                     cfg["head_dim"], cfg["ffn_dim"], cfg["vocab"], float(cfg["rope_theta"]),
                     float(cfg["rms_eps"]), int(cfg.get("n_experts", 0)),
                     int(cfg.get("top_k", 0)))


def decode_step(cfg: dict, model: dict, tokens, positions, kcache: np.ndarray,
                vcache: np.ndarray, nthreads: int = 1, router_out: np.ndarray | None = None):
    """One decode step.  ``model`` holds bf16 (uint16) arrays as produced by
    ``synth.model_host``; kcache/vcache ([L][kv_batch][n_kv][capacity][d]) are
    updated in place.  Returns (logits [B][V], hidden [B][H]) as float64.
    router_out ([B][L][n_experts] float64, mixture of experts) receives the
    router logits."""
    lib = _load()
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    positions = np.ascontiguousarray(positions, dtype=np.int32)
    B = tokens.size
    L, kv_batch, nkv, cap, d = kcache.shape
    assert L == cfg["n_layers"] and nkv == cfg["n_kv_heads"] and d == cfg["head_dim"]
    assert kcache.dtype == np.uint16 and vcache.dtype == np.uint16 and kcache.shape == vcache.shape
    layers = (KloLayer * L)()
    keep = []
    for l in range(L):
        for n in LAYER_FIELDS + BIAS_FIELDS + MOE_FIELDS:
            if n not in model["layers"][l]:
                continue
            a = np.ascontiguousarray(model["layers"][l][n], dtype=np.uint16)
            keep.append(a)
            setattr(layers[l], n, _p(a))
    logits = np.empty((B, cfg["vocab"]), dtype=np.float64)
    hidden = np.empty((B, cfg["hidden"]), dtype=np.float64)
    c = config_struct(cfg)
    rc = lib.klo_decode_step(ctypes.byref(c), _p(model["embed"]), _p(model["final_norm"]),
                             _p(model["lm_head"]), layers, B, _p(tokens), _p(positions),
                             _p(kcache), _p(vcache), kv_batch, cap, _p(logits), _p(hidden),
                             _p(router_out) if router_out is not None else None, nthreads)
    if rc != 0:
        raise ValueError("oracle: token or position out of range")
    return logits, hidden


def argmax(logits) -> int:
    """Greedy sampling, the Sampling block executed once per output token
    (Sec. 2, Fig. 3).  The paper does not fix the sampler; the reading is
    greedy: the index of the largest logit, the lowest such index on ties
    (numpy's argmax returns the first maximum)."""
    x = np.asarray(logits, dtype=np.float64)
    assert x.ndim == 1 and x.size > 0 and not np.isnan(x).any()
    return int(np.argmax(x))


def greedy_decode(cfg: dict, model: dict, tokens, positions, kcache: np.ndarray,
                  vcache: np.ndarray, n_steps: int, nthreads: int = 1, forced=None):
    """n_steps decode steps in a row, each feeding its sampled token to the
    next (the token loop around the step, Sec. 2, Fig. 3): step s runs at
    positions + s on the previous step's argmax (the first step on 'tokens').
    With 'forced' ([n_steps][B] tokens), step s >= 1 runs on forced[s - 1]
    instead (to follow another implementation's choices); the argmax of every
    step is still returned.  The caches are updated in place.  Returns
    (sampled [n_steps][B] int32, logits of every step [n_steps][B][V])."""
    toks = np.asarray(tokens, dtype=np.int32).copy()
    pos = np.asarray(positions, dtype=np.int32)
    B = toks.size
    sampled = np.zeros((n_steps, B), dtype=np.int32)
    all_logits = []
    for s in range(n_steps):
        lg, _ = decode_step(cfg, model, toks, pos + s, kcache, vcache, nthreads=nthreads)
        all_logits.append(lg)
        sampled[s] = [argmax(lg[b]) for b in range(B)]
        toks = (sampled[s] if forced is None else np.asarray(forced[s], dtype=np.int32)).copy()
    return sampled, np.stack(all_logits)


def rel_l2(a, ref) -> float:
    """||a - ref||_2 / ||ref||_2 in fp64."""
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(a - ref) / (den if den > 0 else 1.0))
