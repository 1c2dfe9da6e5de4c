"""The C-ABI library: it loads, exports every declared entry point, and
rejects bad host arguments before touching the GPU (CPU only)."""
import ctypes
import os
import re

import pytest

from paper_2410_23668_amd import binding as kb
from synth.workloads import TINY, LLAMA8B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "kl.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kl_[a-z_]+)\s*\(", text)))


def test_header_declares_the_bound_entry_points():
    assert declared_symbols() == sorted(kb.EXPORTED)


def test_library_exports_every_declared_symbol():
    L = kb.lib()
    for name in declared_symbols():
        assert hasattr(L, name), name


def test_kv_cache_bytes():
    cfg = kb.make_config(LLAMA8B, 1, 4160)
    assert kb.kl_kv_cache_bytes(cfg, 1, 4160) == 32 * 1 * 8 * 4160 * 128 * 2
    assert kb.kl_kv_cache_bytes(cfg, 0, 4160) == 0
    bad = kb.make_config(dict(TINY, head_dim=96), 1, 64)
    assert kb.kl_kv_cache_bytes(bad, 1, 64) == 0


def _load(cfg, weights=None):
    out = ctypes.c_void_p()
    w = weights
    st = kb.lib().kl_load_model(ctypes.byref(cfg) if cfg is not None else None,
                                ctypes.byref(w) if w is not None else None, None,
                                ctypes.byref(out))
    return st, out.value


@pytest.mark.parametrize("over,status,msg", [
    (dict(head_dim=96), kb.KL_ERR_UNSUPPORTED, "head_dim"),
    (dict(n_heads=6, n_kv_heads=4), kb.KL_ERR_UNSUPPORTED, "multiple"),
    (dict(n_heads=6, n_kv_heads=2), kb.KL_ERR_UNSUPPORTED, "1, 2, 4 or 8"),
    (dict(hidden=260), kb.KL_ERR_UNSUPPORTED, "multiples of 8"),
    (dict(n_layers=0), kb.KL_ERR_INVALID_ARGUMENT, ">= 1"),
    (dict(rms_eps=0.0), kb.KL_ERR_INVALID_ARGUMENT, "rms_eps"),
    (dict(rope_theta=float("nan")), kb.KL_ERR_INVALID_ARGUMENT, "rope_theta"),
])
def test_load_model_rejects_bad_configs_before_any_hip_call(over, status, msg):
    cfg = kb.make_config(dict(TINY, **over), 1, 256)
    st, handle = _load(cfg)
    assert st == status and handle is None
    assert msg in kb.kl_last_error()


def test_load_model_rejects_null_arguments():
    st, _ = _load(None)
    assert st == kb.KL_ERR_INVALID_ARGUMENT
    cfg = kb.make_config(TINY, 1, 256)
    st, _ = _load(cfg, None)
    assert st == kb.KL_ERR_INVALID_ARGUMENT and "weight" in kb.kl_last_error()
    layers = (kb.kl_layer_ptrs * TINY["n_layers"])()
    w = kb.kl_weight_ptrs(0x1000, 0x1000, 0x1000, layers)
    st, _ = _load(cfg, w)
    assert st == kb.KL_ERR_INVALID_ARGUMENT and "layer 0" in kb.kl_last_error()
    w = kb.kl_weight_ptrs(0x1001, 0x1000, 0x1000, layers)
    st, _ = _load(cfg, w)
    assert st == kb.KL_ERR_INVALID_ARGUMENT and "aligned" in kb.kl_last_error()


def test_decode_step_rejects_null_state_and_buffers():
    L = kb.lib()
    kv = kb.kl_kv_cache(0x1000, 0x1000, 1, 64)
    assert L.kl_decode_step(None, 0x1000, 0x1000, 1, ctypes.byref(kv), 0x1000, None, None,
                            kb.KL_MODE_LOOPED) == kb.KL_ERR_INVALID_ARGUMENT
    # argument checks that precede any use of the state
    fake_state = ctypes.create_string_buffer(4096)
    addr = ctypes.addressof(fake_state)
    assert L.kl_decode_step(addr, None, 0x1000, 1, ctypes.byref(kv), 0x1000, None, None,
                            kb.KL_MODE_LOOPED) == kb.KL_ERR_INVALID_ARGUMENT
    bad_kv = kb.kl_kv_cache(0x1008, 0x1000, 1, 64)
    assert L.kl_decode_step(addr, 0x1000, 0x1000, 1, ctypes.byref(bad_kv), 0x1000, None, None,
                            kb.KL_MODE_LOOPED) == kb.KL_ERR_INVALID_ARGUMENT
    assert "16-byte" in kb.kl_last_error()
    assert L.kl_decode_step(addr, 0x1002, 0x1000, 1, ctypes.byref(kv), 0x1000, None, None,
                            kb.KL_MODE_LOOPED) == kb.KL_ERR_INVALID_ARGUMENT


def test_get_info_and_error_reject_null():
    info = kb.kl_info()
    assert kb.lib().kl_get_info(None, ctypes.byref(info)) == kb.KL_ERR_INVALID_ARGUMENT
    code = ctypes.c_int32()
    assert kb.lib().kl_get_device_error(None, ctypes.byref(code)) == kb.KL_ERR_INVALID_ARGUMENT
    kb.lib().kl_free_model(None)   # no-op


@pytest.mark.parametrize("buf,nbytes,wg,out,msg", [
    (None, 1024, 256, 64, "null"),
    (4096, 1024, 256, None, "null"),
    (4100, 1024, 256, 64, "multiples of 16"),
    (4096, 1000, 256, 64, "multiples of 16"),
    (4096, 1024, 0, 64, "workgroups"),
    (4096, 1024, 65537, 64, "workgroups"),
])
def test_read_stream_rejects_bad_arguments_before_any_hip_call(buf, nbytes, wg, out, msg):
    st = kb.lib().kl_read_stream(buf, nbytes, wg, out, None)
    assert st == kb.KL_ERR_INVALID_ARGUMENT
    assert msg in kb.lib().kl_last_error().decode()
