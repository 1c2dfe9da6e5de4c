"""Device-memory plumbing around the C ABI (torch is used only to allocate
device buffers and to name the stream).  Every step of the decode path runs
in libkl.so."""
from __future__ import annotations

import numpy as np
import torch

from . import binding as kb


def _dev_u16(a, device) -> torch.Tensor:
    """Host bf16 bit patterns (uint16) -> device int16 tensor with the same bits
    (a device tensor of 16-bit values is taken as it is)."""
    if isinstance(a, torch.Tensor):
        assert a.element_size() == 2 and a.is_contiguous()
        return a.view(torch.int16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device)


def stream_handle(stream: torch.cuda.Stream | None = None) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


class GpuModel:
    """A model loaded into libkl's packed arena."""

    def __init__(self, model_cfg: dict, weights: dict, max_batch: int, max_seq: int,
                 device="cuda", stream: torch.cuda.Stream | None = None):
        if not torch.cuda.is_available():
            raise RuntimeError("GpuModel needs a GPU")
        self.model_cfg = dict(model_cfg)
        self.device = torch.device(device)
        self.cfg = kb.make_config(model_cfg, max_batch, max_seq)
        self.max_batch, self.max_seq = max_batch, max_seq
        src = {}
        layers = []
        for l, lay in enumerate(weights["layers"]):
            ptrs = {}
            for n in kb.PTR_FIELDS:
                if n not in lay:
                    continue
                t = _dev_u16(lay[n], self.device)
                src[(l, n)] = t
                ptrs[n] = t.data_ptr()
            layers.append(ptrs)
        g = {n: _dev_u16(weights[n], self.device) for n in ("embed", "final_norm", "lm_head")}
        torch.cuda.synchronize(self.device)
        self.state = kb.kl_load_model(self.cfg, g["embed"].data_ptr(), g["final_norm"].data_ptr(),
                                      g["lm_head"].data_ptr(), layers, stream_handle(stream))
        del src, g   # kl_load_model copied and repacked everything

    @classmethod
    def from_layers(cls, model_cfg: dict, layer_fn, globals_fn, max_batch: int, max_seq: int,
                    device="cuda", stream: torch.cuda.Stream | None = None) -> "GpuModel":
        """Load one layer at a time (kl_model_create + kl_model_set_layer): only
        one layer's source weights are on the device at once.  layer_fn(l) and
        globals_fn() return host bf16 arrays by name (as in model_host)."""
        if not torch.cuda.is_available():
            raise RuntimeError("GpuModel needs a GPU")
        self = cls.__new__(cls)
        self.model_cfg = dict(model_cfg)
        self.device = torch.device(device)
        self.cfg = kb.make_config(model_cfg, max_batch, max_seq)
        self.max_batch, self.max_seq = max_batch, max_seq
        self.state = kb.kl_model_create(self.cfg)
        h = stream_handle(stream)
        for l in range(model_cfg["n_layers"]):
            lay = layer_fn(l)
            src = {n: _dev_u16(lay[n], self.device)
                   for n in kb.PTR_FIELDS if n in lay}
            torch.cuda.synchronize(self.device)
            kb.kl_model_set_layer(self.state, l, {n: t.data_ptr() for n, t in src.items()}, h)
            del src, lay
        g = globals_fn()
        src = {n: _dev_u16(g[n], self.device) for n in ("embed", "final_norm", "lm_head")}
        torch.cuda.synchronize(self.device)
        kb.kl_model_set_globals(self.state, src["embed"].data_ptr(), src["final_norm"].data_ptr(),
                                src["lm_head"].data_ptr(), h)
        del src, g
        return self

    def info(self) -> kb.kl_info:
        return kb.kl_get_info(self.state)

    def device_error(self) -> int:
        return kb.kl_get_device_error(self.state)

    def step(self, tokens: torch.Tensor, positions: torch.Tensor, kv: "KvCache",
             logits: torch.Tensor, hidden: torch.Tensor | None, mode: int,
             stream: torch.cuda.Stream | None = None) -> None:
        assert tokens.dtype == torch.int32 and positions.dtype == torch.int32
        assert logits.dtype == torch.float32 and logits.is_contiguous()
        B = tokens.numel()
        assert logits.shape == (B, self.model_cfg["vocab"])
        if hidden is not None:
            assert hidden.dtype == torch.float32 and hidden.shape == (B, self.model_cfg["hidden"])
        kb.kl_decode_step(self.state, tokens.data_ptr(), positions.data_ptr(), B,
                          kv.k.data_ptr(), kv.v.data_ptr(), kv.batch, kv.capacity,
                          logits.data_ptr(), hidden.data_ptr() if hidden is not None else None,
                          stream_handle(stream), mode)

    def greedy(self, tokens: torch.Tensor, positions: torch.Tensor, kv: "KvCache", n_steps: int,
               tokens_out: torch.Tensor, logits: torch.Tensor, mode: int,
               stream: torch.cuda.Stream | None = None) -> None:
        assert tokens.dtype == torch.int32 and positions.dtype == torch.int32
        B = tokens.numel()
        assert tokens_out.dtype == torch.int32 and tokens_out.shape == (n_steps, B)
        assert logits.dtype == torch.float32 and logits.shape == (B, self.model_cfg["vocab"])
        kb.kl_decode_greedy(self.state, tokens.data_ptr(), positions.data_ptr(), B, n_steps,
                            kv.k.data_ptr(), kv.v.data_ptr(), kv.batch, kv.capacity,
                            tokens_out.data_ptr(), logits.data_ptr(), stream_handle(stream), mode)

    def close(self):
        if getattr(self, "state", None):
            kb.kl_free_model(self.state)
            self.state = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class KvCache:
    """K and V caches [L][batch][n_kv][capacity][d] bf16 (as int16 tensors)."""

    def __init__(self, model_cfg: dict, batch: int, capacity: int, device="cuda",
                 k_host: np.ndarray | None = None, v_host: np.ndarray | None = None):
        shape = (model_cfg["n_layers"], batch, model_cfg["n_kv_heads"], capacity,
                 model_cfg["head_dim"])
        self.batch, self.capacity = batch, capacity
        if k_host is not None:
            assert k_host.shape == shape and v_host.shape == shape
            self.k = _dev_u16(k_host, device)
            self.v = _dev_u16(v_host, device)
        else:
            self.k = torch.zeros(shape, dtype=torch.int16, device=device)
            self.v = torch.zeros(shape, dtype=torch.int16, device=device)

    def host(self):
        return (self.k.cpu().numpy().view(np.uint16), self.v.cpu().numpy().view(np.uint16))
