"""Bytes and FLOPs of one decode step (the roofline model of the bench).

Two conventions:

* ``paper_table1`` is the paper's operation-intensity model (Sec. 1,
  Table 1): every parameter and every cached KV value is read once per
  token step; parameters are counted from the nominal model size at 2 bytes
  each and reported in GiB; FLOPs are 2 per parameter plus 4 per
  (layer, query head, head dim, cached position) for attention, times the
  batch.
* ``step_bytes`` / ``step_flops`` are the exact algorithmic counts of the
  step this library runs: all layer weights and norm gains, the final norm
  and LM head, one embedding row per sequence, the KV read over the cached
  positions, the KV write of the new slot and the fp32 logits.  The unread
  rows of the embedding table are not counted.  ``step_bytes`` divided by the
  step time is the achieved HBM bandwidth the bench reports against the
  8 TB/s peak (the "% of peak" form of Sec. 4.4).
"""
from __future__ import annotations

GIB = float(1 << 30)


def paper_table1(n_params: float, n_layers: int, n_kv_heads: int, head_dim: int,
                 n_heads: int, batch: int, context: int) -> dict:
    params_gib = n_params * 2 / GIB
    kv_gib = batch * n_layers * 2 * n_kv_heads * head_dim * 2 * context / GIB
    gflops = batch * (2 * n_params + 4 * n_layers * n_heads * head_dim * context) / 1e9
    gbytes = params_gib + kv_gib
    return dict(params_gib=params_gib, kv_gib=kv_gib, gflops=gflops, gbytes=gbytes,
                flops_per_byte=gflops / gbytes)


def active_experts(cfg, batch: int = 1) -> int:
    """Expert MLPs a step reads per layer: 1 for a dense model; with a
    mixture of experts, top_k per token, at most all of them (exact at batch
    1; an upper bound above, where tokens may share experts)."""
    E = cfg.get("n_experts", 0)
    return 1 if E <= 1 else min(E, cfg["top_k"] * batch)


def layer_weight_bytes(cfg, batch: int = 1) -> int:
    H, nq, nkv, d, F = (cfg[k] for k in ("hidden", "n_heads", "n_kv_heads", "head_dim", "ffn_dim"))
    bias = (nq + 2 * nkv) * d if cfg.get("qkv_bias") else 0   # Q/K/V biases (Qwen2.5)
    router = cfg.get("n_experts", 0) * H if cfg.get("n_experts", 0) > 1 else 0
    mlp = active_experts(cfg, batch) * 3 * H * F
    return 2 * (H * nq * d + 2 * H * nkv * d + nq * d * H + mlp + 2 * H + bias + router)


def step_bytes(cfg, batch: int, context: int) -> int:
    """Algorithmic HBM bytes of one step; ``context`` cached positions per sequence."""
    L, H, nkv, d, V = (cfg[k] for k in ("n_layers", "hidden", "n_kv_heads", "head_dim", "vocab"))
    weights = L * layer_weight_bytes(cfg, batch) + 2 * (V * H + H)
    embed_rows = batch * 2 * H
    kv_read = batch * L * 2 * nkv * d * 2 * context
    kv_write = batch * L * 2 * nkv * d * 2
    logits = batch * V * 4
    return weights + embed_rows + kv_read + kv_write + logits


def weight_macs(cfg) -> int:
    """Multiply-adds of the weight products of one step, per sequence."""
    L, H, nq, nkv, d, F, V = (cfg[k] for k in ("n_layers", "hidden", "n_heads", "n_kv_heads",
                                                 "head_dim", "ffn_dim", "vocab"))
    E = cfg.get("n_experts", 0)
    moe = (E * H + active_experts(cfg) * 3 * H * F) if E > 1 else 3 * H * F
    return L * (H * nq * d + 2 * H * nkv * d + nq * d * H + moe) + V * H


def step_flops(cfg, batch: int, context: int) -> int:
    """2 FLOPs per weight MAC per sequence plus 4 * n_heads * d * (context + 1) per layer."""
    L, nq, d = cfg["n_layers"], cfg["n_heads"], cfg["head_dim"]
    attn = L * 4 * nq * d * (context + 1)
    return batch * (2 * weight_macs(cfg) + attn)


def phase_bytes(cfg, batch: int, context: int) -> dict:
    """Algorithmic bytes of each phase of one layer (and of the classifier
    phase), as the step kernel splits the layer: q/k/v (with the attention
    norm gain), attention (the cached K/V read plus the new slot's write), O
    projection, gate/up (with the FFN norm gain), down projection."""
    H, nq, nkv, d, F, V = (cfg[k] for k in ("hidden", "n_heads", "n_kv_heads", "head_dim",
                                            "ffn_dim", "vocab"))
    bias = (nq + 2 * nkv) * d if cfg.get("qkv_bias") else 0
    ne = active_experts(cfg, batch)
    router = cfg.get("n_experts", 0) * H if cfg.get("n_experts", 0) > 1 else 0
    return {
        "qkv": 2 * (H * (nq + 2 * nkv) * d + H + bias),
        "attn": batch * 2 * nkv * d * 2 * (context + 1),
        "oproj": 2 * nq * d * H,
        "gateup": 2 * (ne * 2 * H * F + H + router),
        "down": 2 * ne * F * H,
        "head": 2 * (V * H + H) + batch * V * 4,
    }
