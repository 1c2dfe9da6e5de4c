"""The decode-step workloads, by name, with their shapes and seeds.

Shapes are Llama-style decoder-only models (the paper evaluates Llama 3.1
8B/70B decode, Table 1 and Table 2).  Weights are seeded synthetic stand-ins
for trained checkpoints; decode cost does not depend on the values.
"""
from __future__ import annotations

TINY = dict(n_layers=4, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn_dim=688,
            vocab=1024, rope_theta=10000.0, rms_eps=1e-5)
LLAMA8B = dict(n_layers=32, hidden=4096, n_heads=32, n_kv_heads=8, head_dim=128, ffn_dim=14336,
               vocab=128256, rope_theta=500000.0, rms_eps=1e-5)
LLAMA70B = dict(n_layers=80, hidden=8192, n_heads=64, n_kv_heads=8, head_dim=128, ffn_dim=28672,
                vocab=128256, rope_theta=500000.0, rms_eps=1e-5)
# Table 2's other architectures: Llama 3.2 3B (tied embeddings, 3 query heads
# per KV head) and Qwen2.5-72B (Q/K/V biases)
LLAMA3B = dict(n_layers=28, hidden=3072, n_heads=24, n_kv_heads=8, head_dim=128, ffn_dim=8192,
               vocab=128256, rope_theta=500000.0, rms_eps=1e-5, tie_embeddings=True)
QWEN72B = dict(n_layers=80, hidden=8192, n_heads=64, n_kv_heads=8, head_dim=128, ffn_dim=29568,
               vocab=152064, rope_theta=1000000.0, rms_eps=1e-6, qkv_bias=True)
# and Mixtral 8x7B: a mixture of 8 SwiGLU experts per layer, 2 per token
MIXTRAL = dict(n_layers=32, hidden=4096, n_heads=32, n_kv_heads=8, head_dim=128, ffn_dim=14336,
               vocab=32000, rope_theta=1000000.0, rms_eps=1e-5, n_experts=8, top_k=2)


def _wl(name, model, batch, context, index):
    return dict(name=name, model=dict(model), batch=batch, context=context,
                # new token sits at position = context; capacity rounded up to 64
                capacity=((context + 1 + 63) // 64) * 64,
                seed_weights=1 + 1000 * index, seed_kv=2 + 1000 * index,
                seed_tokens=3 + 1000 * index)


WORKLOADS = {
    "tiny-b1-ctx128": _wl("tiny-b1-ctx128", TINY, 1, 128, 0),
    "llama8b-b1-ctx4096": _wl("llama8b-b1-ctx4096", LLAMA8B, 1, 4096, 1),
    "llama8b-b32-ctx4096": _wl("llama8b-b32-ctx4096", LLAMA8B, 32, 4096, 2),
    "llama8b-b1-ctx65536": _wl("llama8b-b1-ctx65536", LLAMA8B, 1, 65536, 3),
    "llama70b-b1-ctx4096": _wl("llama70b-b1-ctx4096", LLAMA70B, 1, 4096, 4),
    "llama70b-b32-ctx4096": _wl("llama70b-b32-ctx4096", LLAMA70B, 32, 4096, 4),
    # Table 2 variants: other architectures, batch 8 / 16, contexts 8K / 16K
    "llama3b-b1-ctx4096": _wl("llama3b-b1-ctx4096", LLAMA3B, 1, 4096, 5),
    "qwen72b-b1-ctx4096": _wl("qwen72b-b1-ctx4096", QWEN72B, 1, 4096, 6),
    "llama8b-b8-ctx16384": _wl("llama8b-b8-ctx16384", LLAMA8B, 8, 16384, 7),
    "llama8b-b16-ctx8192": _wl("llama8b-b16-ctx8192", LLAMA8B, 16, 8192, 8),
    "mixtral-b1-ctx4096": _wl("mixtral-b1-ctx4096", MIXTRAL, 1, 4096, 9),
    # small batches (the sequences share each GEMV pass)
    "llama8b-b2-ctx4096": _wl("llama8b-b2-ctx4096", LLAMA8B, 2, 4096, 10),
    "llama8b-b4-ctx4096": _wl("llama8b-b4-ctx4096", LLAMA8B, 4, 4096, 11),
}
