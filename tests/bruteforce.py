"""An independent, vectorised fp64 evaluation of a small decode step.

Used only to pin the oracle.  It is written from the mathematics, not from the
oracle's code: bf16 decoding and encoding go through torch's bfloat16 type,
RoPE is a complex rotation z * exp(i * pos * w), attention is a matrix product
over KV heads expanded with np.repeat, softmax and the logistic function come
from scipy, and RMSNorm uses the Euclidean norm.
"""
from __future__ import annotations

import numpy as np
import scipy.special
import torch


def bf16_decode(h: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(h, dtype=np.uint16).view(np.int16))
    return t.view(torch.bfloat16).to(torch.float64).numpy()


def bf16_encode(x: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def rms_normalise(x, gain, eps):
    n = x.shape[-1]
    rms = np.sqrt((np.linalg.norm(x) ** 2) / n + eps)
    return x / rms * gain


def rotate(heads: np.ndarray, pos: int, theta: float) -> np.ndarray:
    """heads: [n, d]; pairs (i, i + d/2) rotated as complex numbers."""
    n, d = heads.shape
    half = d // 2
    z = heads[:, :half] + 1j * heads[:, half:]
    w = theta ** (-np.arange(half) * 2.0 / d)
    z = z * np.exp(1j * pos * w)[None, :]
    return np.concatenate([z.real, z.imag], axis=1)


def decode_step(cfg, model, tokens, positions, K, V):
    """Returns (logits, hidden) and updates K, V ([L][B][nkv][cap][d] bf16) in place."""
    L, H, nq, nkv, d, F = (cfg[k] for k in ("n_layers", "hidden", "n_heads", "n_kv_heads",
                                              "head_dim", "ffn_dim"))
    eps, theta = cfg["rms_eps"], cfg["rope_theta"]
    dec = {}

    def W(l, name):
        key = (l, name)
        if key not in dec:
            src = model["layers"][l][name] if l is not None else model[name]
            dec[key] = bf16_decode(src)
        return dec[key]

    logits, hidden = [], []
    for b, (t, p) in enumerate(zip(tokens, positions)):
        x = bf16_decode(model["embed"])[t].copy()
        for l in range(L):
            u = rms_normalise(x, W(l, "attn_norm"), eps)
            lay = model["layers"][l]
            bias = {n: (W(l, n) if n in lay else 0.0) for n in ("bq", "bk", "bv")}
            q = rotate((W(l, "wq") @ u + bias["bq"]).reshape(nq, d), p, theta)
            k = rotate((W(l, "wk") @ u + bias["bk"]).reshape(nkv, d), p, theta)
            v = (W(l, "wv") @ u + bias["bv"]).reshape(nkv, d)
            K[l, b, :, p, :] = bf16_encode(k)
            V[l, b, :, p, :] = bf16_encode(v)
            Kd = np.repeat(bf16_decode(K[l, b, :, : p + 1, :]), nq // nkv, axis=0)  # [nq, p+1, d]
            Vd = np.repeat(bf16_decode(V[l, b, :, : p + 1, :]), nq // nkv, axis=0)
            scores = np.einsum("hd,hjd->hj", q, Kd) / np.sqrt(d)
            o = np.einsum("hj,hjd->hd", scipy.special.softmax(scores, axis=1), Vd)
            x = x + W(l, "wo") @ o.reshape(-1)
            u = rms_normalise(x, W(l, "ffn_norm"), eps)
            E = cfg.get("n_experts", 0)
            if E > 1:
                # mixture of experts: the top_k router logits (stable sort: the
                # lowest index first among equal ones), softmax over them
                r = W(l, "w_router") @ u
                top = np.argsort(-r, kind="stable")[: cfg["top_k"]]
                wts = scipy.special.softmax(r[top])
                Fd = F
                for e, we in zip(top, wts):
                    g = W(l, "w_gate")[e * Fd:(e + 1) * Fd] @ u
                    m = g * scipy.special.expit(g) * (W(l, "w_up")[e * Fd:(e + 1) * Fd] @ u)
                    x = x + we * (W(l, "w_down")[e * H:(e + 1) * H] @ m)
            else:
                g = W(l, "w_gate") @ u
                m = g * scipy.special.expit(g) * (W(l, "w_up") @ u)
                x = x + W(l, "w_down") @ m
        hidden.append(x)
        logits.append(W(None, "lm_head") @ rms_normalise(x, W(None, "final_norm"), eps))
    return np.array(logits), np.array(hidden)
