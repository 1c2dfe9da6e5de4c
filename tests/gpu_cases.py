"""Shared set-up for the GPU parity tests: seeded inputs, the HIP step through
the C ABI, and the oracle on the same inputs."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import synth
from paper_2410_23668_amd import binding as kb
from paper_2410_23668_amd.device import GpuModel, KvCache

REL_L2_TOL = 1e-2      # tolerance of the decode step (bf16 weights/KV, fp32 accumulation)


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


class Case:
    """One model + KV cache + step inputs, on host (for the oracle) and GPU."""

    def __init__(self, model_cfg, batch, capacity, filled, seed=11, max_batch=None,
                 max_seq=None, nthreads=None, tokens=None):
        self.cfg = dict(model_cfg)
        self.batch, self.capacity = batch, capacity
        self.filled = np.asarray(filled, dtype=np.int32)
        self.weights = synth.model_host(self.cfg, seed, nthreads)
        self.K0, self.V0 = synth.kv_cache_host(self.cfg, seed + 1, batch, capacity, self.filled,
                                               nthreads)
        self.tokens = (synth.tokens(self.cfg, seed + 2, batch) if tokens is None
                       else np.asarray(tokens, dtype=np.int32))
        self.positions = self.filled.copy()          # the new token sits at slot P
        self.model = GpuModel(self.cfg, self.weights, max_batch or batch,
                              max_seq or capacity)

    def gpu_step(self, mode, positions=None, tokens=None, kv=None, with_hidden=True):
        B = self.batch
        kv = kv or KvCache(self.cfg, B, self.capacity, k_host=self.K0, v_host=self.V0)
        toks = torch.from_numpy(self.tokens if tokens is None else tokens).cuda()
        pos = torch.from_numpy(self.positions if positions is None else positions).cuda()
        logits = torch.full((B, self.cfg["vocab"]), float("nan"), device="cuda")
        hidden = (torch.full((B, self.cfg["hidden"]), float("nan"), device="cuda")
                  if with_hidden else None)
        self.model.step(toks, pos, kv, logits, hidden, mode)
        torch.cuda.synchronize()
        K, V = kv.host()
        return (logits.cpu().numpy(), hidden.cpu().numpy() if with_hidden else None, K, V)

    def oracle_step(self, nthreads=1, positions=None, tokens=None):
        K, V = self.K0.copy(), self.V0.copy()
        lg, hd = oracle.decode_step(self.cfg, self.weights,
                                    self.tokens if tokens is None else tokens,
                                    self.positions if positions is None else positions,
                                    K, V, nthreads=nthreads)
        return lg, hd, K, V


def bf16_rel_l2(a_u16, b_u16):
    a = oracle.bf16_to_f64(a_u16)
    b = oracle.bf16_to_f64(b_u16)
    return oracle.rel_l2(a, b)


def check_against_oracle(case: Case, got, ref, positions=None):
    """Per-sequence rel L2 on logits and hidden; written KV slots within the
    tolerance; every other KV slot untouched."""
    lg, hd, K, V = got
    rl, rh, RK, RV = ref
    pos = case.positions if positions is None else positions
    errs = {}
    for b in range(case.batch):
        errs[f"logits[{b}]"] = oracle.rel_l2(lg[b], rl[b])
        if hd is not None:
            errs[f"hidden[{b}]"] = oracle.rel_l2(hd[b], rh[b])
        p = int(pos[b])
        errs[f"k_slot[{b}]"] = bf16_rel_l2(K[:, b, :, p], RK[:, b, :, p])
        errs[f"v_slot[{b}]"] = bf16_rel_l2(V[:, b, :, p], RV[:, b, :, p])
        mask = np.ones(K.shape[3], dtype=bool)
        mask[p] = False
        assert np.array_equal(K[:, b, :, mask], case.K0[:, b, :, mask]), "K slot written outside p"
        assert np.array_equal(V[:, b, :, mask], case.V0[:, b, :, mask]), "V slot written outside p"
    say("  errors: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for k, v in errs.items():
        assert v <= REL_L2_TOL, f"{k}: rel L2 {v:.3e} > {REL_L2_TOL}"
    assert np.isfinite(lg).all()
    return errs


def assert_bit_exact(a, b, what=""):
    for x, y, name in zip(a, b, ("logits", "hidden", "K", "V")):
        if x is None and y is None:
            continue
        assert np.array_equal(np.asarray(x).view(np.uint8), np.asarray(y).view(np.uint8)), \
            f"{what}: {name} differs between modes"


MODES = [("per_layer", kb.KL_MODE_PER_LAYER), ("looped", kb.KL_MODE_LOOPED),
         ("per_op", kb.KL_MODE_PER_OP)]
