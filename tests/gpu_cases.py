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
# Element-wise bound beside the rel-L2 contract: |gpu - ref| <= ELEM_TOL * max|ref| per
# vector.  The rel-L2 norm alone would pass a few wholly wrong elements in a long vector
# (one wrong 8-row group of a 128256-row LM head is rel L2 ~ 0.008); the measured
# element errors are ~1e-6 of the vector's largest magnitude (32 layers, fp32
# accumulation), so 1e-3 leaves a wide margin and still fails any wrong row.
ELEM_TOL = 1e-3
BF16_ULP = 2.0 ** -7   # relative spacing of bf16 values: two roundings may differ by one step


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

    def oracle_step(self, nthreads=1, positions=None, tokens=None, sample=None):
        """The oracle on the same inputs.  With 'sample', only those sequences
        are evaluated (each on its own: sequences of a step are independent);
        the others' logits and hidden rows are NaN and their caches unchanged."""
        toks = self.tokens if tokens is None else np.asarray(tokens, dtype=np.int32)
        pos = self.positions if positions is None else np.asarray(positions, dtype=np.int32)
        K, V = self.K0.copy(), self.V0.copy()
        if sample is None:
            lg, hd = oracle.decode_step(self.cfg, self.weights, toks, pos, K, V,
                                        nthreads=nthreads)
            return lg, hd, K, V
        lg = np.full((self.batch, self.cfg["vocab"]), np.nan)
        hd = np.full((self.batch, self.cfg["hidden"]), np.nan)
        for b in sample:
            Kb, Vb = K[:, b:b + 1].copy(), V[:, b:b + 1].copy()
            l1, h1 = oracle.decode_step(self.cfg, self.weights, toks[b:b + 1], pos[b:b + 1],
                                        Kb, Vb, nthreads=nthreads)
            lg[b], hd[b] = l1[0], h1[0]
            K[:, b:b + 1], V[:, b:b + 1] = Kb, Vb
        return lg, hd, K, V


def bf16_rel_l2(a_u16, b_u16):
    a = oracle.bf16_to_f64(a_u16)
    b = oracle.bf16_to_f64(b_u16)
    return oracle.rel_l2(a, b)


def elem_err(a, ref, ulp=0.0) -> float:
    """max_i (|a_i - ref_i| - ulp |ref_i|) / max_i |ref_i| over one vector (fp64):
    the element-wise error in units of the vector's largest magnitude, beyond
    ulp relative rounding steps."""
    a = np.asarray(a, dtype=np.float64).ravel()
    r = np.asarray(ref, dtype=np.float64).ravel()
    scale = np.abs(r).max()
    if not np.isfinite(a).all():
        return float("inf")
    excess = np.abs(a - r) - ulp * np.abs(r)
    return float(max(excess.max(), 0.0) / (scale if scale > 0 else 1.0))


def check_vectors(errs: dict, elem: dict) -> None:
    say("  rel L2: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    say("  elem:   " + ", ".join(f"{k}={v:.2e}" for k, v in elem.items()))
    for k, v in errs.items():
        assert v <= REL_L2_TOL, f"{k}: rel L2 {v:.3e} > {REL_L2_TOL}"
    for k, v in elem.items():
        assert v <= ELEM_TOL, f"{k}: element error {v:.3e} of max|ref| > {ELEM_TOL}"


def compare_sequence(errs, elem, tag, lg, rl, hd, rh, Kp, RKp, Vp, RVp):
    """Logits, hidden state and the written K/V slots of one sequence against
    the oracle's: rel L2 and the element-wise bound (K/V within one bf16
    rounding step plus the bound)."""
    errs[f"logits{tag}"] = oracle.rel_l2(lg, rl)
    elem[f"logits{tag}"] = elem_err(lg, rl)
    if hd is not None:
        errs[f"hidden{tag}"] = oracle.rel_l2(hd, rh)
        elem[f"hidden{tag}"] = elem_err(hd, rh)
    for name, g, r in (("k_slot", Kp, RKp), ("v_slot", Vp, RVp)):
        gf, rf = oracle.bf16_to_f64(g), oracle.bf16_to_f64(r)
        errs[f"{name}{tag}"] = oracle.rel_l2(gf, rf)
        # per layer and KV head: one head vector is the unit a wrong RoPE pair
        # or a wrong row would show in
        elem[f"{name}{tag}"] = max(elem_err(gf[i, j], rf[i, j], BF16_ULP)
                                   for i in range(gf.shape[0]) for j in range(gf.shape[1]))


def check_against_oracle(case: Case, got, ref, positions=None, skip=(), only=None):
    """Per-sequence rel L2 and element-wise bound on logits and hidden; written
    KV slots within the same bounds; every other KV slot untouched.  Sequences
    in 'skip' (bad token or position) must have NaN outputs and untouched
    caches; with 'only', the other sequences are checked for untouched slots
    outside their position alone (the oracle did not evaluate them)."""
    lg, hd, K, V = got
    rl, rh, RK, RV = ref
    pos = case.positions if positions is None else positions
    errs, elem = {}, {}
    for b in range(case.batch):
        if only is not None and b not in only and b not in skip:
            p = int(pos[b])
            mask = np.ones(K.shape[3], dtype=bool)
            mask[p] = False
            assert np.array_equal(K[:, b, :, mask], case.K0[:, b, :, mask]), "K written outside p"
            assert np.array_equal(V[:, b, :, mask], case.V0[:, b, :, mask]), "V written outside p"
            assert np.isfinite(lg[b]).all()
            continue
        if b in skip:
            assert np.isnan(lg[b]).all(), "a skipped sequence's logits must be NaN"
            if hd is not None:
                assert np.isnan(hd[b]).all(), "a skipped sequence's hidden state must be NaN"
            assert np.array_equal(K[:, b], case.K0[:, b]), "a skipped sequence's K was written"
            assert np.array_equal(V[:, b], case.V0[:, b]), "a skipped sequence's V was written"
            continue
        p = int(pos[b])
        compare_sequence(errs, elem, f"[{b}]", lg[b], rl[b], None if hd is None else hd[b],
                         None if hd is None else rh[b], K[:, b, :, p], RK[:, b, :, p],
                         V[:, b, :, p], RV[:, b, :, p])
        mask = np.ones(K.shape[3], dtype=bool)
        mask[p] = False
        assert np.array_equal(K[:, b, :, mask], case.K0[:, b, :, mask]), "K slot written outside p"
        assert np.array_equal(V[:, b, :, mask], case.V0[:, b, :, mask]), "V slot written outside p"
    check_vectors(errs, elem)
    return errs


def assert_bit_exact(a, b, what=""):
    for x, y, name in zip(a, b, ("logits", "hidden", "K", "V")):
        if x is None and y is None:
            continue
        assert np.array_equal(np.asarray(x).view(np.uint8), np.asarray(y).view(np.uint8)), \
            f"{what}: {name} differs between modes"


MODES = [("per_layer", kb.KL_MODE_PER_LAYER), ("looped", kb.KL_MODE_LOOPED),
         ("per_op", kb.KL_MODE_PER_OP)]
