"""Parity at the benchmarked sizes: the full 8B-shape model (32 layers) at
batch 1 with a 4096- and a 65536-position cache, and at batch 32, against the
oracle.  At batch 32 the oracle evaluates a sample of the sequences (the
sequences of a step are independent, so the oracle runs them on their own:
their tokens, positions and caches), in the launch configuration the bench
times (looped schedule, one launch per step)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2410_23668_amd import binding as kb
from paper_2410_23668_amd.device import GpuModel, KvCache
from synth.workloads import WORKLOADS
from tests.gpu_cases import REL_L2_TOL, bf16_rel_l2, say

pytestmark = pytest.mark.gpu


def run_workload(name, sample):
    wl = WORKLOADS[name]
    cfg, B, P, cap = wl["model"], wl["batch"], wl["context"], wl["capacity"]
    say(f"[{name}] generating inputs")
    weights = synth.model_host(cfg, wl["seed_weights"])
    K0, V0 = synth.kv_cache_host(cfg, wl["seed_kv"], B, cap, [P] * B)
    tokens = synth.tokens(cfg, wl["seed_tokens"], B)
    say(f"[{name}] loading")
    model = GpuModel(cfg, weights, B, cap)
    kv = KvCache(cfg, B, cap, k_host=K0, v_host=V0)
    toks = torch.from_numpy(tokens).cuda()
    pos = torch.full((B,), P, dtype=torch.int32, device="cuda")
    logits = torch.empty((B, cfg["vocab"]), device="cuda")
    hidden = torch.empty((B, cfg["hidden"]), device="cuda")
    say(f"[{name}] GPU step (looped)")
    model.step(toks, pos, kv, logits, hidden, kb.KL_MODE_LOOPED)
    torch.cuda.synchronize()
    assert model.device_error() == 0
    lg, hd = logits.cpu().numpy(), hidden.cpu().numpy()
    K, V = kv.host()
    model.close()
    del kv
    torch.cuda.empty_cache()
    errs = {}
    for b in sample:
        say(f"[{name}] oracle, sequence {b}")
        Kb, Vb = K0[:, b:b + 1].copy(), V0[:, b:b + 1].copy()
        rl, rh = oracle.decode_step(cfg, weights, tokens[b:b + 1], [P], Kb, Vb, nthreads=16)
        errs[f"logits[{b}]"] = oracle.rel_l2(lg[b], rl[0])
        errs[f"hidden[{b}]"] = oracle.rel_l2(hd[b], rh[0])
        errs[f"k_slot[{b}]"] = bf16_rel_l2(K[:, b, :, P], Kb[:, 0, :, P])
        errs[f"v_slot[{b}]"] = bf16_rel_l2(V[:, b, :, P], Vb[:, 0, :, P])
    say("  errors: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for k, v in errs.items():
        assert v <= REL_L2_TOL, f"{k}: rel L2 {v:.3e} > {REL_L2_TOL}"


def test_llama8b_batch1_ctx4096_full_model():
    run_workload("llama8b-b1-ctx4096", [0])


def test_llama8b_batch1_ctx65536_full_model():
    run_workload("llama8b-b1-ctx65536", [0])


def test_llama8b_batch32_full_model_sampled():
    run_workload("llama8b-b32-ctx4096", [0, 17, 31])
