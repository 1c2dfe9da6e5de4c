"""Parity at the benchmarked sizes: the full 8B-shape model (32 layers) at
batch 1 with a 4096- and a 65536-position cache, at batch 4 (the sequences
sharing each GEMV pass) and at batch 32, against the oracle.  At batches 4
and 32 the oracle evaluates a sample of the sequences (the
sequences of a step are independent, so the oracle runs them on their own:
their tokens, positions and caches), in the launch configuration the bench
times (looped schedule, one launch per step).  At batch 1 with 4096 cached
positions, the per-layer and per-op schedules run too and must reproduce the
looped schedule's logits, hidden state and K/V slot writes bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2410_23668_amd import binding as kb
from paper_2410_23668_amd.device import GpuModel, KvCache
from synth.workloads import WORKLOADS
from tests.gpu_cases import check_vectors, compare_sequence, say

pytestmark = pytest.mark.gpu


def run_workload(name, sample, modes=("looped",)):
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
    outs = {}
    for m in modes:
        logits = torch.full((B, cfg["vocab"]), float("nan"), device="cuda")
        hidden = torch.full((B, cfg["hidden"]), float("nan"), device="cuda")
        # (slot P of every layer is reset before each schedule, so each one's
        # writes are seen on their own)
        kv.k[:, :, :, P].zero_()
        kv.v[:, :, :, P].zero_()
        say(f"[{name}] GPU step ({m})")
        model.step(toks, pos, kv, logits, hidden, kb.MODES[m])
        torch.cuda.synchronize()
        assert model.device_error() == 0
        outs[m] = (logits.cpu().numpy(), hidden.cpu().numpy(),
                   kv.k[:, :, :, P].cpu().numpy().view(np.uint16),
                   kv.v[:, :, :, P].cpu().numpy().view(np.uint16))
    model.close()
    del kv
    torch.cuda.empty_cache()
    for m in modes[1:]:
        for x, y, what in zip(outs[modes[0]], outs[m], ("logits", "hidden", "K slot", "V slot")):
            assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), \
                f"{what}: {m} differs from {modes[0]}"
        say(f"[{name}] {m} == {modes[0]} bit for bit")
    lg, hd, Kp, Vp = outs[modes[0]]
    errs, elem = {}, {}
    for b in sample:
        say(f"[{name}] oracle, sequence {b}")
        Kb, Vb = K0[:, b:b + 1].copy(), V0[:, b:b + 1].copy()
        rl, rh = oracle.decode_step(cfg, weights, tokens[b:b + 1], [P], Kb, Vb, nthreads=16)
        compare_sequence(errs, elem, f"[{b}]", lg[b], rl[0], hd[b], rh[0], Kp[:, b], Kb[:, 0, :, P],
                         Vp[:, b], Vb[:, 0, :, P])
    check_vectors(errs, elem)


def test_llama8b_batch1_ctx4096_full_model_all_schedules():
    run_workload("llama8b-b1-ctx4096", [0],
                 modes=("looped", "per_layer", "per_op", "per_layer_graph"))


def test_llama8b_batch1_ctx65536_full_model():
    run_workload("llama8b-b1-ctx65536", [0])


def test_llama8b_batch4_full_model_sampled_two_schedules():
    run_workload("llama8b-b4-ctx4096", [0, 3], modes=("looped", "per_layer"))


def test_llama8b_batch32_full_model_sampled():
    run_workload("llama8b-b32-ctx4096", [0, 17, 31])
