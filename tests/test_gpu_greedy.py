"""Greedy token loop (kl_decode_greedy): the sampled tokens feed the next
step on the device.  Checked against the oracle's greedy loop run on the
same tokens the GPU chose (oracle.greedy_decode with forced tokens): every
sampled token is an argmax of the oracle's logits within the tolerance, and
the oracle's own argmax wherever its top two logits are further apart than
the tolerance; the sampling decision itself is checked in the kernel's
precision against the GPU's own fp32 logits; all schedules give the same
tokens and logits bit for bit."""
import numpy as np
import pytest
import torch

import oracle
from paper_2410_23668_amd import binding as kb
from paper_2410_23668_amd.device import KvCache
from synth.workloads import TINY, WORKLOADS
from tests.gpu_cases import (BF16_ULP, ELEM_TOL, MODES, Case, check_vectors,
                             compare_sequence, elem_err, say)

pytestmark = pytest.mark.gpu


def gpu_greedy(case, n_steps, mode, positions=None):
    B = case.batch
    kv = KvCache(case.cfg, B, case.capacity, k_host=case.K0, v_host=case.V0)
    toks = torch.from_numpy(case.tokens).cuda()
    pos = torch.from_numpy(case.positions if positions is None else positions).cuda()
    out = torch.full((n_steps, B), -7, dtype=torch.int32, device="cuda")
    logits = torch.full((B, case.cfg["vocab"]), float("nan"), device="cuda")
    case.model.greedy(toks, pos, kv, n_steps, out, logits, mode)
    torch.cuda.synchronize()
    K, V = kv.host()
    return out.cpu().numpy(), logits.cpu().numpy(), K, V


def check_greedy(case, n_steps, got, skip=()):
    tokens, last_logits, K, V = got
    good = [b for b in range(case.batch) if b not in skip]
    # the oracle's loop on the tokens the GPU chose (its caches follow the same path)
    Kf, Vf = case.K0[:, good].copy(), case.V0[:, good].copy()
    sampled, logits = oracle.greedy_decode(case.cfg, case.weights, case.tokens[good],
                                           case.positions[good], Kf, Vf, n_steps, nthreads=8,
                                           forced=tokens[:, good])
    exact, near = 0, 0
    for s in range(n_steps):
        for i, b in enumerate(good):
            lg = logits[s, i]
            scale = np.abs(lg).max()
            top2 = np.sort(lg)[-2:]
            gpu_tok = int(tokens[s, b])
            assert 0 <= gpu_tok < case.cfg["vocab"], (s, b, gpu_tok)
            # an argmax within the tolerance
            assert lg[gpu_tok] >= lg.max() - 2 * ELEM_TOL * scale, (s, b, gpu_tok)
            if top2[1] - top2[0] > 2 * ELEM_TOL * scale:
                assert gpu_tok == int(sampled[s, i]), (s, b, gpu_tok, int(sampled[s, i]))
                exact += 1
            else:
                near += 1
    say(f"  tokens: {exact} decided exactly, {near} near-ties within the tolerance")
    errs, elem = {}, {}
    for i, b in enumerate(good):
        # the last step's logits, and the K/V slots of every step
        p = int(case.positions[b]) + n_steps - 1
        compare_sequence(errs, elem, f"[{b}]", last_logits[b], logits[-1, i], None, None,
                         K[:, b, :, p], Kf[:, i, :, p], V[:, b, :, p], Vf[:, i, :, p])
        for s in range(n_steps - 1):
            p = int(case.positions[b]) + s
            for name, g, r in (("k", K[:, b, :, p], Kf[:, i, :, p]), ("v", V[:, b, :, p],
                                                                      Vf[:, i, :, p])):
                gf, rf = oracle.bf16_to_f64(g), oracle.bf16_to_f64(r)
                elem[f"{name}_slot[{b},{s}]"] = max(
                    elem_err(gf[l, h], rf[l, h], BF16_ULP)
                    for l in range(gf.shape[0]) for h in range(gf.shape[1]))
        # the sampling decision in the kernel's precision: the first maximum of
        # the GPU's own fp32 logits
        assert int(np.argmax(last_logits[b])) == int(tokens[-1, b])
    check_vectors(errs, elem)


@pytest.mark.parametrize("batch,n_steps", [(3, 6), (8, 3)])
def test_tiny_greedy_loop_matches_oracle_in_every_schedule(batch, n_steps):
    say(f"[greedy tiny] batch={batch} steps={n_steps}")
    filled = (np.arange(batch, dtype=np.int32) * 31 + 5) % 140
    c = Case(TINY, batch, 160, filled, seed=201 + batch)
    outs = {}
    for name, mode in MODES:
        say(f"  mode={name}")
        outs[name] = gpu_greedy(c, n_steps, mode)
        assert c.model.device_error() == 0
    for name in ("per_layer", "per_op"):
        for x, y, what in zip(outs["looped"], outs[name], ("tokens", "logits", "K", "V")):
            assert np.array_equal(np.asarray(x).view(np.uint8), np.asarray(y).view(np.uint8)), \
                f"{what}: {name} differs from looped"
    check_greedy(c, n_steps, outs["looped"])


def test_llama8b_width_greedy_loop():
    cfg = dict(WORKLOADS["llama8b-b1-ctx4096"]["model"], n_layers=2)
    say("[greedy 8b-width L=2] building")
    c = Case(cfg, 1, 320, [300], seed=211)
    got = gpu_greedy(c, 4, kb.KL_MODE_LOOPED)
    assert c.model.device_error() == 0
    check_greedy(c, 4, got)


def test_greedy_loop_skips_a_sequence_that_runs_out_of_cache():
    # sequence 1 starts 2 slots before the end of its cache: from its third
    # step on it is skipped (position error, token -1), the others go on
    say("[greedy tiny] a sequence reaching the end of its cache")
    c = Case(TINY, 3, 64, [10, 62, 30], seed=221)
    tokens, logits, K, V = gpu_greedy(c, 4, kb.KL_MODE_LOOPED)
    assert c.model.device_error() == kb.KL_DEVERR_POSITION | kb.KL_DEVERR_TOKEN
    assert (tokens[:2, 1] >= 0).all() and (tokens[2:, 1] == -1).all()
    assert np.isnan(logits[1]).all()
    check_greedy(c, 4, (tokens, logits, K, V), skip={1})
