"""Mixture-of-experts decode steps (the Mixtral 8x7B layer of Table 2: a router
over 8 SwiGLU experts, 2 chosen per token) against the oracle: the router's
top-k choice, the softmax weights over the chosen logits and the weighted sum
of the chosen experts' outputs.  The per-layer, looped and graph schedules are
bit-identical.  Each case first checks that the oracle's k-th and (k+1)-th
router logits lie far apart compared with the step's rounding, so the GPU's
fp32 router and the oracle's fp64 router must pick the same experts; the
choice is then checked through the outputs (a wrong expert moves the hidden
state by far more than the tolerance)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2410_23668_amd import binding as kb
from synth.workloads import MIXTRAL, TINY
from tests.gpu_cases import Case, assert_bit_exact, check_against_oracle, say
from tests.test_gpu_greedy import check_greedy, gpu_greedy

pytestmark = pytest.mark.gpu

MOE_MODES = [("per_layer", kb.KL_MODE_PER_LAYER), ("looped", kb.KL_MODE_LOOPED),
             ("per_layer_graph", kb.KL_MODE_PER_LAYER_GRAPH)]
# the router logits carry fp32 rounding of about 1e-6 of their magnitude;
# a gap of 1e-4 of the largest logit leaves the choice unambiguous
ROUTER_GAP = 1e-4


def router_gap(cfg, weights, tokens, positions, K, V) -> float:
    """Smallest gap between the k-th and (k+1)-th router logit over sequences
    and layers, relative to the largest logit of that token and layer (the
    oracle's step on copies of the caches)."""
    B = len(tokens)
    r = np.zeros((B, cfg["n_layers"], cfg["n_experts"]))
    oracle.decode_step(cfg, weights, tokens, positions, K.copy(), V.copy(), nthreads=8,
                       router_out=r)
    k = cfg["top_k"]
    s = -np.sort(-r, axis=2)
    gap = (s[:, :, k - 1] - s[:, :, k]) / np.abs(r).max(axis=2)
    return float(gap.min())


def build(tag, cfg, batch, capacity, seed):
    filled = (np.arange(batch, dtype=np.int32) * 41 + capacity // 3) % (capacity - 1)
    say(f"[{tag}] building")
    c = Case(cfg, batch, capacity, filled, seed=seed)
    gap = router_gap(cfg, c.weights, c.tokens, c.positions, c.K0, c.V0)
    say(f"[{tag}] router gap {gap:.2e}")
    assert gap > ROUTER_GAP, "the seed gives a near-tie in the router"
    return c


def run_case(tag, cfg, batch, capacity, seed):
    c = build(tag, cfg, batch, capacity, seed)
    say(f"[{tag}] oracle")
    ref = c.oracle_step(nthreads=8)
    outs = []
    for name, mode in MOE_MODES:
        say(f"[{tag}] mode={name}")
        outs.append(c.gpu_step(mode))
    check_against_oracle(c, outs[1], ref)
    assert_bit_exact(outs[0], outs[1], "per_layer vs looped")
    assert_bit_exact(outs[2], outs[1], "per_layer_graph vs looped")
    assert c.model.device_error() == 0
    c.model.close()


@pytest.mark.parametrize("batch", [1, 3, 7])
def test_tiny_four_experts_top2(batch):
    run_case(f"tiny E4 top2 B={batch}", dict(TINY, n_layers=2, n_experts=4, top_k=2), batch,
             192, 400 + batch)


def test_tiny_eight_experts_top1():
    run_case("tiny E8 top1 B=2", dict(TINY, n_layers=2, n_experts=8, top_k=1), 2, 192, 412)


def test_tiny_three_experts_top2():
    # an expert count that leaves padding rows in the router's row group
    run_case("tiny E3 top2 B=5", dict(TINY, n_layers=2, n_experts=3, top_k=2), 5, 192, 415)


@pytest.mark.parametrize("batch", [1, 4])
def test_mixtral_width(batch):
    run_case(f"mixtral-width L=2 B={batch}", dict(MIXTRAL, n_layers=2), batch, 256, 420 + batch)


def test_greedy_loop_with_experts():
    cfg = dict(TINY, n_experts=4, top_k=2)
    c = build("tiny E4 greedy B=2", cfg, 2, 192, 431)
    n_steps = 4
    got = {}
    # (the token loop runs the looped and per-layer schedules)
    for name, mode in MOE_MODES[:2]:
        say(f"[greedy E4] mode={name}")
        got[name] = gpu_greedy(c, n_steps, mode)
    toks = got["looped"][0]
    # the routing of every step the GPU took stays clear of near-ties
    K, V = c.K0.copy(), c.V0.copy()
    for s in range(n_steps):
        tk = c.tokens if s == 0 else toks[s - 1]
        pos = c.positions + s
        gap = router_gap(cfg, c.weights, tk, pos, K, V)
        assert gap > ROUTER_GAP, (s, gap)
        oracle.decode_step(cfg, c.weights, tk, pos, K, V, nthreads=8)
    check_greedy(c, n_steps, got["looped"])
    assert_bit_exact(got["per_layer"], got["looped"], "per_layer vs looped")
    assert c.model.device_error() == 0
    c.model.close()


def test_refused_batch_and_per_op():
    """The experts chosen in the gate/up phase stay in LDS for the down phase of
    the same launch on the per-sequence path: batch 8 (the matrix-core path)
    and the per-op schedule are refused before anything runs."""
    cfg = dict(TINY, n_layers=2, n_experts=4, top_k=2)
    c = Case(cfg, 8, 128, np.full(8, 20, dtype=np.int32), seed=441)
    with pytest.raises(kb.KlError) as e:
        c.gpu_step(kb.KL_MODE_LOOPED)
    assert e.value.status == kb.KL_ERR_UNSUPPORTED
    c.batch = 1
    c.tokens, c.positions = c.tokens[:1], c.positions[:1]
    c.K0, c.V0 = c.K0[:, :1].copy(), c.V0[:, :1].copy()
    with pytest.raises(kb.KlError) as e:
        c.gpu_step(kb.KL_MODE_PER_OP)
    assert e.value.status == kb.KL_ERR_UNSUPPORTED
    out = c.gpu_step(kb.KL_MODE_LOOPED)          # and the model still steps
    assert np.isfinite(out[0]).all()
    assert c.model.device_error() == 0
    c.model.close()
