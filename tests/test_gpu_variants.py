"""The Table 2 architecture variants against the oracle, at their layer widths
with 2 layers: Llama 3.2 3B (tied embeddings: the LM head is the embedding
table; 3 query heads per KV head), Qwen2.5-72B (Q/K/V biases), and the
tiny model with biases; the per-sequence and the matrix-core paths, all
schedules bit-identical."""
import numpy as np
import pytest

from synth.workloads import LLAMA3B, LLAMA8B, QWEN72B, TINY
from tests.gpu_cases import MODES, Case, assert_bit_exact, check_against_oracle, say

pytestmark = pytest.mark.gpu


def run_case(tag, cfg, batch, capacity, seed, sample=None):
    filled = (np.arange(batch, dtype=np.int32) * 41 + capacity // 3) % (capacity - 1)
    say(f"[{tag}] building")
    c = Case(cfg, batch, capacity, filled, seed=seed)
    if cfg.get("tie_embeddings"):
        assert c.weights["lm_head"] is c.weights["embed"]
    say(f"[{tag}] oracle")
    ref = c.oracle_step(nthreads=8, sample=sample)
    outs = []
    for name, mode in MODES:
        say(f"[{tag}] mode={name}")
        outs.append(c.gpu_step(mode))
    check_against_oracle(c, outs[1], ref, only=sample)
    assert_bit_exact(outs[0], outs[1], "per_layer vs looped")
    assert_bit_exact(outs[2], outs[1], "per_op vs looped")
    assert c.model.device_error() == 0
    c.model.close()


@pytest.mark.parametrize("batch", [1, 2, 8])
def test_tiny_with_qkv_bias(batch):
    run_case(f"tiny+bias B={batch}", dict(TINY, qkv_bias=True), batch, 192, 301 + batch)


@pytest.mark.parametrize("batch", [1, 4, 8])
def test_llama3b_width_tied_embeddings_group3(batch):
    run_case(f"3b-width L=2 B={batch}", dict(LLAMA3B, n_layers=2), batch, 256, 311 + batch)


@pytest.mark.parametrize("batch", [1, 2, 16])
def test_qwen72b_width_qkv_bias(batch):
    run_case(f"qwen72b-width L=2 B={batch}", dict(QWEN72B, n_layers=2), batch, 256, 321 + batch,
             sample=None if batch <= 2 else [0, 9, 15])


def test_llama8b_width_batch16_ctx8192():
    # Table 2's batch and context range: 16 sequences with 8K caches (ragged fill)
    run_case("8b-width L=2 B=16 ctx8K", dict(LLAMA8B, n_layers=2), 16, 8256, 331,
             sample=[0, 7, 15])
