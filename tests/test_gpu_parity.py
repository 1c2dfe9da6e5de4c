"""Parity of the HIP decode step against the CPU oracle, through the C ABI.

Bar: per-sequence rel L2 <= 1e-2 on logits, hidden state and the written KV
slots (bf16 weights and KV, fp32 accumulation), every other KV slot
untouched, and all three schedules bit-identical with each other.
"""
import numpy as np
import pytest
import torch

import synth
from paper_2410_23668_amd import binding as kb
from paper_2410_23668_amd.device import GpuModel, KvCache
from synth.workloads import TINY, WORKLOADS
from tests.gpu_cases import MODES, Case, assert_bit_exact, check_against_oracle, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tiny():
    w = WORKLOADS["tiny-b1-ctx128"]
    say(f"[tiny] building case capacity={w['capacity']} P={w['context']}")
    return Case(w["model"], 1, w["capacity"], [w["context"]], seed=w["seed_weights"])


def test_tiny_all_modes_match_oracle_and_each_other(tiny):
    ref = tiny.oracle_step()
    outs = {}
    for name, mode in MODES:
        say(f"[tiny] mode={name}")
        outs[name] = tiny.gpu_step(mode)
        check_against_oracle(tiny, outs[name], ref)
    assert_bit_exact(outs["per_layer"], outs["looped"], "per_layer vs looped")
    assert_bit_exact(outs["per_op"], outs["looped"], "per_op vs looped")


def test_tiny_repeated_steps_are_deterministic(tiny):
    say("[tiny] repeat looped x3")
    a = tiny.gpu_step(kb.KL_MODE_LOOPED)
    for _ in range(2):
        assert_bit_exact(a, tiny.gpu_step(kb.KL_MODE_LOOPED), "repeat")


def test_tiny_reports_dispatch_geometry(tiny):
    info = tiny.model.info()
    assert info.n_workgroups == torch.cuda.get_device_properties(0).multi_processor_count
    assert info.threads_per_group % 64 == 0 and 64 <= info.threads_per_group <= 1024
    assert info.lds_bytes <= 160 * 1024
    assert tiny.model.device_error() == 0


@pytest.mark.parametrize("positions", [[0], [1], [127], [190], [191]])
def test_tiny_edge_positions(positions):
    # position 0 attends to one key; 191 is the last slot of the 192-slot cache
    say(f"[tiny-edge] positions={positions}")
    c = Case(TINY, 1, 192, positions, seed=21)
    ref = c.oracle_step()
    outs = [c.gpu_step(mode) for _, mode in MODES]
    check_against_oracle(c, outs[1], ref)
    assert_bit_exact(outs[0], outs[1], "per_layer vs looped")
    assert_bit_exact(outs[2], outs[1], "per_op vs looped")


def test_tiny_batch_with_ragged_positions():
    say("[tiny-batch] batch=5 ragged positions")
    c = Case(TINY, 5, 320, [0, 63, 64, 257, 319], seed=31)
    ref = c.oracle_step()
    outs = [c.gpu_step(mode) for _, mode in MODES]
    check_against_oracle(c, outs[1], ref)
    assert_bit_exact(outs[0], outs[1], "per_layer vs looped")
    assert_bit_exact(outs[2], outs[1], "per_op vs looped")


def test_tiny_batch_smaller_than_allocated():
    # the step's batch may be below max_batch and below the cache's batch extent
    say("[tiny-batch] batch 2 of max 4")
    c = Case(TINY, 4, 128, [5, 100, 17, 60], seed=41, max_batch=4)
    ref = c.oracle_step()
    kv = KvCache(c.cfg, 4, 128, k_host=c.K0, v_host=c.V0)
    toks = torch.from_numpy(c.tokens[:2]).cuda()
    pos = torch.from_numpy(c.positions[:2]).cuda()
    logits = torch.zeros((2, c.cfg["vocab"]), device="cuda")
    c.model.step(toks, pos, kv, logits, None, kb.KL_MODE_LOOPED)
    torch.cuda.synchronize()
    lg = logits.cpu().numpy()
    import oracle
    for b in range(2):
        assert oracle.rel_l2(lg[b], ref[0][b]) <= 1e-2
    K, _ = kv.host()
    assert np.array_equal(K[:, 2:], c.K0[:, 2:]), "sequences beyond the step's batch were written"


def test_device_error_bits_for_bad_token_and_position(tiny):
    # a bad token or position sets its error bit; that sequence is skipped:
    # NaN logits and hidden state, no K/V slot written
    say("[tiny] bad token and position")
    V = tiny.cfg["vocab"]
    for mode, toks, pos, bit in (
            (kb.KL_MODE_LOOPED, [V], None, kb.KL_DEVERR_TOKEN),
            (kb.KL_MODE_LOOPED, [-1], None, kb.KL_DEVERR_TOKEN),
            (kb.KL_MODE_PER_LAYER, None, [tiny.capacity], kb.KL_DEVERR_POSITION),
            (kb.KL_MODE_PER_OP, None, [-3], kb.KL_DEVERR_POSITION)):
        say(f"  mode={mode} tokens={toks} positions={pos}")
        got = tiny.gpu_step(mode, tokens=None if toks is None else np.array(toks, np.int32),
                            positions=None if pos is None else np.array(pos, np.int32))
        assert tiny.model.device_error() == bit
        check_against_oracle(tiny, got, (None, None, None, None), skip={0})
    assert tiny.model.device_error() == 0          # cleared
    ref = tiny.oracle_step()
    check_against_oracle(tiny, tiny.gpu_step(kb.KL_MODE_LOOPED), ref)


@pytest.mark.parametrize("batch", [3, 8])
def test_bad_sequence_is_skipped_and_others_are_exact(batch):
    # one sequence with a bad token and one with a bad position in the same
    # step: both skipped, every other sequence matches the oracle; the GEMV
    # path (batch 3) and the matrix-core path (batch 8), all schedules
    say(f"[tiny-bad] batch={batch}")
    filled = (np.arange(batch, dtype=np.int32) * 29 + 3) % 150
    c = Case(TINY, batch, 160, filled, seed=131 + batch)
    toks, pos = c.tokens.copy(), c.positions.copy()
    toks[1] = c.cfg["vocab"] + 5
    pos[batch - 1] = 160
    good = [b for b in range(batch) if b not in (1, batch - 1)]
    ref = c.oracle_step(sample=good)
    outs = []
    for name, mode in MODES:
        say(f"  mode={name}")
        outs.append(c.gpu_step(mode, tokens=toks, positions=pos))
        assert c.model.device_error() == kb.KL_DEVERR_TOKEN | kb.KL_DEVERR_POSITION
        check_against_oracle(c, outs[-1], ref, positions=pos, skip={1, batch - 1}, only=good)
    assert_bit_exact(outs[0], outs[1], "per_layer vs looped")
    assert_bit_exact(outs[2], outs[1], "per_op vs looped")


def test_host_validation_enqueues_nothing(tiny):
    kv = KvCache(tiny.cfg, 1, tiny.capacity)
    toks = torch.zeros(1, dtype=torch.int32, device="cuda")
    logits = torch.zeros((1, tiny.cfg["vocab"]), device="cuda")
    with pytest.raises(kb.KlError) as e:
        tiny.model.step(toks, toks, kv, logits, None, 7)
    assert e.value.status == kb.KL_ERR_INVALID_ARGUMENT
    with pytest.raises(kb.KlError):
        kb.kl_decode_step(tiny.model.state, toks.data_ptr(), toks.data_ptr(), 2, kv.k.data_ptr(),
                          kv.v.data_ptr(), 1, tiny.capacity, logits.data_ptr(), None, 0,
                          kb.KL_MODE_LOOPED)


def test_llama8b_width_two_layers_long_cache():
    # the 8B layer shapes (d 128, 4 query heads per KV head, K 4096 and 14336,
    # 128256-row LM head) over a 4096-position cache, with 2 layers
    cfg = dict(WORKLOADS["llama8b-b1-ctx4096"]["model"], n_layers=2)
    say("[8b-width L=2] building")
    c = Case(cfg, 1, 4160, [4096], seed=51)
    say("[8b-width L=2] oracle")
    ref = c.oracle_step(nthreads=8)
    outs = []
    for name, mode in MODES:
        say(f"[8b-width L=2] mode={name}")
        outs.append(c.gpu_step(mode))
    check_against_oracle(c, outs[1], ref)
    assert_bit_exact(outs[0], outs[1], "per_layer vs looped")
    assert_bit_exact(outs[2], outs[1], "per_op vs looped")


@pytest.mark.parametrize("batch", [2, 3, 4, 5, 8, 16, 32])
def test_tiny_batched_matrix_core_path(batch):
    # batches 2 .. 4 share each GEMV pass (the attention merge one sequence
    # at a time: their chunks exceed one gather), from 5 on the weight
    # products run on the matrix cores (bf16 activations); ragged
    # positions, all schedules bit-identical
    say(f"[tiny-batched] batch={batch}")
    rng = np.random.default_rng(batch)
    filled = rng.integers(0, 190, size=batch).astype(np.int32)
    c = Case(TINY, batch, 192, filled, seed=61 + batch)
    ref = c.oracle_step(nthreads=8)
    outs = [c.gpu_step(mode) for _, mode in MODES]
    check_against_oracle(c, outs[1], ref)
    assert_bit_exact(outs[0], outs[1], "per_layer vs looped")
    assert_bit_exact(outs[2], outs[1], "per_op vs looped")


def test_batched_path_with_batch_above_one_group():
    # 40 sequences: two groups of the matrix-core path (32 + 8)
    say("[tiny-batched] batch=40")
    filled = (np.arange(40, dtype=np.int32) * 7) % 150
    c = Case(TINY, 40, 192, filled, seed=71)
    ref = c.oracle_step(nthreads=8)
    check_against_oracle(c, c.gpu_step(kb.KL_MODE_LOOPED), ref)


@pytest.mark.parametrize("batch", [2, 3, 4, 5, 8, 16, 32])
def test_llama8b_width_two_layers_batched(batch):
    # the 8B layer shapes, 256-position caches: batches 2 .. 4 on the GEMV
    # path with the sequences sharing each pass (16, 10 and 8 attention
    # chunks per (sequence, KV head), merged in one gather), from 5 on the
    # matrix-core path: below 32 several chunks with the grid-wide merge (6,
    # 4 and 2 chunks), at batch 32 one chunk
    cfg = dict(WORKLOADS["llama8b-b32-ctx4096"]["model"], n_layers=2)
    say(f"[8b-width L=2 B={batch}] building")
    filled = (np.arange(batch, dtype=np.int32) * 37) % 250
    c = Case(cfg, batch, 256, filled, seed=81 + batch)
    say(f"[8b-width L=2 B={batch}] oracle")
    ref = c.oracle_step(nthreads=8)
    outs = []
    for name, mode in MODES:
        say(f"[8b-width L=2 B={batch}] mode={name}")
        outs.append(c.gpu_step(mode))
    check_against_oracle(c, outs[1], ref)
    assert_bit_exact(outs[0], outs[1], "per_layer vs looped")
    assert_bit_exact(outs[2], outs[1], "per_op vs looped")


@pytest.mark.parametrize("batch", [1, 3, 8, 32])
def test_llama70b_width_two_layers(batch):
    # the 70B layer shapes (hidden 8192, 64 query / 8 KV heads: 8 query heads
    # per KV head, FFN 28672) with 2 layers, loaded one layer at a time; at
    # batch 3 the sequences share each GEMV pass (the O projection without
    # its wave split); at batch 32 one attention chunk per (sequence, KV
    # head) with 8 query heads per KV head (the oracle evaluates a sample of
    # the sequences)
    from paper_2410_23668_amd.device import GpuModel
    cfg = dict(WORKLOADS["llama70b-b1-ctx4096"]["model"], n_layers=2)
    say(f"[70b-width L=2 B={batch}] building")
    filled = (np.arange(batch, dtype=np.int32) * 53 + 200) % 250
    c = Case(cfg, batch, 256, filled, seed=91)
    inc = GpuModel.from_layers(cfg, lambda l: c.weights["layers"][l], lambda: c.weights,
                               batch, 256)
    sample = None if batch <= 8 else [0, 13, 31]
    say(f"[70b-width L=2 B={batch}] oracle")
    ref = c.oracle_step(nthreads=8, sample=sample)
    outs = []
    for name, mode in MODES:
        say(f"[70b-width L=2 B={batch}] mode={name}")
        outs.append(c.gpu_step(mode))
    check_against_oracle(c, outs[1], ref, only=sample)
    assert_bit_exact(outs[0], outs[1], "per_layer vs looped")
    assert_bit_exact(outs[2], outs[1], "per_op vs looped")
    # the incrementally loaded copy computes the same bits
    c.model, full = inc, c.model
    assert_bit_exact(c.gpu_step(kb.KL_MODE_LOOPED), outs[1], "incremental vs whole load")
    c.model = full
    inc.close()


@pytest.mark.parametrize("shape", ["tiny-b1", "tiny-b8", "8b-width-b1"])
def test_per_layer_graph_replays_match_looped(shape):
    # the per-layer schedule recorded as a graph: built on the first call with
    # a set of buffers, replayed on the next ones; every replay (with eager
    # steps of the other schedules and synchronizations in between) computes
    # the looped schedule's bits
    say(f"[graph] {shape}")
    if shape == "tiny-b1":
        c = Case(TINY, 1, 192, [150], seed=241)
    elif shape == "tiny-b8":
        c = Case(TINY, 8, 192, (np.arange(8, dtype=np.int32) * 23) % 180, seed=243)
    else:
        cfg = dict(WORKLOADS["llama8b-b1-ctx4096"]["model"], n_layers=2)
        c = Case(cfg, 1, 320, [300], seed=245)
    B, V = c.batch, c.cfg["vocab"]
    kv = KvCache(c.cfg, B, c.capacity, k_host=c.K0, v_host=c.V0)
    toks = torch.from_numpy(c.tokens).cuda()
    pos = torch.from_numpy(c.positions).cuda()
    eager = torch.empty((B, V), device="cuda")
    c.model.step(toks, pos, kv, eager, None, kb.KL_MODE_LOOPED)
    torch.cuda.synchronize()
    want = eager.cpu().numpy()
    graph_out = torch.full((B, V), float("nan"), device="cuda")
    for rep in range(3):
        graph_out.fill_(float("nan"))
        c.model.step(toks, pos, kv, graph_out, None, kb.KL_MODE_PER_LAYER_GRAPH)
        torch.cuda.synchronize()
        assert np.array_equal(graph_out.cpu().numpy().view(np.uint32), want.view(np.uint32)), \
            f"replay {rep} differs from the looped schedule"
        # eager work of the program between the replays
        c.model.step(toks, pos, kv, eager, None, kb.KL_MODE_PER_OP if rep % 2 else kb.KL_MODE_LOOPED)
        torch.cuda.synchronize()
        assert np.array_equal(eager.cpu().numpy().view(np.uint32), want.view(np.uint32))
    assert c.model.device_error() == 0
    # other buffers: the graph is rebuilt for them
    other = torch.empty((B, V), device="cuda")
    c.model.step(toks, pos, kv, other, None, kb.KL_MODE_PER_LAYER_GRAPH)
    torch.cuda.synchronize()
    assert np.array_equal(other.cpu().numpy().view(np.uint32), want.view(np.uint32))
    c.model.close()


def test_matrix_core_batch_per_model():
    """kl_info.mfma_min_batch: a dense model takes the matrix-core path from
    batch 5 (up to 4 sequences share each pass of the GEMV path); with
    experts, the GEMV path (per-token routing) runs below batch 8."""
    for cfg, want in ((dict(TINY, n_layers=1), 5),
                      (dict(TINY, n_layers=1, n_experts=4, top_k=2), 8)):
        weights = synth.model_host(cfg, 5, 4)
        m = GpuModel(cfg, weights, 8, 64)
        assert m.info().mfma_min_batch == want, (cfg, m.info().mfma_min_batch)
        m.close()


@pytest.mark.parametrize("batch", [2, 4])
def test_shared_gemv_pass_in_a_model_sized_for_more(batch):
    """Batches 2 and 4 of a model allocated for 8 sequences (the LDS holds
    both engines' areas): the shared GEMV pass against the oracle, and each
    schedule bit-identical."""
    cfg = dict(WORKLOADS["llama8b-b32-ctx4096"]["model"], n_layers=2)
    say(f"[8b-width L=2 B={batch} of 8] building")
    filled = (np.arange(batch, dtype=np.int32) * 53 + 11) % 250
    c = Case(cfg, batch, 256, filled, seed=91 + batch, max_batch=8)
    ref = c.oracle_step(nthreads=8)
    outs = [c.gpu_step(mode) for _, mode in MODES]
    check_against_oracle(c, outs[1], ref)
    assert_bit_exact(outs[0], outs[1], "per_layer vs looped")
    assert_bit_exact(outs[2], outs[1], "per_op vs looped")
    c.model.close()
