"""kl_decode_step_noalloc (the entry point for callers that cannot allocate)
against kl_decode_step, through the C ABI: the same bits on two calls in a
row, the second with a smaller input, on the per-sequence and on the
matrix-core path, and a request beyond the static scratch refused with
nothing enqueued."""
import numpy as np
import pytest
import torch

from paper_2410_23668_amd import binding as kb
from paper_2410_23668_amd.device import KvCache, stream_handle
from synth.workloads import TINY, WORKLOADS
from tests.gpu_cases import Case, assert_bit_exact, say

pytestmark = pytest.mark.gpu


def run(case, fn, batch, mode, tokens=None, positions=None):
    """One step of the first 'batch' sequences through fn (a C-ABI entry
    point); returns logits, hidden, K, V on the host."""
    kv = KvCache(case.cfg, case.batch, case.capacity, k_host=case.K0, v_host=case.V0)
    toks = torch.from_numpy((case.tokens if tokens is None else tokens)[:batch].copy()).cuda()
    pos = torch.from_numpy((case.positions if positions is None else positions)[:batch].copy()).cuda()
    logits = torch.full((batch, case.cfg["vocab"]), float("nan"), device="cuda")
    hidden = torch.full((batch, case.cfg["hidden"]), float("nan"), device="cuda")
    fn(case.model.state, toks.data_ptr(), pos.data_ptr(), batch, kv.k.data_ptr(), kv.v.data_ptr(),
       kv.batch, kv.capacity, logits.data_ptr(), hidden.data_ptr(), stream_handle(), mode)
    torch.cuda.synchronize()
    K, V = kv.host()
    return logits.cpu().numpy(), hidden.cpu().numpy(), K, V


@pytest.mark.parametrize("batches", [(5, 2), (12, 8), (9, 3)])
def test_noalloc_matches_decode_step_twice_then_smaller(batches):
    # two calls in a row, the second with a smaller batch (so a smaller part
    # of the static scratch, holding the first call's values); (12, 8) stays
    # on the matrix-core path, (9, 3) moves from it to the per-sequence path
    first, second = batches
    say(f"[noalloc] batches {first} then {second}")
    filled = (np.arange(first, dtype=np.int32) * 41 + 7) % 150
    c = Case(TINY, first, 160, filled, seed=151 + first)
    for name, mode in (("looped", kb.KL_MODE_LOOPED), ("per_layer", kb.KL_MODE_PER_LAYER)):
        for b in (first, second):
            say(f"  mode={name} batch={b}")
            want = run(c, kb.kl_decode_step, b, mode)
            got = run(c, kb.kl_decode_step_noalloc, b, mode)
            assert_bit_exact(got, want, f"noalloc vs decode_step, batch {b}, {name}")
            assert np.isfinite(got[0]).all()
    assert c.model.device_error() == 0
    c.model.close()


def test_noalloc_after_another_model_on_the_same_device():
    # the static scratch is shared by every state on the device: a second
    # model of another shape sees the first one's leftovers and must not
    # depend on them
    say("[noalloc] 8B width, 2 layers, batch 1, after a tiny model")
    t = Case(TINY, 4, 160, [3, 50, 99, 140], seed=171)
    run(t, kb.kl_decode_step_noalloc, 4, kb.KL_MODE_LOOPED)
    t.model.close()
    cfg = dict(WORKLOADS["llama8b-b1-ctx4096"]["model"], n_layers=2)
    c = Case(cfg, 1, 320, [300], seed=173)
    want = run(c, kb.kl_decode_step, 1, kb.KL_MODE_LOOPED)
    got = run(c, kb.kl_decode_step_noalloc, 1, kb.KL_MODE_LOOPED)
    assert_bit_exact(got, want, "noalloc vs decode_step, 8B width")
    c.model.close()


def test_noalloc_refuses_a_step_beyond_its_scratch():
    # the 70B layer width at batch 32 needs more than the static scratch:
    # refused on the host, nothing enqueued, the caller's buffers untouched
    cfg = dict(WORKLOADS["llama70b-b1-ctx4096"]["model"], n_layers=1, vocab=256)
    say("[noalloc] 70B width batch 32: over the limit")
    c = Case(cfg, 32, 64, np.full(32, 10, dtype=np.int32), seed=181)
    info = c.model.info()
    assert info.noalloc_scratch_bytes > info.noalloc_scratch_limit == 32 << 20
    kv = KvCache(c.cfg, 32, 64, k_host=c.K0, v_host=c.V0)
    toks = torch.from_numpy(c.tokens).cuda()
    pos = torch.from_numpy(c.positions).cuda()
    logits = torch.full((32, cfg["vocab"]), 7.0, device="cuda")
    with pytest.raises(kb.KlError) as e:
        kb.kl_decode_step_noalloc(c.model.state, toks.data_ptr(), pos.data_ptr(), 32,
                                  kv.k.data_ptr(), kv.v.data_ptr(), 32, 64, logits.data_ptr(),
                                  None, stream_handle(), kb.KL_MODE_LOOPED)
    assert e.value.status == kb.KL_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert (logits.cpu().numpy() == 7.0).all()
    K, _ = kv.host()
    assert np.array_equal(K, c.K0)
    c.model.close()
