"""The seeded input generator: determinism, thread independence, moments (CPU only)."""
import numpy as np

import synth
from tests import bruteforce


def test_splitmix64_output_function_reference_values():
    # word(i) = mix64(key + (i + 1) * G); with key chosen so that the argument
    # is the SplitMix64 state, the first outputs of the published generator
    # seeded with 0 are 0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4.
    G = 0x9E3779B97F4A7C15
    M = (1 << 64) - 1

    def mix(z):
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M
        return z ^ (z >> 31)
    assert mix(G) == 0xE220A8397B1DCDAF
    assert mix((2 * G) & M) == 0x6E789E6AA1B965F4
    key = mix((5 * G + mix(8)) & M)
    assert synth.word(5, 7, 0) == mix((key + G) & M)


def test_normal_is_deterministic_and_thread_count_free():
    a = synth.normal_bf16((100_001,), 11, 3, 0.0, 0.02, nthreads=1)
    b = synth.normal_bf16((100_001,), 11, 3, 0.0, 0.02, nthreads=5)
    np.testing.assert_array_equal(a, b)
    c = synth.normal_bf16((100_001,), 11, 4, 0.0, 0.02, nthreads=1)
    assert (a != c).mean() > 0.9


def test_normal_moments():
    x = bruteforce.bf16_decode(synth.normal_bf16((400_000,), 2, 9, 1.0, 0.01))
    # bf16 spacing near 1 is 2^-7 or 2^-8, so the gains are coarsely quantised
    assert abs(x.mean() - 1.0) < 5e-4
    assert 0.009 < x.std() < 0.0115
    y = bruteforce.bf16_decode(synth.normal_bf16((400_000,), 2, 10, 0.0, 1.0))
    assert abs(y.mean()) < 0.01 and abs(y.std() - 1.0) < 0.01
    assert abs((np.abs(y) < 1).mean() - 0.6827) < 0.005


def test_tokens_in_range_and_uniform():
    t = synth.uniform_int32(200_000, 3, 3_000_000, 0, 1024)
    assert t.min() == 0 and t.max() == 1023
    counts = np.bincount(t, minlength=1024)
    assert counts.std() / counts.mean() < 0.1


def test_kv_cache_slots_beyond_fill_are_zero():
    cfg = dict(n_layers=2, hidden=8, n_heads=2, n_kv_heads=1, head_dim=4, ffn_dim=8, vocab=16,
               rope_theta=1e4, rms_eps=1e-5)
    K, V = synth.kv_cache_host(cfg, 5, 2, 8, [3, 6])
    assert K.shape == (2, 2, 1, 8, 4)
    assert (K[:, 0, :, 3:] == 0).all() and (K[:, 1, :, 6:] == 0).all()
    assert (K[:, 0, :, :3] != 0).mean() > 0.9 and (V[:, 1, :, :6] != 0).mean() > 0.9
