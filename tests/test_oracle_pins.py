"""Pins of the CPU oracle to the mathematics (CPU only).

Each test checks the oracle against something other than itself: a library
routine for a special case, a closed form, an invariant, or an independent
brute-force evaluation on tiny inputs.  They are chosen so that a plausible
slip (a dropped term, a wrong sign or index, a transposed operand, a wrong
head group) fails at least one of them.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests import bruteforce

RNG = np.random.default_rng(1234)


def bf(x):
    return bruteforce.bf16_encode(np.asarray(x, dtype=np.float64))


# ---------------------------------------------------------------- bf16 format

def test_bf16_decode_matches_torch():
    h = RNG.integers(0, 1 << 16, size=20000, dtype=np.uint16)
    h = h[(h & 0x7F80) != 0x7F80]                      # finite patterns only
    np.testing.assert_array_equal(oracle.bf16_to_f64(h), bruteforce.bf16_decode(h))


def test_bf16_encode_matches_torch_on_float32_values():
    # float32 inputs are exact in double, so torch's RNE conversion is the reference
    x = np.concatenate([
        RNG.standard_normal(20000).astype(np.float32),
        (RNG.standard_normal(2000) * 1e-39).astype(np.float32),     # subnormals
        (RNG.standard_normal(2000) * 1e30).astype(np.float32),
        np.array([1.0 + 1 / 256, 1.0 + 3 / 256, -(1.0 + 1 / 256), 2.0 ** -133, 0.0, -0.0,
                  3.3895313892515355e38], dtype=np.float32),          # ties, tiny, max
    ]).astype(np.float64)
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16)
    np.testing.assert_array_equal(oracle.f64_to_bf16(x), ref.numpy().view(np.uint16))


def test_bf16_ties_go_to_even():
    assert oracle.f64_to_bf16(np.array([1.0 + 1 / 256]))[0] == 0x3F80   # down to even
    assert oracle.f64_to_bf16(np.array([1.0 + 3 / 256]))[0] == 0x3F82   # up to even
    # just above a tie rounds up (a float-first conversion would lose this)
    assert oracle.f64_to_bf16(np.array([1.0 + 1 / 256 + 2.0 ** -40]))[0] == 0x3F81


# ---------------------------------------------------------------- RMSNorm

def test_rmsnorm_constant_vector_closed_form():
    n, c, eps = 64, -1.7, 1e-5
    g = bf(1.0 + 0.1 * RNG.standard_normal(n))
    u = oracle.rmsnorm(np.full(n, c), g, eps)
    expect = c / math.sqrt(c * c + eps) * bruteforce.bf16_decode(g)
    np.testing.assert_allclose(u, expect, rtol=1e-14, atol=0)


def test_rmsnorm_one_hot_depends_on_length():
    n, a, eps = 48, 3.0, 1e-2
    x = np.zeros(n)
    x[5] = a
    u = oracle.rmsnorm(x, bf(np.ones(n)), eps)
    assert u[5] == pytest.approx(a / math.sqrt(a * a / n + eps), rel=1e-14)
    assert np.count_nonzero(u) == 1


def test_rmsnorm_scale_invariant_without_eps():
    x = RNG.standard_normal(100)
    g = bf(1 + 0.01 * RNG.standard_normal(100))
    np.testing.assert_allclose(oracle.rmsnorm(7.5 * x, g, 0.0), oracle.rmsnorm(x, g, 0.0),
                               rtol=1e-13)


# ---------------------------------------------------------------- GEMV

def test_gemv_one_hot_selects_column_of_nonsquare_matrix():
    w = bf(RNG.standard_normal((5, 7)))
    wd = bruteforce.bf16_decode(w)
    for j in range(7):
        e = np.zeros(7)
        e[j] = 1.0
        np.testing.assert_array_equal(oracle.gemv(w, e), wd[:, j])


def test_gemv_matches_library_matmul():
    w = bf(RNG.standard_normal((33, 70)) * 0.02)
    u = RNG.standard_normal(70)
    np.testing.assert_allclose(oracle.gemv(w, u), bruteforce.bf16_decode(w) @ u, rtol=1e-12,
                               atol=1e-15)
    np.testing.assert_array_equal(oracle.gemv(w, u, nthreads=4), oracle.gemv(w, u, nthreads=1))


# ---------------------------------------------------------------- RoPE

@pytest.mark.parametrize("d,theta", [(64, 10000.0), (128, 500000.0)])
def test_rope_identity_at_position_zero(d, theta):
    y = RNG.standard_normal(d)
    np.testing.assert_array_equal(oracle.rope(y, theta, 0), y)


@pytest.mark.parametrize("d,theta,pos", [(64, 10000.0, 1), (64, 10000.0, 127),
                                         (128, 500000.0, 4096), (128, 500000.0, 65536)])
def test_rope_is_complex_rotation(d, theta, pos):
    y = RNG.standard_normal(d)
    ref = bruteforce.rotate(y[None, :], pos, theta)[0]
    # the angle pos * omega carries a rounding error of up to a few pos 2^-53
    # radians (two ways of forming omega in double), so the bound grows with pos
    atol = 1e-12 + 8.0 * pos * 2.0 ** -53 * np.abs(y).max()
    np.testing.assert_allclose(oracle.rope(y, theta, pos), ref, rtol=1e-12, atol=atol)


# cos 1 and sin 1 (radians), printed constants
COS1, SIN1 = 0.5403023058681398, 0.8414709848078965


@pytest.mark.parametrize("i", [0, 1, 2, 3])
def test_rope_closed_form_frequencies_and_pairing(i):
    # d = 8, theta = 10^4: pair i has frequency theta^(-2i/d) = 10^-i, so the
    # unit vector e_i at position 10^i turns by exactly 1 radian into the
    # plane of its partner e_(i + d/2) (half-split pairing):
    #   e_i -> cos 1 e_i + sin 1 e_(i+4),   e_(i+4) -> -sin 1 e_i + cos 1 e_(i+4).
    # An interleaved pairing, another exponent or a flipped sign fails this.
    d, p = 8, 10 ** i
    e = np.zeros(d)
    e[i] = 1.0
    want = np.zeros(d)
    want[i], want[i + 4] = COS1, SIN1
    np.testing.assert_allclose(oracle.rope(e, 1e4, p), want, rtol=0, atol=1e-12)
    e = np.zeros(d)
    e[i + 4] = 1.0
    want = np.zeros(d)
    want[i], want[i + 4] = -SIN1, COS1
    np.testing.assert_allclose(oracle.rope(e, 1e4, p), want, rtol=0, atol=1e-12)


def test_rope_first_pair_turns_by_the_position_at_any_theta():
    # pair 0 has frequency theta^0 = 1 whatever theta and d are:
    # e_0 at position 3 -> cos 3 e_0 + sin 3 e_(d/2) (printed constants)
    for d, theta in ((64, 10000.0), (128, 500000.0)):
        e = np.zeros(d)
        e[0] = 1.0
        got = oracle.rope(e, theta, 3)
        assert got[0] == pytest.approx(-0.9899924966004454, abs=1e-13)
        assert got[d // 2] == pytest.approx(0.1411200080598672, abs=1e-13)
        assert np.count_nonzero(got) == 2


def test_rope_preserves_norm_and_relative_position():
    d, theta = 128, 10000.0
    q, k = RNG.standard_normal(d), RNG.standard_normal(d)
    for p in (3, 100, 5000):
        assert np.linalg.norm(oracle.rope(q, theta, p)) == pytest.approx(np.linalg.norm(q), rel=1e-13)
    for p, s in ((10, 3), (700, 699), (4096, 1)):
        lhs = oracle.rope(q, theta, p) @ oracle.rope(k, theta, s)
        rhs = oracle.rope(q, theta, p - s) @ k
        assert lhs == pytest.approx(rhs, rel=1e-10, abs=1e-10)


# ---------------------------------------------------------------- softmax / attention

def test_softmax_closed_form_and_sum():
    a = oracle.softmax(np.array([0.0, math.log(3.0)]))
    np.testing.assert_allclose(a, [0.25, 0.75], rtol=1e-15)
    s = RNG.standard_normal(1000) * 30
    assert oracle.softmax(s).sum() == pytest.approx(1.0, abs=1e-14)
    np.testing.assert_allclose(oracle.softmax(s + 1234.5), oracle.softmax(s), rtol=1e-12)


def _cache(nkv, cap, d, scale=1.0):
    return bf(RNG.standard_normal((nkv, cap, d)) * scale), bf(RNG.standard_normal((nkv, cap, d)))


def test_attention_single_key_returns_value_of_group():
    nq, nkv, d, cap = 8, 2, 16, 4
    K, V = _cache(nkv, cap, d)
    o = oracle.attention(RNG.standard_normal((nq, d)), K, V, pos=0)
    Vd = bruteforce.bf16_decode(V)
    for h in range(nq):
        np.testing.assert_array_equal(o[h], Vd[h // (nq // nkv), 0])


def test_attention_zero_query_is_mean_of_values():
    nq, nkv, d, cap, pos = 4, 4, 8, 16, 9
    K, V = _cache(nkv, cap, d)
    o = oracle.attention(np.zeros((nq, d)), K, V, pos)
    np.testing.assert_allclose(o, bruteforce.bf16_decode(V)[:, : pos + 1].mean(axis=1),
                               rtol=1e-13)


def test_attention_two_keys_closed_form_with_scale():
    d = 4
    K = np.zeros((1, 2, d), dtype=np.uint16)
    K[0, 1, 0] = bf(np.array([2.0]))[0]
    V = bf(np.array([[[1.0, 0, 0, 0], [0, 1.0, 0, 0]]]))
    q = np.array([[1.5, 0, 0, 0]])
    s1 = 1.5 * 2.0 / math.sqrt(d)                # scaled score of key 1; key 0 scores 0
    w1 = math.exp(s1) / (1 + math.exp(s1))
    o = oracle.attention(q, K, V, pos=1)
    np.testing.assert_allclose(o[0], [1 - w1, w1, 0, 0], rtol=1e-14)


def test_attention_gqa_equals_mha_with_repeated_kv():
    nq, nkv, d, cap, pos = 8, 2, 16, 12, 10
    K, V = _cache(nkv, cap, d, scale=0.5)
    q = RNG.standard_normal((nq, d))
    grp = nq // nkv
    o_gqa = oracle.attention(q, K, V, pos)
    o_mha = oracle.attention(q, np.repeat(K, grp, axis=0), np.repeat(V, grp, axis=0), pos)
    np.testing.assert_array_equal(o_gqa, o_mha)


def test_attention_ignores_slots_after_pos_and_order_of_slots():
    nq, nkv, d, cap, pos = 4, 2, 8, 20, 11
    K, V = _cache(nkv, cap, d)
    q = RNG.standard_normal((nq, d))
    o = oracle.attention(q, K, V, pos)
    K2, V2 = K.copy(), V.copy()
    K2[:, pos + 1:] = bf(np.full(1, 1e30))[0]
    V2[:, pos + 1:] = bf(np.full(1, -1e30))[0]
    np.testing.assert_array_equal(oracle.attention(q, K2, V2, pos), o)
    perm = RNG.permutation(pos + 1)
    K3, V3 = K.copy(), V.copy()
    K3[:, : pos + 1] = K[:, perm]
    V3[:, : pos + 1] = V[:, perm]
    np.testing.assert_allclose(oracle.attention(q, K3, V3, pos), o, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------- SwiGLU

def test_swiglu_closed_forms():
    np.testing.assert_array_equal(oracle.swiglu(np.zeros(5), RNG.standard_normal(5)), np.zeros(5))
    m = oracle.swiglu(np.array([1.0, 2.0, -3.0]), np.array([2.0, 1.0, 0.5]))
    silu = lambda z: z / (1 + math.exp(-z))
    np.testing.assert_allclose(m, [silu(1.0) * 2.0, silu(2.0) * 1.0, silu(-3.0) * 0.5],
                               rtol=1e-15)
    assert m[0] != m[1]                          # gate and up are not interchangeable


# ---------------------------------------------------------------- whole step

SMALL = dict(n_layers=2, hidden=16, n_heads=4, n_kv_heads=2, head_dim=4, ffn_dim=24, vocab=32,
             rope_theta=10000.0, rms_eps=1e-5)


def _small_inputs(cfg, batch, cap, positions, seed=7):
    model = synth.model_host(cfg, seed, nthreads=1)
    K, V = synth.kv_cache_host(cfg, seed + 1, batch, cap, positions, nthreads=1)
    toks = synth.tokens(cfg, seed + 2, batch)
    return model, K, V, toks


def test_step_with_zero_updates_keeps_embedding_and_closed_form_logits():
    cfg = dict(SMALL)
    model, K, V, toks = _small_inputs(cfg, 2, 8, [3, 5])
    for lay in model["layers"]:
        lay["wo"][:] = 0
        lay["w_down"][:] = 0
    logits, hidden = oracle.decode_step(cfg, model, toks, [3, 5], K, V)
    E = bruteforce.bf16_decode(model["embed"])
    for b, t in enumerate(toks):
        np.testing.assert_array_equal(hidden[b], E[t])
        u = bruteforce.rms_normalise(E[t], bruteforce.bf16_decode(model["final_norm"]),
                                     cfg["rms_eps"])
        np.testing.assert_allclose(logits[b], bruteforce.bf16_decode(model["lm_head"]) @ u,
                                   rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("cfg_over,positions,cap", [
    ({}, [3, 5], 8),
    ({"qkv_bias": True}, [2, 6], 8),
    ({"tie_embeddings": True, "n_heads": 6, "n_kv_heads": 2}, [4, 1], 8),
    ({"n_heads": 4, "n_kv_heads": 4}, [0, 7], 8),
    ({"n_heads": 6, "n_kv_heads": 2, "head_dim": 8, "hidden": 24, "n_layers": 3}, [1, 2], 4),
    ({"n_experts": 4, "top_k": 2}, [3, 5], 8),
    ({"n_experts": 3, "top_k": 1}, [2, 6], 8),
])
def test_step_matches_independent_brute_force(cfg_over, positions, cap):
    cfg = dict(SMALL, **cfg_over)
    model, K, V, toks = _small_inputs(cfg, len(positions), cap, positions)
    K2, V2 = K.copy(), V.copy()
    logits, hidden = oracle.decode_step(cfg, model, toks, positions, K, V)
    lref, href = bruteforce.decode_step(cfg, model, toks, positions, K2, V2)
    assert oracle.rel_l2(logits, lref) < 1e-12
    assert oracle.rel_l2(hidden, href) < 1e-12
    np.testing.assert_array_equal(K, K2)
    np.testing.assert_array_equal(V, V2)


def test_step_sequences_are_independent_and_thread_count_free():
    cfg = dict(SMALL)
    model, K, V, toks = _small_inputs(cfg, 2, 8, [3, 6])
    Kb, Vb = K.copy(), V.copy()
    logits, hidden = oracle.decode_step(cfg, model, toks, [3, 6], K, V, nthreads=3)
    for b, p in enumerate([3, 6]):
        Ks, Vs = Kb[:, b:b + 1].copy(), Vb[:, b:b + 1].copy()
        ls, hs = oracle.decode_step(cfg, model, toks[b:b + 1], [p], Ks, Vs, nthreads=1)
        np.testing.assert_array_equal(ls[0], logits[b])
        np.testing.assert_array_equal(hs[0], hidden[b])
        np.testing.assert_array_equal(Ks[:, 0], K[:, b])


def test_step_is_idempotent_and_rejects_bad_token():
    cfg = dict(SMALL)
    model, K, V, toks = _small_inputs(cfg, 1, 8, [4])
    l1, h1 = oracle.decode_step(cfg, model, toks, [4], K, V)
    K1, V1 = K.copy(), V.copy()
    l2, h2 = oracle.decode_step(cfg, model, toks, [4], K, V)
    np.testing.assert_array_equal(l1, l2)
    np.testing.assert_array_equal(K1, K)
    with pytest.raises(ValueError):
        oracle.decode_step(cfg, model, np.array([cfg["vocab"]]), [4], K, V)
    with pytest.raises(ValueError):
        oracle.decode_step(cfg, model, toks, [8], K, V)


# ---------------------------------------------------------------- sampling

def test_argmax_lowest_index_on_ties_and_brute_force():
    # ties resolve to the lowest index; -inf and negative values order normally
    assert oracle.argmax([1.0, 3.0, 3.0, 2.0]) == 1
    assert oracle.argmax([-np.inf, -5.0, -5.0]) == 1
    assert oracle.argmax([7.0]) == 0
    assert oracle.argmax([0.0, -0.0]) == 0          # +0 == -0: a tie
    for _ in range(50):                              # brute force on small vectors
        x = RNG.integers(-3, 4, size=int(RNG.integers(1, 12))).astype(np.float64)
        best = max(range(x.size), key=lambda i: (x[i], -i))
        assert oracle.argmax(x) == best


def test_greedy_loop_feeds_each_token_to_the_next_step():
    # a 1-layer toy: step s of the loop equals a single decode step at
    # position p + s on the previous step's argmax, caches carried over
    cfg = dict(n_layers=1, hidden=8, n_heads=2, n_kv_heads=1, head_dim=4, ffn_dim=12, vocab=16,
               rope_theta=10000.0, rms_eps=1e-5)
    import synth
    w = synth.model_host(cfg, 5)
    K0, V0 = synth.kv_cache_host(cfg, 6, 1, 8, [3])
    K, V = K0.copy(), V0.copy()
    sampled, logits = oracle.greedy_decode(cfg, w, [2], [3], K, V, 3)
    Kr, Vr = K0.copy(), V0.copy()
    tok = 2
    for s in range(3):
        lg, _ = oracle.decode_step(cfg, w, [tok], [3 + s], Kr, Vr)
        assert np.array_equal(lg, logits[s])
        tok = oracle.argmax(lg[0])
        assert sampled[s, 0] == tok
    assert np.array_equal(K, Kr) and np.array_equal(V, Vr)


def test_qkv_bias_with_zero_weights_is_the_bias():
    # Q/K/V weights zero: q = bq, k = RoPE(bk) and v = bv exactly; at position 0
    # the single key's softmax weight is 1, so the attention output of every
    # query head is bf16(bv) of its KV head, and with W_o the identity-like
    # one-hot map the residual picks it up exactly
    cfg = dict(SMALL, qkv_bias=True, n_layers=1)
    model, K, V, toks = _small_inputs(cfg, 1, 4, [0])
    lay = model["layers"][0]
    for n in ("wq", "wk", "wv", "w_down"):
        lay[n][:] = 0
    d, nq, nkv, H = cfg["head_dim"], cfg["n_heads"], cfg["n_kv_heads"], cfg["hidden"]
    wo = np.zeros((H, nq * d))
    wo[np.arange(nq * d), np.arange(nq * d)] = 1.0          # x[i] += o[i] for i < nq d
    lay["wo"][:] = oracle.f64_to_bf16(wo)
    _, hidden = oracle.decode_step(cfg, model, toks, [0], K, V)
    E = bruteforce.bf16_decode(model["embed"])[toks[0]]
    bv = oracle.bf16_to_f64(oracle.f64_to_bf16(bruteforce.bf16_decode(lay["bv"])))
    o = np.repeat(bv.reshape(nkv, d), nq // nkv, axis=0).reshape(-1)
    want = E.copy()
    want[: nq * d] += o
    np.testing.assert_array_equal(hidden[0], want)
    # the new key slot holds bf16(RoPE at 0 of bk) = bf16(bk)
    np.testing.assert_array_equal(K[0, 0, :, 0, :], lay["bk"].reshape(nkv, d))


def test_route_top_k_ties_and_softmax():
    # the largest logits, the lowest index first among equal ones, weighted
    # by the softmax of the chosen logits
    idx, w = oracle.route([0.5, 2.0, -1.0, 2.0, 1.0], 2)
    assert list(idx) == [1, 3]
    np.testing.assert_allclose(w, [0.5, 0.5], rtol=0, atol=1e-15)
    idx, w = oracle.route([0.0, 1.0, 3.0, 2.0], 2)
    assert list(idx) == [2, 3]
    np.testing.assert_allclose(w, [1 / (1 + np.exp(-1.0)), 1 / (1 + np.exp(1.0))], rtol=1e-15)
    idx, w = oracle.route([4.0, 1.0, 3.0], 1)
    assert list(idx) == [0] and w[0] == 1.0


def test_experts_all_equal_reduce_to_the_dense_mlp():
    # every expert the same MLP: any routing weights summing to 1 give the
    # dense model's step exactly up to rounding of the weighted sum
    E = 4
    cfg_d = dict(SMALL, n_layers=2)
    cfg_m = dict(cfg_d, n_experts=E, top_k=2)
    model, K, V, toks = _small_inputs(cfg_d, 2, 8, [3, 5])
    moe = {k: v for k, v in model.items() if k != "layers"}
    moe["layers"] = []
    for l, lay in enumerate(model["layers"]):
        ml = dict(lay)
        for n in ("w_gate", "w_up", "w_down"):
            ml[n] = np.ascontiguousarray(np.concatenate([lay[n]] * E, axis=0))
        ml["w_router"] = synth.normal_bf16((E, cfg_d["hidden"]), 77, l, 0.0, 0.02)
        moe["layers"].append(ml)
    Km, Vm = K.copy(), V.copy()
    ld, hd = oracle.decode_step(cfg_d, model, toks, [3, 5], K, V)
    lm, hm = oracle.decode_step(cfg_m, moe, toks, [3, 5], Km, Vm)
    assert oracle.rel_l2(hm, hd) < 1e-14 and oracle.rel_l2(lm, ld) < 1e-14
    np.testing.assert_array_equal(K, Km)


def test_router_logits_are_reported_and_drive_the_choice():
    # the reported router logits decide the experts: zeroing every expert's
    # down projection except the two chosen ones leaves the step unchanged
    cfg = dict(SMALL, n_layers=1, n_experts=4, top_k=2)
    model, K, V, toks = _small_inputs(cfg, 1, 8, [3])
    router = np.zeros((1, 1, 4))
    K2, V2 = K.copy(), V.copy()
    l1, h1 = oracle.decode_step(cfg, model, toks, [3], K, V, router_out=router)
    chosen, _ = oracle.route(router[0, 0], 2)
    H, F = cfg["hidden"], cfg["ffn_dim"]
    lay = model["layers"][0]
    for e in range(4):
        if e not in chosen:
            lay["w_down"][e * H:(e + 1) * H] = 0
    l2, h2 = oracle.decode_step(cfg, model, toks, [3], K2, V2)
    np.testing.assert_array_equal(h1, h2)
