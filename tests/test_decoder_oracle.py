"""Pins of the decoder-loop oracle (oracle/decoder.py): rotary embedding
closed forms and its relative-position property, grouped-query attention
special cases (one key, equal keys, a dominant key, group mapping,
causality), bf16 rounding against the generator's, Norm against the C
oracle, and the layer's reduction when the attention output is zero."""
import numpy as np
import pytest

import synth


def test_rope_closed_forms():
    from oracle import decoder
    x = np.array([[1.0, 0.0]])
    # D = 2: one pair rotated by the angle p * base^0 = p
    np.testing.assert_allclose(decoder.rope(x, np.pi / 2, 10000.0), [[0.0, 1.0]], atol=1e-15)
    np.testing.assert_allclose(decoder.rope(x, np.pi, 10000.0), [[-1.0, 0.0]], atol=1e-15)
    rng = np.random.default_rng(0)
    q = rng.standard_normal((3, 64))
    assert np.array_equal(decoder.rope(q, 0, 1e6), q)
    r = decoder.rope(q, 37, 1e6)
    # each (i, i + D/2) pair keeps its length
    np.testing.assert_allclose(r[:, :32] ** 2 + r[:, 32:] ** 2, q[:, :32] ** 2 + q[:, 32:] ** 2, rtol=1e-12)
    # pair i turns by p * base^(-2i/D): i = 1 at D = 64, base 1e6
    ang = 37 * 1e6 ** (-2.0 / 64)
    np.testing.assert_allclose(r[0, 1], q[0, 1] * np.cos(ang) - q[0, 33] * np.sin(ang), rtol=1e-12)


def test_rope_scores_depend_on_relative_position_only():
    from oracle import decoder
    rng = np.random.default_rng(1)
    q, k = rng.standard_normal((1, 128)), rng.standard_normal((1, 128))
    base = 1e6
    for m, n, s in ((5, 2, 100), (0, 0, 31), (300, 17, 999)):
        a = decoder.rope(q, m, base) @ decoder.rope(k, n, base).T
        b = decoder.rope(q, m + s, base) @ decoder.rope(k, n + s, base).T
        np.testing.assert_allclose(a, b, rtol=1e-9)


def test_attend_special_cases():
    from oracle import decoder
    rng = np.random.default_rng(2)
    Hq, Hkv, D = 4, 2, 8
    q = rng.standard_normal((Hq, D))
    K = rng.standard_normal((Hkv, 6, D))
    V = rng.standard_normal((Hkv, 6, D))
    # one key: every head returns its group's value row
    o = decoder.attend(q, K, V, 1)
    np.testing.assert_allclose(o, V[[0, 0, 1, 1], 0], rtol=1e-14)
    # equal keys: uniform weights, the mean of the value rows
    Ke = np.repeat(K[:, :1], 6, axis=1)
    np.testing.assert_allclose(decoder.attend(q, Ke, V, 5), V[[0, 0, 1, 1], :5].mean(axis=1), rtol=1e-12)
    # a key aligned with q and scaled up dominates the softmax
    Kd = K.copy()
    Kd[0, 3] = 60.0 * q[0] / np.linalg.norm(q[0])
    assert np.allclose(decoder.attend(q, Kd, V, 6)[0], V[0, 3], atol=1e-6)


def test_attention_is_causal_and_incremental():
    """Token t sees positions <= pos0 + t only: a batch of T new tokens gives
    the same outputs as appending them one at a time."""
    from oracle import decoder
    rng = np.random.default_rng(3)
    d, Hq, Hkv, D, base = 64, 4, 2, 16, 1e4
    wqkv = 0.1 * rng.standard_normal(((Hq + 2 * Hkv) * D, d))
    wo = 0.1 * rng.standard_normal((d, Hq * D))
    x = rng.standard_normal((5, d))
    c1 = decoder.Cache(Hkv, 16, D)
    full = decoder.attention(x, wqkv, wo, c1, 2, Hq, Hkv, D, base)
    c2 = decoder.Cache(Hkv, 16, D)
    rows = [decoder.attention(x[t:t + 1], wqkv, wo, c2, 2 + t, Hq, Hkv, D, base)["att"][0] for t in range(5)]
    np.testing.assert_allclose(full["att"], np.array(rows), rtol=1e-12, atol=1e-14)
    assert np.array_equal(c1.K, c2.K) and np.array_equal(c1.V, c2.V)
    # entries past the last position never matter
    c3 = decoder.Cache(Hkv, 16, D)
    c3.K[:, 8:] = 1e3
    c3.V[:, 8:] = -1e3
    np.testing.assert_allclose(decoder.attention(x, wqkv, wo, c3, 2, Hq, Hkv, D, base)["att"], full["att"], rtol=1e-12)


def test_bf16_round_matches_the_generator():
    from oracle import decoder
    rng = np.random.default_rng(4)
    x = (rng.standard_normal(10000) * 10.0 ** rng.integers(-4, 4, 10000)).astype(np.float32)
    ref = synth.bf16_to_f32(synth.bf16_bits(x)).astype(np.float64)
    assert np.array_equal(decoder.bf16_round(x), ref)


def test_rmsnorm_matches_the_c_oracle():
    import oracle
    from oracle import decoder
    rng = np.random.default_rng(5)
    x = rng.standard_normal((3, 128))
    np.testing.assert_allclose(decoder.rmsnorm(x), oracle.residual_rmsnorm(x, np.zeros_like(x)), rtol=1e-12)


def test_layer_without_attention_output_is_the_moe_glue():
    """W_o = 0 makes Att(x) = 0: h = Norm(x) and x' = Norm(h + MoE(h))."""
    from oracle import decoder
    rng = np.random.default_rng(6)
    d, Hq, Hkv, D = 64, 2, 1, 32
    lw = dict(w_qkv=rng.standard_normal(((Hq + 2 * Hkv) * D, d)), w_o=np.zeros((d, Hq * D)))
    x = decoder.bf16_round(rng.standard_normal((2, d)))
    moe = lambda h: 0.5 * h  # noqa: E731  (a stand-in module with a closed form)
    xo, h = decoder.layer(x, lw, decoder.Cache(Hkv, 4, D), 0, dict(Hq=Hq, Hkv=Hkv, D=D, base=1e4), moe)
    np.testing.assert_allclose(h, decoder.bf16_round(decoder.rmsnorm(x)), rtol=0)
    np.testing.assert_allclose(xo, decoder.bf16_round(decoder.rmsnorm(1.5 * h)), rtol=0)


def test_head_argmax_takes_the_lowest_index_on_ties():
    from oracle import decoder
    w = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 0.0]])
    _, idx = decoder.head_argmax(np.array([[2.0, 1.0], [1.0, 3.0]]), w)
    assert idx.tolist() == [0, 1]
