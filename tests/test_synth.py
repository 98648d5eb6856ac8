"""Seeded input generators: bf16 round-to-nearest-even and determinism."""
import numpy as np

import synth


def test_bf16_round_to_nearest_even():
    bits = np.array([0x3F800000, 0x3F808000, 0x3F818000, 0x3F807FFF, 0x3F808001,
                     0xBF800000, 0x00000000, 0x80000000, 0x7F7FFFFF], np.uint32)
    want = [0x3F80, 0x3F80, 0x3F82, 0x3F80, 0x3F81, 0xBF80, 0x0000, 0x8000, 0x7F80]
    got = synth.bf16_bits(bits.view(np.float32))
    assert got.tolist() == want


def test_bf16_roundtrip_is_exact_on_bf16_values():
    x = synth.bf16_to_f32(np.arange(0, 0x7F80, 7, dtype=np.uint16))
    assert np.array_equal(synth.bf16_bits(x), np.arange(0, 0x7F80, 7, dtype=np.uint16))


def test_generators_are_deterministic_and_distinct():
    s = synth.TINY
    a = synth.expert(s, 0, 0, 1)
    b = synth.expert(s, 0, 0, 1)
    c = synth.expert(s, 0, 0, 2)
    for x, y, z in zip(a.f32, b.f32, c.f32):
        assert np.array_equal(x, y) and not np.array_equal(x, z)
    assert a.f32[0].shape == (256, 512) and a.f32[2].shape == (512, 256)
    raw, f = synth.hidden(synth.MIXTRAL, 0, 3)
    assert raw.dtype == np.uint16 and np.array_equal(synth.bf16_to_f32(raw), f)


def test_zipf_bias_softmax_is_zipf():
    s = synth.QWEN3
    b = synth.router_bias(s, 0, 3).astype(np.float64)
    p = np.exp(b) / np.exp(b).sum()
    ranks = np.sort(p)[::-1]
    ref = np.arange(1, s.n_experts + 1, dtype=np.float64) ** -1.1
    np.testing.assert_allclose(ranks, ref / ref.sum(), rtol=1e-6)
    assert synth.router_bias(synth.MIXTRAL, 0, 0) is None


def test_walk_keeps_unit_variance():
    steps = synth.walk(synth.TINY, 0, 200, T=4)
    x = np.stack([f for _, f in steps])
    assert abs(x.std() - 1.0) < 0.05
    # consecutive tokens correlated at about sqrt(1 - 0.3^2)
    c = np.corrcoef(x[:-1].reshape(-1), x[1:].reshape(-1))[0, 1]
    assert abs(c - np.sqrt(1 - 0.09)) < 0.02
