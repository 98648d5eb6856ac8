"""Pins of the quantized-expert oracle (oracle/quant.py): the code format on
hand-worked rows, fp16 metadata against numpy's float16, the orientation of
the three matrices, agreement with the plain C oracle where the dequantized
weights are exact in fp32, and the synthetic quantizer's packing."""
import json
import os

import numpy as np
import pytest

import synth

HERE = os.path.dirname(os.path.abspath(__file__))


def _golden():
    with open(os.path.join(HERE, "golden", "quant_cases.json")) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", _golden(), ids=lambda c: c["name"][:12])
def test_dequantize_hand_worked_rows(case):
    from oracle import quant
    packed = np.frombuffer(bytes.fromhex(case["packed_hex"]), np.uint8).reshape(1, -1)
    meta = np.array(case["meta"], np.uint16).reshape(1, -1, 2)
    w = quant.dequantize(packed, meta, case["bits"], case["n"])
    for g, period in enumerate(case["expect_period"]):
        grp = w[0, g * 64:(g + 1) * 64]
        expect = np.tile(np.array(period), 64 // len(period))
        assert np.array_equal(grp, expect), "group %d" % g


def test_fp16_meta_matches_numpy_float16():
    from oracle import quant
    rng = np.random.default_rng(3)
    vals = rng.standard_normal(1000).astype(np.float16)
    assert np.array_equal(quant.fp16_values(vals.view(np.uint16)), vals.astype(np.float64))


@pytest.mark.parametrize("bits", [2, 4])
def test_codes_round_trip_through_the_packing(bits):
    """synth.pack_codes and oracle.quant.unpack_codes are written apart; with
    scale 1 and zero 0 the dequantized row is the codes themselves."""
    from oracle import quant
    rng = np.random.default_rng(bits)
    q = rng.integers(0, 2 ** bits, size=(3, 192))
    packed = synth.pack_codes(q, bits)
    assert packed.shape == (3, 192 * bits // 8)
    assert np.array_equal(quant.unpack_codes(packed, bits, 192), q)
    meta = np.zeros((3, 3, 2), np.uint16)
    meta[:, :, 0] = np.float16(1.0).view(np.uint16)
    assert np.array_equal(quant.dequantize(packed, meta, bits, 192), q.astype(np.float64))


def test_matrix_orientation():
    """gate/up are given [F][d] and down [d][F]: with all codes 0 and zero
    -f on row f, W_gate[k][f] = f for every k (a transposed reading would
    vary with k), and W_down[f][c] = c."""
    from oracle import quant
    d, F, bits = 64, 128, 2
    zg = np.zeros((F, 1, 2), np.uint16)
    zg[:, 0, 0] = np.float16(1.0).view(np.uint16)
    zg[:, 0, 1] = (-np.arange(F, dtype=np.float16)).view(np.uint16)
    zd = np.zeros((d, F // 64, 2), np.uint16)
    zd[:, :, 0] = np.float16(1.0).view(np.uint16)
    zd[:, :, 1] = (-np.arange(d, dtype=np.float16)).view(np.uint16)[:, None]
    codes = (np.zeros((F, d * bits // 8), np.uint8), np.zeros((F, d * bits // 8), np.uint8),
             np.zeros((d, F * bits // 8), np.uint8))
    wg, wu, wd = quant.expert_weights(codes, (zg, zg, zd), bits, d, F)
    assert wg.shape == (d, F) and wd.shape == (F, d)
    assert np.array_equal(wg, np.tile(np.arange(F, dtype=np.float64), (d, 1)))
    assert np.array_equal(wd, np.tile(np.arange(d, dtype=np.float64), (F, 1)))


@pytest.mark.parametrize("bits", [2, 4])
def test_expert_matches_the_plain_oracle_on_exact_weights(bits):
    """Scale 2^-5 and zeros in {0.5, 1, 1.5, 2}: every dequantized weight is
    exact in fp32, so the C oracle's expert on those fp32 weights and the
    fp64 numpy expert here compute the same function (to rounding order)."""
    import oracle
    from oracle import quant
    rng = np.random.default_rng(11 + bits)
    d, F = 128, 192
    codes, metas = [], []
    for rows, n in ((F, d), (F, d), (d, F)):
        q = rng.integers(0, 2 ** bits, size=(rows, n))
        codes.append(synth.pack_codes(q, bits))
        m = np.zeros((rows, n // 64, 2), np.uint16)
        m[:, :, 0] = np.float16(2.0 ** -5).view(np.uint16)
        m[:, :, 1] = rng.choice(np.array([0.5, 1.0, 1.5, 2.0], np.float16), size=(rows, n // 64)).view(np.uint16)
        metas.append(m)
    ws = quant.expert_weights(codes, metas, bits, d, F)
    assert all(np.array_equal(w.astype(np.float32).astype(np.float64), w) for w in ws)
    for t in range(3):
        h = rng.standard_normal(d).astype(np.float32)
        y = quant.expert(h, ws)
        ref = oracle.expert(h, tuple(w.astype(np.float32) for w in ws))
        np.testing.assert_allclose(y, ref, rtol=1e-10, atol=1e-12 * np.abs(ref).max())


def test_zero_input_gives_zero_output():
    from oracle import quant
    shape = synth.ModelShape("q-tiny", 1, 128, 128, 4, 2, expert_bits=2)
    qe = synth.quant_expert(shape, 0, 0, 1, 2)
    ws = quant.expert_weights(qe.codes, qe.meta, 2, 128, 128)
    assert np.array_equal(quant.expert(np.zeros(128, np.float32), ws), np.zeros(128))


@pytest.mark.parametrize("bits", [2, 4])
def test_synthetic_quantizer_stays_within_half_a_step(bits):
    """Round-to-nearest over [min, max]: every dequantized weight is within
    half a quantization step (plus the fp16 rounding of scale and zero) of
    the N(0, 0.02) draw it stands for."""
    from oracle import quant
    rng = np.random.default_rng(5)
    w = (0.02 * rng.standard_normal((16, 256))).astype(np.float32)
    packed, meta = synth.quantize_rows(w, bits)
    deq = quant.dequantize(packed, meta, bits, 256)
    s = quant.fp16_values(meta[:, :, 0])
    z = quant.fp16_values(meta[:, :, 1])
    step = np.repeat(s, 64, axis=1)
    # rounding of the zero to fp16 shifts the grid by up to half an fp16 ulp of z
    slack = np.repeat(np.abs(z) * 2.0 ** -11 * s, 64, axis=1)
    assert np.all(np.abs(deq - w) <= 0.5 * step * (1 + 1e-3) + slack + 1e-12)


@pytest.mark.parametrize("bits", [2, 4])
def test_expert_ranges_sum_to_the_expert(bits):
    """Split identity (Sec. 3.1): the range form over [0, F_top) plus
    [F_top, F) equals the full expert, within fp64 rounding, for every
    chunk-aligned split point."""
    from oracle import quant
    shape = synth.ModelShape("q-split", 1, 256, 320, 4, 2, expert_bits=bits)
    qe = synth.quant_expert(shape, 1, 0, 2, bits)
    ws = quant.expert_weights(qe.codes, qe.meta, bits, 256, 320)
    h = np.random.default_rng(7).standard_normal(256).astype(np.float32)
    full = quant.expert(h, ws)
    for top in range(0, 321, 64):
        y = (quant.expert_range(h, qe.codes, qe.meta, bits, 256, 320, 0, top)
             + quant.expert_range(h, qe.codes, qe.meta, bits, 256, 320, top, 320))
        np.testing.assert_allclose(y, full, rtol=1e-12, atol=1e-14 * np.abs(full).max())
