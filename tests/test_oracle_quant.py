"""Pins of the oracle's decoding of group-quantised experts (Sec. 5.1: 2-bit
codes, groups of 16, compressed zero points)."""
import numpy as np
import pytest

from oracle import quant
from paper_2511_05814_amd import workload as wl


def _matrix(rows, cols, codes, scale_bits, zero_codes):
    """Stored bytes from explicit planes (codes already packed per byte)."""
    return np.concatenate([np.asarray(codes, np.uint8).ravel(),
                           np.asarray(scale_bits, "<u2").view(np.uint8).ravel(),
                           np.asarray(zero_codes, np.uint8).ravel()])


def test_hand_worked_group():
    # byte 0b11_10_01_00 holds codes 0, 1, 2, 3 for columns 0..3; scale 0.5
    # (fp16 0x3800), zero code 96 -> zero point 1.5: w = (q - 1.5) * 0.5
    buf = _matrix(1, 16, [0b11100100] * 4, [0x3800], [96])
    w = quant.dequantize(buf, 1, 16)
    assert w.tolist() == [[-0.75, -0.25, 0.25, 0.75] * 4]


def test_scale_bits_decode_exactly():
    # q = 1 everywhere (byte 0b01010101), zero code 0: w = scale
    for bits, value in ((0x3C00, 1.0), (0x0001, 2.0 ** -24), (0x7BFF, 65504.0), (0x2E66, 0.0999755859375)):
        w = quant.dequantize(_matrix(1, 16, [0x55] * 4, [bits], [0]), 1, 16)
        assert np.all(w == value)


def test_zero_point_on_a_code_gives_zeros():
    # zero code 128 = 2.0 and every q = 2 (byte 0b10101010)
    w = quant.dequantize(_matrix(2, 32, [0xAA] * 16, [0x4500] * 4, [128] * 4), 2, 32)
    assert np.all(w == 0.0)


def test_plane_and_bit_order():
    # row r, group g gets scale 2^(r*2+g) and zero 0; column c of each group
    # gets code c % 4 (so byte = 0b11100100 everywhere): w = (c % 4) * 2^(2r+g)
    rows, cols = 2, 32
    scale_bits = [0x3C00 + ((2 * r + g) << 10) for r in range(rows) for g in range(cols // 16)]
    w = quant.dequantize(_matrix(rows, cols, [0b11100100] * (rows * cols // 4), scale_bits,
                                 [0] * (rows * cols // 16)), rows, cols)
    for r in range(rows):
        for c in range(cols):
            assert w[r, c] == (c % 4) * 2.0 ** (2 * r + c // 16)
    # a single code moved: column 5 of row 1 (byte 1, field 1) set to 3
    codes = np.full(rows * cols // 4, 0b11100100, np.uint8)
    codes[cols // 4 + 1] = 0b11101100
    w2 = quant.dequantize(_matrix(rows, cols, codes, scale_bits, [0] * (rows * cols // 16)), rows, cols)
    diff = np.argwhere(w2 != w)
    assert diff.tolist() == [[1, 5]] and w2[1, 5] == 3 * 4.0


def test_expert_split_order():
    # W1, W3, W2 of a tiny expert get scales 1, 2, 4 (codes 1, zero 0)
    d, d_ff = 16, 32
    parts = []
    for bits, rows, cols in ((0x3C00, d_ff, d), (0x4000, d_ff, d), (0x4400, d, d_ff)):
        parts.append(_matrix(rows, cols, [0x55] * (rows * cols // 4), [bits] * (rows * cols // 16),
                             [0] * (rows * cols // 16)))
    w1, w3, w2 = quant.split_expert(np.concatenate(parts), d, d_ff)
    assert w1.shape == (d_ff, d) and w3.shape == (d_ff, d) and w2.shape == (d, d_ff)
    assert np.all(w1 == 1.0) and np.all(w3 == 2.0) and np.all(w2 == 4.0)


def test_round_trip_error_bound_against_the_quantiser():
    # The generator's quantiser (separate code) and the oracle's decoder must
    # agree on the format: each weight is within half a step of its group's
    # scale plus the zero point's rounding (1/128 of a step), wherever the
    # group spans zero (zero code not clipped).
    rng = np.random.default_rng(5)
    w = (rng.standard_normal((64, 256)) * 0.02).astype(np.float32)
    codes, scales, zeros = wl.quantize_q2g16(w)
    buf = np.concatenate([codes.ravel(), scales.view(np.uint8).ravel(), zeros.ravel()])
    deq = quant.dequantize(buf, 64, 256)
    s = np.repeat(scales.astype(np.float64), 16, axis=1)
    g = w.reshape(64, 16, 16)
    spans_zero = np.repeat((g.min(axis=2) <= 0) & (g.max(axis=2) >= 0), 16, axis=1)
    err = np.abs(deq - w.astype(np.float64))
    bound = s * (0.5 + 1.0 / 128) * (1 + 1e-3)  # fp16 rounding of the scale
    assert spans_zero.mean() > 0.99
    assert np.all(err[spans_zero] <= bound[spans_zero])


def test_dequantised_values_are_exact_in_fp32():
    # (q - z) has at most 9 significant bits and the fp16 scale 11, so every
    # weight is an fp32 number: fp32 and fp64 evaluation agree bit for bit
    c = wl.CONFIGS["tiny-q2"]
    flat = wl.expert_weights(c, 1, 3)
    for m in quant.split_expert(flat, c.d_model, c.d_ff):
        assert np.array_equal(m.astype(np.float32).astype(np.float64), m)


@pytest.mark.parametrize("name", ["tiny-q2", "mixtral-layer-q2"])
def test_stored_size(name):
    c = wl.CONFIGS[name]
    assert c.expert_bytes == 3 * quant.matrix_bytes(c.d_ff, c.d_model) == 3 * c.d_model * c.d_ff * 7 // 16
