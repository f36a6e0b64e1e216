"""Pins for the oracle's group-64 cache quantiser (Sec. 4.5 stand-in scheme)."""
import numpy as np
import pytest

import oracle


@pytest.mark.parametrize("bits", [2, 4])
def test_round_trip_error_is_at_most_half_a_step(bits):
    rng = np.random.default_rng(bits)
    x = rng.standard_normal((50, 3, 128)).astype(np.float32)
    codes, meta = oracle.quantize_g64(x, bits)
    xh = oracle.dequantize_g64(codes, meta)
    scale = meta[..., 0].astype(np.float64)
    zero = meta[..., 1].astype(np.float64)
    g = x.reshape(50, 3, 2, 64).astype(np.float64)
    err = np.abs(xh.reshape(g.shape) - g)
    # half a step, plus what fp16 rounding of zero and scale can add at the top code
    slack = np.abs(g.min(-1) - zero) + (2 ** bits - 1) * np.abs(
        (g.max(-1) - g.min(-1)) / (2 ** bits - 1) - scale)
    assert np.all(err <= (scale / 2 + slack)[..., None] * (1 + 1e-6) + 1e-7)
    assert codes.max() <= 2 ** bits - 1


def test_exact_grid_round_trips_exactly():
    x = np.tile(np.arange(16, dtype=np.float32) * 0.5 - 2.0, 4)[None]   # 64 values on a 0.5 grid
    codes, meta = oracle.quantize_g64(x, 4)
    assert float(meta[0, 0, 0]) == 0.5 and float(meta[0, 0, 1]) == -2.0
    np.testing.assert_array_equal(codes[0], np.tile(np.arange(16), 4))
    np.testing.assert_array_equal(oracle.dequantize_g64(codes, meta), x)


def test_constant_group_has_zero_scale():
    x = np.full((1, 64), 0.3, dtype=np.float32)
    codes, meta = oracle.quantize_g64(x, 2)
    assert float(meta[0, 0, 0]) == 0.0 and not codes.any()
    np.testing.assert_allclose(oracle.dequantize_g64(codes, meta), np.float16(0.3), rtol=0)


def test_packing_order_low_bits_first():
    c4 = np.array([[1, 2, 3, 4]], dtype=np.uint8)
    assert list(oracle.pack_codes(c4, 4)[0]) == [0x21, 0x43]
    c2 = np.array([[1, 2, 3, 0, 3, 3, 3, 3]], dtype=np.uint8)
    assert list(oracle.pack_codes(c2, 2)[0]) == [0b00111001, 0xFF]
    rng = np.random.default_rng(0)
    for bits in (2, 4):
        c = rng.integers(0, 2 ** bits, size=(5, 128)).astype(np.uint8)
        np.testing.assert_array_equal(oracle.unpack_codes(oracle.pack_codes(c, bits), bits), c)


def test_half_way_codes_round_to_even():
    # values on exact half steps: (x - zero) / scale = 0.5, 1.5, 2.5 -> 0, 2, 2
    x = np.zeros((1, 64), dtype=np.float32)
    x[0, :4] = [0.5, 1.5, 2.5, 0.0]
    x[0, 4] = 3.0                      # max 3, min 0, scale 1 with 2 bits
    codes, meta = oracle.quantize_g64(x, 2)
    assert float(meta[0, 0, 0]) == 1.0
    assert list(codes[0, :5]) == [0, 2, 2, 0, 3]
