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


# ---- FP8 (E4M3) group-64 scheme ----------------------------------------------------------

def _torch_e4m3_values():
    import torch
    return torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def test_e4m3_values_match_torch_for_every_byte():
    """The plain definition of the format against torch's own float8_e4m3fn type."""
    ours = oracle.e4m3_value(np.arange(256))
    ref = _torch_e4m3_values()
    np.testing.assert_array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    np.testing.assert_array_equal(ours[ok], ref[ok])
    assert np.isnan(ours).sum() == 2  # S.1111.111 only


def test_e4m3_closed_forms():
    v = oracle.e4m3_value
    assert v(0x7E) == 448.0 and v(0xFE) == -448.0      # largest finite
    assert v(0x38) == 1.0 and v(0x40) == 2.0
    assert v(0x08) == 2.0 ** -6                         # smallest normal
    assert v(0x01) == 2.0 ** -9 and v(0x07) == 7 / 8 * 2.0 ** -6   # subnormals
    assert v(0x00) == 0.0 and np.signbit(v(0x80))


def test_e4m3_code_round_trips_every_finite_byte():
    c = np.array([b for b in range(256) if (b & 0x7F) != 0x7F], dtype=np.uint8)
    np.testing.assert_array_equal(oracle.e4m3_code(oracle.e4m3_value(c)), c)


def test_e4m3_code_matches_torch_rounding():
    """Round-half-even on random values and on every midpoint between neighbours."""
    import torch
    rng = np.random.default_rng(5)
    pos = oracle.e4m3_value(np.arange(0x7F))
    mids = (pos[:-1] + pos[1:]) / 2
    x = np.concatenate([rng.uniform(-448, 448, 20000), rng.standard_normal(20000) * 0.01,
                        mids, -mids]).astype(np.float32)
    ours = oracle.e4m3_code(x)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    np.testing.assert_array_equal(ours, ref)


def test_e4m3_group_quantiser_bounds():
    rng = np.random.default_rng(6)
    x = (rng.standard_normal((40, 2, 128)) * rng.uniform(0.01, 10, (40, 2, 1))).astype(np.float32)
    codes, meta = oracle.quantize_e4m3_g64(x)
    assert np.all(meta[..., 1] == 0)
    xh = oracle.dequantize_e4m3_g64(codes, meta)
    scale = meta[..., 0].astype(np.float64)
    g = x.reshape(40, 2, 2, 64).astype(np.float64)
    e = np.abs(xh.reshape(g.shape) - g)
    # 3 mantissa bits: half a unit in the last place is 2^-4 of the value in the normal
    # range; below 2^-6 (subnormal) it is scale * 2^-10 absolute
    bound = np.maximum(np.abs(g) * 2.0 ** -4, scale[..., None] * 2.0 ** -10)
    assert np.all(e <= bound * (1 + 1e-6) + 1e-12)
    # the group maximum lands on (or one step below, after fp16 rounding of the scale) 448
    top = np.abs(oracle.e4m3_value(codes)).reshape(g.shape).max(-1)
    assert np.all(top >= 416.0)


def test_e4m3_zero_group_and_saturation():
    x = np.zeros((1, 64), np.float32)
    codes, meta = oracle.quantize_e4m3_g64(x)
    assert np.all(codes == 0) and float(meta[0, 0, 0]) == 0.0
    with pytest.raises(ValueError):
        oracle.e4m3_code(np.array([449.0]))
