"""Oracle for the group-64 asymmetric cache quantiser and its dequantiser.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. 4.5 composes the reuse path with low-bit KV caches (KIVI / OTT 2- and 4-bit,
FP8): the cache is stored quantised and the probe offset then also absorbs the
mean quantisation error. The stand-in scheme here quantises every group of 64
consecutive head-dim elements of one (token, KV head) row:

  zero  = fp16(min of the group)
  scale = fp16((max - min) / (2^B - 1))          (fp32 arithmetic, then fp16)
  code  = clamp(round-half-even((x - zero) / scale), 0, 2^B - 1), 0 if scale == 0
  x_hat = scale * code + zero

The code decision is taken in fp32, the precision the GPU quantiser uses, so both
sides round identically. Codes are packed low bits first: with 4 bits element 2k
is the low nibble of byte k; with 2 bits element 4k sits in bits 0-1 of byte k.
"""
from __future__ import annotations

import numpy as np

GROUP = 64


def quantize_g64(x: np.ndarray, bits: int):
    """Quantise the last axis of x (length a multiple of 64).

    Returns (codes uint8 [..., hd], meta float16 [..., hd/64, 2] holding (scale, zero)).
    Codes are unpacked here; pack_codes packs them.
    """
    if bits not in (2, 4):
        raise ValueError("bits must be 2 or 4")
    x32 = np.asarray(x, dtype=np.float32)
    hd = x32.shape[-1]
    if hd % GROUP:
        raise ValueError("last axis must be a multiple of 64")
    g = x32.reshape(x32.shape[:-1] + (hd // GROUP, GROUP))
    mn = g.min(axis=-1)
    mx = g.max(axis=-1)
    levels = np.float32(2 ** bits - 1)
    zero16 = mn.astype(np.float16)
    scale16 = ((mx - mn) / levels).astype(np.float32).astype(np.float16)
    zero = zero16.astype(np.float32)[..., None]
    scale = scale16.astype(np.float32)[..., None]
    with np.errstate(divide="ignore", invalid="ignore"):
        t = (g - zero) / np.where(scale == 0, np.float32(1), scale)
    code = np.clip(np.rint(t), 0, 2 ** bits - 1)
    code = np.where(scale == 0, 0, code).astype(np.uint8)
    meta = np.stack([scale16, zero16], axis=-1)
    return code.reshape(x32.shape), meta


def dequantize_g64(codes: np.ndarray, meta: np.ndarray) -> np.ndarray:
    """x_hat = scale * code + zero per group of 64, in fp64 (exact for these operands)."""
    c = np.asarray(codes, dtype=np.float64)
    hd = c.shape[-1]
    g = c.reshape(c.shape[:-1] + (hd // GROUP, GROUP))
    scale = np.asarray(meta[..., 0], dtype=np.float64)[..., None]
    zero = np.asarray(meta[..., 1], dtype=np.float64)[..., None]
    return (g * scale + zero).reshape(c.shape)


def pack_codes(codes: np.ndarray, bits: int) -> np.ndarray:
    """Pack unpacked codes [..., hd] into bytes [..., hd * bits / 8], low bits first."""
    per = 8 // bits
    c = np.asarray(codes, dtype=np.uint8)
    c = c.reshape(c.shape[:-1] + (c.shape[-1] // per, per))
    out = np.zeros(c.shape[:-1], dtype=np.uint8)
    for k in range(per):
        out |= (c[..., k] << (bits * k)).astype(np.uint8)
    return out


def unpack_codes(packed: np.ndarray, bits: int) -> np.ndarray:
    per = 8 // bits
    p = np.asarray(packed, dtype=np.uint8)
    mask = (1 << bits) - 1
    parts = [(p >> (bits * k)) & mask for k in range(per)]
    return np.stack(parts, axis=-1).reshape(p.shape[:-1] + (p.shape[-1] * per,))


# ---- FP8 (E4M3) cache with one scale per 64 values ------------------------------------
# Sec. 4.5 lists FP8 (E4M3) among the cache formats the reuse path composes with; the
# paper does not say how values are scaled into the format. The reading taken here uses
# the same group-64 rows as the integer schemes, symmetric (no zero point):
#
#   scale = fp16(max|x| / 448)        (fp32 arithmetic, then fp16; 448 = largest E4M3)
#   code  = E4M3 of clamp(x / scale, -448, 448), round half to even, 0 if scale == 0
#   x_hat = scale * value(code)
#
# meta keeps the (scale, zero) pair layout of the integer schemes with zero = 0.

E4M3_MAX = 448.0


def e4m3_value(code) -> np.ndarray:
    """The number an E4M3 byte denotes (OCP FP8 E4M3: 1 sign, 4 exponent bits with bias
    7, 3 mantissa bits; exponent field 0 is subnormal; S.1111.111 is NaN; no infinity)."""
    c = np.asarray(code, dtype=np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 15
    m = (c & 7).astype(np.float64)
    mag = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * np.exp2(e.astype(np.float64) - 7))
    mag = np.where((e == 15) & ((c & 7) == 7), np.nan, mag)
    return sign * mag


_E4M3_POS = e4m3_value(np.arange(0x7F))  # the 127 finite non-negative values, increasing


def e4m3_code(v) -> np.ndarray:
    """Nearest E4M3 byte to each value (|v| <= 448), ties to the even code (the one whose
    last mantissa bit is 0: consecutive codes are consecutive values). The sign bit
    follows the sign of v, also when the magnitude rounds to zero."""
    v = np.asarray(v, dtype=np.float64)
    a = np.abs(v)
    if np.any(a > E4M3_MAX) or np.any(np.isnan(a)):
        raise ValueError("e4m3_code needs |v| <= 448")
    hi = np.searchsorted(_E4M3_POS, a, side="left")  # first value >= a
    hi = np.minimum(hi, len(_E4M3_POS) - 1)
    lo = np.maximum(hi - 1, 0)
    d_lo = a - _E4M3_POS[lo]
    d_hi = _E4M3_POS[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    mag = np.where(pick_hi, hi, lo)
    mag = np.where(a == _E4M3_POS[hi], hi, mag)
    return (mag | np.where(np.signbit(v), 0x80, 0)).astype(np.uint8)


def quantize_e4m3_g64(x: np.ndarray):
    """FP8 (E4M3) group-64 quantiser of the last axis (see the reading above).

    Returns (codes uint8 [..., hd], meta float16 [..., hd/64, 2] holding (scale, 0))."""
    x32 = np.asarray(x, dtype=np.float32)
    hd = x32.shape[-1]
    if hd % GROUP:
        raise ValueError("last axis must be a multiple of 64")
    g = x32.reshape(x32.shape[:-1] + (hd // GROUP, GROUP))
    amax = np.abs(g).max(axis=-1)
    scale16 = (amax / np.float32(E4M3_MAX)).astype(np.float32).astype(np.float16)
    scale = scale16.astype(np.float32)[..., None]
    with np.errstate(divide="ignore", invalid="ignore"):
        t = g / np.where(scale == 0, np.float32(1), scale)
    t = np.clip(t, np.float32(-E4M3_MAX), np.float32(E4M3_MAX))
    code = np.where(scale == 0, np.uint8(0), e4m3_code(np.where(scale == 0, 0, t)))
    meta = np.stack([scale16, np.zeros_like(scale16)], axis=-1)
    return code.astype(np.uint8).reshape(x32.shape), meta


def dequantize_e4m3_g64(codes: np.ndarray, meta: np.ndarray) -> np.ndarray:
    """x_hat = scale * value(code) per group of 64, in fp64."""
    v = e4m3_value(codes)
    hd = v.shape[-1]
    g = v.reshape(v.shape[:-1] + (hd // GROUP, GROUP))
    scale = np.asarray(meta[..., 0], dtype=np.float64)[..., None]
    return (g * scale).reshape(v.shape)
