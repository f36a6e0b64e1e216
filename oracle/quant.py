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
