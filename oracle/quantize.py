"""Quantizer into Q4NX (oracle, NumPy, CPU).  Test infrastructure only.

The paper converts the model's weights offline into the Q4NX format, whose
groups follow the Q4_1 scheme: per group of 32 consecutive input columns a
minimal-value offset m and a step d, so that w is approximated by d*q + m with
a 4-bit code q (Sec. 3.1.1, Eq. 3).  It fixes neither how d and m are rounded
to bf16 nor how q is chosen.  Reading used here (and by the GPU quantizer):

  clamp   w -> 0 if NaN, else to [-2^100, 2^100]   (keeps d and m in the
          format's value domain; |m| <= 2^100 < 2^101, d < 2^98)
  lo, hi = min and max of the group's 32 (clamped) float32 values (a zero
          minimum is taken as +0)
  d32    = RN_f32( RN_f32(hi - lo) / 15 )           float32 arithmetic
  d      = RNE_bf16(d32),  m = RNE_bf16(lo)         the stored scale / offset
          (a magnitude below 2^-100 becomes a zero of the same sign)
  q      = the code 0..15 whose Eq. 3 value RN_f32(d*q + m) is nearest to w,
          distances taken as float64 differences, the smaller code on a tie

so every code is the best one for the stored (rounded) d and m.
"""
from __future__ import annotations

import numpy as np

from .q4nx import GROUP, bf16_to_f32, f32_to_bf16

CLAMP = np.float32(2.0 ** 100)
_MIN_MAG_BITS = 27 << 7  # bf16 bits of 2^-100


def _flush_tiny(bits: np.ndarray) -> np.ndarray:
    """Magnitudes below 2^-100 -> a zero of the same sign (bf16 bits)."""
    bits = np.asarray(bits, dtype=np.uint16).copy()
    tiny = (bits & 0x7FFF) < _MIN_MAG_BITS
    bits[tiny] &= 0x8000
    return bits


def clamp_weights(W: np.ndarray) -> np.ndarray:
    """NaN -> 0, everything else clamped to [-2^100, 2^100] (float32)."""
    W = np.asarray(W, dtype=np.float32)
    W = np.where(np.isnan(W), np.float32(0.0), W)
    return np.clip(W, -CLAMP, CLAMP).astype(np.float32)


def group_scale_offset(W: np.ndarray):
    """Scales and offsets (bf16 bits, [N][K/32]) of the clamped weights [N][K]."""
    N, K = W.shape
    g = W.reshape(N, K // GROUP, GROUP)
    lo = g.min(axis=2) + np.float32(0.0)   # -0 + +0 = +0: a zero minimum is +0
    hi = g.max(axis=2)
    d32 = (hi - lo) / np.float32(15.0)           # two float32 roundings
    scales = _flush_tiny(f32_to_bf16(d32))
    offsets = _flush_tiny(f32_to_bf16(lo))
    return scales, offsets


def quantize(W: np.ndarray, rows_per_chunk: int = 256):
    """float32 weights [N][K] (K % 32 == 0) -> codes u8[N][K], scales and
    offsets (bf16 bits, u16[N][K/32]), ready for the packer."""
    W = clamp_weights(W)
    N, K = W.shape
    if K % GROUP:
        raise ValueError("K must be a multiple of 32")
    scales, offsets = group_scale_offset(W)
    d = bf16_to_f32(scales)
    m = bf16_to_f32(offsets)
    q16 = np.arange(16, dtype=np.float32)
    codes = np.empty((N, K), dtype=np.uint8)
    for r0 in range(0, N, rows_per_chunk):
        r1 = min(N, r0 + rows_per_chunk)
        # Eq. 3 levels of each group: RN_f32(d*q + m) (d*q is exact).
        levels = d[r0:r1, :, None] * q16 + m[r0:r1, :, None]            # [n][G][16] float32
        w = W[r0:r1].reshape(r1 - r0, K // GROUP, GROUP)
        dist = np.abs(levels[:, :, None, :].astype(np.float64) - w[:, :, :, None].astype(np.float64))
        codes[r0:r1] = np.argmin(dist, axis=3).reshape(r1 - r0, K)      # first minimum: smaller code
    return codes, scales, offsets
