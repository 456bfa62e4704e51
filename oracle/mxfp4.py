"""MXFP4 variant of the Q4NX block (oracle, NumPy, CPU).  Test infrastructure only.

The paper notes that Q4NX can be extended to MXFP4 (Sec. 3.1.1) without
defining it.  The element and scale encodings follow the OCP Microscaling
(MX) format specification v1.0 for MXFP4: blocks of 32 elements, each a 4-bit
FP4 E2M1 value (1 sign, 2 exponent bits with bias 1, 1 mantissa bit; values
0, 0.5, 1, 1.5, 2, 3, 4, 6 and their negatives), sharing one 8-bit E8M0
scale X = 2^(e - 127).  Reading used for the Q4NX-shaped variant:

  * the same 32 x 256 blocks, strip-major order, nibble layout and group
    (32 consecutive input columns of one row) as Q4NX;
  * a block holds [codes 4096 B][scales 256 B] -- the E8M0 byte of (row r,
    group c) at index 8r + c -- 4352 bytes; there is no offset; padding is
    code 0 with scale byte 127 (value +0);
  * w = X * fp4(q), exact in float32 and bf16 inside the value domain
    e in [27, 227] (X in [2^-100, 2^100]), which the packer enforces;
  * quantizer (the specification's conversion): per group amax = max |w|;
    the shared exponent is floor(log2(amax)) - 2 (2 = the largest FP4
    exponent), clamped to [-100, 100] (0 for an all-zero group); each element
    is w / X rounded to the nearest FP4 value, ties to the even mantissa,
    saturating at +-6.  Inputs are first taken into the domain exactly as
    for the Q4NX quantizer: NaN -> 0, everything else clamped to
    [-2^100, 2^100].
"""
from __future__ import annotations

import numpy as np

from .q4nx import BLOCK_ROWS, BLOCK_COLS, GROUP, GROUPS_PER_BLOCK_ROW, CODE_BYTES, _ceil_div
from .quantize import clamp_weights

MX_SCALE_BYTES = BLOCK_ROWS * GROUPS_PER_BLOCK_ROW  # 256 E8M0 bytes
MX_BLOCK_BYTES = CODE_BYTES + MX_SCALE_BYTES        # 4352
MX_EXP_MIN, MX_EXP_MAX = 27, 227                     # accepted E8M0 codes (2^-100 .. 2^100)


def fp4_value(code: np.ndarray) -> np.ndarray:
    """FP4 E2M1 code (0..15) -> its value (float64), from the bit fields."""
    code = np.asarray(code, dtype=np.int64)
    sign = np.where(code & 8, -1.0, 1.0)
    e = (code >> 1) & 3
    m = code & 1
    mag = np.where(e == 0, 0.5 * m, (1.0 + 0.5 * m) * np.exp2(e - 1.0))
    return sign * mag


def e8m0_value(e: np.ndarray) -> np.ndarray:
    return np.exp2(np.asarray(e, dtype=np.float64) - 127.0)


def mx_packed_size(N: int, K: int) -> int:
    return _ceil_div(N, BLOCK_ROWS) * _ceil_div(K, BLOCK_COLS) * MX_BLOCK_BYTES


def mx_pack(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """codes u8[N][K] (0..15), scales u8[N][K/32] (E8M0) -> blob (uint8)."""
    N, K = codes.shape
    if K % GROUP or scales.shape != (N, K // GROUP):
        raise ValueError("bad shapes")
    if codes.max(initial=0) > 15 or scales.min(initial=MX_EXP_MIN) < MX_EXP_MIN or scales.max(initial=0) > MX_EXP_MAX:
        raise ValueError("value outside the domain")
    NS, KB = _ceil_div(N, BLOCK_ROWS), _ceil_div(K, BLOCK_COLS)
    Np, Kp = NS * BLOCK_ROWS, KB * BLOCK_COLS
    c = np.zeros((Np, Kp), np.uint8)
    c[:N, :K] = codes
    s = np.full((Np, Kp // GROUP), 127, np.uint8)  # padding: code 0 with scale 1 (value +0)
    s[:N, :K // GROUP] = scales
    blob = np.zeros(NS * KB * MX_BLOCK_BYTES, np.uint8)
    for i in range(NS):
        for j in range(KB):
            base = (i * KB + j) * MX_BLOCK_BYTES
            cb = c[32 * i:32 * i + 32, 256 * j:256 * j + 256]
            blob[base:base + CODE_BYTES] = (cb[:, 0::2] | (cb[:, 1::2] << 4)).reshape(-1)
            blob[base + CODE_BYTES:base + MX_BLOCK_BYTES] = s[32 * i:32 * i + 32, 8 * j:8 * j + 8].reshape(-1)
    return blob


def mx_unpack(blob: np.ndarray, N: int, K: int):
    NS, KB = _ceil_div(N, BLOCK_ROWS), _ceil_div(K, BLOCK_COLS)
    c = np.zeros((NS * BLOCK_ROWS, KB * BLOCK_COLS), np.uint8)
    s = np.zeros((NS * BLOCK_ROWS, KB * GROUPS_PER_BLOCK_ROW), np.uint8)
    for i in range(NS):
        for j in range(KB):
            base = (i * KB + j) * MX_BLOCK_BYTES
            b = blob[base:base + CODE_BYTES].reshape(32, 128)
            c[32 * i:32 * i + 32, 256 * j:256 * j + 256:2] = b & 0xF
            c[32 * i:32 * i + 32, 256 * j + 1:256 * j + 256:2] = b >> 4
            s[32 * i:32 * i + 32, 8 * j:8 * j + 8] = blob[base + CODE_BYTES:base + MX_BLOCK_BYTES].reshape(32, 8)
    return c[:N, :K], s[:N, :K // GROUP]


def mx_dequant_f32(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """w = X * fp4(q), exact (float32)."""
    N, K = codes.shape
    X = np.repeat(e8m0_value(scales), GROUP, axis=1)
    return (fp4_value(codes) * X).astype(np.float32)


def _round_fp4(r: np.ndarray) -> np.ndarray:
    """Nearest FP4 E2M1 code of r (float64), ties to the even mantissa,
    saturating at +-6."""
    mags = fp4_value(np.arange(8))               # 0, .5, 1, 1.5, 2, 3, 4, 6
    a = np.minimum(np.abs(r), 6.0)
    dist = np.abs(a[..., None] - mags)
    best = dist.min(axis=-1, keepdims=True)
    tied = dist == best
    # among equally near magnitudes take the one with an even mantissa bit
    even = tied & ((np.arange(8) & 1) == 0)
    pick = np.where(even.any(axis=-1), np.argmax(even, axis=-1), np.argmax(tied, axis=-1))
    return (pick | np.where(r < 0, 8, 0)).astype(np.uint8)


def mx_quantize(W: np.ndarray):
    """float32 W[N][K] -> codes u8[N][K], E8M0 scales u8[N][K/32]."""
    W = clamp_weights(W).astype(np.float64)
    N, K = W.shape
    g = W.reshape(N, K // GROUP, GROUP)
    amax = np.abs(g).max(axis=2)
    _, e2 = np.frexp(amax)                      # amax = f * 2^e2, f in [0.5, 1): floor(log2) = e2 - 1
    ex = np.where(amax > 0, e2 - 1 - 2, 0)
    ex = np.clip(ex, MX_EXP_MIN - 127, MX_EXP_MAX - 127).astype(np.int64)
    scales = (ex + 127).astype(np.uint8)
    codes = _round_fp4(g / np.exp2(ex)[:, :, None]).reshape(N, K)
    return codes, scales
