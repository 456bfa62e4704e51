"""Q4NX oracle (NumPy, CPU).  Test infrastructure only; see the package header.

Everything here follows the plain definition of the operation, step by step:

  unpack code q[n,k] from its block            (Q4NX block, Sec. 3.1.1)
  d = scale[n, k/32], m = offset[n, k/32]      (group size 32, Sec. 3.1.1)
  w32[n,k] = RN_fp32(d*q + m)                  (Eq. 3)
  y[m,n]   = sum_k f64(x[m,k]) * f64(w32[n,k]) (Eq. 14/15; MM of Sec. 3.1.2)

Readings where the paper is silent (stated once here, used throughout):
  * A block is 32 output rows x 256 input columns (FusedDQP, Sec. 3.2.1); a
    quantization group is 32 consecutive input columns of one row, so a block
    row holds 8 groups and a block 256 groups (= 256 scales, 256 offsets).
  * Bytes inside a block: [codes 4096 B][scales 512 B][offsets 512 B].  Codes
    are row-major, row r owning bytes 128r..128r+127; byte j of a row holds
    column 2j in bits 0-3 and column 2j+1 in bits 4-7.  scale/offset index of
    (row r, group c) is 8r + c; bf16 values are stored little-endian.
  * Blocks are stored strip-major: block (i, j) (i = 32-row strip, j = 256-col
    block along K) starts at byte (i*KB + j)*5120 with KB = ceil(K/256).
  * K must be a multiple of 32.  N is padded to a multiple of 32 and K to a
    multiple of 256 with code 0, scale +0 and offset +0 (padded w = +0).
  * w32 is Eq. 3 evaluated in float32; the product d*q is exact (d has 8
    significant bits, q at most 4), so one rounding happens, at the addition.
  * The bf16 dequantized weight is RNE_bf16(w32).
"""
from __future__ import annotations

import numpy as np

BLOCK_ROWS = 32            # output rows per block (Sec. 3.1.1 / 3.2.1)
BLOCK_COLS = 256           # input columns per block
GROUP = 32                 # weights sharing one scale and one offset
GROUPS_PER_BLOCK_ROW = BLOCK_COLS // GROUP
CODE_BYTES = BLOCK_ROWS * BLOCK_COLS // 2           # 4096 (int4)
SCALE_BYTES = BLOCK_ROWS * GROUPS_PER_BLOCK_ROW * 2  # 512 (256 bf16)
OFFSET_BYTES = SCALE_BYTES                           # 512 (256 bf16)
BLOCK_BYTES = CODE_BYTES + SCALE_BYTES + OFFSET_BYTES  # 5120 (Sec. 3.1.1)


# ----------------------------------------------------------------------------
# bfloat16 <-> float32 at the bit level
# ----------------------------------------------------------------------------
def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float32: the bf16 bits are the top half."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest, ties to even.

    Adding 0x7FFF plus the lowest kept bit, then dropping the low 16 bits,
    rounds the magnitude to nearest with ties going to the even pattern.
    NaN inputs map to a quiet NaN of the same sign.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    if nan.any():
        r = r.copy()
        r[nan] = ((u[nan] >> np.uint64(16)).astype(np.uint16) | np.uint16(0x0040))
    return r


# ----------------------------------------------------------------------------
# format
# ----------------------------------------------------------------------------
def _ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def packed_size(N: int, K: int) -> int:
    """Bytes of a Q4NX matrix: one 5120-byte block per 32x256 tile (padded)."""
    if N <= 0 or K <= 0 or K % GROUP:
        return 0
    return _ceil_div(N, BLOCK_ROWS) * _ceil_div(K, BLOCK_COLS) * BLOCK_BYTES


def _padded(N: int, K: int):
    NS = _ceil_div(N, BLOCK_ROWS)
    KB = _ceil_div(K, BLOCK_COLS)
    return NS, KB, NS * BLOCK_ROWS, KB * BLOCK_COLS


def pack(codes: np.ndarray, scales: np.ndarray, offsets: np.ndarray) -> np.ndarray:
    """codes u8[N][K] (0..15), scales/offsets bf16 bits u16[N][K/32] -> blob u8."""
    codes = np.asarray(codes, dtype=np.uint8)
    N, K = codes.shape
    if K % GROUP or N <= 0:
        raise ValueError("need N > 0 and K a multiple of 32")
    if (codes > 15).any():
        raise ValueError("codes must lie in 0..15")
    G = K // GROUP
    scales = np.asarray(scales, dtype=np.uint16).reshape(N, G)
    offsets = np.asarray(offsets, dtype=np.uint16).reshape(N, G)
    NS, KB, Np, Kp = _padded(N, K)

    c = np.zeros((Np, Kp), dtype=np.uint8)
    c[:N, :K] = codes
    s = np.zeros((Np, Kp // GROUP), dtype=np.uint16)
    s[:N, :G] = scales
    o = np.zeros((Np, Kp // GROUP), dtype=np.uint16)
    o[:N, :G] = offsets

    # tile into (strip i, block j, row r, column within block)
    cb = c.reshape(NS, BLOCK_ROWS, KB, BLOCK_COLS).transpose(0, 2, 1, 3)
    nib = (cb[..., 0::2] | (cb[..., 1::2] << 4)).astype(np.uint8)       # (NS,KB,32,128)
    sb = s.reshape(NS, BLOCK_ROWS, KB, GROUPS_PER_BLOCK_ROW).transpose(0, 2, 1, 3)
    ob = o.reshape(NS, BLOCK_ROWS, KB, GROUPS_PER_BLOCK_ROW).transpose(0, 2, 1, 3)

    blob = np.empty((NS, KB, BLOCK_BYTES), dtype=np.uint8)
    blob[:, :, :CODE_BYTES] = nib.reshape(NS, KB, CODE_BYTES)
    blob[:, :, CODE_BYTES:CODE_BYTES + SCALE_BYTES] = (
        np.ascontiguousarray(sb).astype("<u2").reshape(NS, KB, -1).view(np.uint8))
    blob[:, :, CODE_BYTES + SCALE_BYTES:] = (
        np.ascontiguousarray(ob).astype("<u2").reshape(NS, KB, -1).view(np.uint8))
    return blob.reshape(-1)


def unpack(blob: np.ndarray, N: int, K: int):
    """blob -> (codes u8[N][K], scales u16[N][K/32], offsets u16[N][K/32])."""
    blob = np.asarray(blob, dtype=np.uint8)
    NS, KB, Np, Kp = _padded(N, K)
    if blob.size < NS * KB * BLOCK_BYTES:
        raise ValueError("blob too small")
    b = blob[:NS * KB * BLOCK_BYTES].reshape(NS, KB, BLOCK_BYTES)
    nib = b[:, :, :CODE_BYTES].reshape(NS, KB, BLOCK_ROWS, BLOCK_COLS // 2)
    cb = np.empty((NS, KB, BLOCK_ROWS, BLOCK_COLS), dtype=np.uint8)
    cb[..., 0::2] = nib & 0x0F
    cb[..., 1::2] = nib >> 4
    codes = cb.transpose(0, 2, 1, 3).reshape(Np, Kp)[:N, :K]

    def _vals(lo, hi):
        v = np.ascontiguousarray(b[:, :, lo:hi]).view("<u2").astype(np.uint16)
        v = v.reshape(NS, KB, BLOCK_ROWS, GROUPS_PER_BLOCK_ROW).transpose(0, 2, 1, 3)
        return v.reshape(Np, Kp // GROUP)[:N, :K // GROUP]

    scales = _vals(CODE_BYTES, CODE_BYTES + SCALE_BYTES)
    offsets = _vals(CODE_BYTES + SCALE_BYTES, BLOCK_BYTES)
    return np.ascontiguousarray(codes), np.ascontiguousarray(scales), np.ascontiguousarray(offsets)


# ----------------------------------------------------------------------------
# Eq. 3 and the projection
# ----------------------------------------------------------------------------
def dequant_f32(codes: np.ndarray, scales: np.ndarray, offsets: np.ndarray) -> np.ndarray:
    """Eq. 3 in float32: w = d_g * q + m_g with d_g, m_g the group's bf16 values."""
    q = np.asarray(codes, dtype=np.uint8).astype(np.float32)
    d = np.repeat(bf16_to_f32(scales), GROUP, axis=1)
    m = np.repeat(bf16_to_f32(offsets), GROUP, axis=1)
    prod = (d * q).astype(np.float32)       # exact: <= 12 significant bits
    return (prod + m).astype(np.float32)    # the single rounding


def dequant_bf16(codes, scales, offsets) -> np.ndarray:
    """Dequantized weights as bf16 bits: RNE_bf16 of the float32 Eq. 3 value."""
    return f32_to_bf16(dequant_f32(codes, scales, offsets))


def dequant_blob_f32(blob, N: int, K: int) -> np.ndarray:
    return dequant_f32(*unpack(blob, N, K))


def gemv_f64(w32: np.ndarray, x_bits: np.ndarray) -> np.ndarray:
    """Eq. 14: y = W x with x given as bf16 bits, accumulated in float64."""
    x = bf16_to_f32(np.asarray(x_bits).reshape(-1)).astype(np.float64)
    return np.asarray(w32, dtype=np.float64) @ x


def gemm_f64(X_bits: np.ndarray, w32: np.ndarray) -> np.ndarray:
    """Y[M][N] = X[M][K] . W[N][K]^T in float64 (C = A x B with B = W^T)."""
    X = bf16_to_f32(np.asarray(X_bits)).astype(np.float64)
    return X @ np.asarray(w32, dtype=np.float64).T


def abs_bound(X_bits: np.ndarray, w32: np.ndarray) -> np.ndarray:
    """sum_k |x[m,k] * w[n,k]| in float64: the scale of each output's error."""
    X = np.abs(bf16_to_f32(np.asarray(X_bits)).astype(np.float64))
    W = np.abs(np.asarray(w32, dtype=np.float64))
    if X.ndim == 1:
        return W @ X
    return X @ W.T


REL_TOL = 2e-3
ABS_TOL = 1e-5


def tolerance(bound: np.ndarray, y_ref: np.ndarray | None = None,
              bf16_out: bool = False) -> np.ndarray:
    """|y - y_ref| <= 2e-3 * bound + 1e-5, plus half a bf16 ulp of y_ref when
    the output itself is rounded to bf16."""
    tol = REL_TOL * np.asarray(bound, dtype=np.float64) + ABS_TOL
    if bf16_out:
        a = np.abs(np.asarray(y_ref, dtype=np.float64))
        tol = tol + a * 2.0 ** -8  # half ulp of an 8-bit significand, relative
    return tol


def check_close(y: np.ndarray, y_ref: np.ndarray, bound: np.ndarray,
                bf16_out: bool = False):
    """Return (ok, worst ratio |err| / tol)."""
    y = np.asarray(y, dtype=np.float64)
    err = np.abs(y - np.asarray(y_ref, dtype=np.float64))
    tol = tolerance(bound, y_ref, bf16_out)
    ratio = err / tol
    worst = float(np.nanmax(ratio)) if ratio.size else 0.0
    return bool(np.all(np.isfinite(y)) and worst <= 1.0), worst
