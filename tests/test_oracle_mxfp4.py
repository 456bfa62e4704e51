"""Pins of the MXFP4-variant oracle (oracle.mxfp4).

  * the FP4 E2M1 value table and the E8M0 scale as the OCP MX specification
    lists them (a literal table, not the bit-field formula);
  * block layout: packed size 4352 B per 32 x 256 block, a hand-derived byte
    map of a small matrix, pack/unpack round trip;
  * dequantization is exact (X * value, powers of two);
  * quantizer: exactly representable groups are recovered, the
    round-to-nearest-even cases of the FP4 grid, saturation at 6, and the
    per-element error bound.
"""
import numpy as np
import pytest

from oracle import mxfp4 as mx

SPEC_FP4 = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0, -0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0]


def test_fp4_table_and_e8m0():
    v = mx.fp4_value(np.arange(16))
    assert np.array_equal(v, SPEC_FP4)
    assert np.signbit(v[8]) and not np.signbit(v[0])
    assert mx.e8m0_value(127) == 1.0 and mx.e8m0_value(128) == 2.0 and mx.e8m0_value(27) == 2.0 ** -100


def test_block_size_and_hand_layout():
    assert mx.MX_BLOCK_BYTES == 4352 and mx.mx_packed_size(32, 256) == 4352
    assert mx.mx_packed_size(33, 288) == 2 * 2 * 4352
    N, K = 33, 288
    codes = np.zeros((N, K), np.uint8)
    scales = np.full((N, K // 32), 127, np.uint8)
    codes[0, 0], codes[0, 1] = 0x3, 0xA        # block (0,0) byte 0 = 0xA3
    codes[5, 257] = 0x7                         # block (0,1): row 5, col 1 -> byte 128*5 + 0, high nibble
    scales[32, 8] = 200                         # block (1,1): row 0, group 0 -> byte 4096 + 0
    scales[1, 3] = 28                           # block (0,0): row 1, group 3 -> byte 4096 + 11
    blob = mx.mx_pack(codes, scales)
    assert blob[0] == 0xA3
    assert blob[4352 + 640] == 0x70
    assert blob[3 * 4352 + 4096] == 200
    assert blob[4096 + 11] == 28
    assert blob[4096] == 127
    # padding: rows >= 33 in strip 1, columns >= 288 in column block 1: code 0, scale 127
    assert blob[3 * 4352 + 4096 + 8 * 5] == 127 and blob[3 * 4352 + 128 * 5] == 0
    c2, s2 = mx.mx_unpack(blob, N, K)
    assert np.array_equal(c2, codes) and np.array_equal(s2, scales)


def test_dequant_exact():
    rng = np.random.default_rng(0)
    codes = rng.integers(0, 16, (64, 512)).astype(np.uint8)
    scales = rng.integers(27, 228, (64, 16)).astype(np.uint8)
    w = mx.mx_dequant_f32(codes, scales).astype(np.float64)
    ref = np.array(SPEC_FP4)[codes] * np.repeat(2.0 ** (scales.astype(np.float64) - 127), 32, axis=1)
    assert np.array_equal(w, ref)


def test_quantize_recovers_representable_groups():
    rng = np.random.default_rng(1)
    N, K = 16, 256
    codes = rng.integers(0, 16, (N, K)).astype(np.uint8)
    codes.reshape(N, 8, 32)[:, :, 0] = 7        # +6 in every group: amax = 6 X
    scales = rng.integers(40, 200, (N, 8)).astype(np.uint8)
    W = mx.mx_dequant_f32(codes, scales)
    c, s = mx.mx_quantize(W)
    assert np.array_equal(s, scales)
    assert np.array_equal(mx.fp4_value(c), mx.fp4_value(codes))   # -0 and +0 may differ in code
    assert np.array_equal(mx.mx_dequant_f32(c, s), W)


@pytest.mark.parametrize("r,expect", [(0.25, 0.0), (0.75, 1.0), (1.25, 1.0), (1.75, 2.0), (2.5, 2.0),
                                      (3.5, 4.0), (5.0, 4.0), (7.9, 6.0), (-2.5, -2.0), (-5.0, -4.0),
                                      (0.26, 0.5), (2.6, 3.0), (5.1, 6.0)])
def test_fp4_rounding_ties_to_even_and_saturation(r, expect):
    W = np.zeros((1, 32), np.float32)
    W[0, 0] = 4.0          # amax in [4, 8): X = 1
    W[0, 1] = r
    c, s = mx.mx_quantize(W)
    assert s[0, 0] == 127
    assert mx.fp4_value(c[0, 1]) == expect


def test_quantize_error_bound_and_zero_group():
    rng = np.random.default_rng(2)
    W = (rng.standard_normal((32, 512)) * 0.02).astype(np.float32)
    W[3, :32] = 0.0
    c, s = mx.mx_quantize(W)
    assert (s[3, 0] == 127) and (c[3, :32] == 0).all()
    w_hat = mx.mx_dequant_f32(c, s).astype(np.float64)
    X = np.repeat(mx.e8m0_value(s), 32, axis=1)
    a = np.abs(W.astype(np.float64))
    bound = np.where(a <= 6 * X, X, a - 6 * X)   # half the largest FP4 spacing (2) below 6, saturation above
    assert (np.abs(w_hat - W) <= bound + 1e-30).all()


def test_quantize_domain_and_exponent_clamps():
    """Out-of-domain inputs follow the Q4NX quantizer's reading (NaN -> 0,
    clamp to +-2^100); the shared exponent is clamped to [-100, 100]."""
    W = np.zeros((1, 128), np.float32)
    W[0, 0:32] = np.nan                       # group 0: all NaN -> an all-zero group
    W[0, 32] = np.inf                         # group 1: clamped to 2^100 -> X = 2^98, code of 4.0
    W[0, 33] = -np.inf
    W[0, 64] = np.float32(2.0 ** -120)        # group 2: floor(log2) - 2 = -122 -> clamped to -100
    W[0, 96] = np.float32(3.0)                # group 3: floor(log2 3) - 2 = -1 -> X = 1/2, 3 / (1/2) = 6
    c, s = mx.mx_quantize(W)
    assert s[0].tolist() == [127, 127 + 98, 27, 126]
    assert (c[0, :32] == 0).all()
    assert c[0, 32] == 6 and c[0, 33] == 14   # +4.0 and -4.0
    assert c[0, 64] == 0                       # 2^-120 / 2^-100 rounds to 0
    assert c[0, 96] == 7                       # 6.0
    assert mx.mx_dequant_f32(c, s)[0, 32] == np.float32(2.0 ** 100)
