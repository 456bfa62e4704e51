"""Pins of the quantizer oracle (oracle.quantize): what it must reproduce
independently of its own code.

  * closed form: weights that lie exactly on a Q4NX grid (d a power of two,
    m a multiple of it, every group reaching codes 0 and 15) are recovered
    exactly -- codes, scale and offset;
  * brute force: an exact-rational re-implementation of the reading
    (oracle/brute.py) on tiny inputs, with ties, zeros, constant groups,
    clamped (NaN, inf, huge) and flushed (tiny) values;
  * bounds and properties: the dequantized weight is within half a step of w
    (plus the bf16 rounding of d and m), codes are monotone in w, a constant
    group has d = 0, an exact tie picks the smaller code.
"""
import struct

import numpy as np
import pytest

import oracle
from oracle import brute


def bf16_bits(x: float) -> int:
    b = struct.unpack("<I", struct.pack("<f", x))[0]
    assert b & 0xFFFF == 0, "test value must be exactly representable in bf16"
    return b >> 16


@pytest.mark.parametrize("e,mult", [(-7, -20), (-3, 5), (0, -7), (-12, 0), (4, -100)])
def test_exact_grid_is_recovered(e, mult):
    rng = np.random.default_rng(abs(e) * 100 + mult + 1000)
    N, K = 8, 128
    d = 2.0 ** e
    m = mult * d
    codes = rng.integers(0, 16, size=(N, K)).astype(np.uint8)
    codes.reshape(N, K // 32, 32)[:, :, 0] = 0
    codes.reshape(N, K // 32, 32)[:, :, 1] = 15
    W = (codes.astype(np.float64) * d + m).astype(np.float32)
    assert np.array_equal(W.astype(np.float64), codes.astype(np.float64) * d + m)  # exact grid
    c, s, o = oracle.quantize(W)
    assert np.array_equal(c, codes)
    assert (s == bf16_bits(d)).all()
    expect_m = bf16_bits(m) if m != 0 else 0
    assert (o == expect_m).all()


def _brute_quantize(W):
    N, K = W.shape
    Wc = oracle.clamp_weights(W)
    codes = np.zeros((N, K), np.uint8)
    s = np.zeros((N, K // 32), np.uint16)
    o = np.zeros((N, K // 32), np.uint16)
    for n in range(N):
        for g in range(K // 32):
            cb, sb, mb = brute.quantize_group_exact([float(v) for v in Wc[n, 32 * g:32 * g + 32]])
            codes[n, 32 * g:32 * g + 32] = cb
            s[n, g], o[n, g] = sb, mb
    return codes, s, o


def test_matches_exact_brute_force_on_tiny_inputs():
    rng = np.random.default_rng(7)
    W = (rng.standard_normal((6, 96)) * 0.03).astype(np.float32)
    W[0, :32] = 0.25                                    # constant group
    W[1, :32] = rng.integers(-3, 4, 32).astype(np.float32)  # many exact ties
    W[1, 5] = -0.0
    W[2, 32:64] = np.float32(2.0 ** -110) * rng.standard_normal(32).astype(np.float32)  # flushed d and m
    W[3, 64:] = rng.standard_normal(32).astype(np.float32) * np.float32(1e30)  # large, clamped
    W[3, 64] = np.inf
    W[3, 65] = -np.inf
    W[3, 66] = np.nan
    W[4, :32] = -np.abs(W[4, :32])                      # all negative
    W[5, 32:64] = 0.0                                   # all zero
    W[5, 40] = -0.0
    got = oracle.quantize(W)
    want = _brute_quantize(W)
    for a, b in zip(got, want):
        assert np.array_equal(a, b)


def test_error_within_half_step_plus_rounding():
    rng = np.random.default_rng(3)
    W = (rng.standard_normal((64, 512)) * 0.02).astype(np.float32)
    c, s, o = oracle.quantize(W)
    w_hat = oracle.dequant_f32(c, s, o).astype(np.float64)
    g = W.reshape(64, 16, 32).astype(np.float64)
    lo, hi = g.min(axis=2), g.max(axis=2)
    d = oracle.bf16_to_f32(s).astype(np.float64)
    bound = 0.5 * d + 2.0 ** -8 * (np.abs(lo) + (hi - lo)) + 2.0 ** -22 * np.maximum(np.abs(lo), np.abs(hi))
    err = np.abs(w_hat.reshape(64, 16, 32) - g).max(axis=2)
    assert (err <= bound).all()
    # an off-by-one code would cost about a whole step, which the bound excludes
    assert (bound < 0.9 * d).all()


def test_codes_are_monotone_in_w():
    rng = np.random.default_rng(5)
    W = (rng.standard_normal((16, 256)) * 0.02).astype(np.float32)
    c, _, _ = oracle.quantize(W)
    g = W.reshape(16, 8, 32)
    cg = c.reshape(16, 8, 32)
    order = np.argsort(g, axis=2, kind="stable")
    cs = np.take_along_axis(cg, order, axis=2).astype(int)
    assert (np.diff(cs, axis=2) >= 0).all()


def test_tie_takes_the_smaller_code():
    W = np.zeros((1, 32), np.float32)
    W[0, 0], W[0, 1] = 0.0, 15.0      # d = 1, m = 0: levels 0..15
    W[0, 2:] = np.float32(2.5)        # exactly between levels 2 and 3
    c, s, o = oracle.quantize(W)
    assert s[0, 0] == bf16_bits(1.0) and o[0, 0] == 0
    assert (c[0, 2:] == 2).all() and c[0, 0] == 0 and c[0, 1] == 15


def test_constant_group_has_zero_step():
    W = np.full((2, 64), np.float32(-0.375))
    c, s, o = oracle.quantize(W)
    assert (s == 0).all() and (c == 0).all() and (o == bf16_bits(-0.375)).all()
