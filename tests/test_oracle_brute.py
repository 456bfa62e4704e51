"""The NumPy oracle against the pure-Python exact-rational brute force on tiny
shapes: the dequantized float32 bits must be identical (signed zeros
included) and the float64 projections within 1e-12 of the exact sums."""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import brute
from workloads import gen_weights, gen_activations, gen_edge_weights


CASES = [(1, 32, "zp"), (32, 256, "literal"), (33, 288, "zp"), (5, 1152, "zp"),
         (64, 64, "edge"), (3, 544, "edge")]


@pytest.mark.parametrize("N,K,mode", CASES)
def test_dequant_bits_and_projection_match_brute_force(N, K, mode):
    if mode == "edge":
        codes, s, o = gen_edge_weights(N, K, seed=N + K)
    else:
        codes, s, o = gen_weights(N, K, seed=N * 7 + K, offset_mode=mode)
    blob = oracle.pack(codes, s, o)
    bl = blob.tolist()
    w_brute = np.array(brute.dequant_bits(bl, N, K), dtype=np.uint32)
    w = oracle.dequant_blob_f32(blob, N, K)
    assert np.array_equal(w.view(np.uint32), w_brute)

    M = 2
    X = gen_activations((M, K), seed=N + 3 * K)
    Y = oracle.gemm_f64(X, w)
    bound = oracle.abs_bound(X, w)
    Yx = brute.project_exact(bl, N, K, X.tolist())
    for m in range(M):
        for n in range(N):
            err = abs(Fraction(float(Y[m, n])) - Yx[m][n])
            assert err <= Fraction(1e-12) * Fraction(float(bound[m, n])) + Fraction(1, 10 ** 300), (m, n)


def test_brute_rounding_helper_against_struct():
    """round_to_f32 agrees with the platform's binary64 -> binary32 conversion
    on values that are exact in binary64."""
    import struct
    rng = np.random.default_rng(0)
    for v in rng.standard_normal(2000) * 10.0 ** rng.integers(-30, 30, 2000):
        want = struct.unpack("<f", struct.pack("<f", float(v)))[0]
        assert brute.round_to_f32(Fraction(float(v))) == Fraction(want)
