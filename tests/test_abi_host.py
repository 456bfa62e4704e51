"""The C ABI on the host: the library loads and exports every entry point the
header declares; q4nx_pack / q4nx_unpack agree with the oracle byte for byte;
every argument error is reported before any HIP call (so these run without a
GPU: the device entry points are only called with invalid arguments)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_2602_06063_amd as q4
from workloads import gen_weights, gen_edge_weights, gen_mx_weights, MODELS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "q4nx.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(q4nx_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = _declared_functions()
    assert len(names) >= 9
    for n in names:
        assert hasattr(q4.lib, n), n
    assert sorted(q4.EXPORTED) == names


@pytest.mark.parametrize("N,K", [(1, 32), (32, 256), (33, 288), (1024, 1152), (1024, 2560), (300, 5376), (64, 21504)])
def test_packed_size_matches_oracle(N, K):
    assert q4.q4nx_packed_size(N, K) == oracle.packed_size(N, K)


def test_packed_size_rejects():
    for N, K in [(0, 256), (-1, 256), (32, 0), (32, 33), (32, 48), (1 << 31, 256), (32, 1 << 31)]:
        assert q4.q4nx_packed_size(N, K) == 0


SHAPES = [(1, 32, "zp"), (32, 256, "zp"), (33, 288, "literal"), (100, 1152, "zp"), (1024, 1152, "zp"),
          (256, 2560, "literal"), (64, 5376, "zp"), (40, 10240, "zp"), (70, 800, "edge")]


@pytest.mark.parametrize("N,K,mode", SHAPES)
def test_pack_bit_exact_vs_oracle_and_roundtrip(N, K, mode):
    if mode == "edge":
        codes, s, o = gen_edge_weights(N, K, seed=1)
    else:
        codes, s, o = gen_weights(N, K, seed=N + K, offset_mode=mode)
    blob = q4.q4nx_pack(codes, s, o)
    ref = oracle.pack(codes, s, o)
    assert blob.size == ref.size
    assert np.array_equal(blob, ref)
    c2, s2, o2 = q4.q4nx_unpack(blob, N, K)
    assert np.array_equal(c2, codes) and np.array_equal(s2, s) and np.array_equal(o2, o)


def test_pack_full_size_projection_shape_is_bit_exact():
    # a real Gemma3-4B shape (gate 10240 x 2560) through the threaded packer
    N, K = MODELS["4b"]["proj"][4][1:]
    codes, s, o = gen_weights(N, K, seed=0, layer=0, proj=4)
    assert np.array_equal(q4.q4nx_pack(codes, s, o), oracle.pack(codes, s, o))


def test_stacked_matrix_blob_is_the_blobs_back_to_back():
    """Blocks are stored strip by strip, so the blob of row-stacked matrices
    whose N are multiples of 32 is their blobs concatenated (the prefill runs
    q/k/v and gate/up as one product over such a stacked blob)."""
    K = 800
    parts = [gen_weights(N, K, seed=20 + i) for i, N in enumerate((64, 32, 96))]
    stacked = q4.q4nx_pack(*(np.concatenate([p[j] for p in parts]) for j in range(3)))
    assert np.array_equal(stacked, np.concatenate([q4.q4nx_pack(*p) for p in parts]))
    mparts = [gen_mx_weights(N, K, seed=30 + i) for i, N in enumerate((64, 32, 96))]
    mstacked = q4.q4nx_mx_pack(*(np.concatenate([p[j] for p in mparts]) for j in range(2)))
    assert np.array_equal(mstacked, np.concatenate([q4.q4nx_mx_pack(*p) for p in mparts]))


def _raw_pack(codes, s, o, N, K, blob_bytes):
    blob = np.zeros(max(blob_bytes, 1), np.uint8)
    st = q4.lib.q4nx_pack(q4._np_ptr(codes), q4._np_ptr(s), q4._np_ptr(o), N, K, q4._np_ptr(blob), blob_bytes)
    return st, blob


def test_pack_error_paths():
    N, K = 32, 256
    codes, s, o = gen_weights(N, K, seed=3)
    size = q4.q4nx_packed_size(N, K)
    st, _ = _raw_pack(codes, s, o, N, K, size)
    assert st == q4.Q4NX_OK
    # shapes
    assert _raw_pack(codes, s, o, 0, K, size)[0] == q4.Q4NX_ERR_SHAPE
    assert _raw_pack(codes, s, o, N, 48, size)[0] == q4.Q4NX_ERR_SHAPE
    assert _raw_pack(codes, s, o, N, -32, size)[0] == q4.Q4NX_ERR_SHAPE
    # blob too small
    assert _raw_pack(codes, s, o, N, K, size - 1)[0] == q4.Q4NX_ERR_BUFFER_TOO_SMALL
    # NULL pointers
    blob = np.zeros(size, np.uint8)
    for args in [(None, q4._np_ptr(s), q4._np_ptr(o)), (q4._np_ptr(codes), None, q4._np_ptr(o)),
                 (q4._np_ptr(codes), q4._np_ptr(s), None)]:
        assert q4.lib.q4nx_pack(*args, N, K, q4._np_ptr(blob), size) == q4.Q4NX_ERR_INVALID_ARG
    assert q4.lib.q4nx_pack(q4._np_ptr(codes), q4._np_ptr(s), q4._np_ptr(o), N, K, None, size) == q4.Q4NX_ERR_INVALID_ARG
    # a code above 15 anywhere, checked before anything is written
    bad = codes.copy()
    bad[17, 201] = 16
    st, blob = _raw_pack(bad, s, o, N, K, size)
    assert st == q4.Q4NX_ERR_INVALID_ARG and not blob.any()
    assert "code" in q4.lib.q4nx_last_error().decode()
    # scales / offsets outside {0} U [2^-100, 2^101): inf, nan, 2^-101, 2^101, subnormal
    for bits in (0x7F80, 0xFF80, 0x7FC0, 0x0D00, 0x8D00, 0x7200, 0xF200, 0x0001):
        s2 = s.copy()
        s2[5, 3] = bits
        assert _raw_pack(codes, s2, o, N, K, size)[0] == q4.Q4NX_ERR_INVALID_ARG, hex(bits)
        o2 = o.copy()
        o2[31, 7] = bits
        assert _raw_pack(codes, s, o2, N, K, size)[0] == q4.Q4NX_ERR_INVALID_ARG, hex(bits)
    # domain edges are accepted: +-0, +-2^-100, just below +-2^101
    for bits in (0x0000, 0x8000, 0x0D80, 0x8D80, 0x71FF, 0xF1FF):
        s2 = s.copy()
        s2[0, 0] = bits
        assert _raw_pack(codes, s2, o, N, K, size)[0] == q4.Q4NX_OK, hex(bits)


def test_unpack_error_paths():
    N, K = 32, 256
    codes, s, o = gen_weights(N, K, seed=3)
    blob = q4.q4nx_pack(codes, s, o)
    c = np.empty((N, K), np.uint8)
    ss = np.empty((N, K // 32), np.uint16)
    oo = np.empty((N, K // 32), np.uint16)
    P = q4._np_ptr
    assert q4.lib.q4nx_unpack(P(blob), blob.size - 1, N, K, P(c), P(ss), P(oo)) == q4.Q4NX_ERR_BUFFER_TOO_SMALL
    assert q4.lib.q4nx_unpack(None, blob.size, N, K, P(c), P(ss), P(oo)) == q4.Q4NX_ERR_INVALID_ARG
    assert q4.lib.q4nx_unpack(P(blob), blob.size, N, 40, P(c), P(ss), P(oo)) == q4.Q4NX_ERR_SHAPE


# Device entry points: only invalid arguments here, which must be rejected on
# the host before any HIP call (pointers below are never dereferenced).
A16 = 0x10000
MIS = 0x10002


def test_device_calls_validate_before_hip():
    L = q4.lib
    # dequant
    assert L.q4nx_dequant(None, 32, 256, A16, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_dequant(A16, 32, 250, A16, 0, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_dequant(A16, 0, 256, A16, 0, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_dequant(MIS, 32, 256, A16, 0, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_dequant(A16, 32, 256, MIS, 1, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_dequant(A16, 32, 256, A16, 7, None) == q4.Q4NX_ERR_INVALID_ARG
    # gemv
    assert L.q4nx_gemv(None, A16, A16, 0, 32, 256, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_gemv(A16, None, A16, 0, 32, 256, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_gemv(A16, A16, None, 0, 32, 256, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_gemv(A16, A16, A16, 0, 32, 100, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_gemv(A16, A16, A16, 0, -5, 256, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_gemv(A16, A16, A16, 0, 32, (1 << 30) + 32, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_gemv(MIS, A16, A16, 0, 32, 256, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_gemv(A16, MIS, A16, 0, 32, 256, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_gemv(A16, A16, MIS, 0, 32, 256, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_gemv(A16, A16, A16, 2, 32, 256, None) == q4.Q4NX_ERR_INVALID_ARG
    # gemv_batched
    arr = (q4.q4nx_gemv_desc * 9)()
    for i in range(9):
        arr[i] = q4.q4nx_gemv_desc(A16, A16, A16, 32, 256)
    assert L.q4nx_gemv_batched(arr, 0, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_gemv_batched(arr, 9, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_gemv_batched(None, 1, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    arr[2] = q4.q4nx_gemv_desc(A16, A16, A16, 32, 40)
    assert L.q4nx_gemv_batched(arr, 3, 0, None) == q4.Q4NX_ERR_SHAPE
    arr[2] = q4.q4nx_gemv_desc(A16, MIS, A16, 32, 256)
    assert L.q4nx_gemv_batched(arr, 3, 0, None) == q4.Q4NX_ERR_ALIGNMENT
    # gemm
    assert L.q4nx_gemm(0, 32, 256, A16, A16, A16, 0, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_gemm(4, 32, 80, A16, A16, A16, 0, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_gemm(4, 32, 256, None, A16, A16, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_gemm(4, 32, 256, A16, None, A16, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_gemm(4, 32, 256, A16, A16, None, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_gemm(4, 32, 256, MIS, A16, A16, 0, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_gemm(4, 32, 256, A16, MIS, A16, 0, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_gemm(4, 32, 256, A16, A16, MIS, 0, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_gemm(4, 32, 256, A16, A16, A16, 3, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_quantize(A16, 32, 80, A16, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_quantize(A16, 0, 256, A16, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_quantize(None, 32, 256, A16, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_quantize(A16, 32, 256, None, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_quantize(MIS, 32, 256, A16, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_quantize(A16, 32, 256, MIS, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_gemm_bf16(0, 32, 256, A16, A16, A16, 0, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_gemm_bf16(4, 32, 80, A16, A16, A16, 0, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_gemm_bf16(4, 32, 256, None, A16, A16, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_gemm_bf16(4, 32, 256, A16, None, A16, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_gemm_bf16(4, 32, 256, A16, A16, None, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_gemm_bf16(4, 32, 256, A16, MIS, A16, 0, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_gemm_bf16(4, 32, 256, A16, A16, A16, 3, None) == q4.Q4NX_ERR_INVALID_ARG


# ----------------------------------------------------------------- MXFP4 variant
@pytest.mark.parametrize("N,K", [(1, 32), (32, 256), (33, 288), (300, 5376), (64, 21504)])
def test_mx_packed_size_matches_oracle(N, K):
    assert q4.q4nx_mx_packed_size(N, K) == oracle.mx_packed_size(N, K)
    assert q4.q4nx_mx_packed_size(N, K) == ((N + 31) // 32) * ((K + 255) // 256) * 4352


def test_mx_packed_size_rejects():
    for N, K in [(0, 256), (-1, 256), (32, 0), (32, 33), (1 << 31, 256), (32, 1 << 31)]:
        assert q4.q4nx_mx_packed_size(N, K) == 0


@pytest.mark.parametrize("N,K,mode", [(1, 32, "model"), (32, 256, "model"), (33, 288, "edge"), (100, 1152, "model"),
                                      (70, 800, "edge"), (64, 5376, "model")])
def test_mx_pack_bit_exact_vs_oracle_and_roundtrip(N, K, mode):
    codes, sc = gen_mx_weights(N, K, seed=N + K, mode=mode)
    blob = q4.q4nx_mx_pack(codes, sc)
    ref = oracle.mx_pack(codes, sc)
    assert blob.size == ref.size
    assert np.array_equal(blob, ref)
    c2, s2 = q4.q4nx_mx_unpack(blob, N, K)
    assert np.array_equal(c2, codes) and np.array_equal(s2, sc)


def test_mx_pack_full_size_projection_shape_is_bit_exact():
    N, K = MODELS["4b"]["proj"][4][1:]
    codes, sc = gen_mx_weights(N, K, seed=0, proj=4)
    assert np.array_equal(q4.q4nx_mx_pack(codes, sc), oracle.mx_pack(codes, sc))


def test_mx_pack_error_paths():
    N, K = 32, 256
    codes, sc = gen_mx_weights(N, K, seed=3)
    size = q4.q4nx_mx_packed_size(N, K)
    P = q4._np_ptr

    def raw(c, s, n, k, nbytes):
        blob = np.zeros(max(nbytes, 1), np.uint8)
        return q4.lib.q4nx_mx_pack(P(c), P(s), n, k, P(blob), nbytes), blob

    assert raw(codes, sc, N, K, size)[0] == q4.Q4NX_OK
    assert raw(codes, sc, 0, K, size)[0] == q4.Q4NX_ERR_SHAPE
    assert raw(codes, sc, N, 48, size)[0] == q4.Q4NX_ERR_SHAPE
    assert raw(codes, sc, N, K, size - 1)[0] == q4.Q4NX_ERR_BUFFER_TOO_SMALL
    blob = np.zeros(size, np.uint8)
    assert q4.lib.q4nx_mx_pack(None, P(sc), N, K, P(blob), size) == q4.Q4NX_ERR_INVALID_ARG
    assert q4.lib.q4nx_mx_pack(P(codes), None, N, K, P(blob), size) == q4.Q4NX_ERR_INVALID_ARG
    assert q4.lib.q4nx_mx_pack(P(codes), P(sc), N, K, None, size) == q4.Q4NX_ERR_INVALID_ARG
    bad = codes.copy()
    bad[17, 201] = 16
    st, blob = raw(bad, sc, N, K, size)
    assert st == q4.Q4NX_ERR_INVALID_ARG and not blob.any()
    for e in (0, 1, 26, 228, 254, 255):        # outside [27, 227]; 255 is NaN in E8M0
        s2 = sc.copy()
        s2[5, 3] = e
        st, blob = raw(codes, s2, N, K, size)
        assert st == q4.Q4NX_ERR_INVALID_ARG and not blob.any(), e
        assert "scale" in q4.lib.q4nx_last_error().decode()
    for e in (27, 127, 227):
        s2 = sc.copy()
        s2[0, 0] = e
        assert raw(codes, s2, N, K, size)[0] == q4.Q4NX_OK, e
    c = np.empty((N, K), np.uint8)
    ss = np.empty((N, K // 32), np.uint8)
    good = q4.q4nx_mx_pack(codes, sc)
    assert q4.lib.q4nx_mx_unpack(P(good), good.size - 1, N, K, P(c), P(ss)) == q4.Q4NX_ERR_BUFFER_TOO_SMALL
    assert q4.lib.q4nx_mx_unpack(None, good.size, N, K, P(c), P(ss)) == q4.Q4NX_ERR_INVALID_ARG
    assert q4.lib.q4nx_mx_unpack(P(good), good.size, N, 40, P(c), P(ss)) == q4.Q4NX_ERR_SHAPE


def test_mx_device_calls_validate_before_hip():
    L = q4.lib
    assert L.q4nx_mx_quantize(A16, 32, 80, A16, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_mx_quantize(None, 32, 256, A16, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_mx_quantize(A16, 32, 256, None, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_mx_quantize(MIS, 32, 256, A16, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_mx_quantize(A16, 32, 256, MIS, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_mx_dequant(None, 32, 256, A16, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_mx_dequant(A16, 32, 250, A16, 0, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_mx_dequant(MIS, 32, 256, A16, 0, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_mx_dequant(A16, 32, 256, A16, 7, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_mx_gemv(None, A16, A16, 0, 32, 256, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_mx_gemv(A16, A16, A16, 0, 32, 100, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_mx_gemv(A16, MIS, A16, 0, 32, 256, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_mx_gemv(A16, A16, A16, 2, 32, 256, None) == q4.Q4NX_ERR_INVALID_ARG
    arr = (q4.q4nx_gemv_desc * 9)()
    for i in range(9):
        arr[i] = q4.q4nx_gemv_desc(A16, A16, A16, 32, 256)
    assert L.q4nx_mx_gemv_batched(arr, 0, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_mx_gemv_batched(arr, 9, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    arr[1] = q4.q4nx_gemv_desc(A16, A16, A16, 32, 40)
    assert L.q4nx_mx_gemv_batched(arr, 2, 0, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_mx_gemm(0, 32, 256, A16, A16, A16, 0, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_mx_gemm(4, 32, 80, A16, A16, A16, 0, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_mx_gemm(4, 32, 256, A16, None, A16, 0, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_mx_gemm(4, 32, 256, A16, MIS, A16, 0, None) == q4.Q4NX_ERR_ALIGNMENT
    assert L.q4nx_mx_gemm(4, 32, 256, A16, A16, A16, 3, None) == q4.Q4NX_ERR_INVALID_ARG


def test_gemm_ex_workspace_size_and_validation():
    """The split-K plan (device of 256 CUs: the planner's fallback without a
    GPU) and every argument error of q4nx_gemm_ex before any launch."""
    ws = q4.q4nx_gemm_workspace_size
    Q, MX, BF = q4.Q4NX_WEIGHTS_Q4NX, q4.Q4NX_WEIGHTS_MXFP4, q4.Q4NX_WEIGHTS_BF16
    for M, N, K in [(0, 256, 256), (4, 0, 256), (4, 32, 80), (-1, 32, 256), (4, 32, (1 << 30) + 32)]:
        assert ws(Q, M, N, K) == 0
    assert ws(7, 2048, 2560, 10240) == 0  # unknown format
    for f in (MX, BF):
        assert ws(f, 4096, 8192, 5376) == 0   # 512 tiles: two full rounds, nothing to split
    # Q4NX: W is dequantized to bf16 in the workspace first where the fused
    # kernel's Eq. 3 work would cost more than the dequantization pass -- every
    # product at M = 4096, the large 4B products at M = 2048 -- and not for the
    # short-K 4B q/k/v and o products or at M = 1024 (the fused kernel).
    assert ws(Q, 4096, 8192, 5376) == 8192 * 5376 * 2
    assert ws(Q, 2048, 20480, 2560) == 20480 * 2560 * 2
    assert ws(Q, 2048, 4096, 2560) == 0 and ws(Q, 2048, 2560, 2048) == 0
    assert ws(Q, 1024, 43008, 5376) == 0
    w = ws(BF, 2048, 2560, 10240)             # 80 tiles over a long K: split
    assert w > 0 and w % (4 * 2048 * 2560) == 0 and 2 <= w // (4 * 2048 * 2560) <= 4
    assert ws(MX, 2048, 2560, 10240) == w
    assert ws(Q, 2048, 2560, 10240) == 2560 * 10240 * 2 + w   # bf16 W, then the partials
    L = q4.lib
    args = lambda fmt, M, N, K, work, nbytes: (fmt, M, N, K, A16, A16, A16, 0, work, nbytes, None)
    assert L.q4nx_gemm_ex(*args(3, 4, 32, 256, None, 0)) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_gemm_ex(*args(-1, 4, 32, 256, None, 0)) == q4.Q4NX_ERR_INVALID_ARG
    for fmt in (q4.Q4NX_WEIGHTS_Q4NX, q4.Q4NX_WEIGHTS_MXFP4, q4.Q4NX_WEIGHTS_BF16):
        assert L.q4nx_gemm_ex(*args(fmt, 0, 32, 256, None, 0)) == q4.Q4NX_ERR_SHAPE
        assert L.q4nx_gemm_ex(*args(fmt, 4, 32, 80, None, 0)) == q4.Q4NX_ERR_SHAPE
        assert L.q4nx_gemm_ex(fmt, 4, 32, 256, None, A16, A16, 0, None, 0, None) == q4.Q4NX_ERR_INVALID_ARG
        assert L.q4nx_gemm_ex(fmt, 4, 32, 256, A16, MIS, A16, 0, None, 0, None) == q4.Q4NX_ERR_ALIGNMENT
        wf = ws(fmt, 2048, 2560, 10240)
        assert L.q4nx_gemm_ex(*args(fmt, 2048, 2560, 10240, MIS, wf)) == q4.Q4NX_ERR_ALIGNMENT
        assert L.q4nx_gemm_ex(*args(fmt, 2048, 2560, 10240, A16, wf - 1)) == q4.Q4NX_ERR_BUFFER_TOO_SMALL
        assert L.q4nx_gemm_ex(*args(fmt, 2048, 2560, 10240, A16, 0)) == q4.Q4NX_ERR_BUFFER_TOO_SMALL


def test_stream_read_validation():
    L = q4.lib
    assert L.q4nx_stream_read(None, 16, A16, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_stream_read(A16, 16, None, None) == q4.Q4NX_ERR_INVALID_ARG
    assert L.q4nx_stream_read(A16, 0, A16, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_stream_read(A16, 24, A16, None) == q4.Q4NX_ERR_SHAPE
    assert L.q4nx_stream_read(MIS, 16, A16, None) == q4.Q4NX_ERR_ALIGNMENT


def test_status_strings():
    for st in range(6):
        assert q4.lib.q4nx_status_str(st).decode()
    assert q4.lib.q4nx_status_str(99).decode() == "unknown status"


def test_single_hip_runtime_in_process():
    """The library must share torch's HIP runtime, not load a second one."""
    maps = open("/proc/self/maps").read()
    paths = {line.split()[-1] for line in maps.splitlines() if "libamdhip64" in line}
    assert len(paths) == 1, paths
    import torch
    torch_lib = os.path.join(os.path.dirname(torch.__file__), "lib")
    assert next(iter(paths)).startswith(torch_lib), paths


def test_flowkv_workspace_size_and_validation():
    import paper_2602_06063_amd as q4
    L = q4.lib
    assert L.q4nx_flowkv_workspace_size(8, 256, 1) == 8 * 1 * 260 * 4
    assert L.q4nx_flowkv_workspace_size(8, 256, 257) == 8 * 17 * 260 * 4
    assert L.q4nx_flowkv_workspace_size(32, 128, 32768) == 32 * 2048 * 132 * 4
    assert L.q4nx_flowkv_workspace_size(0, 256, 10) == 0 and L.q4nx_flowkv_workspace_size(8, 256, 0) == 0
    A = ctypes.c_void_p(1 << 20)      # aligned, never dereferenced: every call below fails validation
    MIS = ctypes.c_void_p((1 << 20) + 2)
    W = 1 << 30

    def call(q=A, k=A, v=A, H=8, G=4, d=256, Lc=1024, t=10, win=0, scale=0.0625, o=A, odt=0, work=A, wb=W):
        return L.q4nx_flowkv_decode(q, k, v, H, G, d, Lc, t, win, scale, o, odt, work, wb, None)
    assert call(q=None) == q4.Q4NX_ERR_INVALID_ARG
    assert call(work=None) == q4.Q4NX_ERR_INVALID_ARG
    assert call(odt=5) == q4.Q4NX_ERR_INVALID_ARG
    assert call(scale=float("inf")) == q4.Q4NX_ERR_INVALID_ARG
    assert call(H=6, G=4) == q4.Q4NX_ERR_SHAPE
    assert call(H=48, G=3) == q4.Q4NX_ERR_SHAPE        # H/G = 16
    assert call(d=96) == q4.Q4NX_ERR_SHAPE
    assert call(t=1024) == q4.Q4NX_ERR_SHAPE
    assert call(t=-1) == q4.Q4NX_ERR_SHAPE
    assert call(win=-2) == q4.Q4NX_ERR_SHAPE
    assert call(k=MIS) == q4.Q4NX_ERR_ALIGNMENT
    assert call(work=MIS) == q4.Q4NX_ERR_ALIGNMENT
    assert call(wb=8 * 260 * 4 - 1) == q4.Q4NX_ERR_BUFFER_TOO_SMALL


def test_flowkv_static_validates_before_hip():
    """The entry point that allocates nothing checks every argument before any
    HIP call (these run without a GPU: each call fails validation)."""
    import paper_2602_06063_amd as q4
    L = q4.lib
    A = ctypes.c_void_p(1 << 20)
    MIS = ctypes.c_void_p((1 << 20) + 2)

    def call(q=A, k=A, v=A, H=8, G=4, d=256, Lc=1024, t=10, win=0, scale=0.0625, o=A, odt=0):
        return L.q4nx_flowkv_decode_static(q, k, v, H, G, d, Lc, t, win, scale, o, odt, None)
    assert call(q=None) == q4.Q4NX_ERR_INVALID_ARG
    assert call(o=None) == q4.Q4NX_ERR_INVALID_ARG
    assert call(odt=7) == q4.Q4NX_ERR_INVALID_ARG
    assert call(scale=float("nan")) == q4.Q4NX_ERR_INVALID_ARG
    assert call(H=6, G=4) == q4.Q4NX_ERR_SHAPE
    assert call(d=96) == q4.Q4NX_ERR_SHAPE
    assert call(t=1024) == q4.Q4NX_ERR_SHAPE
    assert call(win=-1) == q4.Q4NX_ERR_SHAPE
    assert call(v=MIS) == q4.Q4NX_ERR_ALIGNMENT
    assert "q4nx_flowkv_decode_static" in L.q4nx_last_error().decode()
