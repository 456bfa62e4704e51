"""Pins of the CPU oracle against facts fixed outside it: the constants the
paper prints, hand-worked Eq. 3 values, the hand-derived byte layout, special
cases with textbook answers, and an independent bf16 rounding routine."""
import os

import numpy as np
import pytest

import oracle
from workloads import gen_weights, gen_activations, gen_edge_weights, MODELS


def _read_kv(path):
    out = {}
    for line in open(path):
        line = line.split("#", 1)[0].strip()
        if line:
            k, v = line.split()
            out[k] = int(v)
    return out


def _hexfloat(tok):
    return float.fromhex(tok) if "0x" in tok else float(tok)


# ---------------------------------------------------------------- PIN1/PIN2
def test_block_geometry_matches_paper(golden_dir):
    c = _read_kv(os.path.join(golden_dir, "paper_constants.txt"))
    assert oracle.BLOCK_ROWS == c["block_rows"]
    assert oracle.BLOCK_COLS == c["block_cols"]
    assert oracle.GROUP == c["group_size"]
    assert oracle.BLOCK_BYTES == c["block_bytes"]
    assert oracle.packed_size(32, 256) == c["block_bytes"]
    # 5 bits per weight: 4-bit code plus (2 + 2 bytes) / 32 weights
    assert oracle.packed_size(32, 256) * 8 / (32 * 256) == 5.0
    # a block's 256 groups give exactly 256 scales and 256 offsets
    codes = np.zeros((32, 256), np.uint8)
    s = np.arange(256, dtype=np.uint16).reshape(32, 8) + 0x3F80
    o = np.arange(256, dtype=np.uint16).reshape(32, 8) + 0x4000
    blob = oracle.pack(codes, s, o)
    _, s2, o2 = oracle.unpack(blob, 32, 256)
    assert s2.size == c["scales_per_block"] and o2.size == c["offsets_per_block"]
    assert len(set(s2.ravel().tolist())) == 256


def test_packed_size_rules():
    assert oracle.packed_size(1024, 1152) == 32 * 5 * 5120      # K=1152: 4.5 blocks -> 5
    assert oracle.packed_size(33, 256) == 2 * 5120
    assert oracle.packed_size(1, 32) == 5120
    assert oracle.packed_size(0, 256) == 0
    assert oracle.packed_size(32, 0) == 0
    assert oracle.packed_size(32, 48) == 0                       # K % 32 != 0


def test_gemma3_4b_attention_shapes_follow_paper(golden_dir):
    c = _read_kv(os.path.join(golden_dir, "paper_constants.txt"))
    m = MODELS["4b"]
    p = dict((n, (N, K)) for n, N, K in m["proj"])
    D, H, G, d = c["model_dim"], c["heads"], c["kv_groups"], c["head_dim"]
    assert m["layers"] == c["layers_4b"]
    assert p["q"] == (H * d, D)
    assert p["k"] == (G * d, D) and p["v"] == (G * d, D)
    assert p["o"] == (D, H * d)
    assert p["gate"][1] == D and p["up"][1] == D and p["down"][0] == D


# ---------------------------------------------------------------- PIN3
def test_eq3_closed_form(golden_dir):
    rows = []
    for line in open(os.path.join(golden_dir, "eq3_closed_form.txt")):
        line = line.split("#", 1)[0].strip()
        if line:
            t = line.split()
            rows.append((int(t[0], 16), int(t[1], 16), [_hexfloat(v) for v in t[2:]]))
    assert len(rows) == 9
    for d_bits, m_bits, expect in rows:
        assert len(expect) == 16
        codes = np.tile(np.arange(16, dtype=np.uint8), 2).reshape(1, 32)
        s = np.array([[d_bits]], np.uint16)
        o = np.array([[m_bits]], np.uint16)
        w = oracle.dequant_f32(codes, s, o)[0, :16]
        want = np.array(expect, dtype=np.float32)
        # bitwise, so the sign of zero counts
        assert np.array_equal(w.view(np.uint32), want.view(np.uint32)), (hex(d_bits), hex(m_bits), w, want)


def test_dequant_bf16_is_rne_of_f32():
    codes, s, o = gen_weights(64, 512, seed=3)
    w32 = oracle.dequant_f32(codes, s, o)
    w16 = oracle.dequant_bf16(codes, s, o)
    import torch
    ref = torch.from_numpy(w32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(w16, ref)


# ---------------------------------------------------------------- layout
def test_block_layout_hand_bytes(golden_dir):
    cases, cur = [], None
    for line in open(os.path.join(golden_dir, "block_layout_bytes.txt")):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        t = line.split()
        if t[0] == "case":
            cur = (int(t[1]), int(t[2]), int(t[3]), [])
            cases.append(cur)
        else:
            cur[3].append((int(t[0]), int(t[1], 16)))
    assert len(cases) == 2
    for N, K, total, pairs in cases:
        G = K // 32
        n = np.arange(N)[:, None]
        k = np.arange(K)[None, :]
        codes = ((n + 3 * k) % 16).astype(np.uint8)
        g = np.arange(G)[None, :]
        s = (0x3F80 + g + G * n).astype(np.uint16)
        o = (0xC000 + g + G * n).astype(np.uint16)
        blob = oracle.pack(codes, s, o)
        assert blob.size == total == oracle.packed_size(N, K)
        for off, val in pairs:
            assert blob[off] == val, (N, K, off, hex(blob[off]), hex(val))


# ---------------------------------------------------------------- PIN4
@pytest.mark.parametrize("N,K", [(1, 32), (32, 256), (33, 288), (64, 1152), (100, 544)])
def test_pack_roundtrip_and_zero_padding(N, K):
    codes, s, o = gen_weights(N, K, seed=11)
    blob = oracle.pack(codes, s, o)
    c2, s2, o2 = oracle.unpack(blob, N, K)
    assert np.array_equal(c2, codes) and np.array_equal(s2, s) and np.array_equal(o2, o)
    # all bytes that belong to padded rows / columns are zero
    NS, KB = -(-N // 32), -(-K // 256)
    pad_codes = np.zeros((NS * 32, KB * 256), bool)
    pad_codes[N:, :] = True
    pad_codes[:, K:] = True
    b = blob.reshape(NS, KB, 5120)
    nib = b[:, :, :4096].reshape(NS, KB, 32, 128)
    lo = (nib & 15).transpose(0, 2, 1, 3).reshape(NS * 32, KB * 128)
    hi = (nib >> 4).transpose(0, 2, 1, 3).reshape(NS * 32, KB * 128)
    assert not lo[pad_codes[:, 0::2]].any() and not hi[pad_codes[:, 1::2]].any()
    sv = b[:, :, 4096:].copy().view("<u2").reshape(NS, KB, 2, 32, 8)
    sv = sv.transpose(2, 0, 3, 1, 4).reshape(2, NS * 32, KB * 8)
    pad_groups = np.zeros((NS * 32, KB * 8), bool)
    pad_groups[N:, :] = True
    pad_groups[:, K // 32:] = True
    assert not sv[:, pad_groups].any()


def test_pack_is_injective():
    codes, s, o = gen_weights(32, 256, seed=5)
    base = oracle.pack(codes, s, o)
    rng = np.random.default_rng(0)
    for _ in range(50):
        c2, s2, o2 = codes.copy(), s.copy(), o.copy()
        which = rng.integers(0, 3)
        if which == 0:
            i, j = rng.integers(0, 32), rng.integers(0, 256)
            c2[i, j] = (c2[i, j] + 1 + rng.integers(0, 15)) % 16
        elif which == 1:
            i, j = rng.integers(0, 32), rng.integers(0, 8)
            s2[i, j] ^= np.uint16(1 << int(rng.integers(0, 16)))
        else:
            i, j = rng.integers(0, 32), rng.integers(0, 8)
            o2[i, j] ^= np.uint16(1 << int(rng.integers(0, 16)))
        assert not np.array_equal(oracle.pack(c2, s2, o2), base)


def test_pack_rejects_bad_input():
    with pytest.raises(ValueError):
        oracle.pack(np.full((32, 256), 16, np.uint8), np.zeros((32, 8), np.uint16), np.zeros((32, 8), np.uint16))
    with pytest.raises(ValueError):
        oracle.pack(np.zeros((32, 48), np.uint8), np.zeros((32, 1), np.uint16), np.zeros((32, 1), np.uint16))


# ---------------------------------------------------------------- PIN5
def test_unit_scale_zero_offset_is_integer_matvec():
    rng = np.random.default_rng(1)
    N, K = 48, 544
    codes = rng.integers(0, 16, (N, K)).astype(np.uint8)
    s = np.full((N, K // 32), 0x3F80, np.uint16)   # d = 1
    o = np.zeros((N, K // 32), np.uint16)           # m = +0
    xi = rng.integers(-8, 9, K)
    x = oracle.f32_to_bf16(xi.astype(np.float32))
    w = oracle.dequant_blob_f32(oracle.pack(codes, s, o), N, K)
    assert np.array_equal(w, codes.astype(np.float32))
    y = oracle.gemv_f64(w, x)
    assert np.array_equal(y, (codes.astype(np.int64) @ xi).astype(np.float64))


def test_zero_scale_gives_offset_times_group_sums():
    codes, s, o = gen_weights(40, 1152, seed=7)
    s[:] = 0
    x = gen_activations(1152, seed=7)
    w = oracle.dequant_f32(codes, s, o)
    y = oracle.gemv_f64(w, x)
    xf = oracle.bf16_to_f32(x).astype(np.float64)
    S = xf.reshape(-1, 32).sum(axis=1)                       # group sums of x
    m = oracle.bf16_to_f32(o).astype(np.float64)
    assert np.allclose(y, m @ S, rtol=1e-12, atol=1e-12)


def test_unit_vector_extracts_column_and_ones_give_row_sums():
    N, K = 70, 800
    codes, s, o = gen_weights(N, K, seed=9)
    blob = oracle.pack(codes, s, o)
    w = oracle.dequant_blob_f32(blob, N, K)
    for k in (0, 1, 31, 32, 255, 256, 257, 799):
        e = np.zeros(K, np.uint16)
        e[k] = 0x3F80
        y = oracle.gemv_f64(w, e)
        assert np.array_equal(y, w[:, k].astype(np.float64))
        # the column is Eq. 3 of that column's code and group values
        g = k // 32
        col = (oracle.bf16_to_f32(s[:, g]) * codes[:, k].astype(np.float32)) + oracle.bf16_to_f32(o[:, g])
        assert np.array_equal(y, col.astype(np.float32).astype(np.float64))
    ones = np.full(K, 0x3F80, np.uint16)
    assert np.allclose(oracle.gemv_f64(w, ones), w.astype(np.float64).sum(axis=1), rtol=1e-13)


def test_gemm_rows_equal_gemv():
    N, K, M = 40, 576, 5
    codes, s, o = gen_weights(N, K, seed=2)
    w = oracle.dequant_f32(codes, s, o)
    X = gen_activations((M, K), seed=2)
    Y = oracle.gemm_f64(X, w)
    b = oracle.abs_bound(X, w)
    for m in range(M):
        assert np.all(np.abs(Y[m] - oracle.gemv_f64(w, X[m])) <= 1e-13 * b[m])
    assert Y.shape == (M, N)


# ---------------------------------------------------------------- PIN8
def test_bf16_rounding_matches_torch():
    import torch
    rng = np.random.default_rng(0)
    bits = rng.integers(0, 2 ** 32, 200000, dtype=np.uint64).astype(np.uint32)
    edge = np.array([0x00000000, 0x80000000, 0x3F808000, 0x3F818000, 0x3F80FFFF, 0x3F7FFFFF,
                     0x7F7FFFFF, 0x00008000, 0x00018000, 0x7F800000, 0xFF800000, 0x7F7F8000,
                     0x3F807FFF, 0xBF808000, 0x4B000000, 0x34000001], np.uint32)
    bits = np.concatenate([bits, edge])
    f = bits.view(np.float32)
    finite = np.isfinite(f)
    ours = oracle.f32_to_bf16(f[finite])
    ref = torch.from_numpy(f[finite].copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    # round trip of every bf16 pattern that is finite
    allb = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    fin = np.isfinite(oracle.bf16_to_f32(allb))
    assert np.array_equal(oracle.f32_to_bf16(oracle.bf16_to_f32(allb[fin])), allb[fin])


def test_edge_weights_stay_finite_and_exact():
    codes, s, o = gen_edge_weights(64, 512)
    w = oracle.dequant_f32(codes, s, o)
    assert np.isfinite(w).all()
    # d*q + m with the product exact: compare against the same sum done in float64
    d = np.repeat(oracle.bf16_to_f32(s), 32, 1).astype(np.float64)
    m = np.repeat(oracle.bf16_to_f32(o), 32, 1).astype(np.float64)
    exact64 = d * codes + m      # exact in float64 for these magnitudes
    assert np.array_equal(w, exact64.astype(np.float32)) or np.allclose(w, exact64, rtol=2 ** -24)


def test_tolerance_check_catches_planted_errors():
    N, K = 64, 1152
    codes, s, o = gen_weights(N, K, seed=4)
    w = oracle.dequant_f32(codes, s, o)
    x = gen_activations(K, seed=4)
    y = oracle.gemv_f64(w, x)
    b = oracle.abs_bound(x, w)
    ok, worst = oracle.check_close(y.astype(np.float32), y, b)
    assert ok and worst < 1e-3
    # a dropped offset term, a sign flip of one row, a transposed group layout
    w_no_off = oracle.dequant_f32(codes, s, np.zeros_like(o))
    assert not oracle.check_close(oracle.gemv_f64(w_no_off, x), y, b)[0]
    y2 = y.copy()
    y2[3] = -y2[3]
    assert not oracle.check_close(y2, y, b)[0]
    s_t = s.reshape(N, -1)[:, ::-1].copy()
    assert not oracle.check_close(oracle.gemv_f64(oracle.dequant_f32(codes, s_t, o), x), y, b)[0]


def test_abs_bound_and_tolerance_hand_values():
    """abs_bound, tolerance and check_close on a worked example (bf16-exact
    values, sums done by hand): bound_n = sum_k |x_k w_nk|; tol = 2e-3 bound
    + 1e-5 (+ |y_ref| 2^-8 for bf16 outputs); a result passes at 0.999 tol
    and fails at 1.001 tol, and a NaN never passes."""
    x = oracle.f32_to_bf16(np.array([1.0, -2.0, 0.5], dtype=np.float32))
    w = np.array([[1.0, 2.0, -4.0], [0.25, 0.0, 3.0]], dtype=np.float32)
    # row 0: |1*1| + |-2*2| + |0.5*-4| = 1 + 4 + 2 = 7; row 1: 0.25 + 0 + 1.5 = 1.75
    assert np.array_equal(oracle.abs_bound(x, w), np.array([7.0, 1.75]))
    # y = W x: row 0: 1 - 4 - 2 = -5; row 1: 0.25 + 0 + 1.5 = 1.75
    y = oracle.gemv_f64(w, x)
    assert np.array_equal(y, np.array([-5.0, 1.75]))
    tol = oracle.tolerance(np.array([7.0, 1.75]))
    assert np.allclose(tol, [2e-3 * 7 + 1e-5, 2e-3 * 1.75 + 1e-5], rtol=0, atol=1e-15)
    tol16 = oracle.tolerance(np.array([7.0, 1.75]), y_ref=y, bf16_out=True)
    assert np.allclose(tol16 - tol, [5.0 / 256, 1.75 / 256], rtol=0, atol=1e-15)
    b = oracle.abs_bound(x, w)
    ok, worst = oracle.check_close(y + 0.999 * tol, y, b)
    assert ok and abs(worst - 0.999) < 1e-9
    ok, worst = oracle.check_close(y - 1.001 * tol, y, b)
    assert not ok and abs(worst - 1.001) < 1e-9
    assert not oracle.check_close(np.array([np.nan, 1.75]), y, b)[0]
    # the matrix form: X[m] . W[n] over rows of X
    X = oracle.f32_to_bf16(np.array([[1.0, -2.0, 0.5], [0.0, 1.0, -1.0]], dtype=np.float32))
    # row 1 of X: |0| + |1*2| + |-1*-4| = 6 against W row 0; |0| + 0 + |-1*3| = 3 against W row 1
    assert np.array_equal(oracle.abs_bound(X, w), np.array([[7.0, 1.75], [6.0, 3.0]]))
    assert np.array_equal(oracle.gemm_f64(X, w), np.array([[-5.0, 1.75], [6.0, -3.0]]))
