"""Parity of the MXFP4-variant kernels (through the C ABI) with the CPU oracle.

  * q4nx_mx_dequant: bit-exact (float32 and bf16 outputs; every value is
    exact in both).
  * q4nx_mx_gemv / q4nx_mx_gemv_batched: the projection tolerance
    |y - y_ref| <= 2e-3 * sum_k |x_k w_k| + 1e-5 against the float64 oracle;
    unit vectors extract a column exactly (bit for bit but for the sign of a
    zero); batched launches are reproducible and meet the same tolerance.
  * q4nx_mx_gemm: the same tolerance, the tight bound against the float64
    product (the bf16 weights are exact here), and bitwise equality with
    q4nx_mx_dequant (bf16) followed by q4nx_gemm_bf16.
Shapes: tiny, ragged, every launch plan of the matrix product, Gemma3
projection shapes at full size, scales over the whole accepted range.
"""
import numpy as np
import pytest

import oracle
from workloads import gen_mx_weights, gen_activations, MODELS

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def q4():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_06063_amd as mod
    return mod


def _say(*a):
    print("[case]", *a, flush=True)


def dev_u8(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def host_f32(t):
    torch.cuda.synchronize()
    return t.float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()


def host_bits16(t):
    torch.cuda.synchronize()
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


# ----------------------------------------------------------------- dequant
@pytest.mark.parametrize("N,K,mode", [(1, 32, "model"), (32, 256, "model"), (33, 288, "edge"), (1024, 1152, "model"),
                                      (100, 544, "edge"), (2048, 5376, "model"), (65, 21504, "edge")])
def test_mx_dequant_bit_exact(q4, N, K, mode):
    _say("mx dequant", N, K, mode)
    codes, sc = gen_mx_weights(N, K, seed=N + K, mode=mode)
    blob = dev_u8(q4.q4nx_mx_pack(codes, sc))
    w32 = oracle.mx_dequant_f32(codes, sc)
    W = torch.empty((N, K), dtype=torch.float32, device="cuda")
    q4.q4nx_mx_dequant(blob, N, K, W)
    assert np.array_equal(host_f32(W).view(np.uint32), w32.view(np.uint32))
    Wb = torch.empty((N, K), dtype=torch.bfloat16, device="cuda")
    q4.q4nx_mx_dequant(blob, N, K, Wb)
    assert np.array_equal(host_bits16(Wb), oracle.f32_to_bf16(w32))


# ----------------------------------------------------------------- gemv
def _gemv_case(q4, N, K, seed, mode="model", bf16_out=False, proj=0):
    codes, sc = gen_mx_weights(N, K, seed=seed, proj=proj, mode=mode)
    blob = q4.q4nx_mx_pack(codes, sc)
    x = gen_activations(K, seed=seed, proj=proj)
    w32 = oracle.mx_dequant_f32(codes, sc)
    y = torch.empty(N, dtype=torch.bfloat16 if bf16_out else torch.float32, device="cuda")
    q4.q4nx_mx_gemv(dev_u8(blob), dev_bf16(x), y, N, K)
    return oracle.check_close(host_f32(y), oracle.gemv_f64(w32, x), oracle.abs_bound(x, w32), bf16_out=bf16_out)


# (2561, 2080) and (5088, 1056): launches of 81 and 159 strips (the persistent
# streaming form) with a ragged last strip and K tails.
@pytest.mark.parametrize("N,K", [(1, 32), (32, 256), (33, 288), (64, 512), (1024, 1152), (257, 1184), (8, 4096),
                                 (3000, 256), (40, 21504), (40, 22560), (33, 51232), (2561, 2080), (5088, 1056)])
@pytest.mark.parametrize("mode", ["model", "edge"])
def test_mx_gemv_parity_small(q4, N, K, mode):
    _say("mx gemv", N, K, mode)
    ok, worst = _gemv_case(q4, N, K, seed=N * 3 + K, mode=mode)
    assert ok, worst


@pytest.mark.parametrize("model,p", [(m, p) for m in ("4b", "27b") for p in range(7)])
def test_mx_gemv_every_projection_full_size(q4, model, p):
    name, N, K = MODELS[model]["proj"][p]
    _say("mx gemv full", model, name, N, K)
    ok, worst = _gemv_case(q4, N, K, seed=0, proj=p)
    assert ok, (model, name, worst)


def test_mx_gemv_bf16_output(q4):
    for N, K in [(1024, 1152), (2560, 10240)]:
        _say("mx gemv bf16 out", N, K)
        ok, worst = _gemv_case(q4, N, K, seed=5, bf16_out=True)
        assert ok, worst


def test_mx_gemv_unit_vectors_extract_columns_bit_exact(q4):
    N, K = 96, 1184
    _say("mx gemv unit vectors", N, K)
    codes, sc = gen_mx_weights(N, K, seed=4, mode="edge")
    blob = dev_u8(q4.q4nx_mx_pack(codes, sc))
    w32 = oracle.mx_dequant_f32(codes, sc)
    for k in (0, 1, 31, 32, 255, 256, 1000, K - 1):
        x = np.zeros(K, np.uint16)
        x[k] = 0x3F80  # 1.0
        y = torch.empty(N, dtype=torch.float32, device="cuda")
        q4.q4nx_mx_gemv(blob, dev_bf16(x), y, N, K)
        # exact values; FP4 code 8 is -0, which a float32 sum starting at +0 returns as +0
        got = host_f32(y)
        assert np.array_equal(got, w32[:, k]), k
        nz = w32[:, k] != 0
        assert np.array_equal(got[nz].view(np.uint32), w32[nz, k].view(np.uint32)), k


def test_mx_gemv_batched_reproducible_and_within_tolerance(q4):
    shapes = [(2560, 2560), (1024, 2560), (10240, 2560), (2560, 10240)]
    _say("mx gemv batched", shapes)
    items = []
    for i, (N, K) in enumerate(shapes):
        codes, sc = gen_mx_weights(N, K, seed=7, proj=i)
        blob = dev_u8(q4.q4nx_mx_pack(codes, sc))
        x = dev_bf16(gen_activations(K, seed=7, proj=i))
        yb = torch.empty(N, dtype=torch.float32, device="cuda")
        items.append((blob, x, yb, N, K))
    q4.q4nx_mx_gemv_batched(items)
    torch.cuda.synchronize()
    first = [it[2].clone() for it in items]
    q4.q4nx_mx_gemv_batched(items)
    torch.cuda.synchronize()
    for a, it in zip(first, items):
        assert torch.equal(a.view(torch.int32), it[2].view(torch.int32))
    # the batch launch splits like a single launch over the same total strips,
    # so each output also meets the oracle's tolerance
    for i, (blob, x, yb, N, K) in enumerate(items):
        codes, sc = gen_mx_weights(N, K, seed=7, proj=i)
        w32 = oracle.mx_dequant_f32(codes, sc)
        xb = gen_activations(K, seed=7, proj=i)
        ok, worst = oracle.check_close(host_f32(yb), oracle.gemv_f64(w32, xb), oracle.abs_bound(xb, w32))
        assert ok, (N, K, worst)


# ----------------------------------------------------------------- gemm
def _gemm_case(q4, M, N, K, seed, mode="model", bf16_out=False, rows=None, proj=0):
    codes, sc = gen_mx_weights(N, K, seed=seed, proj=proj, mode=mode)
    blob = q4.q4nx_mx_pack(codes, sc)
    X = gen_activations((M, K), seed=seed, proj=proj)
    Y = torch.empty((M, N), dtype=torch.bfloat16 if bf16_out else torch.float32, device="cuda")
    q4.q4nx_mx_gemm(M, N, K, dev_bf16(X), dev_u8(blob), Y)
    Yh = host_f32(Y)
    if rows is not None:
        X, Yh = X[rows], Yh[rows]
    w32 = oracle.mx_dequant_f32(codes, sc)
    ref = oracle.gemm_f64(X, w32)
    bound = oracle.abs_bound(X, w32)
    ok, worst = oracle.check_close(Yh, ref, bound, bf16_out=bf16_out)
    tight = np.abs(Yh.astype(np.float64) - ref) <= (
        1e-5 * bound + 1e-6 + (2.0 ** -8 * np.abs(ref) if bf16_out else 0))
    return ok, worst, bool(tight.all())


@pytest.mark.parametrize("M,N,K", [(1, 32, 256), (5, 33, 288), (130, 200, 1152), (64, 1024, 1152), (256, 512, 2560),
                                   (129, 257, 1184), (128, 128, 64), (7, 3000, 96), (300, 96, 5376)])
@pytest.mark.parametrize("mode", ["model", "edge"])
def test_mx_gemm_parity_small(q4, M, N, K, mode):
    _say("mx gemm", M, N, K, mode)
    ok, worst, tight = _gemm_case(q4, M, N, K, seed=M + N + K, mode=mode)
    assert ok, worst
    assert tight


@pytest.mark.parametrize("model,p", [("4b", 0), ("4b", 4), ("4b", 6), ("27b", 0), ("27b", 3), ("27b", 4),
                                     ("27b", 6)])
def test_mx_gemm_full_size_sampled_rows(q4, model, p):
    M = 2048 if model == "4b" else 4096
    name, N, K = MODELS[model]["proj"][p]
    rng = np.random.default_rng(1)
    rows = np.unique(np.concatenate([np.arange(32), M - 32 + np.arange(32), rng.integers(0, M, 64)]))
    _say("mx gemm full", model, name, M, N, K)
    ok, worst, tight = _gemm_case(q4, M, N, K, seed=0, rows=rows, proj=p)
    assert ok, (name, worst)
    assert tight, name


# Shapes that take each launch plan of the matrix product on a 256-CU device
# (one launch of 256 x 256 tiles with a K tail; a row split; a column split;
# K a multiple of 64).
@pytest.mark.parametrize("M,N,K", [(3996, 4080, 5344), (4000, 5344, 2080), (4096, 21472, 96), (1024, 16384, 128)])
@pytest.mark.parametrize("bf16_out", [False, True])
def test_mx_gemm_launch_plans_sampled_rows(q4, M, N, K, bf16_out):
    rng = np.random.default_rng(2)
    rows = np.concatenate([np.arange(32), M - 32 + np.arange(32), rng.integers(0, M, 32)])
    if M > 3072 + 32:
        rows = np.concatenate([rows, 3072 - 32 + np.arange(64)])
    rows = np.unique(rows)
    _say("mx gemm plan", M, N, K, "bf16" if bf16_out else "f32")
    ok, worst, tight = _gemm_case(q4, M, N, K, seed=M + N, rows=rows, bf16_out=bf16_out)
    assert ok, worst
    assert tight


@pytest.mark.parametrize("M,N,K", [(5, 33, 288), (130, 200, 1152), (300, 96, 5376), (3996, 4080, 544),
                                   (4000, 5344, 224), (4096, 21472, 96), (2040, 4000, 2560)])
def test_mx_gemm_equals_dequant_then_gemm_bf16_bitwise(q4, M, N, K):
    """Same bf16 weights, same MFMA chain over K: the same bits."""
    _say("mx two-phase", M, N, K)
    codes, sc = gen_mx_weights(N, K, seed=M + K, mode="edge")
    blob = dev_u8(q4.q4nx_mx_pack(codes, sc))
    X = dev_bf16(gen_activations((M, K), seed=M + K))
    W = torch.empty((N, K), dtype=torch.bfloat16, device="cuda")
    Y1 = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    Y2 = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    q4.q4nx_mx_gemm(M, N, K, X, blob, Y1)
    q4.q4nx_mx_dequant(blob, N, K, W)
    q4.q4nx_gemm_bf16(M, N, K, X, W, Y2)
    torch.cuda.synchronize()
    assert torch.equal(Y1.view(torch.int32), Y2.view(torch.int32))


# ----------------------------------------------------------------- quantizer
def _mx_edge_weights(N, K, seed):
    """Groups on the FP4 grid's midpoints (ties), saturating values, zeros,
    signed zeros, tiny and huge magnitudes, NaN and infinities."""
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 7.0], np.float32)
    for n in range(N):
        for g in range(K // 32):
            sl = W[n, 32 * g:32 * g + 32]
            kind = rng.integers(0, 8)
            X = np.float32(2.0 ** int(rng.integers(-20, 20)))
            if kind == 1:
                sl[:] = (mids[rng.integers(0, 8, 32)] * X * np.where(rng.random(32) < 0.5, -1, 1)).astype(np.float32)
                sl[0] = 7.0 * X                                        # keeps the exponent at log2(X)
            elif kind == 2:
                sl[:] = 0.0
                sl[5] = -0.0
            elif kind == 3:
                sl[:] = (rng.standard_normal(32) * 2.0 ** -110).astype(np.float32)   # exponent clamped at -100
            elif kind == 4:
                sl[:] = (rng.standard_normal(32) * 1e31).astype(np.float32)        # clamped to 2^100
                sl[3], sl[4], sl[5] = np.inf, -np.inf, np.nan
            elif kind == 5:
                sl[:] = np.float32(1e-42)                                         # denormal inputs
                sl[1] = -np.float32(1e-42)
    return W


@pytest.mark.parametrize("N,K,kind", [(1, 32, "normal"), (33, 288, "edge"), (64, 1152, "edge"),
                                      (1024, 1152, "normal"), (2048, 5376, "normal"), (100, 21504, "edge")])
def test_mx_quantize_bit_exact(q4, N, K, kind):
    _say("mx quantize", N, K, kind)
    if kind == "edge":
        W = _mx_edge_weights(N, K, seed=N + K)
    else:
        W = (np.random.default_rng(N).standard_normal((N, K)) * 0.02).astype(np.float32)
    want = oracle.mx_pack(*oracle.mx_quantize(W))
    blob = torch.full((q4.q4nx_mx_packed_size(N, K),), 0xAB, dtype=torch.uint8, device="cuda")
    q4.q4nx_mx_quantize(torch.from_numpy(W).cuda(), N, K, blob)
    torch.cuda.synchronize()
    assert np.array_equal(blob.cpu().numpy(), want)
