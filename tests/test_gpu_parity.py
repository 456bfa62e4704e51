"""Parity of the HIP path (through the C ABI) with the CPU oracle.

  * q4nx_dequant: bit-exact, float32 and bf16 outputs.
  * q4nx_gemv / q4nx_gemv_batched: |y - y_ref| <= 2e-3 * sum_k |x_k w_k| + 1e-5
    per output (bf16 outputs: plus half a bf16 ulp of y_ref); unit vectors
    extract a column bit-exactly; batched == single bit for bit; repeated
    calls are bitwise identical.
  * q4nx_gemm: the same tolerance against the float64 oracle, and a tighter
    diagnostic against the float64 product with the bf16-rounded weights the
    matrix cores consume.
Shapes: tiny, ragged (N % 32 != 0, K % 256 != 0, M not a tile multiple),
every Gemma3 projection shape at full size, edge-valued weights.
"""
import numpy as np
import pytest

import oracle
from workloads import gen_weights, gen_activations, gen_edge_weights, MODELS

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


def make(N, K, seed=0, mode="zp", layer=0, proj=0):
    if mode == "edge":
        codes, s, o = gen_edge_weights(N, K, seed=seed)
    else:
        codes, s, o = gen_weights(N, K, seed=seed, layer=layer, proj=proj, offset_mode=mode)
    return codes, s, o


# ----------------------------------------------------------------- dequant
DEQ_SHAPES = [(1, 32, "zp"), (32, 256, "zp"), (33, 288, "literal"), (1024, 1152, "zp"), (100, 544, "edge"),
              (2048, 5376, "zp"), (65, 21504, "zp")]


@pytest.mark.parametrize("N,K,mode", DEQ_SHAPES)
def test_dequant_bit_exact(q4, N, K, mode):
    _say("dequant", N, K, mode)
    codes, s, o = make(N, K, seed=N + K, mode=mode)
    blob = q4.q4nx_pack(codes, s, o)
    w32 = oracle.dequant_f32(codes, s, o)
    db = dev_u8(blob)
    W = torch.empty((N, K), dtype=torch.float32, device="cuda")
    q4.q4nx_dequant(db, N, K, W)
    assert np.array_equal(host_f32(W).view(np.uint32), w32.view(np.uint32))
    Wb = torch.empty((N, K), dtype=torch.bfloat16, device="cuda")
    q4.q4nx_dequant(db, N, K, Wb)
    assert np.array_equal(host_bits16(Wb), oracle.f32_to_bf16(w32))


# ----------------------------------------------------------------- gemv
def _gemv_case(q4, N, K, seed, mode="zp", bf16_out=False, layer=0, proj=0):
    codes, s, o = make(N, K, seed=seed, mode=mode, layer=layer, proj=proj)
    blob = q4.q4nx_pack(codes, s, o)
    x = gen_activations(K, seed=seed, layer=layer, proj=proj)
    w32 = oracle.dequant_f32(codes, s, o)
    y_ref = oracle.gemv_f64(w32, x)
    bound = oracle.abs_bound(x, w32)
    y = torch.empty(N, dtype=torch.bfloat16 if bf16_out else torch.float32, device="cuda")
    q4.q4nx_gemv(dev_u8(blob), dev_bf16(x), y, N, K)
    ok, worst = oracle.check_close(host_f32(y), y_ref, bound, bf16_out=bf16_out)
    return ok, worst


# K = 22560 and 51232 span 89 and 201 blocks: the weights are read in more than one chunk.
# N = 2561, 5088 and 2600 give launches of 81, 159 and 82 strips, which take the
# persistent streaming form (80-159 strips), here with a ragged last strip and
# K tails (2080 = 8 blocks + 32 columns, 1056 = 4 blocks + 32 columns) and
# with the longest K it takes (88 blocks).
GEMV_SHAPES = [(1, 32), (32, 256), (33, 288), (64, 512), (1024, 1152), (100, 544), (257, 1184), (8, 4096),
               (3000, 256), (40, 21504), (40, 22560), (33, 51232), (2561, 2080), (5088, 1056), (2600, 22528)]


@pytest.mark.parametrize("N,K", GEMV_SHAPES)
@pytest.mark.parametrize("mode", ["zp", "literal", "edge"])
def test_gemv_parity_small(q4, N, K, mode):
    _say("gemv", N, K, mode)
    ok, worst = _gemv_case(q4, N, K, seed=N * 3 + K, mode=mode)
    assert ok, worst


FULL = [(m, p) for m in ("1b", "4b", "27b") for p in range(7)]


@pytest.mark.parametrize("model,p", FULL)
def test_gemv_parity_every_projection_full_size(q4, model, p):
    name, N, K = MODELS[model]["proj"][p]
    _say("gemv full", model, name, N, K)
    ok, worst = _gemv_case(q4, N, K, seed=0, layer=0, proj=p)
    assert ok, (model, name, worst)


def test_gemv_bf16_output(q4):
    for N, K in [(1024, 1152), (2560, 10240), (33, 288)]:
        _say("gemv bf16 out", N, K)
        ok, worst = _gemv_case(q4, N, K, seed=5, bf16_out=True)
        assert ok, worst


def test_gemv_lm_head_sampled_rows(q4):
    """4B lm_head 262144 x 2560 at full size; the oracle checks sampled strips."""
    N, K = MODELS["4b"]["lm_head"][1:]
    _say("gemv lm_head", N, K)
    codes, s, o = gen_weights(N, K, seed=0, layer=34, proj=7)
    blob = q4.q4nx_pack(codes, s, o)
    x = gen_activations(K, seed=0, layer=34, proj=7)
    y = torch.empty(N, dtype=torch.float32, device="cuda")
    q4.q4nx_gemv(dev_u8(blob), dev_bf16(x), y, N, K)
    yh = host_f32(y)
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([np.arange(64), N - 64 + np.arange(64), rng.integers(0, N, 2048)]))
    w32 = oracle.dequant_f32(codes[rows], s[rows], o[rows])
    ok, worst = oracle.check_close(yh[rows], oracle.gemv_f64(w32, x), oracle.abs_bound(x, w32))
    assert ok, worst


def test_gemv_unit_vectors_extract_columns_bit_exact(q4):
    N, K = 300, 1184
    _say("gemv e_k", N, K)
    codes, s, o = make(N, K, seed=8)
    blob = dev_u8(q4.q4nx_pack(codes, s, o))
    w32 = oracle.dequant_f32(codes, s, o)
    for k in (0, 1, 31, 32, 255, 256, 511, 1024, 1183):
        e = np.zeros(K, np.uint16)
        e[k] = 0x3F80
        y = torch.empty(N, dtype=torch.float32, device="cuda")
        q4.q4nx_gemv(blob, dev_bf16(e), y, N, K)
        assert np.array_equal(host_f32(y), w32[:, k]), k  # == treats +0 and -0 alike


def test_gemv_integer_case_exact(q4):
    """d = 1, m = 0 and small integer x: every partial sum is an exact integer."""
    rng = np.random.default_rng(3)
    N, K = 200, 2560
    _say("gemv integer", N, K)
    codes = rng.integers(0, 16, (N, K)).astype(np.uint8)
    s = np.full((N, K // 32), 0x3F80, np.uint16)
    o = np.zeros((N, K // 32), np.uint16)
    xi = rng.integers(-4, 5, K)
    x = oracle.f32_to_bf16(xi.astype(np.float32))
    y = torch.empty(N, dtype=torch.float32, device="cuda")
    q4.q4nx_gemv(dev_u8(q4.q4nx_pack(codes, s, o)), dev_bf16(x), y, N, K)
    assert np.array_equal(host_f32(y), (codes.astype(np.int64) @ xi).astype(np.float32))


def test_gemv_batched_matches_single_and_is_deterministic(q4):
    shapes = MODELS["4b"]["proj"][:3] + [("x", 33, 288), ("y", 1000, 21504)]
    items, singles = [], []
    for p, (name, N, K) in enumerate(shapes):
        codes, s, o = make(N, K, seed=p)
        blob = dev_u8(q4.q4nx_pack(codes, s, o))
        x = dev_bf16(gen_activations(K, seed=p))
        yb = torch.empty(N, dtype=torch.float32, device="cuda")
        ys = torch.empty(N, dtype=torch.float32, device="cuda")
        items.append((blob, x, yb, N, K))
        singles.append((blob, x, ys, N, K))
    _say("gemv batched", [s[1:] for s in shapes])
    q4.q4nx_gemv_batched(items)
    for blob, x, ys, N, K in singles:
        q4.q4nx_gemv(blob, x, ys, N, K)
    for p, ((_, x, yb, N, K), (_, _, ys, _, _)) in enumerate(zip(items, singles)):
        codes, s, o = make(N, K, seed=p)
        w32 = oracle.dequant_f32(codes, s, o)
        xb = gen_activations(K, seed=p)
        ref, bound = oracle.gemv_f64(w32, xb), oracle.abs_bound(xb, w32)
        assert oracle.check_close(host_f32(yb), ref, bound)[0]
        assert oracle.check_close(host_f32(ys), ref, bound)[0]
    first = [host_f32(it[2]).copy() for it in items]
    for _ in range(3):
        q4.q4nx_gemv_batched(items)
    for f, it in zip(first, items):
        assert np.array_equal(f.view(np.uint32), host_f32(it[2]).view(np.uint32))


# ----------------------------------------------------------------- gemm
def _gemm_case(q4, M, N, K, seed, mode="zp", bf16_out=False, rows=None, layer=0, proj=0):
    codes, s, o = make(N, K, seed=seed, mode=mode, layer=layer, proj=proj)
    blob = q4.q4nx_pack(codes, s, o)
    X = gen_activations((M, K), seed=seed, layer=layer, proj=proj)
    Y = torch.empty((M, N), dtype=torch.bfloat16 if bf16_out else torch.float32, device="cuda")
    q4.q4nx_gemm(M, N, K, dev_bf16(X), dev_u8(blob), Y)
    Yh = host_f32(Y)
    if rows is not None:
        X, Yh = X[rows], Yh[rows]
    w32 = oracle.dequant_f32(codes, s, o)
    ref = oracle.gemm_f64(X, w32)
    ok, worst = oracle.check_close(Yh, ref, oracle.abs_bound(X, w32), bf16_out=bf16_out)
    # diagnostic: the float64 product with the bf16 weights the MFMA consumes
    w16 = oracle.bf16_to_f32(oracle.f32_to_bf16(w32))
    ref16 = oracle.gemm_f64(X, w16)
    tight = np.abs(Yh.astype(np.float64) - ref16) <= (
        1e-5 * oracle.abs_bound(X, w16) + 1e-6 + (2.0 ** -8 * np.abs(ref16) if bf16_out else 0))
    return ok, worst, bool(tight.all())


GEMM_SHAPES = [(1, 32, 256), (5, 33, 288), (130, 200, 1152), (64, 1024, 1152), (256, 512, 2560), (129, 257, 1184),
               (128, 128, 64), (7, 3000, 96), (300, 96, 5376)]


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
@pytest.mark.parametrize("mode", ["zp", "edge"])
def test_gemm_parity_small(q4, M, N, K, mode):
    _say("gemm", M, N, K, mode)
    ok, worst, tight = _gemm_case(q4, M, N, K, seed=M + N + K, mode=mode)
    assert ok, worst
    assert tight


def test_gemm_bf16_output(q4):
    _say("gemm bf16 out")
    ok, worst, tight = _gemm_case(q4, 96, 320, 1152, seed=1, bf16_out=True)
    assert ok and tight, worst


def test_gemm_single_row_matches_gemv_within_tolerance(q4):
    M, N, K = 1, 2048, 2560
    _say("gemm M=1 vs gemv")
    codes, s, o = make(N, K, seed=12)
    blob = dev_u8(q4.q4nx_pack(codes, s, o))
    x = gen_activations(K, seed=12)
    y = torch.empty(N, dtype=torch.float32, device="cuda")
    Y = torch.empty((1, N), dtype=torch.float32, device="cuda")
    q4.q4nx_gemv(blob, dev_bf16(x), y, N, K)
    q4.q4nx_gemm(M, N, K, dev_bf16(x), blob, Y)
    w32 = oracle.dequant_f32(codes, s, o)
    b = oracle.abs_bound(x, w32)
    assert oracle.check_close(host_f32(Y)[0], host_f32(y), b)[0]


@pytest.mark.parametrize("model,p", [(m, p) for m in ("4b", "27b") for p in range(7)])
def test_gemm_full_size_sampled_rows(q4, model, p):
    """Every projection shape at the prefill chunk size (4B: 2048 token rows,
    27B: 4096); the oracle checks the first and last 32 rows and 64 random
    ones, all N outputs each."""
    M = 2048 if model == "4b" else 4096
    name, N, K = MODELS[model]["proj"][p]
    rng = np.random.default_rng(1)
    rows = np.unique(np.concatenate([np.arange(32), M - 32 + np.arange(32), rng.integers(0, M, 64)]))
    _say("gemm full", model, name, M, N, K)
    ok, worst, tight = _gemm_case(q4, M, N, K, seed=0, rows=rows, layer=0, proj=p)
    assert ok, (name, worst)
    assert tight, name


# The stacked prefill products (q/k/v and gate/up of one layer as one GEMM):
# 27B 4096 x 8192 and 4096 x 43008 (columns 0..40959 in 256 x 256 tiles, the
# rest in 256 x 128), 4B 2048 x 4096 and 2048 x 20480, all at the model's K.
@pytest.mark.parametrize("M,N,K", [(4096, 8192, 5376), (4096, 43008, 5376), (2048, 4096, 2560), (2048, 20480, 2560)])
def test_gemm_stacked_prefill_shapes_sampled_rows(q4, M, N, K):
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([np.arange(16), M - 16 + np.arange(16), rng.integers(0, M, 32)]))
    _say("gemm stacked", M, N, K)
    ok, worst, tight = _gemm_case(q4, M, N, K, seed=N, rows=rows)
    assert ok, worst
    assert tight


# Shapes that take each launch plan of q4nx_gemm on a 256-CU device, with
# ragged M and N and a K that is not a multiple of the 64-column step:
#   3996 x 4080 x 5344  one launch of 256 x 256 tiles (the K-tail variant)
#   4000 x 5344 x 2080  rows 0..3071 in 256 x 256 tiles, the rest in 256 x 128
#   4096 x 21472 x 96   columns 0..20479 in 256 x 256 tiles, the rest in 128 x 128
#   1024 x 16384 x 128  one launch of 256 x 256 tiles, K a multiple of 64
PLAN_SHAPES = [(3996, 4080, 5344), (4000, 5344, 2080), (4096, 21472, 96), (1024, 16384, 128)]


@pytest.mark.parametrize("M,N,K", PLAN_SHAPES)
@pytest.mark.parametrize("bf16_out", [False, True])
def test_gemm_launch_plans_sampled_rows(q4, M, N, K, bf16_out):
    """The oracle checks the first and last 32 rows, the 32 rows on each side
    of a row split at 3072, and 32 random rows, all N outputs each."""
    rng = np.random.default_rng(2)
    rows = np.concatenate([np.arange(32), M - 32 + np.arange(32), rng.integers(0, M, 32)])
    if M > 3072 + 32:
        rows = np.concatenate([rows, 3072 - 32 + np.arange(64)])
    rows = np.unique(rows)
    _say("gemm plan", M, N, K, "bf16" if bf16_out else "f32")
    ok, worst, tight = _gemm_case(q4, M, N, K, seed=M + N, rows=rows, bf16_out=bf16_out)
    assert ok, worst
    assert tight


@pytest.mark.parametrize("N", [(1 << 21) - 256, (1 << 21) + 256])
def test_gemm_wide_rows_either_side_of_the_fast_store_stride(q4, N):
    """Tiles inside the output store through 32-bit buffer offsets while the
    row stride is below 2^21 elements, and element by element with 64-bit
    addresses beyond it.  All 256 rows are checked at sampled columns around
    2^21 and at both ends, float32 and bf16 outputs.  K is one group (32) to
    keep W small; with so few terms one weight's bf16 rounding (up to 2^-8
    relative) can exceed the projection tolerance, so the reference is the
    float64 product of the bf16 weights the matrix cores consume, within the
    tight bound (a misplaced or missing store fails it by orders of
    magnitude)."""
    M, K = 256, 32
    _say("gemm wide rows", M, N, K)
    codes, s, o = make(N, K, seed=21)
    blob = dev_u8(q4.q4nx_pack(codes, s, o))
    Xh = gen_activations((M, K), seed=21)
    X = dev_bf16(Xh)
    rng = np.random.default_rng(21)
    cols = np.unique(np.concatenate([np.arange(64), (1 << 21) - 320 + np.arange(128), N - 64 + np.arange(64),
                                     rng.integers(0, N, 64)]))
    cols = cols[cols < N]
    w16 = oracle.bf16_to_f32(oracle.f32_to_bf16(oracle.dequant_f32(codes[cols], s[cols], o[cols])))
    ref, bound = oracle.gemm_f64(Xh, w16), oracle.abs_bound(Xh, w16)
    idx = torch.from_numpy(cols).cuda()
    for bf16_out in (False, True):
        Y = torch.full((M, N), float("nan"), dtype=torch.bfloat16 if bf16_out else torch.float32, device="cuda")
        q4.q4nx_gemm(M, N, K, X, blob, Y)
        Yh = host_f32(Y.index_select(1, idx)).astype(np.float64)
        tol = 1e-5 * bound + 1e-6 + (2.0 ** -8 * np.abs(ref) if bf16_out else 0)
        err = np.abs(Yh - ref)
        assert (err <= tol).all(), (bf16_out, float(np.nanmax(err / tol)))
        del Y
        torch.cuda.empty_cache()


# ----------------------------------------------------------------- two-phase prefill
# q4nx_dequant (bf16) then q4nx_gemm_bf16: the paper's dequantize-then-MM
# structure.  Same bf16 weights and the same MFMA chain over K as the fused
# q4nx_gemm, hence the same bits.
TWO_PHASE_SHAPES = [(5, 33, 288), (130, 200, 1152), (300, 96, 5376), (4096, 2048, 256), (3996, 4080, 544),
                    (4000, 5344, 224), (4096, 21472, 96), (2040, 4000, 2560)]


@pytest.mark.parametrize("M,N,K", TWO_PHASE_SHAPES)
@pytest.mark.parametrize("bf16_out", [False, True])
def test_two_phase_prefill_equals_fused_bitwise(q4, M, N, K, bf16_out):
    _say("two-phase", M, N, K, "bf16" if bf16_out else "f32")
    codes, s, o = make(N, K, seed=M + K, mode="zp")
    blob = dev_u8(q4.q4nx_pack(codes, s, o))
    X = dev_bf16(gen_activations((M, K), seed=M + K))
    ydt = torch.bfloat16 if bf16_out else torch.float32
    W = torch.empty((N, K), dtype=torch.bfloat16, device="cuda")
    Y1 = torch.full((M, N), float("nan"), dtype=ydt, device="cuda")
    Y2 = torch.full((M, N), float("nan"), dtype=ydt, device="cuda")
    q4.q4nx_gemm(M, N, K, X, blob, Y1)
    q4.q4nx_dequant(blob, N, K, W)
    q4.q4nx_gemm_bf16(M, N, K, X, W, Y2)
    torch.cuda.synchronize()
    it = torch.int16 if bf16_out else torch.int32
    assert torch.equal(Y1.view(it), Y2.view(it))


@pytest.mark.parametrize("M,N,K", [(7, 40, 96), (129, 257, 1184), (512, 640, 2048)])
def test_gemm_bf16_arbitrary_weights_vs_float64(q4, M, N, K):
    """Any bf16 W (not only dequantized ones): the float64 product of the bf16
    values, with the GEMM tolerance and the tight diagnostic bound."""
    _say("gemm_bf16", M, N, K)
    rng = np.random.default_rng(M * N)
    w32 = rng.standard_normal((N, K), dtype=np.float32) * np.float32(0.05)
    wbits = oracle.f32_to_bf16(w32)
    w16 = oracle.bf16_to_f32(wbits)
    X = gen_activations((M, K), seed=N)
    Y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    q4.q4nx_gemm_bf16(M, N, K, dev_bf16(X), dev_bf16(wbits), Y)
    Yh = host_f32(Y)
    ref = oracle.gemm_f64(X, w16)
    ok, worst = oracle.check_close(Yh, ref, oracle.abs_bound(X, w16))
    assert ok, worst
    assert (np.abs(Yh.astype(np.float64) - ref) <= 1e-5 * oracle.abs_bound(X, w16) + 1e-6).all()


# ----------------------------------------------------------------- quantizer
def _edge_weights(N, K, seed):
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    G = K // 32
    kinds = rng.integers(0, 9, size=(N, G))
    for n in range(N):
        for g in range(G):
            sl = W[n, 32 * g:32 * g + 32]
            k = kinds[n, g]
            if k == 1:
                sl[:] = np.float32(0.125)                                  # constant
            elif k == 2:
                sl[:] = rng.integers(-4, 5, 32).astype(np.float32)         # ties on an integer grid
                sl[0], sl[1] = -4.0, 11.0
            elif k == 3:
                sl[:] = (rng.standard_normal(32) * 2.0 ** -110).astype(np.float32)  # d, m flushed
            elif k == 4:
                sl[:] = (rng.standard_normal(32) * 1e31).astype(np.float32)        # clamped
                sl[3], sl[4], sl[5] = np.inf, -np.inf, np.nan
            elif k == 5:
                sl[:] = 0.0
                sl[7] = -0.0
            elif k == 6:
                sl[:] = -np.abs(sl) - np.float32(3.0)                       # offset far from zero
            elif k == 7:
                # d far below the float32 spacing at m (0.125 at 2^20): Eq. 3 levels repeat, and
                # the inputs sit on that spacing, so many are equal to a level or halfway between
                sl[:] = np.float32(2.0 ** 20) + rng.integers(0, 8, 32).astype(np.float32) * np.float32(0.125)
                sl[0], sl[1] = np.float32(2.0 ** 20), np.float32(2.0 ** 20 + 0.875)
    return W


@pytest.mark.parametrize("N,K,kind", [(1, 32, "normal"), (33, 288, "edge"), (64, 1152, "edge"),
                                      (1024, 1152, "normal"), (2048, 5376, "normal"), (100, 21504, "edge")])
def test_quantize_bit_exact(q4, N, K, kind):
    _say("quantize", N, K, kind)
    if kind == "edge":
        W = _edge_weights(N, K, seed=N + K)
    else:
        W = (np.random.default_rng(N).standard_normal((N, K)) * 0.02).astype(np.float32)
    want = oracle.pack(*oracle.quantize(W))
    blob = torch.full((q4.q4nx_packed_size(N, K),), 0xAB, dtype=torch.uint8, device="cuda")
    q4.q4nx_quantize(torch.from_numpy(W).cuda(), N, K, blob)
    torch.cuda.synchronize()
    got = blob.cpu().numpy()
    assert np.array_equal(got, want)


# ----------------------------------------------------------------- measurement aid
def test_stream_read_folds_every_word(q4):
    """q4nx_stream_read reads every 16-byte piece exactly once: its per-wave
    XOR fold equals the fold computed on the host."""
    n16 = 2048 * 37 + 5            # slices of unequal length, some workgroups past the end
    data = np.random.default_rng(8).integers(0, 2 ** 32, size=4 * n16, dtype=np.uint32)
    src = torch.from_numpy(data.view(np.uint8)).cuda()
    sink = torch.empty(8192, dtype=torch.float32, device="cuda")
    q4.q4nx_stream_read(src, sink)
    got = sink.cpu().numpy().view(np.uint32)
    per = -(-n16 // 2048)
    words = data.reshape(n16, 4)
    want = np.zeros(8192, np.uint32)
    for b in range(2048):
        lo, hi = b * per, min(n16, (b + 1) * per)
        for w in range(4):
            idx = [p for p in range(lo, hi) if (p - lo) % 256 // 64 == w]
            want[4 * b + w] = np.bitwise_xor.reduce(words[idx].reshape(-1)) if idx else 0
    assert np.array_equal(got, want & np.uint32(0x3FFFFFFF))
