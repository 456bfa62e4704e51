"""q4nx_gemm_ex through the C ABI: the matrix product with a caller workspace,
where the launch plan splits K for shapes with few output tiles.

  * every case here takes a split plan (q4nx_gemm_workspace_size > 0), with
    ragged M and N, K not a multiple of 64, float32 and bf16 outputs;
  * parity with the float64 oracle: the projection tolerance and the tight
    bound against the product of the bf16 weights;
  * the three weight formats give the same bits for the same bf16 weights
    (same plan, same partial products, same order of the final sum);
  * the workspace starts filled with NaN, so a partial that is read before it
    is written would show; repeated calls are bitwise identical;
  * without a workspace the result equals q4nx_gemm bit for bit;
  * Q4NX products with a large M dequantize W to bf16 in the workspace first
    (each weight once) and give the fused kernel's bits.
"""
import numpy as np
import pytest

import oracle
from workloads import gen_weights, gen_mx_weights, gen_activations

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


def work_for(q4, M, N, K, fmt=None):
    """A NaN-filled workspace big enough for every weight format."""
    fmts = [fmt] if fmt is not None else [q4.Q4NX_WEIGHTS_Q4NX, q4.Q4NX_WEIGHTS_MXFP4, q4.Q4NX_WEIGHTS_BF16]
    nbytes = max(q4.q4nx_gemm_workspace_size(f, M, N, K) for f in fmts)
    assert nbytes > 0, "this shape is meant to use a workspace"
    return torch.full((nbytes // 4,), float("nan"), dtype=torch.float32, device="cuda")


def work_if_any(q4, M, N, K, fmt):
    """The workspace the planner asks for (NaN-filled), or None when its plan
    takes none."""
    nbytes = q4.q4nx_gemm_workspace_size(fmt, M, N, K)
    return torch.full((nbytes // 4,), float("nan"), dtype=torch.float32, device="cuda") if nbytes else None


# (M, N, K, rows checked by the oracle: None = all)
SPLIT_SHAPES = [(512, 512, 16384, None), (512, 512, 16352, None), (300, 520, 20000, None), (260, 257, 12000, None),
                (1, 256, 20480, None), (2048, 2560, 10240, 64), (2048, 2560, 10208, 64), (4096, 5376, 21504, 48)]


def _rows(M, n):
    if n is None:
        return None
    rng = np.random.default_rng(M)
    return np.unique(np.concatenate([np.arange(8), M - 8 + np.arange(8), rng.integers(0, M, n)]))


@pytest.mark.parametrize("M,N,K,nrows", SPLIT_SHAPES)
@pytest.mark.parametrize("bf16_out", [False, True])
def test_gemm_ex_split_parity(q4, M, N, K, nrows, bf16_out):
    _say("gemm_ex split", M, N, K, "bf16" if bf16_out else "f32")
    codes, s, o = gen_weights(N, K, seed=M + K)
    blob = dev_u8(q4.q4nx_pack(codes, s, o))
    X = gen_activations((M, K), seed=N + K)
    Y = torch.empty((M, N), dtype=torch.bfloat16 if bf16_out else torch.float32, device="cuda")
    q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_Q4NX, M, N, K, dev_bf16(X), blob, Y, work=work_for(q4, M, N, K))
    Yh = host_f32(Y)
    rows = _rows(M, nrows)
    if rows is not None:
        X, Yh = X[rows], Yh[rows]
    w32 = oracle.dequant_f32(codes, s, o)
    ok, worst = oracle.check_close(Yh, oracle.gemm_f64(X, w32), oracle.abs_bound(X, w32), bf16_out=bf16_out)
    assert ok, worst
    w16 = oracle.bf16_to_f32(oracle.f32_to_bf16(w32))
    ref16 = oracle.gemm_f64(X, w16)
    tight = np.abs(Yh.astype(np.float64) - ref16) <= (
        1e-5 * oracle.abs_bound(X, w16) + 1e-6 + (2.0 ** -8 * np.abs(ref16) if bf16_out else 0))
    assert tight.all()


@pytest.mark.parametrize("M,N,K", [(300, 520, 20000), (260, 257, 12000), (2048, 2560, 10208)])
def test_gemm_ex_formats_agree_bitwise(q4, M, N, K):
    """Q4NX and MXFP4-variant blobs against the bf16 weights they dequantize
    to, all through split plans: identical bits."""
    _say("gemm_ex formats", M, N, K)
    X = dev_bf16(gen_activations((M, K), seed=M))
    work = work_for(q4, M, N, K)
    W = torch.empty((N, K), dtype=torch.bfloat16, device="cuda")
    Y1 = torch.empty((M, N), dtype=torch.float32, device="cuda")
    Y2 = torch.empty((M, N), dtype=torch.float32, device="cuda")
    codes, s, o = gen_weights(N, K, seed=K)
    blob = dev_u8(q4.q4nx_pack(codes, s, o))
    q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_Q4NX, M, N, K, X, blob, Y1, work=work)
    q4.q4nx_dequant(blob, N, K, W)
    work.fill_(float("nan"))
    q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_BF16, M, N, K, X, W, Y2, work=work)
    torch.cuda.synchronize()
    assert torch.equal(Y1.view(torch.int32), Y2.view(torch.int32))
    mcodes, msc = gen_mx_weights(N, K, seed=K, mode="edge")
    mblob = dev_u8(q4.q4nx_mx_pack(mcodes, msc))
    work.fill_(float("nan"))
    q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_MXFP4, M, N, K, X, mblob, Y1, work=work)
    q4.q4nx_mx_dequant(mblob, N, K, W)
    q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_BF16, M, N, K, X, W, Y2, work=work)
    torch.cuda.synchronize()
    assert torch.equal(Y1.view(torch.int32), Y2.view(torch.int32))
    w32 = oracle.mx_dequant_f32(mcodes, msc)
    Xh = gen_activations((M, K), seed=M)
    ok, worst = oracle.check_close(host_f32(Y1), oracle.gemm_f64(Xh, w32), oracle.abs_bound(Xh, w32))
    assert ok, worst


def test_gemm_ex_repeatable_and_unsplit_without_workspace(q4):
    M, N, K = 512, 512, 16352
    _say("gemm_ex repeat / no workspace", M, N, K)
    codes, s, o = gen_weights(N, K, seed=9)
    blob = dev_u8(q4.q4nx_pack(codes, s, o))
    X = dev_bf16(gen_activations((M, K), seed=9))
    work = work_for(q4, M, N, K)
    Ys = [torch.empty((M, N), dtype=torch.float32, device="cuda") for _ in range(4)]
    q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_Q4NX, M, N, K, X, blob, Ys[0], work=work)
    q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_Q4NX, M, N, K, X, blob, Ys[1], work=work)
    q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_Q4NX, M, N, K, X, blob, Ys[2])      # no workspace: nothing split
    q4.q4nx_gemm(M, N, K, X, blob, Ys[3])
    torch.cuda.synchronize()
    assert torch.equal(Ys[0].view(torch.int32), Ys[1].view(torch.int32))
    assert torch.equal(Ys[2].view(torch.int32), Ys[3].view(torch.int32))
    # split and unsplit differ only by the order of the float32 sums
    d = (Ys[0] - Ys[3]).abs().max().item()
    assert d <= 1e-4 * Ys[3].abs().max().item()


@pytest.mark.parametrize("M,N,K,split", [(4096, 1024, 4096, False), (4096, 5376, 21504, True),
                                         (2048, 20480, 2560, False)])
def test_gemm_ex_dequantize_then_multiply(q4, M, N, K, split):
    """Shapes whose Q4NX workspace holds bf16 W (M = 4096, and the 4B gate/up
    product at M = 2048): the result equals the fused product of the same plan
    bit for bit (q4nx_gemm when nothing is split,
    the bf16-weight product of the dequantized W when K is split), and meets
    the oracle on sampled rows."""
    _say("gemm_ex two-phase", M, N, K)
    nbytes = q4.q4nx_gemm_workspace_size(q4.Q4NX_WEIGHTS_Q4NX, M, N, K)
    assert nbytes >= N * K * 2
    codes, s, o = gen_weights(N, K, seed=N)
    blob = dev_u8(q4.q4nx_pack(codes, s, o))
    Xh = gen_activations((M, K), seed=K)
    X = dev_bf16(Xh)
    work = torch.full((nbytes // 4,), float("nan"), dtype=torch.float32, device="cuda")
    Y1 = torch.empty((M, N), dtype=torch.float32, device="cuda")
    Y2 = torch.empty((M, N), dtype=torch.float32, device="cuda")
    q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_Q4NX, M, N, K, X, blob, Y1, work=work)
    if split:
        W = torch.empty((N, K), dtype=torch.bfloat16, device="cuda")
        q4.q4nx_dequant(blob, N, K, W)
        q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_BF16, M, N, K, X, W, Y2, work=work_for(q4, M, N, K, q4.Q4NX_WEIGHTS_BF16))
    else:
        q4.q4nx_gemm(M, N, K, X, blob, Y2)
    torch.cuda.synchronize()
    assert torch.equal(Y1.view(torch.int32), Y2.view(torch.int32))
    rows = _rows(M, 24)
    w32 = oracle.dequant_f32(codes, s, o)
    ok, worst = oracle.check_close(host_f32(Y1)[rows], oracle.gemm_f64(Xh[rows], w32), oracle.abs_bound(Xh[rows], w32))
    assert ok, worst


# Shapes whose tiles do not fill whole rounds of the 256 CUs, where the plan
# mixes tile shapes or splits K: a round and a few tiles (4352 x 4096), two
# rounds and a part (4352 x 8448), the Gemma3-4B o shape (80 tiles), few tiles
# over a long K with M and N ragged (2000 x 1100 x 6912), and a K tail with a
# ragged M (1999 x 2500 x 2016).
# Ragged prefill-sized shapes; the planner takes a different plan for each:
# dequantize-once with a partial last wave of tiles (the first two), the
# direct fused launch (the third and fifth), split K (the fourth), and one
# round of 256 x 128 tiles with M and N ragged (the sixth and seventh, N a
# multiple of 32 or not: the one-wave-per-SIMD 256 x 128 kernel's edge tiles).
PLANNED_SHAPES = [(4352, 4096, 2560, 32), (4352, 8448, 2560, 32), (2048, 2560, 2048, 48), (2000, 1100, 6912, 48),
                  (1999, 2500, 2016, 48), (2040, 4000, 2560, 48), (2040, 3999, 2560, 48)]


@pytest.mark.parametrize("M,N,K,nrows", PLANNED_SHAPES)
@pytest.mark.parametrize("bf16_out", [False, True])
def test_gemm_ex_planned_parity(q4, M, N, K, nrows, bf16_out):
    """The planned launches against the oracle on sampled rows, against the
    bf16-weight product within the tight bound, and against the launch without
    a workspace (no split) within the order of float32 sums."""
    _say("gemm_ex planned", M, N, K, "bf16" if bf16_out else "f32")
    codes, s, o = gen_weights(N, K, seed=M + 3 * K)
    blob = dev_u8(q4.q4nx_pack(codes, s, o))
    Xh = gen_activations((M, K), seed=N + 5)
    X = dev_bf16(Xh)
    odt = torch.bfloat16 if bf16_out else torch.float32
    Y = torch.empty((M, N), dtype=odt, device="cuda")
    Y0 = torch.empty((M, N), dtype=odt, device="cuda")
    q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_Q4NX, M, N, K, X, blob, Y, work=work_if_any(q4, M, N, K, q4.Q4NX_WEIGHTS_Q4NX))
    q4.q4nx_gemm(M, N, K, X, blob, Y0)
    Yh, Y0h = host_f32(Y), host_f32(Y0)
    assert np.isfinite(Yh).all()
    rows = _rows(M, nrows)
    w32 = oracle.dequant_f32(codes, s, o)
    ok, worst = oracle.check_close(Yh[rows], oracle.gemm_f64(Xh[rows], w32), oracle.abs_bound(Xh[rows], w32),
                                   bf16_out=bf16_out)
    assert ok, worst
    w16 = oracle.bf16_to_f32(oracle.f32_to_bf16(w32))
    ref16 = oracle.gemm_f64(Xh[rows], w16)
    tight = np.abs(Yh[rows].astype(np.float64) - ref16) <= (
        1e-5 * oracle.abs_bound(Xh[rows], w16) + 1e-6 + (2.0 ** -8 * np.abs(ref16) if bf16_out else 0))
    assert tight.all()
    # Every element, split or not, against the unsplit launch: the same
    # products summed in another order (float32), or equal after bf16 rounding.
    scale = np.abs(Y0h).max()
    assert np.abs(Yh - Y0h).max() <= (1e-4 if not bf16_out else 2.0 ** -7) * scale


@pytest.mark.parametrize("M,N,K", [(2048, 4096, 2560), (2048, 2560, 2048), (2048, 20480, 2560), (2048, 2560, 10240)])
def test_gemm_ex_gemma3_4b_products(q4, M, N, K):
    """The four stacked Gemma3-4B prefill products at M = 2048 (q/k/v, o,
    gate/up, down) through the plans the benchmark runs, against the oracle on
    sampled rows."""
    _say("gemm_ex 4B", M, N, K)
    codes, s, o = gen_weights(N, K, seed=N + K)
    blob = dev_u8(q4.q4nx_pack(codes, s, o))
    Xh = gen_activations((M, K), seed=K + 1)
    Y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_Q4NX, M, N, K, dev_bf16(Xh), blob, Y,
                    work=work_if_any(q4, M, N, K, q4.Q4NX_WEIGHTS_Q4NX))
    rows = _rows(M, 24)
    w32 = oracle.dequant_f32(codes, s, o)
    ok, worst = oracle.check_close(host_f32(Y)[rows], oracle.gemm_f64(Xh[rows], w32), oracle.abs_bound(Xh[rows], w32))
    assert ok, worst


def test_gemm_ex_split_repeats_with_workspace_cleared(q4):
    """Ten calls of a split-K plan in a row, the workspace refilled with NaN
    before each: a partial read before its writer finished, or one left over
    from the previous call, would show as a NaN or a changed bit."""
    M, N, K = 2000, 1100, 6912
    _say("gemm_ex split repeats", M, N, K)
    codes, s, o = gen_weights(N, K, seed=77)
    blob = dev_u8(q4.q4nx_pack(codes, s, o))
    X = dev_bf16(gen_activations((M, K), seed=78))
    work = work_for(q4, M, N, K, q4.Q4NX_WEIGHTS_Q4NX)
    ref = torch.empty((M, N), dtype=torch.float32, device="cuda")
    q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_Q4NX, M, N, K, X, blob, ref, work=work)
    Y = torch.empty_like(ref)
    for _ in range(10):
        work.fill_(float("nan"))
        Y.fill_(float("nan"))
        q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_Q4NX, M, N, K, X, blob, Y, work=work)
        torch.cuda.synchronize()
        assert torch.equal(Y.view(torch.int32), ref.view(torch.int32))
    # And ten back to back without clearing (the partials of the previous
    # call in place).
    outs = [torch.empty_like(ref) for _ in range(10)]
    for y in outs:
        q4.q4nx_gemm_ex(q4.Q4NX_WEIGHTS_Q4NX, M, N, K, X, blob, y, work=work)
    torch.cuda.synchronize()
    assert all(torch.equal(y.view(torch.int32), ref.view(torch.int32)) for y in outs)
