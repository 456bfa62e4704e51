"""The entry point that allocates nothing (q4nx_flowkv_decode_static) against
the one with a caller workspace (q4nx_flowkv_decode), through the C ABI.

Both run the same kernels, so the outputs must be equal bit for bit; the
static entry point's outputs are also checked against the float64 oracle
with the FlowKV tolerance.  Two calls in a row, the second on a smaller
input, because every call on a device shares the one static array and it
keeps the previous call's contents.
"""
import ctypes

import numpy as np
import pytest

import oracle
from oracle.attention import decode_attention, attended_range

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def q4():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_06063_amd as mod
    return mod


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()


def _inputs(H, G, d, L, seed):
    rng = np.random.default_rng(seed)
    q = oracle.f32_to_bf16(rng.standard_normal((H, d), dtype=np.float32))
    K = oracle.f32_to_bf16(rng.standard_normal((G, L, d), dtype=np.float32))
    V = oracle.f32_to_bf16(rng.standard_normal((G, L, d), dtype=np.float32))
    return q, K, V


def _both(q4, H, G, d, L, t, window, seed, odt):
    """Runs both entry points on one input; returns (static, workspace) outputs
    and the host inputs."""
    q, K, V = _inputs(H, G, d, L, seed)
    qd, Kd, Vd = _dev(q), _dev(K), _dev(V)
    scale = ctypes.c_float(1.0 / np.sqrt(d))
    tdt = torch.float32 if odt == q4.Q4NX_F32 else torch.bfloat16
    o_static = torch.full((H, d), float("nan"), dtype=tdt, device="cuda")
    o_work = torch.full((H, d), float("nan"), dtype=tdt, device="cuda")
    j0, j1 = attended_range(t, window)
    wb = q4.lib.q4nx_flowkv_workspace_size(H, d, j1 - j0)
    work = torch.empty(wb // 4, dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    st = q4.lib.q4nx_flowkv_decode_static(qd.data_ptr(), Kd.data_ptr(), Vd.data_ptr(), H, G, d, L, t, window,
                                          scale, o_static.data_ptr(), odt, s)
    assert st == q4.Q4NX_OK, q4.lib.q4nx_last_error()
    st = q4.lib.q4nx_flowkv_decode(qd.data_ptr(), Kd.data_ptr(), Vd.data_ptr(), H, G, d, L, t, window, scale,
                                   o_work.data_ptr(), odt, work.data_ptr(), wb, s)
    assert st == q4.Q4NX_OK, q4.lib.q4nx_last_error()
    torch.cuda.synchronize()
    return o_static, o_work, (q, K, V, scale.value)


@pytest.mark.parametrize("odt_name", ["f32", "bf16"])
def test_static_scratch_equals_workspace_twice(q4, odt_name):
    odt = q4.Q4NX_F32 if odt_name == "f32" else q4.Q4NX_BF16
    # First a long context (27B geometry, 512-position chunks, many partials),
    # then a smaller one (4B geometry, windowed): the second call must not see
    # anything of the first in the shared array.
    for (H, G, d, L, t, window, seed) in [(32, 16, 128, 32768, 30000, 0, 11), (8, 4, 256, 4096, 2500, 1024, 12)]:
        print("[case] flowkv static", odt_name, H, G, d, L, t, window, flush=True)
        o_s, o_w, (q, K, V, scale) = _both(q4, H, G, d, L, t, window, seed, odt)
        view = torch.int32 if odt == q4.Q4NX_F32 else torch.int16
        assert torch.equal(o_s.view(view), o_w.view(view))
        ref, bound = decode_attention(q, K, V, t, window, scale)
        got = o_s.float().cpu().numpy().astype(np.float64)
        tol = 2e-3 * bound + 1e-6 + (2.0 ** -8 * np.abs(ref) if odt == q4.Q4NX_BF16 else 0.0)
        assert (np.abs(got - ref) <= tol).all()


def test_static_scratch_rejects_oversized(q4):
    # 27B geometry at 2^20 attended positions needs 32 heads x 2048 chunks of
    # 512 x 132 floats = 34.6 MB of partials > 16 MiB: rejected before launch.
    H, G, d, L = 32, 16, 128, 1 << 20
    big = torch.empty(16, dtype=torch.int16, device="cuda")
    o = torch.empty((H, d), dtype=torch.float32, device="cuda")
    st = q4.lib.q4nx_flowkv_decode_static(big.data_ptr(), big.data_ptr(), big.data_ptr(), H, G, d, L, L - 1, 0,
                                          ctypes.c_float(0.1), o.data_ptr(), q4.Q4NX_F32, None)
    assert st == q4.Q4NX_ERR_BUFFER_TOO_SMALL
    assert "static scratch" in q4.lib.q4nx_last_error().decode()
