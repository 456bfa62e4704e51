"""FlowKV decode attention (q4nx_flowkv_decode) against the float64 oracle.

Tolerance per output element: |o - o_ref| <= 2e-3 * sum_j p_j |v_j| + 1e-6
(plus half a bf16 ulp of o_ref for bf16 outputs).  Scores are float32 sums of
exact bf16 products (relative error below d * 2^-24 of sum |q k|); the
weighted sums run over up to 2^15 positions in float32 (below L * 2^-24
relative to sum p |v| in the worst case, far less in practice); the chunk
merge adds a few roundings more.
"""
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


def _case(H, G, d, L, seed):
    rng = np.random.default_rng(seed)
    q = oracle.f32_to_bf16(rng.standard_normal((H, d), dtype=np.float32))
    K = oracle.f32_to_bf16(rng.standard_normal((G, L, d), dtype=np.float32))
    V = oracle.f32_to_bf16(rng.standard_normal((G, L, d), dtype=np.float32))
    return q, K, V


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()


CASES = [
    # (H, G, d, L, t, window)  -- Gemma3 1B (4 heads, 1 group, d 256), 4B (8, 4, 256), 27B (32, 16, 128)
    (8, 4, 256, 4096, 0, 0),
    (8, 4, 256, 4096, 255, 0),
    (8, 4, 256, 4096, 256, 0),
    (8, 4, 256, 4096, 1000, 0),
    (8, 4, 256, 4096, 4095, 0),
    (8, 4, 256, 4096, 4095, 1024),
    (8, 4, 256, 4096, 700, 1024),
    (8, 4, 256, 4096, 2000, 1),
    (4, 1, 256, 2048, 1500, 0),
    (32, 16, 128, 4096, 3000, 0),
    (32, 16, 128, 4096, 3000, 1024),
    (8, 1, 64, 1024, 777, 0),
    (8, 4, 256, 32768, 32767, 0),
    # 1B geometry at 30K: 469 chunks of 64, more than a merge slice holds in
    # registers (the two-pass merge)
    (4, 1, 256, 32768, 30000, 0),
    (32, 16, 128, 32768, 20000, 0),
    # sliding windows of 1000 positions (a ragged last chunk: 40 positions
    # of a 64-position chunk, or 8 of a 32-position one) with at least 64
    # chunk workgroups: K and V requested with the query
    (32, 16, 128, 4096, 1500, 1000),
    (64, 16, 64, 2048, 1500, 1000),
    (8, 4, 256, 4096, 3000, 1000),
    # grids of 64-position chunks below one workgroup per CU take 32-position
    # chunks (K and V requested with the query from 64 workgroups): d = 128
    # and d = 64, whole and ragged last chunks
    (16, 4, 128, 2048, 1023, 1024),
    (16, 8, 64, 2048, 2000, 1000),
    # one KV group: 16-position chunks, with K and V requested early (64
    # chunks) and without (63, a ragged last chunk of 8), d = 256 and 128
    (4, 1, 256, 2048, 2047, 1024),
    (4, 1, 256, 2048, 1500, 1000),
    (8, 1, 128, 4096, 3000, 1024),
    # many heads: the merge takes 64, 128 and 256 dims per workgroup
    (64, 16, 128, 2048, 1999, 0),
    (128, 16, 128, 1024, 900, 0),
    (128, 16, 256, 1024, 1000, 0),
]


@pytest.mark.parametrize("H,G,d,L,t,window", CASES)
def test_flowkv_decode_vs_oracle(q4, H, G, d, L, t, window):
    print("[case] flowkv", H, G, d, L, t, window, flush=True)
    q, K, V = _case(H, G, d, L, seed=H * 1000 + t)
    scale = 1.0 / np.sqrt(d)
    j0, j1 = attended_range(t, window)
    work = torch.empty(q4.q4nx_flowkv_workspace_size(H, d, j1 - j0) // 4, dtype=torch.float32, device="cuda")
    o = torch.full((H, d), float("nan"), dtype=torch.float32, device="cuda")
    q4.q4nx_flowkv_decode(_dev(q), _dev(K), _dev(V), H, G, d, L, t, window, float(scale), o, work)
    torch.cuda.synchronize()
    ref, bound = decode_attention(q, K, V, t, window, scale)
    got = o.cpu().numpy().astype(np.float64)
    err = np.abs(got - ref)
    tol = 2e-3 * bound + 1e-6
    assert (err <= tol).all(), float((err / tol).max())


def test_flowkv_bf16_output_and_repeatable(q4):
    H, G, d, L, t = 8, 4, 256, 4096, 3333
    q, K, V = _case(H, G, d, L, seed=5)
    scale = 1.0 / 16.0
    work = torch.empty(q4.q4nx_flowkv_workspace_size(H, d, t + 1) // 4, dtype=torch.float32, device="cuda")
    o = torch.empty((H, d), dtype=torch.bfloat16, device="cuda")
    qd, Kd, Vd = _dev(q), _dev(K), _dev(V)
    q4.q4nx_flowkv_decode(qd, Kd, Vd, H, G, d, L, t, 0, scale, o, work)
    first = o.clone()
    q4.q4nx_flowkv_decode(qd, Kd, Vd, H, G, d, L, t, 0, scale, o, work)
    torch.cuda.synchronize()
    assert torch.equal(first.view(torch.int16), o.view(torch.int16))
    ref, bound = decode_attention(q, K, V, t, 0, scale)
    got = o.float().cpu().numpy().astype(np.float64)
    assert (np.abs(got - ref) <= 2e-3 * bound + 1e-6 + 2.0 ** -8 * np.abs(ref)).all()
