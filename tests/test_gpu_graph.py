"""HIP-graph capture of the projection launches: every replay (with eager
launches and synchronizations in between) must equal the eager result bit
for bit.  The library records no memset nodes; the kernels overwrite their
outputs completely."""
import numpy as np
import pytest

from workloads import gen_weights, gen_activations

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def test_graph_replay_matches_eager():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_06063_amd as q4
    print("[case] graph replay: gemv_batched + gemv + gemm", flush=True)
    s = torch.cuda.Stream()
    torch.cuda.set_stream(s)
    shapes = [(2048, 2560), (1024, 2560), (1024, 2560), (2560, 2048)]
    blobs, xs, ys = [], [], []
    for p, (N, K) in enumerate(shapes):
        codes, sc, of = gen_weights(N, K, seed=p)
        blobs.append(torch.from_numpy(q4.q4nx_pack(codes, sc, of)).cuda())
        xs.append(torch.from_numpy(gen_activations(K, seed=p).view(np.int16)).cuda())
        ys.append(torch.empty(N, dtype=torch.float32, device="cuda"))
    M = 96
    X = torch.from_numpy(gen_activations((M, 2048), seed=9).view(np.int16)).cuda()
    Y = torch.empty((M, 2560), dtype=torch.float32, device="cuda")

    def run():
        q4.q4nx_gemv_batched([(blobs[i], xs[i], ys[i], *shapes[i]) for i in range(3)], stream=s)
        q4.q4nx_gemv(blobs[3], xs[3], ys[3], *shapes[3], stream=s)
        q4.q4nx_gemm(M, 2560, 2048, X, blobs[3], Y, stream=s)

    run()
    torch.cuda.synchronize()
    ref = [y.clone() for y in ys] + [Y.clone()]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        run()
    for _ in range(3):
        for t in ys + [Y]:
            t.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(ys + [Y], ref):
            assert torch.equal(a.view(torch.int32), b.view(torch.int32))
        run()  # eager work between replays
        torch.cuda.synchronize()
