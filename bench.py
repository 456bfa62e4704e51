#!/usr/bin/env python3
"""Benchmark of the Q4NX projection path on one MI355X.

One step = one pass of the whole path over one batch of synthetic input:
  * decode: the FusedDQP mat-vec of every projection of every layer, in layer
    order -- per layer q/k/v in one batched launch, o, gate/up in one batched
    launch, down (+ lm_head once for the 4B decode step);
  * prefill: the fused dequant-GEMM of every projection of every layer on an
    M-token chunk; projections that read the same input (q/k/v, gate/up) run
    as one GEMM over their stacked weights, as an inference engine lays them
    out (a stacked Q4NX matrix is the projections' blobs back to back, since
    blocks are stored strip by strip and every N is a multiple of 32); each
    GEMM is q4nx_gemm_ex with a workspace, so shapes with few output tiles
    over a long K (the down projections) are split along K, and at M = 4096
    the Q4NX weights are dequantized to bf16 once per product before the
    bf16 plan runs (same bits as the fused kernel).
Inputs (packed weights, activations) are resident in HBM before the timed
region; every (layer, projection) has its own independently seeded weights and
activations.  Timing uses HIP events on the stream the kernels run on; the K
timed steps run their decode halves back to back and then their prefill
halves, so that each phase is timed in its steady state.

Prints one JSON line: value = decode weight GB/s (0.625 B per weight: the
4-bit code plus the per-32 bf16 scale and offset); the prefill TFLOP/s
(2*M*N*K per projection) is reported beside it.  The same steps over weights
in the MXFP4 variant of the block (0.53125 B per weight: the FP4 code plus the
per-32 E8M0 scale) are timed and reported under "mxfp4".

    python bench.py [--config 4] [--steps 5] [--warmup 2] [--gpus 1]

--config 0 times one GEMV launch (1B q_proj) cold and warm instead of a step.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import re
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0           # MI355X HBM3E
BF16_MFMA_PEAK_TFLOPS = 2516.6  # 256 CU x 4096 flop/clk x 2.4 GHz, dense
WEIGHT_BYTES = 0.625            # per weight: 0.5 code + 1/16 scale + 1/16 offset
MX_WEIGHT_BYTES = 0.53125       # MXFP4 variant: 0.5 code + 1/32 E8M0 scale
# Projections of a layer that read the same input, in order: q/k/v, o, gate/up, down.
GROUPS = [[0, 1, 2], [3], [4, 5], [6]]


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=4, choices=[0, 1, 2, 3, 4])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--offset-mode", default="zp", choices=["zp", "literal"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-layers", type=int, default=6, help="layers of the oracle CPU sample")
    ap.add_argument("--decode-graph", type=int, default=1, help="replay the decode step as a HIP graph")
    ap.add_argument("--two-phase", type=int, default=1,
                    help="also time the two-phase prefill (q4nx_dequant to bf16, then q4nx_gemm_bf16)")
    ap.add_argument("--fused", type=int, default=1,
                    help="also time the prefill step through q4nx_gemm alone (fused dequant-GEMM, no workspace)")
    ap.add_argument("--bf16-out", type=int, default=1,
                    help="also time the prefill step with bf16 outputs (the paper keeps every activation in bf16)")
    ap.add_argument("--quantize", type=int, default=1,
                    help="also time q4nx_quantize on the model's largest projection (float32 -> Q4NX)")
    ap.add_argument("--flowkv", type=int, default=1,
                    help="also time FlowKV decode attention over every layer at --context positions")
    ap.add_argument("--context", type=int, default=32768, help="decode position + 1 for the FlowKV timing")
    ap.add_argument("--mx", type=int, default=1,
                    help="also time the decode and prefill steps over MXFP4-variant weights")
    ap.add_argument("--with-4b", type=int, default=1,
                    help="with the default 27B configuration, also run the 4B decode step and prefill chunk "
                         "(configurations 2 and 3) and report them beside it")
    ap.add_argument("--pmc-pass", action="store_true",
                    help="run one eager decode step, one prefill step and a 1 GiB device copy (for rocprofv3 "
                         "counter passes), then exit")
    ap.add_argument("--trace-summary", nargs=2, metavar=("TRACE_DIR", "BENCH_JSON"),
                    help="summarise a rocprofv3 --kernel-trace --stats run of this benchmark as markdown")
    ap.add_argument("--pmc-summary", nargs="+", metavar="DIR",
                    help="summarise the rocprofv3 --pmc output folders of --pmc-pass runs as markdown: "
                         "FETCH_DIR WRITE_DIR MFMA_DIR [LDS_DIR]")
    return ap.parse_args()


def build_weights(model, cfg, seed, mode, q4, torch, mx=False):
    """Generate, pack (q4nx_pack, or q4nx_mx_pack for the MXFP4 variant) and
    upload every projection's weights.  The blobs of a group of projections
    that share an input lie back to back in one device buffer, which is the
    packed blob of the stacked matrix; returns ({(layer, proj): blob view},
    {(layer, group): stacked blob})."""
    from workloads import gen_weights, gen_mx_weights
    L = model["layers"]
    tasks = [(l, p, N, K) for l in range(L) for p, (_, N, K) in enumerate(model["proj"])]
    if cfg.get("lm_head"):
        tasks.append((L, 7, model["lm_head"][1], model["lm_head"][2]))

    def work(t):
        l, p, N, K = t
        if mx:
            return q4.q4nx_mx_pack(*gen_mx_weights(N, K, seed=seed, layer=l, proj=p))
        codes, s, o = gen_weights(N, K, seed=seed, layer=l, proj=p, offset_mode=mode)
        return q4.q4nx_pack(codes, s, o)

    size = q4.q4nx_mx_packed_size if mx else q4.q4nx_packed_size
    out, stacked = {}, {}
    for l in range(L):
        for gi, g in enumerate(GROUPS):
            buf = torch.empty(sum(size(model["proj"][p][1], model["proj"][p][2]) for p in g), dtype=torch.uint8,
                              device="cuda")
            stacked[(l, gi)] = buf
            off = 0
            for p in g:
                n = size(model["proj"][p][1], model["proj"][p][2])
                out[(l, p)] = buf[off:off + n]
                off += n
    t0 = time.time()
    workers = max(1, min(16, len(os.sched_getaffinity(0))))
    with ThreadPoolExecutor(workers) as ex:
        for i, (t, blob) in enumerate(zip(tasks, ex.map(work, tasks))):
            key = (t[0], t[1])
            if key in out:
                out[key].copy_(torch.from_numpy(blob))
            else:
                out[key] = torch.from_numpy(blob).cuda()
            if (i + 1) % 50 == 0 or i + 1 == len(tasks):
                log(f"{'MXFP4 ' if mx else ''}weights {i + 1}/{len(tasks)} packed+uploaded ({time.time() - t0:.0f}s)")
    return out, stacked


class Step:
    """Prebuilt C-ABI calls of one step (pointers marshalled once)."""

    def __init__(self, q4, stream, mx=False):
        self.q4 = q4
        self.s = ctypes.c_void_p(stream)
        self.calls = []
        self.keep = []
        # weight format of the packed launches: Q4NX or the MXFP4 variant
        self.size = q4.q4nx_mx_packed_size if mx else q4.q4nx_packed_size
        self.gemv_fn = q4.lib.q4nx_mx_gemv_batched if mx else q4.lib.q4nx_gemv_batched
        self.wformat = q4.Q4NX_WEIGHTS_MXFP4 if mx else q4.Q4NX_WEIGHTS_Q4NX
        self.work = None  # GEMM workspace (q4nx_gemm_ex may split K with it), shared by the step's launches

    def _work(self, fmt, M, N, K):
        need = self.q4.q4nx_gemm_workspace_size(fmt, M, N, K)
        have = 0 if self.work is None else self.work.numel() * 4
        if need > have:
            raise ValueError(f"GEMM workspace: {have} bytes, {M}x{N}x{K} needs {need}")
        return (self.work.data_ptr() if self.work is not None else None), have

    def gemv_batched(self, items, ydt):
        arr = (self.q4.q4nx_gemv_desc * len(items))()
        for i, (blob, x, y, N, K) in enumerate(items):
            self.q4._need(blob, self.size(N, K), "blob")
            self.q4._need(x, 2 * K, "x")
            self.q4._need(y, N * y.element_size(), "y")
            arr[i] = self.q4.q4nx_gemv_desc(blob.data_ptr(), x.data_ptr(), y.data_ptr(), N, K)
        self.keep.append(arr)
        self.calls.append((self.gemv_fn, (arr, len(items), ydt, self.s)))

    def gemm(self, M, N, K, X, blob, Y, ydt):
        self.q4._need(blob, self.size(N, K), "blob")
        self.q4._need(X, 2 * M * K, "X")
        self.q4._need(Y, M * N * Y.element_size(), "Y")
        wp, wn = self._work(self.wformat, M, N, K)
        self.calls.append((self.q4.lib.q4nx_gemm_ex, (self.wformat, M, N, K, X.data_ptr(), blob.data_ptr(),
                                                      Y.data_ptr(), ydt, wp, wn, self.s)))

    def gemm_fused(self, M, N, K, X, blob, Y, ydt):
        """q4nx_gemm: the fused dequant-GEMM, no workspace (no split K, no dequantize-once)."""
        self.q4._need(blob, self.size(N, K), "blob")
        self.q4._need(X, 2 * M * K, "X")
        self.q4._need(Y, M * N * Y.element_size(), "Y")
        self.calls.append((self.q4.lib.q4nx_gemm, (M, N, K, X.data_ptr(), blob.data_ptr(), Y.data_ptr(), ydt, self.s)))

    def dequant_bf16(self, blob, N, K, W):
        self.q4._need(blob, self.q4.q4nx_packed_size(N, K), "blob")
        self.q4._need(W, 2 * N * K, "W")
        self.calls.append((self.q4.lib.q4nx_dequant, (blob.data_ptr(), N, K, W.data_ptr(), self.q4.Q4NX_BF16, self.s)))

    def gemm_bf16(self, M, N, K, X, W, Y, ydt):
        self.q4._need(W, 2 * N * K, "W")
        self.q4._need(X, 2 * M * K, "X")
        self.q4._need(Y, M * N * Y.element_size(), "Y")
        wp, wn = self._work(self.q4.Q4NX_WEIGHTS_BF16, M, N, K)
        self.calls.append((self.q4.lib.q4nx_gemm_ex, (self.q4.Q4NX_WEIGHTS_BF16, M, N, K, X.data_ptr(), W.data_ptr(),
                                                      Y.data_ptr(), ydt, wp, wn, self.s)))

    def run(self):
        for fn, args in self.calls:
            st = fn(*args)
            if st:
                raise RuntimeError(f"{fn.__name__}: status {st}: {self.q4.lib.q4nx_last_error().decode()}")


def time_steps(torch, stream, fn, steps):
    """Runs fn `steps` times back to back, each between an event pair on
    `stream`; returns (median ms, min ms)."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    for a, b in evs:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    ts = sorted(a.elapsed_time(b) for a, b in evs)
    return ts[len(ts) // 2], ts[0]


def capture(torch, stream, fn):
    """fn captured as a HIP graph on `stream` (run once eagerly first)."""
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        fn()
    return g


def faster_launch_mode(torch, stream, run, outputs, warmup):
    """The decode step as a HIP graph, checked bit for bit against eager
    launches on three replays (outputs cleared in between), and the faster
    of graph and eager by a short timing; returns (fn, info)."""
    run()
    torch.cuda.synchronize()
    ref = [y.clone() for y in outputs]
    g = capture(torch, stream, run)
    ok = True
    for _ in range(3):
        for y in outputs:
            y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        ok = ok and all(torch.equal(a.view(torch.int32), b.view(torch.int32)) for a, b in zip(outputs, ref))
        run()
        torch.cuda.synchronize()
    info = {"replays_checked": 3, "bitwise_equal_to_eager": bool(ok)}
    if not ok:
        return run, dict(info, launch="eager")
    for _ in range(warmup):
        g.replay()
        run()
    gm, _ = time_steps(torch, stream, g.replay, 3)
    em, _ = time_steps(torch, stream, run, 3)
    info["calibration_ms"] = {"graph": round(gm, 4), "eager": round(em, 4)}
    if gm <= em:
        return g.replay, dict(info, launch="hip graph replay", graph=g)
    return run, dict(info, launch="eager", graph=g)


def launch_floor(q4, torch, stream, blobs, steps, warmup):
    """q4nx_stream_read over each decode launch's weight bytes, one launch per
    GEMV launch (the faster of graph and eager): the time a plain streaming
    kernel needs for the same bytes in the same launch structure."""
    sink = torch.empty(8192, dtype=torch.float32, device="cuda")
    fl = Step(q4, stream.cuda_stream)
    for b in blobs:
        fl.calls.append((q4.lib.q4nx_stream_read, (b.data_ptr(), b.numel(), sink.data_ptr(), fl.s)))
    g = capture(torch, stream, fl.run)
    fn = g.replay if time_steps(torch, stream, g.replay, 3)[0] < time_steps(torch, stream, fl.run, 3)[0] else fl.run
    for _ in range(warmup):
        fn()
    ms, _ = time_steps(torch, stream, fn, steps)
    nbytes = sum(b.numel() for b in blobs)
    return {"what": "q4nx_stream_read (a plain streaming read with the GEMV's load pattern) over each decode "
                    "launch's weight bytes, one launch per GEMV launch, graph or eager (the faster)",
            "launches": len(blobs), "ms_median": round(ms, 4), "GB_per_s": round(nbytes / (ms * 1e-3) / 1e9, 1)}


def run_4b(args, q4, torch, stream):
    """The Gemma3-4B workloads beside the default 27B line: the decode step
    (34 layers + lm_head 262144 x 2560, M = 1) and the prefill chunk (34
    layers, M = 2048), timed like the 27B steps, each with its roofline
    fraction, and checked in the same run against the oracle: every output of
    layers 0 and 33 and 4096 sampled lm_head rows at decode, every element of
    layer 0's four prefill products and 256 sampled token rows of layer 33's."""
    import numpy as np
    import oracle
    from workloads import MODELS, CONFIGS, gen_weights, gen_activations, gen_activations_device
    cfg = CONFIGS[2]
    model = MODELS[cfg["model"]]
    L = model["layers"]
    F32 = q4.Q4NX_F32
    log(f"gemma3-4b: {L} layers, decode step with lm_head and prefill chunk at M = 2048")
    weights, stacked = build_weights(model, cfg, args.seed, args.offset_mode, q4, torch)
    out = {}
    # ---- decode step
    xs, ys, dec_bytes = {}, {}, 0.0
    keys = [(l, p) for l in range(L) for p in range(len(model["proj"]))] + [(L, 7)]
    for (l, p) in keys:
        _, N, K = model["lm_head"] if p == 7 else model["proj"][p]
        xs[(l, p)] = torch.from_numpy(gen_activations(K, seed=args.seed, layer=l, proj=p).view("int16")).cuda()
        ys[(l, p)] = torch.empty(N, dtype=torch.float32, device="cuda")
        dec_bytes += N * K * WEIGHT_BYTES
    dec = Step(q4, stream.cuda_stream)
    for l in range(L):
        it = lambda p: (weights[(l, p)], xs[(l, p)], ys[(l, p)], model["proj"][p][1], model["proj"][p][2])
        for g in GROUPS:
            dec.gemv_batched([it(p) for p in g], F32)
    _, Nh, Kh = model["lm_head"]
    dec.gemv_batched([(weights[(L, 7)], xs[(L, 7)], ys[(L, 7)], Nh, Kh)], F32)
    for _ in range(args.warmup):
        dec.run()
    fn, info = faster_launch_mode(torch, stream, dec.run, list(ys.values()), args.warmup)
    info.pop("graph", None)
    ms, ms_min = time_steps(torch, stream, fn, args.steps)
    gbs = dec_bytes / (ms * 1e-3) / 1e9
    floor = launch_floor(q4, torch, stream, [stacked[(l, gi)] for l in range(L) for gi in range(len(GROUPS))]
                         + [weights[(L, 7)]], args.steps, args.warmup)
    floor["decode_ms_median_over_floor"] = round(ms / floor["ms_median"], 4)
    out["decode"] = {"workload": cfg["name"], "ms_median": round(ms, 4), "ms_min": round(ms_min, 4),
                     "weight_GB": round(dec_bytes / 1e9, 4), "GB_per_s": round(gbs, 2),
                     "frac_hbm": round(gbs / HBM_PEAK_GBS, 4), "launches": len(dec.calls), "launch": info["launch"],
                     "graph_check": info, "launch_floor": floor,
                     "target": "70% of 8 TB/s = 0.433 ms"}
    st = stored_traffic(2)
    if st and "gemv" in st["families"]:
        out["decode"]["traffic"] = round(st["families"]["gemv"]["hbm_bytes_per_step"])
        out["decode"]["traffic_note"] = ("HBM bytes per step of the GEMV launches from rocprofv3 FETCH_SIZE/WRITE_SIZE "
                                         "scaled by a copy-kernel calibration: "
                                         + os.path.relpath(traffic_file(2), ROOT))
    log(f"4b decode {ms:.3f} ms ({gbs:.0f} GB/s), floor {floor['ms_median']:.3f} ms")
    # ---- prefill chunk
    M = 2048
    shapes = [(sum(model["proj"][p][1] for p in g), model["proj"][g[0]][2]) for g in GROUPS]
    Xs = {(l, gi): gen_activations_device((M, K), seed=args.seed, layer=l, proj=GROUPS[gi][0])
          for l in range(L) for gi, (N, K) in enumerate(shapes)}
    Ys = [torch.empty((M, N), dtype=torch.float32, device="cuda") for N, _ in shapes]
    wb = max(q4.q4nx_gemm_workspace_size(q4.Q4NX_WEIGHTS_Q4NX, M, N, K) for N, K in shapes)
    pre = Step(q4, stream.cuda_stream)
    pre.work = torch.empty(max(wb // 4, 1), dtype=torch.float32, device="cuda")
    flops = 0.0
    for l in range(L):
        for gi, (N, K) in enumerate(shapes):
            pre.gemm(M, N, K, Xs[(l, gi)], stacked[(l, gi)], Ys[gi], F32)
            flops += 2.0 * M * N * K
    for _ in range(args.warmup):
        pre.run()
    pms, pms_min = time_steps(torch, stream, pre.run, args.steps)
    tf = flops / (pms * 1e-3) / 1e12
    out["prefill"] = {"workload": CONFIGS[3]["name"], "ms_median": round(pms, 4), "ms_min": round(pms_min, 4),
                      "M": M, "TFLOP": round(flops / 1e12, 4), "TFLOP_per_s": round(tf, 2),
                      "frac_mfma": round(tf / BF16_MFMA_PEAK_TFLOPS, 4), "launches": len(pre.calls),
                      "gemms": ", ".join(f"{N}x{K}" for N, K in shapes), "target": "50% of 2516.6 TFLOP/s = 10.45 ms"}
    st = stored_traffic(3)
    if st and "gemm" in st["families"]:
        e = st["families"]["gemm"]
        out["prefill"]["traffic"] = round(e["hbm_bytes_per_step"])
        out["prefill"]["traffic_note"] = ("HBM bytes per step of the GEMM launches from rocprofv3 FETCH_SIZE/WRITE_SIZE "
                                          "scaled by a copy-kernel calibration: " + os.path.relpath(traffic_file(3), ROOT))
        if "mfma_busy_fraction" in e:
            out["prefill"]["mfma_busy_counter"] = round(e["mfma_busy_fraction"], 4)
    log(f"4b prefill {pms:.3f} ms ({tf:.0f} TFLOP/s)")
    if args.no_cpu_baseline:
        return out
    # ---- parity against the oracle, same run
    checks = []
    for l in (0, L - 1):
        for c in dec.calls[4 * l:4 * l + 4]:
            c[0](*c[1])
    dec.calls[-1][0](*dec.calls[-1][1])
    for gi in range(len(GROUPS)):
        pre.calls[gi][0](*pre.calls[gi][1])
    torch.cuda.synchronize()
    y0 = {k: ys[k].cpu().numpy() for k in ys if k[0] in (0, L - 1, L)}
    Yl0 = [Y.cpu().numpy() for Y in Ys]
    rng = np.random.default_rng(args.seed)
    rows = np.unique(np.concatenate([[0, M - 1], rng.integers(0, M, 254)]))
    for gi in range(len(GROUPS)):   # last layer's products on sampled rows (run after layer 0's are copied)
        pre.calls[4 * (L - 1) + gi][0](*pre.calls[4 * (L - 1) + gi][1])
    torch.cuda.synchronize()
    idx = torch.tensor(rows, device="cuda")
    Ylast = [Y.index_select(0, idx).cpu().numpy() for Y in Ys]
    for l in (0, L - 1):
        wl = []
        for p, (_, N, K) in enumerate(model["proj"]):
            codes, sc, of = gen_weights(N, K, seed=args.seed, layer=l, proj=p, offset_mode=args.offset_mode)
            w = oracle.dequant_f32(codes, sc, of)
            x = gen_activations(K, seed=args.seed, layer=l, proj=p)
            ok, worst = oracle.check_close(y0[(l, p)], oracle.gemv_f64(w, x), oracle.abs_bound(x, w))
            checks.append(("decode", ok, worst))
            wl.append(w)
        for gi, g in enumerate(GROUPS):
            w = np.concatenate([wl[p] for p in g])
            X = Xs[(l, gi)].view(torch.int16).cpu().numpy().view("uint16")
            if l == 0:
                ok, worst = oracle.check_close(Yl0[gi], oracle.gemm_f64(X, w), oracle.abs_bound(X, w))
            else:
                ok, worst = oracle.check_close(Ylast[gi], oracle.gemm_f64(X[rows], w), oracle.abs_bound(X[rows], w))
            checks.append(("prefill", ok, worst))
        log(f"4b oracle check: layer {l} done")
        del wl
    codes, sc, of = gen_weights(Nh, Kh, seed=args.seed, layer=L, proj=7, offset_mode=args.offset_mode)
    hr = np.unique(np.concatenate([[0, Nh - 1], rng.integers(0, Nh, 4094)]))
    w = oracle.dequant_f32(codes[hr], sc[hr], of[hr])
    x = gen_activations(Kh, seed=args.seed, layer=L, proj=7)
    ok, worst = oracle.check_close(y0[(L, 7)][hr], oracle.gemv_f64(w, x), oracle.abs_bound(x, w))
    checks.append(("decode", ok, worst))
    out["parity_check"] = {
        "tolerance": "|y - y_ref| <= 2e-3 * sum_k |x_k w_k| + 1e-5 per output, float64 oracle",
        "decode": f"every output of layers 0 and {L - 1} (7 projections each) and {len(hr)} sampled lm_head rows",
        "prefill": f"every element of layer 0's 4 products, {len(rows)} sampled token rows of layer {L - 1}'s",
        "decode_worst_err_over_tol": float(f"{max(c[2] for c in checks if c[0] == 'decode'):.3g}"),
        "prefill_worst_err_over_tol": float(f"{max(c[2] for c in checks if c[0] == 'prefill'):.3g}"),
        "ok": all(c[1] for c in checks)}
    del weights, stacked, Xs, Ys, pre, dec
    torch.cuda.empty_cache()
    return out


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:  # pragma: no cover
        pass
    return "unknown"


def blas_thread_count():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        return 1


def cpu_baseline(model, cfg, seed, mode, layers, do_decode, do_prefill, M_prefill):
    """The oracle, untuned, on a bounded sample: `layers` layer(s) of the
    workload's projections, timed on this host's cores (16 token rows of the
    prefill chunk)."""
    import oracle
    from workloads import gen_weights, gen_activations
    blas_threads = blas_thread_count()
    dec_t = dec_bytes = 0.0
    pre_t = pre_flops = 0.0
    deq_total = mv_total = mm_total = 0.0   # the oracle's dequant, mat-vec and matmul separately
    rows = 16
    first = {p: g[0] for g in GROUPS for p in g}   # projections of a group share the prefill input
    for l in range(layers):
        for p, (_, N, K) in enumerate(model["proj"]):
            codes, s, o = gen_weights(N, K, seed=seed, layer=l, proj=p, offset_mode=mode)
            blob = oracle.pack(codes, s, o)
            x = gen_activations(K, seed=seed, layer=l, proj=p)
            X = gen_activations((rows, K), seed=seed, layer=l, proj=first[p])
            t0 = time.perf_counter()
            w = oracle.dequant_blob_f32(blob, N, K)
            t_deq = time.perf_counter() - t0
            deq_total += t_deq
            if do_decode:
                t0 = time.perf_counter()
                oracle.gemv_f64(w, x)
                t_mv = time.perf_counter() - t0
                mv_total += t_mv
                dec_t += t_deq + t_mv
                dec_bytes += N * K * WEIGHT_BYTES
            if do_prefill:
                t0 = time.perf_counter()
                oracle.gemm_f64(X, w)
                t_mm = time.perf_counter() - t0
                mm_total += t_mm
                pre_t += t_deq + t_mm
                pre_flops += 2.0 * rows * N * K
            log(f"oracle sample: layer {l} projection {p} ({N}x{K}) done")
    out = {"cores": int(blas_threads), "kind": "oracle", "cpu_model": cpu_model(),
           "affinity_cpus": len(os.sched_getaffinity(0)),
           "seconds_split": {"dequant": round(deq_total, 4), "matvec": round(mv_total, 4),
                             "matmul": round(mm_total, 4)}}
    what = f"{layers} layer(s) x {len(model['proj'])} projections of {cfg['name']}"
    if do_decode:
        out.update(value=dec_bytes / dec_t / 1e9, unit="GB/s",
                   sample=f"decode M=1 over {what}: NumPy float32 Eq. 3 dequant + float64 mat-vec "
                          f"(dequant single-threaded, mat-vec on {blas_threads} BLAS threads)",
                   seconds=dec_t)
    if do_prefill:
        pf = {"value": pre_flops / pre_t / 1e12, "unit": "TFLOP/s", "seconds": pre_t,
              "sample": f"prefill {rows} of {M_prefill} token rows over {what}: float32 dequant + float64 matmul"}
        if do_decode:
            out["prefill"] = pf
        else:
            out.update(value=pf["value"], unit=pf["unit"], sample=pf["sample"], seconds=pre_t)
    return out


def parity_check(model, seed, mode, gpu):
    """The timed steps' outputs against the oracle (untimed): at decode every
    output of the layers in gpu["decode"]; at prefill every element of the
    product in gpu["prefill_full"] and the sampled token rows of the last
    layer's products in gpu["prefill"]."""
    import numpy as np
    import oracle
    from workloads import gen_weights, gen_activations
    checks = []
    layers = sorted(set([l for l, _ in gpu.get("decode", {})] + ([gpu["prefill_layer"]] if "prefill" in gpu else [])
                        + ([gpu["prefill_full"][0]] if "prefill_full" in gpu else [])))
    for l in layers:
        ws = {}
        for p, (_, N, K) in enumerate(model["proj"]):
            codes, sc, of = gen_weights(N, K, seed=seed, layer=l, proj=p, offset_mode=mode)
            ws[p] = oracle.dequant_f32(codes, sc, of)
            if (l, p) in gpu.get("decode", {}):
                x = gen_activations(K, seed=seed, layer=l, proj=p)
                ok, worst = oracle.check_close(gpu["decode"][(l, p)], oracle.gemv_f64(ws[p], x),
                                               oracle.abs_bound(x, ws[p]))
                checks.append(("decode", ok, worst))
        if "prefill_full" in gpu and gpu["prefill_full"][0] == l:
            _, gi, X, Y = gpu["prefill_full"]
            w = np.concatenate([ws[p] for p in GROUPS[gi]])
            ok, worst = oracle.check_close(Y, oracle.gemm_f64(X, w), oracle.abs_bound(X, w))
            checks.append(("prefill", ok, worst))
        if "prefill" in gpu and gpu["prefill_layer"] == l:
            for gi, (Xr, Yr) in gpu["prefill"].items():
                w = np.concatenate([ws[p] for p in GROUPS[gi]])
                ok, worst = oracle.check_close(Yr, oracle.gemm_f64(Xr, w), oracle.abs_bound(Xr, w))
                checks.append(("prefill", ok, worst))
        log(f"oracle check: layer {l} done")
        del ws
    pc = {"tolerance": "|y - y_ref| <= 2e-3 * sum_k |x_k w_k| + 1e-5 per output, float64 oracle"}
    if "decode" in gpu:
        dl = sorted(set(l for l, _ in gpu["decode"]))
        pc["decode"] = f"every output of layers {dl} ({len(gpu['decode'])} projections)"
    if "prefill_full" in gpu or "prefill" in gpu:
        parts = []
        if "prefill_full" in gpu:
            l, gi, X, _ = gpu["prefill_full"]
            parts.append(f"every element of layer {l}'s product {gi} ({X.shape[0]} x {gpu['prefill_full'][3].shape[1]})")
        if "prefill" in gpu:
            parts.append(f"{gpu['prefill_rows']} sampled token rows of each of layer {gpu['prefill_layer']}'s "
                         f"{len(gpu['prefill'])} stacked products")
        pc["prefill"] = "; ".join(parts)
    for kind in ("decode", "prefill"):
        cs = [c for c in checks if c[0] == kind]
        if cs:
            pc[f"{kind}_worst_err_over_tol"] = float(f"{max(c[2] for c in cs):.3g}")
    pc["ok"] = all(c[1] for c in checks)
    return pc


KERNEL_SOURCE = os.path.join(ROOT, "paper_2602_06063_amd", "csrc", "q4nx_kernels.hip")
PROFILES = os.path.join(ROOT, "profiles")
CALIB_BYTES = 1 << 30  # the calibration copy reads and writes this many bytes


def kernel_code_text(text):
    """The kernel source with comments, trailing blanks and empty lines taken
    out: what the counters depend on (a comment edit leaves them valid)."""
    import re
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    lines = [re.sub(r"//.*$", "", l).rstrip() for l in text.splitlines()]
    return "\n".join(l for l in lines if l)


def kernel_source_sha256(text=None):
    import hashlib
    if text is None:
        with open(KERNEL_SOURCE) as f:
            text = f.read()
    return hashlib.sha256(kernel_code_text(text).encode()).hexdigest()


# Counter summaries, named for the workload of each configuration.
WORKLOAD_SLUG = {1: "gemma3-1b_decode-M1", 2: "gemma3-4b_decode-M1", 3: "gemma3-4b_prefill-M2048",
                 4: "gemma3-27b_decode-M1_prefill-M4096"}


def traffic_file(config):
    return os.path.join(PROFILES, f"hbm-traffic_{WORKLOAD_SLUG.get(config, f'config{config}')}.md")


# The prefill step's launches: the products, their partial sums and the
# dequant pass of products that dequantize first.
PREFILL_KERNELS = ("gemm256_kernel", "gemm256x128_kernel", "gemm_kernel", "splitk_sum_kernel", "dequant_kernel")


def kernel_family(name):
    # (The counter passes run only the decode and prefill steps, so no other
    # step launches these.)
    if any(k in name for k in PREFILL_KERNELS):
        return "gemm"
    if re.search(r"gemv(_stream)?_kernel<", name):
        return "gemv"
    return None


def kernel_base_name(name):
    """`void q4nx::gemm256_kernel<false, 0>(...)` -> `gemm256_kernel`."""
    base = name.split("(")[0].split("<")[0].strip()
    return base.split()[-1].split("::")[-1] if base else name


def trace_summary(trace_dir, bench_json):
    """Markdown summary of a rocprofv3 --kernel-trace --stats run of this
    benchmark (its *kernel_stats.csv) next to the JSON line the same run
    printed: per-kernel calls and durations, and the per-step time of the
    roofline kernels against the benchmark's own HIP-event time."""
    import csv
    import glob
    paths = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)
    if not paths:
        raise SystemExit(f"no *kernel_stats.csv under {trace_dir}")
    rows = list(csv.DictReader(open(paths[0])))
    r = json.loads(open(bench_json).read().strip().splitlines()[-1])
    runs = r["warmup"] + r["steps"]
    kern = [(row["Name"], int(row["Calls"]), float(row["TotalDurationNs"]) / 1e6) for row in rows]
    total = sum(k[2] for k in kern)
    out = ["| kernel | calls | avg (us) | total (ms) | share |", "|---|---:|---:|---:|---:|"]
    for n, c, t in sorted(kern, key=lambda k: -k[2])[:14]:
        short = n.split("(")[0].replace("q4nx::", "")
        out.append(f"| `{short[:90]}` | {c} | {1e3 * t / c:.1f} | {t:.1f} | {100 * t / total:.2f}% |")
    lines = ["\n".join(out), ""]
    # The prefill step's kernels: the products, their partial sums and, where a
    # Q4NX product dequantizes first, the dequant pass.  Other steps that use
    # them (the two-phase comparison, the MXFP4 variant) must be off in the
    # profiled run, or the attribution would mix them in.
    pf = r.get("prefill", {})
    if pf.get("two_phase") or pf.get("bf16_outputs") or pf.get("fused_only") or "prefill" in (r.get("mxfp4") or {}):
        raise SystemExit("profile with --two-phase 0 --mx 0 --bf16-out 0 --fused 0: those steps launch the same "
                         "kernels")
    fam = PREFILL_KERNELS
    gemm = [(n, c, t) for n, c, t in kern if any(f in n.split("(")[0] for f in fam)]
    gemm_t, gemm_c = sum(k[2] for k in gemm), sum(k[1] for k in gemm)
    if "prefill" in r:
        per = gemm_t / runs
        tflop = r["prefill"]["TFLOP"]
        lines.append(f"Prefill kernels ({', '.join('`' + f + '`' for f in fam)}): {gemm_c} launches, "
                     f"{gemm_t:.1f} ms over the {runs} runs of the prefill step (warm-up + timed) = {per:.2f} ms "
                     f"per step; the benchmark's HIP-event time of the step (median): {r['prefill']['ms_median']:.2f} ms.")
        lines.append(f"Achieved: {tflop:.2f} TFLOP per step / {per:.2f} ms = {tflop / per * 1e3:.0f} TFLOP/s "
                     f"(benchmark: {r['prefill']['TFLOP_per_s']:.0f} TFLOP/s, "
                     f"{100 * r['prefill']['frac_mfma']:.1f}% of {BF16_MFMA_PEAK_TFLOPS} TFLOP/s dense bf16).")
    # Q4NX GEMV launches: gemv_kernel and gemv_stream_kernel with the Q4NX
    # format (last template argument 1; 2 is the MXFP4 variant).
    gv = [(n, c, t) for n, c, t in kern if re.search(r"gemv(_stream)?_kernel<", n.split("(")[0])
          and n.split("(")[0].rstrip().endswith("1>")]
    if gv and "decode" in r:
        c = sum(k[1] for k in gv)
        t = sum(k[2] for k in gv)
        d = r["decode"]
        per = 1e3 * t / c * d["launches"] / 1e3
        lines.append(f"Q4NX GEMV (`gemv_kernel`, `gemv_stream_kernel`): {c} launches, average {1e3 * t / c:.2f} us; "
                     f"x {d['launches']} launches per decode step = {per:.3f} ms of kernel time per step = "
                     f"{d['weight_GB'] / per * 1e3:.0f} GB/s ({d['weight_GB'] / per * 1e3 / HBM_PEAK_GBS * 100:.1f}% of "
                     f"8 TB/s) for {d['weight_GB']:.3f} GB. The benchmark's own step time in this profiled run "
                     f"({d['launch']}, median): {d['ms_median']:.3f} ms (the tracer adds time between dispatches).")
    return "\n".join(lines) + "\n"


def read_pmc(folder):
    """Per-dispatch counter values of a rocprofv3 --pmc csv folder:
    {dispatch_id: (kernel_name, {counter: value})}."""
    import csv
    import glob
    out = {}
    for path in glob.glob(os.path.join(folder, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                d = int(r["Dispatch_Id"])
                name, ctr = out.setdefault(d, (r["Kernel_Name"], {}))
                ctr[r["Counter_Name"]] = ctr.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return out


LDS_COUNTERS = ("SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", "SQ_WAIT_INST_LDS", "SQ_WAIT_ANY", "SQ_WAVE_CYCLES",
                "SQ_LDS_DATA_FIFO_FULL", "GRBM_GUI_ACTIVE")


def pmc_summary(config, fetch_dir, write_dir, mfma_dir, lds_dir=None):
    """Markdown summary of the counter passes, with a JSON block that bench.py
    reads back (only while the kernel source is unchanged).  FETCH_SIZE and
    WRITE_SIZE are KiB per dispatch; each is scaled by bytes / counter of the
    calibration copy (the last dispatch of the pass).  The optional fourth pass
    gives, per kernel family, the share of LDS cycles lost to bank conflicts
    and the shares of wave cycles spent waiting to issue an LDS instruction
    and waiting on a memory counter (s_waitcnt)."""
    fetch, write, mfma = read_pmc(fetch_dir), read_pmc(write_dir), read_pmc(mfma_dir)
    lds = read_pmc(lds_dir) if lds_dir else {}

    def calib(pass_, counter):
        # Copy dispatches after the last kernel of the path: the calibration copy.
        last = max(d for d, (n, _) in pass_.items() if kernel_family(n))
        return sum(c[counter] for d, (n, c) in pass_.items() if d > last and "copy" in n.lower())
    calib_f, calib_w = calib(fetch, "FETCH_SIZE"), calib(write, "WRITE_SIZE")
    cf = CALIB_BYTES / (calib_f * 1024.0)
    cw = CALIB_BYTES / (calib_w * 1024.0)
    fam = {}
    for d, (name, c) in fetch.items():
        k = kernel_family(name)
        if k:
            fam.setdefault(k, {"dispatches": 0, "fetch_kib": 0.0, "write_kib": 0.0, "mfma_busy": 0.0, "gui_active": 0.0,
                               "valu_active": 0.0})
            fam[k]["dispatches"] += 1
            fam[k]["fetch_kib"] += c["FETCH_SIZE"]
    for d, (name, c) in write.items():
        k = kernel_family(name)
        if k:
            fam[k]["write_kib"] += c["WRITE_SIZE"]
    for d, (name, c) in mfma.items():
        k = kernel_family(name)
        if k:
            fam[k]["mfma_busy"] += c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
            fam[k]["gui_active"] += c.get("GRBM_GUI_ACTIVE", 0.0)
            fam[k]["valu_active"] += c.get("SQ_ACTIVE_INST_VALU", 0.0)
    # The LDS / wait pass is kept per kernel (the family mixes the products
    # with the streaming dequant and partial-sum passes).
    per_kernel = {}
    for d, (name, c) in lds.items():
        if kernel_family(name):
            kn = kernel_base_name(name)
            acc = per_kernel.setdefault(kn, {})
            for ctr in LDS_COUNTERS[:-1]:
                acc[ctr] = acc.get(ctr, 0.0) + c.get(ctr, 0.0)
    data = {"config": config, "kernel_source_sha256": kernel_source_sha256(),
            "calibration": {"bytes": CALIB_BYTES, "fetch_kib": calib_f, "write_kib": calib_w,
                            "fetch_scale": cf, "write_scale": cw},
            "families": {}}
    for k, v in fam.items():
        fb, wb = v["fetch_kib"] * 1024.0 * cf, v["write_kib"] * 1024.0 * cw
        e = {"dispatches_per_step": v["dispatches"], "fetch_bytes_per_step": fb, "write_bytes_per_step": wb,
             "hbm_bytes_per_step": fb + wb}
        if v["mfma_busy"] > 0:
            # SQ_VALU_MFMA_BUSY_CYCLES is summed over all SIMDs; GRBM_GUI_ACTIVE over the 8 XCDs.
            e["mfma_busy_fraction"] = v["mfma_busy"] / (1024.0 * v["gui_active"] / 8.0)
        if v["valu_active"] > 0:
            # rocprofv3's VALUBusy: sum of SQ_ACTIVE_INST_VALU / CUs / GRBM_GUI_ACTIVE (per XCD).
            e["valu_busy_fraction"] = v["valu_active"] / (256.0 * v["gui_active"] / 8.0)
        data["families"][k] = e
    if per_kernel:
        data["kernels_lds"] = {}
        for kn, v in sorted(per_kernel.items()):
            e = {}
            if v.get("SQ_LDS_IDX_ACTIVE", 0.0) > 0:
                e["lds_bank_conflict_fraction"] = v["SQ_LDS_BANK_CONFLICT"] / v["SQ_LDS_IDX_ACTIVE"]
            if v.get("SQ_WAVE_CYCLES", 0.0) > 0:
                e["wait_lds_issue_fraction"] = v["SQ_WAIT_INST_LDS"] / v["SQ_WAVE_CYCLES"]
                e["wait_memory_fraction"] = v["SQ_WAIT_ANY"] / v["SQ_WAVE_CYCLES"]
            data["kernels_lds"][kn] = e
    lines = [f"# HBM traffic, MFMA and VALU busy counters: {WORKLOAD_SLUG.get(config, config)}", "",
             "%s rocprofv3 counter passes over `python3 bench.py --config %d --pmc-pass` (one eager step of "
             "each kind the configuration has, decode and/or prefill, then a 1 GiB device-to-device copy used "
             "as the calibration):" % ("Four" if lds_dir else "Three", config), "",
             "```", "cd /tmp && export TMPDIR=/tmp && cd /root/repo",
             f"rocprofv3 --pmc FETCH_SIZE --output-format csv -d {fetch_dir} -o run -- python3 bench.py --config {config} --pmc-pass",
             f"rocprofv3 --pmc WRITE_SIZE --output-format csv -d {write_dir} -o run -- python3 bench.py --config {config} --pmc-pass",
             f"rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES SQ_ACTIVE_INST_VALU GRBM_GUI_ACTIVE --output-format csv -d {mfma_dir} -o run -- python3 bench.py --config {config} --pmc-pass",
             *([f"rocprofv3 --pmc {' '.join(LDS_COUNTERS)} --output-format csv -d {lds_dir} -o run -- python3 bench.py --config {config} --pmc-pass"]
               if lds_dir else []),
             f"python3 bench.py --config {config} --pmc-summary {fetch_dir} {write_dir} {mfma_dir}" + (f" {lds_dir}" if lds_dir else ""),
             "```", "",
             "Calibration copy: FETCH_SIZE %.0f KiB and WRITE_SIZE %.0f KiB for %d bytes each way, so counter bytes are "
             "scaled by %.4f (fetch) and %.4f (write)." % (data["calibration"]["fetch_kib"], data["calibration"]["write_kib"],
                                                        CALIB_BYTES, cf, cw), "",
             "| kernels | dispatches per step | HBM read (GB/step) | HBM write (GB/step) | MFMA busy | VALU busy |",
             "|---|---:|---:|---:|---:|---:|"]
    for k, e in data["families"].items():
        mb = "%.1f%%" % (100 * e["mfma_busy_fraction"]) if "mfma_busy_fraction" in e else "-"
        vb = "%.1f%%" % (100 * e["valu_busy_fraction"]) if "valu_busy_fraction" in e else "-"
        lines.append(f"| {k} | {e['dispatches_per_step']} | {e['fetch_bytes_per_step'] / 1e9:.3f} | "
                     f"{e['write_bytes_per_step'] / 1e9:.3f} | {mb} | {vb} |")
    lines += ["", "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES (summed over the 1024 SIMDs) / (1024 x GRBM_GUI_ACTIVE / 8), "
              "i.e. the fraction of the kernels' busy cycles in which a SIMD's matrix core is working. "
              "VALU busy = rocprofv3's derived VALUBusy, SQ_ACTIVE_INST_VALU (summed) / (256 CUs x GRBM_GUI_ACTIVE / 8)."]
    if lds:
        lines += ["", "| kernel | LDS bank conflicts (of LDS cycles) | waiting to issue an LDS instruction | waiting on memory (s_waitcnt) |",
                  "|---|---:|---:|---:|"]
        for k, e in data.get("kernels_lds", {}).items():
            if "wait_lds_issue_fraction" in e:
                lines.append(f"| {k} | {100 * e.get('lds_bank_conflict_fraction', 0.0):.1f}% | "
                             f"{100 * e['wait_lds_issue_fraction']:.1f}% | {100 * e['wait_memory_fraction']:.1f}% |")
        lines += ["", "Shares: SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE, and SQ_WAIT_INST_LDS and SQ_WAIT_ANY over "
                  "SQ_WAVE_CYCLES (all summed over the kernel's dispatches in the step, every template instance)."]
    lines += ["",
              "bench.py reads the block below while the kernel source, comments and blank lines aside, still has this SHA-256:", "",
              "```json", json.dumps(data, indent=1), "```", ""]
    return "\n".join(lines)


def stored_traffic(config):
    """The counter summary for this configuration, if taken on the current kernels."""
    path = traffic_file(config)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    try:
        block = text.split("```json", 1)[1].split("```", 1)[0]
        data = json.loads(block)
    except (IndexError, ValueError):
        return None
    if data.get("config") != config or data.get("kernel_source_sha256") != kernel_source_sha256():
        return None
    return data


def run_single(args, cfg, q4, torch):
    """Config 0: one GEMV launch (1B q_proj, 1024 x 1152, 819,200 stored bytes),
    launch-latency-bound.  Timed warm (the same weights every launch: they sit
    in L2) and cold (512 distinct copies, 419 MB, more than the 4 MB L2s and the
    256 MB memory-side cache together), each as a HIP graph of back-to-back
    launches; `value` is the cold rate.  The output of every copy is checked
    against the float64 oracle (full N)."""
    import numpy as np
    from workloads import gen_weights, gen_activations
    _, N, K = cfg["single"]
    codes, s, o = gen_weights(N, K, seed=args.seed, layer=0, proj=0, offset_mode=args.offset_mode)
    x_h = gen_activations(K, seed=args.seed, layer=0, proj=0)
    blob_h = q4.q4nx_pack(codes, s, o)
    stream = torch.cuda.Stream()
    torch.cuda.set_stream(stream)
    st = ctypes.c_void_p(stream.cuda_stream)
    copies = 512
    blobs = torch.from_numpy(blob_h).cuda().repeat(copies).view(copies, -1)
    x = torch.from_numpy(x_h.view("int16")).cuda()
    ys = torch.empty((copies, N), dtype=torch.float32, device="cuda")
    gemv = q4.lib.q4nx_gemv

    def launches(which):
        for i in which:
            assert gemv(blobs[i].data_ptr(), x.data_ptr(), ys[i].data_ptr(), q4.Q4NX_F32, N, K, st) == 0

    def graph_ms(which, reps):
        launches(which)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            launches(which)
        for _ in range(args.warmup):
            g.replay()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            g.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) / len(which))
        return sorted(ts)[len(ts) // 2], min(ts)

    cold_ms, cold_min = graph_ms(list(range(copies)), args.steps)
    warm_ms, warm_min = graph_ms([0] * copies, args.steps)
    wbytes = N * K * WEIGHT_BYTES
    cold_gbs, warm_gbs = wbytes / (cold_ms * 1e-3) / 1e9, wbytes / (warm_ms * 1e-3) / 1e9
    log(f"single GEMV {N}x{K}: cold {cold_ms * 1e3:.2f} us, warm {warm_ms * 1e3:.2f} us per launch")
    result = {
        "metric": "Q4NX dequant-GEMV weight GB/s (% HBM peak); dequant-GEMM TFLOP/s (% MFMA)",
        "value": round(cold_gbs, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(cold_ms, 6), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": cfg["name"], "N": N, "K": K, "M": [1], "offset_mode": args.offset_mode,
                   "seed": args.seed},
        "single": {"what": "one q4nx_gemv launch per step; per-launch time from a HIP graph of 512 launches",
                   "cold_us": round(cold_ms * 1e3, 3), "cold_us_min": round(cold_min * 1e3, 3),
                   "warm_us": round(warm_ms * 1e3, 3), "warm_us_min": round(warm_min * 1e3, 3),
                   "cold_GB_per_s": round(cold_gbs, 2), "warm_GB_per_s": round(warm_gbs, 2),
                   "weight_bytes": int(wbytes), "stored_bytes": int(blob_h.nbytes), "copies_cold": copies},
        "roofline": {"kernel": "gemv_kernel", "bound": "hbm", "achieved": round(cold_gbs, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(cold_gbs / HBM_PEAK_GBS, 4), "traffic": None,
                     "algorithmic_bytes": int(wbytes + 2 * K + 4 * N),
                     "note": "launch-latency-bound: 0.1 us of streaming at 8 TB/s against a few us per launch"},
    }
    if not args.no_cpu_baseline:
        import oracle
        torch.cuda.synchronize()
        y_gpu = ys.cpu().numpy()
        reps, t = 0, 0.0
        while t < 2.0:
            t0 = time.perf_counter()
            w = oracle.dequant_blob_f32(blob_h, N, K)
            y_ref = oracle.gemv_f64(w, x_h)
            t += time.perf_counter() - t0
            reps += 1
        bound = oracle.abs_bound(x_h, w)
        worst = 0.0
        ok = True
        for i in range(copies):
            good, wr = oracle.check_close(y_gpu[i], y_ref, bound)
            ok = ok and good
            worst = max(worst, wr)
        result["cpu_baseline"] = {
            "value": reps * wbytes / t / 1e9, "unit": "GB/s", "cores": int(blas_thread_count()), "kind": "oracle",
            "sample": f"{reps} runs of the oracle's float32 Eq. 3 dequant (single-threaded) + float64 mat-vec "
                      f"(BLAS threads) of this GEMV",
            "seconds": t,
            "parity_check": {"tolerance": "|y - y_ref| <= 2e-3 * sum_k |x_k w_k| + 1e-5 per output",
                             "outputs": f"all {N} outputs of every one of the {copies} launches",
                             "worst_err_over_tol": float(f"{worst:.3g}"), "ok": bool(ok)}}
    print(json.dumps(result), flush=True)


def main():
    args = parse()
    if args.pmc_summary:
        if len(args.pmc_summary) not in (3, 4):
            sys.exit("--pmc-summary takes FETCH_DIR WRITE_DIR MFMA_DIR [LDS_DIR]")
        print(pmc_summary(args.config, *args.pmc_summary))
        return
    if args.trace_summary:
        print(trace_summary(*args.trace_summary), end="")
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the library implements and measures the single-GPU path "
              "(how it would shard over several GPUs is described, not implemented).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2602_06063_amd as q4
    from workloads import MODELS, CONFIGS, gen_activations, gen_activations_device

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    cfg = CONFIGS[args.config]
    if "single" in cfg:
        return run_single(args, cfg, q4, torch)
    model = MODELS[cfg["model"]]
    L = model["layers"]
    Ms = cfg["M"]
    do_decode = 1 in Ms
    M_pre = max(m for m in Ms) if any(m > 1 for m in Ms) else 0
    do_prefill = M_pre > 0
    log(f"config {args.config}: {cfg['name']}, {L} layers, M={Ms}")

    weights, stacked = build_weights(model, cfg, args.seed, args.offset_mode, q4, torch)
    stream = torch.cuda.Stream()      # every launch, capture and event lives here
    torch.cuda.set_stream(stream)
    F32 = q4.Q4NX_F32

    # ---------------------------------------------------------------- decode
    dec = Step(q4, stream.cuda_stream)
    dec_bytes = 0.0
    dec_launches = 0
    if do_decode:
        xs, ys = {}, {}
        for l in range(L):
            for p, (_, N, K) in enumerate(model["proj"]):
                xs[(l, p)] = torch.from_numpy(gen_activations(K, seed=args.seed, layer=l, proj=p).view("int16")).cuda()
                ys[(l, p)] = torch.empty(N, dtype=torch.float32, device="cuda")
                dec_bytes += N * K * WEIGHT_BYTES
        if cfg.get("lm_head"):
            _, N, K = model["lm_head"]
            xs[(L, 7)] = torch.from_numpy(gen_activations(K, seed=args.seed, layer=L, proj=7).view("int16")).cuda()
            ys[(L, 7)] = torch.empty(N, dtype=torch.float32, device="cuda")
            dec_bytes += N * K * WEIGHT_BYTES

        def decode_calls(step, wts):
            for l in range(L):
                it = lambda p: (wts[(l, p)], xs[(l, p)], ys[(l, p)], model["proj"][p][1], model["proj"][p][2])
                step.gemv_batched([it(0), it(1), it(2)], F32)   # q, k, v
                step.gemv_batched([it(3)], F32)                 # o
                step.gemv_batched([it(4), it(5)], F32)          # gate, up
                step.gemv_batched([it(6)], F32)                 # down
            if cfg.get("lm_head"):
                _, N, K = model["lm_head"]
                step.gemv_batched([(wts[(L, 7)], xs[(L, 7)], ys[(L, 7)], N, K)], F32)

        decode_calls(dec, weights)
        dec_launches = len(dec.calls)

    # ---------------------------------------------------------------- prefill
    pre = Step(q4, stream.cuda_stream)
    two = Step(q4, stream.cuda_stream)   # two-phase: dequant to bf16 W, then the plain bf16 GEMM
    pre16 = Step(q4, stream.cuda_stream)  # the prefill step with bf16 outputs
    fus = Step(q4, stream.cuda_stream)    # the prefill step through q4nx_gemm alone
    mpre = Step(q4, stream.cuda_stream, mx=True)
    pre_flops = 0.0
    alg_pre = 0.0
    # One GEMM per group of projections that share an input: N = the group's
    # stacked outputs, X drawn per (layer, first projection of the group).
    shapes = [(sum(model["proj"][p][1] for p in g), model["proj"][g[0]][2]) for g in GROUPS]
    if do_prefill:
        Xs = {}
        Ys = [torch.empty((M_pre, N), dtype=torch.float32, device="cuda") for N, _ in shapes]
        Ys16 = [torch.empty((M_pre, N), dtype=torch.bfloat16, device="cuda") for N, _ in shapes] if args.bf16_out else None
        Wtmp = torch.empty(max(N * K for N, K in shapes), dtype=torch.bfloat16, device="cuda")
        # One workspace for every GEMM of the steps (they run one after another):
        # split-K partials, and bf16 W where a Q4NX product dequantizes first.
        work_bytes = max(q4.q4nx_gemm_workspace_size(f, M_pre, N, K) for N, K in shapes
                         for f in (q4.Q4NX_WEIGHTS_Q4NX, q4.Q4NX_WEIGHTS_MXFP4, q4.Q4NX_WEIGHTS_BF16))
        gemm_work = torch.empty(max(work_bytes // 4, 1), dtype=torch.float32, device="cuda")
        pre.work = two.work = mpre.work = pre16.work = gemm_work
        for l in range(L):
            for gi, (N, K) in enumerate(shapes):
                Xs[(l, gi)] = gen_activations_device((M_pre, K), seed=args.seed, layer=l, proj=GROUPS[gi][0])
                pre.gemm(M_pre, N, K, Xs[(l, gi)], stacked[(l, gi)], Ys[gi], F32)
                if args.bf16_out:
                    pre16.gemm(M_pre, N, K, Xs[(l, gi)], stacked[(l, gi)], Ys16[gi], q4.Q4NX_BF16)
                if args.fused:
                    fus.gemm_fused(M_pre, N, K, Xs[(l, gi)], stacked[(l, gi)], Ys[gi], F32)
                two.dequant_bf16(stacked[(l, gi)], N, K, Wtmp)
                two.gemm_bf16(M_pre, N, K, Xs[(l, gi)], Wtmp, Ys[gi], F32)
                pre_flops += 2.0 * M_pre * N * K
                alg_pre += 2 * M_pre * K + N * K * WEIGHT_BYTES + 4 * M_pre * N
    # MXFP4 variant: the same steps over MXFP4-variant weights (same
    # activations and outputs).
    mdec = Step(q4, stream.cuda_stream, mx=True)
    mweights = None
    if args.mx and not args.pmc_pass:
        mweights, mstacked = build_weights(model, cfg, args.seed, args.offset_mode, q4, torch, mx=True)
        if do_decode:
            decode_calls(mdec, mweights)
        if do_prefill:
            for l in range(L):
                for gi, (N, K) in enumerate(shapes):
                    mpre.gemm(M_pre, N, K, Xs[(l, gi)], mstacked[(l, gi)], Ys[gi], F32)
    torch.cuda.synchronize()
    log(f"inputs resident: {sum(t.numel() for t in weights.values()) / 1e9:.2f} GB of packed weights"
        + (f" + {sum(t.numel() for t in mweights.values()) / 1e9:.2f} GB MXFP4-variant" if mweights else ""))

    if args.pmc_pass:
        # Exactly one step of each kind, then the calibration copy as the last dispatch.
        dec.run()
        pre.run()
        torch.cuda.synchronize()
        src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log("pmc pass done")
        return

    # ---------------------------------------------------------------- timing
    for _ in range(args.warmup):
        pre.run()
    for _ in range(args.warmup):
        dec.run()
    torch.cuda.synchronize()
    log("warmup done")

    graphs = []

    def graph_of(step):
        """Capture a decode step once and replay it (no per-launch host cost).
        Every replay is checked bit for bit against the eager result (the
        kernels are deterministic), with eager work between replays; on a
        mismatch the eager launches are timed instead."""
        step.run()
        torch.cuda.synchronize()
        ref = [y.clone() for y in ys.values()]
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            step.run()
        graphs.append(g)
        ok = True
        for _ in range(3):
            for y in ys.values():
                y.fill_(float("nan"))
            g.replay()
            torch.cuda.synchronize()
            ok = ok and all(torch.equal(a.view(torch.int32), b.view(torch.int32)) for a, b in zip(ys.values(), ref))
            step.run()
            torch.cuda.synchronize()
        info = {"replays_checked": 3, "bitwise_equal_to_eager": bool(ok), "graph_usable": bool(ok)}
        fn = g.replay if ok else step.run
        if not ok:
            log("graph replay differs from eager: timing eager launches")
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        return fn, info

    def quick_ms(fn, n=3):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(n):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    # (Bound methods are compared through this flag: `dec.run is dec.run` is
    # False, every attribute access makes a new method object.)
    use_graph = False
    decode_fn = dec.run
    graph_info = None
    if do_decode and args.decode_graph:
        decode_fn, graph_info = graph_of(dec)
        use_graph = graph_info["graph_usable"]
        # Graph replay removes host launch cost but its node dispatch is not
        # always faster than back-to-back eager launches: time both briefly
        # and keep the faster for the timed steps (both are reported).
        if use_graph:
            g_ms, e_ms = quick_ms(decode_fn), quick_ms(dec.run)
            graph_info.update(calibration_ms={"graph": round(g_ms, 4), "eager": round(e_ms, 4)})
            if e_ms < g_ms:
                use_graph = False
                decode_fn = dec.run

    def timed(run_dec, run_pre, steps):
        """K decode steps back to back, then K prefill chunks back to back,
        all inside one synchronized region, with an event pair per step of
        each phase.  Each phase is timed in its steady state, as a serving loop
        runs it: a decode step put right after a 170 ms prefill chunk measured a
        median of 3.62-3.84 ms, against 3.45-3.48 ms after another decode step
        (same kernels)."""
        evd = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        evp = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        for a, b in evd:
            a.record(stream)
            run_dec()
            b.record(stream)
        for a, b in evp:
            a.record(stream)
            run_pre()
            b.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        return [a.elapsed_time(b) for a, b in evd], [a.elapsed_time(b) for a, b in evp], wall

    dec_ms, pre_ms, wall = timed(decode_fn, pre.run, args.steps)
    step_ms = [d + p for d, p in zip(dec_ms, pre_ms)]
    mean = lambda v: sum(v) / len(v)
    med = lambda v: sorted(v)[len(v) // 2]
    log(f"timed {args.steps} steps in {wall:.2f}s wall; decode {mean(dec_ms):.3f} ms, prefill {mean(pre_ms):.3f} ms")
    other_dec_ms = None   # the launch mode not used in the timed steps
    if do_decode and graph_info and "calibration_ms" in graph_info:
        other = dec.run if use_graph else graphs[0].replay
        other_dec_ms, _, _ = timed(other, lambda: None, args.steps)
    two_ms = None
    gemm_only_ms = None
    if do_prefill and args.two_phase:
        for _ in range(args.warmup):
            two.run()
        _, two_ms, _ = timed(lambda: None, two.run, args.steps)
        # The bf16 GEMM launches alone: an event pair around every
        # q4nx_gemm_bf16 call of the two-phase step (the dequantization
        # passes run between them, outside the pairs).
        per_step = []
        for _ in range(args.steps):
            pairs = []
            for fn, a in two.calls:
                if fn is q4.lib.q4nx_gemm_ex:
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    e0.record(stream)
                    fn(*a)
                    e1.record(stream)
                    pairs.append((e0, e1))
                else:
                    fn(*a)
            torch.cuda.synchronize()
            per_step.append(sum(x.elapsed_time(y) for x, y in pairs))
        gemm_only_ms = sorted(per_step)[len(per_step) // 2]
    fus_ms = None
    if do_prefill and args.fused:
        for _ in range(args.warmup):
            fus.run()
        _, fus_ms, _ = timed(lambda: None, fus.run, args.steps)
    b16_ms, b16_equal = None, None
    if do_prefill and args.bf16_out:
        for _ in range(args.warmup):
            pre16.run()
        _, b16_ms, _ = timed(lambda: None, pre16.run, args.steps)
        # The same accumulation rounded once: the bf16 outputs of the last
        # layer's products must equal the float32 outputs rounded to bf16.
        for fn, a in pre.calls[-len(GROUPS):] + pre16.calls[-len(GROUPS):]:
            fn(*a)
        torch.cuda.synchronize()
        b16_equal = all(torch.equal(y16.view(torch.int16), y32.to(torch.bfloat16).view(torch.int16))
                        for y16, y32 in zip(Ys16, Ys))

    # Bytes the launches must move at least once (operands in, results out).
    alg_dec = sum(N * K * WEIGHT_BYTES + 2 * K + 4 * N for _, N, K in model["proj"]) * L if do_decode else 0
    if do_decode and cfg.get("lm_head"):
        _, N, K = model["lm_head"]
        alg_dec += N * K * WEIGHT_BYTES + 2 * K + 4 * N
    mx = None
    if mweights is not None:
        mx = {"what": "the same decode and prefill steps over MXFP4-variant weights (FP4 E2M1 codes, one E8M0 "
                      "scale per 32 weights; q4nx_mx_gemv_batched / q4nx_mx_gemm)"}
        if do_decode:
            mdec_fn, minfo = graph_of(mdec) if args.decode_graph else (mdec.run, None)
            mdec_ms, _, _ = timed(mdec_fn, lambda: None, args.steps)
            if minfo and minfo["graph_usable"]:   # keep the faster launch mode, as for the Q4NX step
                eager_ms, _, _ = timed(mdec.run, lambda: None, args.steps)
                minfo.update(graph_ms=round(med(mdec_ms), 4), eager_ms=round(med(eager_ms), 4))
                if med(eager_ms) < med(mdec_ms):
                    mdec_ms = eager_ms
            mbytes = dec_bytes / WEIGHT_BYTES * MX_WEIGHT_BYTES
            t = med(mdec_ms)
            mx["decode"] = {"ms_median": round(t, 4), "ms_min": round(min(mdec_ms), 4), "weight_GB": round(mbytes / 1e9, 4),
                            "GB_per_s": round(mbytes / (t * 1e-3) / 1e9, 2),
                            "frac_hbm": round(mbytes / (t * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                            "launches": len(mdec.calls), "graph_check": minfo,
                            "bytes": "0.53125 B per weight (FP4 code + E8M0 scale per 32)"}
        if do_prefill:
            for _ in range(args.warmup):
                mpre.run()
            _, mpre_ms, _ = timed(lambda: None, mpre.run, args.steps)
            t = med(mpre_ms)
            mx["prefill"] = {"ms_median": round(t, 4), "ms_min": round(min(mpre_ms), 4), "M": M_pre,
                             "TFLOP_per_s": round(pre_flops / (t * 1e-3) / 1e12, 2),
                             "frac_mfma": round(pre_flops / (t * 1e-3) / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4),
                             "launches": len(mpre.calls)}


    quant = None
    if args.quantize:
        # The offline conversion on the GPU: one float32 matrix of the largest
        # projection shape (N(0, 0.02) values), timed like the steps.
        _, Nq, Kq = max(model["proj"] + ([model["lm_head"]] if cfg.get("lm_head") else []), key=lambda p: p[1] * p[2])
        gq = torch.Generator(device="cuda")
        gq.manual_seed(args.seed)
        Wq = torch.randn((Nq, Kq), generator=gq, device="cuda", dtype=torch.float32) * 0.02
        Bq = torch.empty(q4.q4nx_packed_size(Nq, Kq), dtype=torch.uint8, device="cuda")
        sq = Step(q4, stream.cuda_stream)
        sq.calls.append((q4.lib.q4nx_quantize, (Wq.data_ptr(), Nq, Kq, Bq.data_ptr(), sq.s)))
        for _ in range(args.warmup):
            sq.run()
        _, q_ms, _ = timed(lambda: None, sq.run, args.steps)
        tq = med(q_ms)
        qbytes = Nq * Kq * (4 + WEIGHT_BYTES)
        quant = {"shape": [Nq, Kq], "ms_median": round(tq, 4), "ms_min": round(min(q_ms), 4),
                 "Gweights_per_s": round(Nq * Kq / (tq * 1e-3) / 1e9, 2),
                 "GB_per_s": round(qbytes / (tq * 1e-3) / 1e9, 2),
                 "frac_hbm": round(qbytes / (tq * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                 "bytes": "4 B read + 0.625 B written per weight"}
        # The MXFP4 variant's quantizer on the same matrix.
        Bm = torch.empty(q4.q4nx_mx_packed_size(Nq, Kq), dtype=torch.uint8, device="cuda")
        sm = Step(q4, stream.cuda_stream)
        sm.calls.append((q4.lib.q4nx_mx_quantize, (Wq.data_ptr(), Nq, Kq, Bm.data_ptr(), sm.s)))
        for _ in range(args.warmup):
            sm.run()
        _, m_ms, _ = timed(lambda: None, sm.run, args.steps)
        tm = med(m_ms)
        mbytes = Nq * Kq * (4 + MX_WEIGHT_BYTES)
        quant["mxfp4"] = {"ms_median": round(tm, 4), "Gweights_per_s": round(Nq * Kq / (tm * 1e-3) / 1e9, 2),
                          "GB_per_s": round(mbytes / (tm * 1e-3) / 1e9, 2),
                          "frac_hbm": round(mbytes / (tm * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                          "bytes": "4 B read + 0.53125 B written per weight"}
        del Wq, Bq, Bm

    fkv = None
    if args.flowkv and do_decode:
        from workloads import ATTENTION, SWA_WINDOW, is_global_layer
        A = ATTENTION[cfg["model"]]
        H, G, d = A["H"], A["G"], A["d"]
        gk = torch.Generator(device="cuda")
        gk.manual_seed(args.seed + 7)
        sk = Step(q4, stream.cuda_stream)
        kv_bytes, bufs = 0, []
        T = args.context
        wbytes = q4.q4nx_flowkv_workspace_size(H, d, T)
        work = torch.empty(wbytes // 4, dtype=torch.float32, device="cuda")
        for l in range(L):
            glob = is_global_layer(l)
            Lc = T if glob else min(T, SWA_WINDOW)   # a sliding-window layer keeps the last 1024 positions
            t = Lc - 1
            win = 0 if glob else SWA_WINDOW
            Kc = (torch.randn((G, Lc, d), generator=gk, device="cuda")).to(torch.bfloat16)
            Vc = (torch.randn((G, Lc, d), generator=gk, device="cuda")).to(torch.bfloat16)
            qv = (torch.randn((H, d), generator=gk, device="cuda")).to(torch.bfloat16)
            ov = torch.empty((H, d), dtype=torch.float32, device="cuda")
            bufs += [Kc, Vc, qv, ov]
            sk.calls.append((q4.lib.q4nx_flowkv_decode,
                             (qv.data_ptr(), Kc.data_ptr(), Vc.data_ptr(), H, G, d, Lc, t, win,
                              ctypes.c_float(1.0 / d ** 0.5), ov.data_ptr(), q4.Q4NX_F32, work.data_ptr(),
                              wbytes, sk.s)))
            kv_bytes += 2 * G * min(Lc, T) * d * 2
        for _ in range(args.warmup):
            sk.run()
        _, k_ms, _ = timed(lambda: None, sk.run, args.steps)
        tk = med(k_ms)
        fkv = {"context": T, "layers": L, "global_layers": sum(is_global_layer(l) for l in range(L)),
               "window": SWA_WINDOW, "heads": H, "kv_groups": G, "head_dim": d,
               "ms_median": round(tk, 4), "ms_min": round(min(k_ms), 4), "kv_GB": round(kv_bytes / 1e9, 4),
               "GB_per_s": round(kv_bytes / (tk * 1e-3) / 1e9, 2),
               "frac_hbm": round(kv_bytes / (tk * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
               "launches": 2 * L, "bytes": "K and V rows of the attended positions, bf16"}
        del bufs, work

    dec_gbs = dec_bytes / (med(dec_ms) * 1e-3) / 1e9 if do_decode else None
    pre_tflops = pre_flops / (med(pre_ms) * 1e-3) / 1e12 if do_prefill else None

    result = {
        "metric": "Q4NX dequant-GEMV weight GB/s (% HBM peak); dequant-GEMM TFLOP/s (% MFMA)",
        "value": round(dec_gbs, 2) if do_decode else round(pre_tflops, 2),
        "unit": "GB/s" if do_decode else "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(med(step_ms), 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": cfg["name"],
            "layers": L,
            "projections": [list(p) for p in model["proj"]] + ([list(model["lm_head"])] if cfg.get("lm_head") else []),
            "M": Ms,
            "offset_mode": args.offset_mode,
            "seed": args.seed,
        },
    }
    if do_decode:
        result["decode"] = {"ms_median": round(med(dec_ms), 4), "ms_min": round(min(dec_ms), 4),
                            "ms_mean": round(mean(dec_ms), 4),
                            "weight_GB": round(dec_bytes / 1e9, 4), "GB_per_s": round(dec_gbs, 2),
                            "frac_hbm": round(dec_gbs / HBM_PEAK_GBS, 4), "launches": dec_launches,
                            "launch": "hip graph replay" if use_graph else "eager",
                            "graph_check": graph_info,
                            "dtype": "exact bf16 codes times bf16 x (v_dot2), float32 accumulation"}
        if other_dec_ms:
            key = "eager" if use_graph else "graph"
            result["decode"][f"{key}_ms_median"] = round(med(other_dec_ms), 4)
            result["decode"][f"{key}_GB_per_s"] = round(dec_bytes / (med(other_dec_ms) * 1e-3) / 1e9, 2)
    if do_prefill:
        result["prefill"] = {"ms_median": round(med(pre_ms), 4), "ms_min": round(min(pre_ms), 4),
                             "ms_mean": round(mean(pre_ms), 4), "M": M_pre,
                             "TFLOP": round(pre_flops / 1e12, 4), "TFLOP_per_s": round(pre_tflops, 2),
                             "frac_mfma": round(pre_tflops / BF16_MFMA_PEAK_TFLOPS, 4),
                             "launches": len(pre.calls), "dtype": "bf16 MFMA, f32 accumulate",
                             "gemms": "per layer: q/k/v stacked, o, gate/up stacked, down ("
                                      + ", ".join(f"{N}x{K}" for N, K in shapes) + ")"}
        if two_ms:
            t = med(two_ms)
            result["prefill"]["two_phase"] = {
                "ms_median": round(t, 4), "ms_min": round(min(two_ms), 4),
                "TFLOP_per_s": round(pre_flops / (t * 1e-3) / 1e12, 2),
                "launches": len(two.calls),
                "what": "per GEMM: q4nx_dequant to a bf16 W buffer, then q4nx_gemm_bf16 (same bits as q4nx_gemm)"}
        if fus_ms:
            t = sorted(fus_ms)[len(fus_ms) // 2]
            result["prefill"]["fused_only"] = {
                "ms_median": round(t, 4), "ms_min": round(min(fus_ms), 4),
                "TFLOP_per_s": round(pre_flops / (t * 1e-3) / 1e12, 2),
                "what": "every product through q4nx_gemm: the fused dequant-GEMM (Eq. 3 in the tile loads), no "
                        "workspace, so no split K and no dequantize-once"}
        if b16_ms:
            t = sorted(b16_ms)[len(b16_ms) // 2]
            result["prefill"]["bf16_outputs"] = {
                "ms_median": round(t, 4), "ms_min": round(min(b16_ms), 4),
                "TFLOP_per_s": round(pre_flops / (t * 1e-3) / 1e12, 2),
                "frac_mfma": round(pre_flops / (t * 1e-3) / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4),
                "equal_to_rounded_f32_outputs": bool(b16_equal),
                "what": "the same step with bf16 outputs (the paper keeps every activation in bf16); each output "
                        "is the float32 accumulation rounded once to bf16 by the kernels"}
        if do_decode:
            result["value_gemm"] = round(pre_tflops, 2)
    # Dominant kernel by time: the GEMM when the step has a prefill chunk.
    if do_prefill:
        result["roofline"] = {"kernel": "the prefill step's q4nx_gemm_ex launches (" + ", ".join(PREFILL_KERNELS) +
                                        ")", "bound": "mfma",
                              "achieved": round(pre_tflops, 2), "peak": BF16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                              "frac": round(pre_tflops / BF16_MFMA_PEAK_TFLOPS, 4), "traffic": None,
                              "algorithmic_bytes": round(alg_pre)}
        if gemm_only_ms:
            t = gemm_only_ms
            result["roofline"]["dominant_kernel"] = {
                "what": "the same products' bf16 MFMA launches alone (gemm256_kernel, gemm256x128_kernel, "
                        "gemm_kernel and the split-K sum, the dequantization pass excluded): HIP events around every q4nx_gemm_bf16 call of "
                        "the two-phase step, summed per step, median over the steps",
                "ms_median": round(t, 4), "achieved": round(pre_flops / (t * 1e-3) / 1e12, 2),
                "frac": round(pre_flops / (t * 1e-3) / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4)}
    if do_decode:
        r = {"kernel": "gemv_kernel", "bound": "hbm", "achieved": round(dec_gbs, 2), "peak": HBM_PEAK_GBS,
             "unit": "GB/s", "frac": round(dec_gbs / HBM_PEAK_GBS, 4), "traffic": None,
             "algorithmic_bytes": round(alg_dec)}
        result["roofline" if not do_prefill else "roofline_gemv"] = r

    if mx:
        result["mxfp4"] = mx
    if do_decode:
        # Read bandwidth a plain streaming kernel reaches on this device (the
        # library's measurement aid, the GEMV's load pattern over 4 GiB).
        src = torch.empty(1 << 32, dtype=torch.uint8, device="cuda")
        sink = torch.empty(8192, dtype=torch.float32, device="cuda")
        sr = Step(q4, stream.cuda_stream)
        sr.calls.append((q4.lib.q4nx_stream_read, (src.data_ptr(), src.numel(), sink.data_ptr(), sr.s)))
        for _ in range(args.warmup):
            sr.run()
        _, sr_ms, _ = timed(lambda: None, sr.run, args.steps)
        t = sorted(sr_ms)[len(sr_ms) // 2]
        rkey = "roofline_gemv" if do_prefill else "roofline"
        result[rkey]["stream_read_GB_per_s"] = round(src.numel() / (t * 1e-3) / 1e9, 1)
        del src
        # The same weight bytes read by the plain streaming kernel in the
        # decode step's launch structure: one dependent launch per GEMV launch,
        # over the very blobs that launch reads.  Each launch pays its ramp and
        # drain, so this is the ceiling for a step of that many launches.
        blobs = [stacked[(l, gi)] for l in range(L) for gi in range(len(GROUPS))]
        if cfg.get("lm_head"):
            blobs.append(weights[(L, 7)])
        floor = launch_floor(q4, torch, stream, blobs, args.steps, args.warmup)
        floor["decode_ms_median_over_floor"] = round(med(dec_ms) / floor["ms_median"], 4)
        result[rkey]["launch_floor"] = floor
        del sink
    if quant:
        result["quantize"] = quant
    if fkv:
        result["flowkv_decode_attention"] = fkv
    stored = stored_traffic(args.config)
    for key, fam in (("roofline", "gemm" if do_prefill else "gemv"), ("roofline_gemv", "gemv")):
        if key in result and stored and fam in stored["families"]:
            e = stored["families"][fam]
            result[key]["traffic"] = round(e["hbm_bytes_per_step"])
            result[key]["traffic_note"] = ("HBM bytes per step (read + write) of these launches, from rocprofv3 "
                                           "FETCH_SIZE/WRITE_SIZE scaled by a copy-kernel calibration: "
                                           + os.path.relpath(traffic_file(args.config), ROOT))
            if "mfma_busy_fraction" in e:
                result[key]["mfma_busy_counter"] = round(e["mfma_busy_fraction"], 4)

    parity_ok = True
    if not args.no_cpu_baseline:
        # Outputs of the timed GPU steps for the oracle to check, each launch
        # run once more because later steps reuse the output buffers: every
        # decode output of the first and last layers, every element of the
        # first layer's o product, and sampled rows of the last layer's
        # prefill products.
        import numpy as np
        gpu = {}
        if do_decode:
            for l in (0, L - 1):
                for fn, a in dec.calls[len(GROUPS) * l:len(GROUPS) * (l + 1)]:
                    fn(*a)
            torch.cuda.synchronize()
            gpu["decode"] = {(l, p): ys[(l, p)].cpu().numpy() for l in (0, L - 1) for p in range(len(model["proj"]))}
        if do_prefill:
            fn, a = pre.calls[1]                  # layer 0, the o product (group 1)
            fn(*a)
            torch.cuda.synchronize()
            gpu["prefill_full"] = (0, 1, Xs[(0, 1)].view(torch.int16).cpu().numpy().view("uint16"),
                                   Ys[1].cpu().numpy())
            for fn, a in pre.calls[-len(GROUPS):]:
                fn(*a)
            torch.cuda.synchronize()
            rng = np.random.default_rng(args.seed)
            rows = np.unique(np.concatenate([[0, 1, M_pre // 2, M_pre - 1], rng.integers(0, M_pre, 252)]))
            idx = torch.tensor(rows, device="cuda")
            gpu["prefill_layer"], gpu["prefill_rows"] = L - 1, len(rows)
            gpu["prefill"] = {gi: (Xs[(L - 1, gi)].index_select(0, idx).view(torch.int16).cpu().numpy().view("uint16"),
                                   Ys[gi].index_select(0, idx).cpu().numpy()) for gi in range(len(GROUPS))}
        log("timing the CPU oracle sample")
        result["cpu_baseline"] = cpu_baseline(model, cfg, args.seed, args.offset_mode, args.cpu_layers,
                                              do_decode, do_prefill, M_pre)
        result["cpu_baseline"]["parity_check"] = parity_check(model, args.seed, args.offset_mode, gpu)
        parity_ok = result["cpu_baseline"]["parity_check"]["ok"]
    if args.config == 4 and args.with_4b:
        del weights, stacked
        if mweights is not None:
            del mweights, mstacked
        if do_prefill:
            del Xs, Ys, gemm_work
        torch.cuda.empty_cache()
        result["gemma3_4b"] = run_4b(args, q4, torch, stream)
        if "parity_check" in result["gemma3_4b"]:
            parity_ok = parity_ok and result["gemma3_4b"]["parity_check"]["ok"]
    result["parity_ok"] = bool(parity_ok)
    print(json.dumps(result), flush=True)
    if not parity_ok:
        log("parity check FAILED: the numbers above are not valid")
        sys.exit(1)


if __name__ == "__main__":
    main()
