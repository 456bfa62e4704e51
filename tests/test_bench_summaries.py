"""The benchmark's profile tooling on synthetic rocprofv3 output (CPU).

trace_summary turns a --kernel-trace --stats run into the per-step kernel time
of the prefill products; pmc_summary turns three counter passes into HBM bytes
per step (scaled by the calibration copy), MFMA busy and VALU busy.  These
figures end up in the committed profiles and in the benchmark's `traffic`
field, so their arithmetic is checked here on hand-made inputs whose results
are worked out below.
"""
import csv
import json
import os
import re

import pytest

import bench

STATS_FIELDS = ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs", "StdDev"]
PMC_FIELDS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
              "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
              "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _write_csv(path, fields, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=fields)
        w.writeheader()
        for r in rows:
            w.writerow({k: r.get(k, 0) for k in fields})


def _bench_json(path, **extra):
    r = {"warmup": 2, "steps": 5,
         "prefill": {"TFLOP": 209.7, "ms_median": 180.0, "TFLOP_per_s": 1165.0, "frac_mfma": 0.463},
         "decode": {"launch": "eager", "launches": 248, "ms_median": 3.6, "weight_GB": 16.0, "GB_per_s": 4444.0, "frac_hbm": 0.555}}
    for k, v in extra.items():
        r["prefill"][k] = v
    with open(path, "w") as f:
        f.write(json.dumps(r) + "\n")


def test_trace_summary_per_step_prefill_time(tmp_path):
    stats = tmp_path / "trace" / "run_kernel_stats.csv"
    # 7 runs (2 warm-up + 5 timed): gemm 700 ms + split sums 7 ms + dequant 63 ms = 770 ms -> 110 ms per step
    _write_csv(str(stats), STATS_FIELDS, [
        {"Name": "void q4nx::gemm256_kernel<false, 0>(unsigned short const*)", "Calls": 70, "TotalDurationNs": 700e6},
        {"Name": "q4nx::splitk_sum_kernel(float const*)", "Calls": 7, "TotalDurationNs": 7e6},
        {"Name": "void q4nx::dequant_kernel<1>(unsigned char const*)", "Calls": 28, "TotalDurationNs": 63e6},
        {"Name": "void q4nx::gemv_kernel<4, 1, 1>(q4nx::GemvArgs)", "Calls": 1736, "TotalDurationNs": 24.304e6},
        {"Name": "void q4nx::gemv_kernel<4, 1, 2>(q4nx::GemvArgs)", "Calls": 100, "TotalDurationNs": 5e6},
        {"Name": "void q4nx::gemv_stream_kernel<4, 1, 1>(q4nx::GemvArgs)", "Calls": 264, "TotalDurationNs": 3.696e6},
    ])
    js = tmp_path / "b.json"
    _bench_json(str(js))
    md = bench.trace_summary(str(tmp_path / "trace"), str(js))
    assert "770.0 ms over the 7 runs" in md and "110.00 ms per step" in md
    assert "= 1906 TFLOP/s" in md                        # 209.7 TFLOP / 110 ms
    assert "2000 launches, average 14.00 us" in md       # the Q4NX GEMVs (both kernels), not the MXFP4 one
    assert "= 3.472 ms of kernel time per step" in md    # 14 us x 248 launches
    _bench_json(str(js), bf16_outputs={"ms_median": 1.0})
    with pytest.raises(SystemExit):
        bench.trace_summary(str(tmp_path / "trace"), str(js))


def _pmc_pass(folder, counter_rows):
    rows = []
    for d, (name, counters) in enumerate(counter_rows, start=1):
        for cname, values in counters.items():
            for v in values:   # one row per XCD / shader engine instance
                rows.append({"Correlation_Id": d, "Dispatch_Id": d, "Kernel_Name": name,
                             "Counter_Name": cname, "Counter_Value": v})
    _write_csv(os.path.join(folder, "run_counter_collection.csv"), PMC_FIELDS, rows)


def test_pmc_summary_scaling_and_busy_fractions(tmp_path, monkeypatch):
    gemv, gemm = "void q4nx::gemv_kernel<4, 1, 1>(q4nx::GemvArgs)", "void q4nx::gemm256_kernel<false, 0>(x)"
    copy = "__amd_rocclr_copyBuffer"
    gvs = "void q4nx::gemv_stream_kernel<2, 3, 1>(q4nx::GemvArgs)"   # counted with the GEMV launches
    f, w, m = (str(tmp_path / n) for n in ("fetch", "write", "mfma"))
    # Calibration copy of 1 GiB each way: FETCH_SIZE reads half (512 MiB in KiB), WRITE_SIZE all of it.
    _pmc_pass(f, [(gemv, {"FETCH_SIZE": [1000.0, 500.0]}), (gvs, {"FETCH_SIZE": [500.0]}), (gemm, {"FETCH_SIZE": [3000.0]}),
                  (copy, {"FETCH_SIZE": [262144.0, 262144.0]})])
    _pmc_pass(w, [(gemv, {"WRITE_SIZE": [3.0]}), (gvs, {"WRITE_SIZE": [1.0]}), (gemm, {"WRITE_SIZE": [500.0]}),
                  (copy, {"WRITE_SIZE": [1048576.0]})])
    # 8 XCDs each report GRBM_GUI_ACTIVE = 1000 cycles -> 8000 summed
    _pmc_pass(m, [(gemv, {"GRBM_GUI_ACTIVE": [600.0] * 8, "SQ_ACTIVE_INST_VALU": [15360.0]}),
                  (gvs, {"GRBM_GUI_ACTIVE": [400.0] * 8, "SQ_ACTIVE_INST_VALU": [10240.0]}),
                  (gemm, {"GRBM_GUI_ACTIVE": [1000.0] * 8, "SQ_VALU_MFMA_BUSY_CYCLES": [512000.0],
                          "SQ_ACTIVE_INST_VALU": [51200.0]}),
                  (copy, {"GRBM_GUI_ACTIVE": [10.0] * 8})])
    lds = str(tmp_path / "lds")
    # gemm: 250 of 1000 LDS cycles in conflicts; 100 and 50 of 1000 wave cycles waiting on LDS issue / memory
    _pmc_pass(lds, [(gemv, {"SQ_WAVE_CYCLES": [500.0], "SQ_WAIT_INST_LDS": [0.0], "SQ_WAIT_ANY": [200.0]}),
                    (gvs, {"SQ_WAVE_CYCLES": [100.0], "SQ_WAIT_INST_LDS": [0.0], "SQ_WAIT_ANY": [10.0]}),
                    (gemm, {"SQ_LDS_BANK_CONFLICT": [125.0, 125.0], "SQ_LDS_IDX_ACTIVE": [500.0, 500.0],
                            "SQ_WAVE_CYCLES": [1000.0], "SQ_WAIT_INST_LDS": [100.0], "SQ_WAIT_ANY": [50.0]})])
    md = bench.pmc_summary(4, f, w, m, lds)
    data = json.loads(re.search(r"```json\n(.*?)\n```", md, re.S).group(1))
    kl = data["kernels_lds"]
    assert kl["gemm256_kernel"]["lds_bank_conflict_fraction"] == pytest.approx(0.25)
    assert kl["gemm256_kernel"]["wait_lds_issue_fraction"] == pytest.approx(0.1)
    assert kl["gemm256_kernel"]["wait_memory_fraction"] == pytest.approx(0.05)
    assert kl["gemv_kernel"]["wait_memory_fraction"] == pytest.approx(0.4)
    assert kl["gemv_stream_kernel"]["wait_memory_fraction"] == pytest.approx(0.1)
    assert data["families"]["gemv"]["dispatches_per_step"] == 2
    assert "| gemm256_kernel | 25.0% | 10.0% | 5.0% |" in md and md.startswith("# HBM") and "Four rocprofv3" in md
    assert "Three rocprofv3" in bench.pmc_summary(4, f, w, m)
    assert data["calibration"]["fetch_scale"] == pytest.approx(2.0)
    assert data["calibration"]["write_scale"] == pytest.approx(1.0)
    gv, gm = data["families"]["gemv"], data["families"]["gemm"]
    assert gv["fetch_bytes_per_step"] == pytest.approx(2000.0 * 1024 * 2.0)
    assert gv["write_bytes_per_step"] == pytest.approx(4.0 * 1024)
    assert gm["hbm_bytes_per_step"] == pytest.approx(3000.0 * 1024 * 2.0 + 500.0 * 1024)
    assert gm["mfma_busy_fraction"] == pytest.approx(512000.0 / (1024 * 8000.0 / 8))   # 0.5
    assert gm["valu_busy_fraction"] == pytest.approx(51200.0 / (256 * 8000.0 / 8))     # 0.2
    assert gv["valu_busy_fraction"] == pytest.approx(0.1)
    assert "mfma_busy_fraction" not in gv
    assert data["kernel_source_sha256"] == bench.kernel_source_sha256()
    # The stored block is read back only while the kernel code is unchanged.
    monkeypatch.setattr(bench, "traffic_file", lambda config: str(tmp_path / "t.md"))
    (tmp_path / "t.md").write_text(md)
    assert bench.stored_traffic(4)["families"]["gemm"]["dispatches_per_step"] == 1
    (tmp_path / "t.md").write_text(md.replace(data["kernel_source_sha256"], "0" * 64))
    assert bench.stored_traffic(4) is None


def test_kernel_hash_ignores_comments_only():
    src = "int a; // one\n/* two\n three */\nint b;\n\n   \n"
    assert bench.kernel_source_sha256(src) == bench.kernel_source_sha256("int a;\nint b;\n")
    assert bench.kernel_source_sha256(src) != bench.kernel_source_sha256("int a;\nint c;\n")


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU: --gpus N > 1 (or a WORLD_SIZE above 1) exits
    with status 2 and says why, before touching any device."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    for extra_env, args in (({}, ["--gpus", "2"]), ({"WORLD_SIZE": "4"}, [])):
        env = dict(os.environ, **extra_env)
        r = subprocess.run([sys.executable, os.path.join(root, "bench.py")] + args, cwd=root, env=env,
                           capture_output=True, text=True, timeout=120)
        assert r.returncode == 2, (r.returncode, r.stderr[-2000:])
        assert "one GPU only" in r.stderr
        assert r.stdout == ""
