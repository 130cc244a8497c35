"""bench.py's host logic without a GPU: the contract's refusal of more than
one GPU, and the mapping of rocprofv3's demangled kernel names onto the names
the library's own launch timer records."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_kernel_key_maps_profiler_names():
    k = bench.kernel_key
    assert k("void mpq::(anonymous namespace)::fit_hist_kernel<512, 9, true, true, false>"
             "(mpq::HistBatch)") == "fit_hist_kernel<512,9,lattice>"
    assert k("fit_hist_kernel<64, 2, true, false, false>(mpq::HistBatch)") == "fit_hist_kernel<64,2,linear>"
    assert k("fit_hist_kernel<256, 4, false, false, false>(x)") == "fit_hist_kernel<256,4,grid>"
    assert k("fit_hist_kernel<1024, 32, true, true, true>(x)") == "fit_hist_kernel<1024,32,lattice,rebuilt>"
    assert k("void mpq::(anonymous namespace)::gemm_err_kernel<true>(mpq::ErrGroup)") == "gemm_err_kernel"
    assert bench.stage_of("form_d_kernel") == "output_error"
    assert bench.stage_of("fit_hist_kernel<64,1,linear>") == "fit"
    assert k("void mpq::(anonymous namespace)::fit_small_kernel<9>(mpq::HistBatch, int)") == "fit_small_kernel<9>"
    assert bench.stage_of("fit_small_kernel<16>") == "fit"
    assert bench.stage_of("zero_i32_kernel") is None
    assert k("void mpq::(anonymous namespace)::int_forward_kernel<0>(mpq::IntGroup)") == "int_forward_kernel<16>"
    assert k("int_forward_kernel<2>(mpq::IntGroup)") == "int_forward_kernel<1>"
    assert k("void mpq::(anonymous namespace)::int_forward_kernel<1, 8>(mpq::IntGroup)") == "int_forward_kernel<4>"
    assert bench.stage_of("int_forward_kernel<16>") == "deploy"


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2 and "one GPU" in p.stderr


def _pmc_csv(path, rows):
    import csv
    cols = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id",
            "Grid_Size", "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size",
            "Scratch_Size", "VGPR_Count", "Accum_VGPR_Count", "SGPR_Count", "Counter_Name",
            "Counter_Value", "Start_Timestamp", "End_Timestamp"]
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "p_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=cols)
        w.writeheader()
        for did, name, grid, c, v, t0, t1 in rows:
            w.writerow({"Correlation_Id": did, "Dispatch_Id": did, "Agent_Id": "Agent 1", "Queue_Id": 1,
                        "Process_Id": 1, "Thread_Id": 1, "Grid_Size": grid, "Kernel_Id": 1,
                        "Kernel_Name": name, "Workgroup_Size": 256, "LDS_Block_Size": 0,
                        "Scratch_Size": 0, "VGPR_Count": 8, "Accum_VGPR_Count": 0, "SGPR_Count": 16,
                        "Counter_Name": c, "Counter_Value": v, "Start_Timestamp": t0,
                        "End_Timestamp": t1})


def test_counter_summary_arithmetic(tmp_path, capsys):
    """The counter summary scales FETCH_SIZE / WRITE_SIZE by the calibration
    copy, averages per dispatch, divides FLOP counts by the dispatch's own
    duration, and takes shares of SQ_WAVE_CYCLES."""
    gemm = "void mpq::(anonymous namespace)::gemm_err_kernel<true>(mpq::ErrGroup)"
    fit = "void mpq::(anonymous namespace)::fit_hist_kernel<512, 9, true, true, false>(mpq::HistBatch)"
    copy = "__amd_rocclr_copyBuffer"
    a, b, c = (str(tmp_path / x) for x in "abc")
    # pass a: SQ shares, two fit dispatches of 100 us and 300 us
    _pmc_csv(a, [(1, fit, 512, "SQ_WAVE_CYCLES", 1000.0, 0, 100000),
                 (1, fit, 512, "SQ_ACTIVE_INST_VALU", 250.0, 0, 100000),
                 (1, fit, 512, "SQ_WAIT_ANY", 500.0, 0, 100000),
                 (2, fit, 512, "SQ_WAVE_CYCLES", 3000.0, 0, 300000),
                 (2, fit, 512, "SQ_ACTIVE_INST_VALU", 750.0, 0, 300000),
                 (2, fit, 512, "SQ_WAIT_ANY", 1500.0, 0, 300000),
                 (1, fit, 512, "SQ_BUSY_CU_CYCLES", 400.0, 0, 100000),
                 (2, fit, 512, "SQ_BUSY_CU_CYCLES", 1600.0, 0, 300000)])
    # pass b: FLOP counts (1e9 FP32, 2e9 FP64 FLOP per dispatch)
    _pmc_csv(b, [(1, fit, 512, "SQ_INSTS_VALU_FLOPS_FP32", 1e9, 0, 200000),
                 (1, fit, 512, "SQ_INSTS_VALU_FLOPS_FP64", 2e9, 0, 200000)])
    # pass c: FETCH_SIZE with a copy that reads 256 MiB but counts half of it
    _pmc_csv(c, [(1, copy, 131072, "FETCH_SIZE", 131072.0, 0, 10),
                 (2, gemm, 1024, "FETCH_SIZE", 1000.0, 0, 50000)])
    d = str(tmp_path / "d")
    _pmc_csv(d, [(1, copy, 131072, "WRITE_SIZE", 262144.0, 0, 10),
                 (2, gemm, 1024, "WRITE_SIZE", 10.0, 0, 50000)])
    bench.summarize_counters([a, b, c, d], "resnet50", steps=1)
    out = capsys.readouterr().out
    import json
    blob = json.loads(next(l for l in out.splitlines() if l.startswith("counters-json: "))[15:])
    f = blob["fit_hist_kernel<512,9,lattice>"]
    assert abs(f["valu_active_share"] - 0.25) < 1e-12 and abs(f["wait_any_share"] - 0.5) < 1e-12
    # SIMD VALU busy: mean SQ_ACTIVE_INST_VALU (500) over mean SQ_BUSY_CU_CYCLES (1000)
    assert abs(f["valu_busy_per_cu_busy"] - 0.5) < 1e-12
    # 1e9 FLOP over the pass-b dispatch's 200 us = 5 TFLOP/s
    assert abs(f["valu_fp32_tflops"] - 5.0) < 1e-9 and abs(f["valu_fp64_tflops"] - 10.0) < 1e-9
    g = blob["gemm_err_kernel"]
    assert abs(g["fetch_size_bytes"] - 2 * 1000.0 * 1024) < 1e-6     # the copy read 2x its count
    assert abs(g["write_size_bytes"] - 10.0 * 1024) < 1e-6
    assert "sources: " in out


def test_bench_table(tmp_path, capsys):
    """The workload table reads each bench line's rate, roofline, traffic,
    longest fit, search counters and CPU sample stride."""
    import json
    line = {"value": 2.5e6, "ms_per_step": 1.25, "steps": 20, "warmup": 3,
            "config": {"workload": "resnet18", "points_per_step": 3125},
            "roofline": {"achieved": 90.0, "frac": 0.5722, "peak": 157.3, "avg_launch_us": 250.0,
                         "traffic": 4.36e8},
            "kernels": {"fit_hist_kernel<512,9,lattice>": {"stage": "fit", "us_per_step": 240.0,
                                                           "avg_us": 240.0, "launches_per_step": 1.0},
                        "gemm_err_kernel": {"stage": "output_error", "us_per_step": 250.0,
                                            "avg_us": 250.0, "launches_per_step": 1.0}},
            "search": {"kernel": "fit_hist_kernel<512,9,lattice>",
                       "counters": {"valu_busy_per_cu_busy": 0.503}},
            "cpu_baseline": {"value": 12360.0, "cores": 16,
                             "sample": "every 8th channel of each of the 21 layers of resnet18"}}
    p = tmp_path / "resnet18.json"
    p.write_text(json.dumps(line))
    bench.summarize_benches([str(p)])
    out = capsys.readouterr().out
    row = next(l for l in out.splitlines() if l.startswith("| resnet18 |"))
    assert "2.50 M" in row and "1.250" in row and "90.0 TFLOP/s (57% of 157.3)" in row
    assert "436 MB" in row and "50.3%" in row and "12.36 k (16)" in row
    assert "resnet18 8;" in out
