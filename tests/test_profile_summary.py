"""The rocprofv3 summarizer of bench.py (--summarize-profile) on synthetic
CSV files laid out as rocprofv3 writes them: kernel averages, the counter
calibration on the run's device copies, HBM bytes per dispatch, the
assignment of a layer's GEMM dispatches to its four matrices, and the MFMA
counter ratios."""
import csv
import os

import pytest

import bench

TRACE_COLS = ["Kind", "Agent_Id", "Queue_Id", "Stream_Id", "Thread_Id", "Dispatch_Id", "Kernel_Id", "Kernel_Name",
              "Correlation_Id", "Start_Timestamp", "End_Timestamp", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
              "Accum_VGPR_Count", "SGPR_Count", "Workgroup_Size_X", "Workgroup_Size_Y", "Workgroup_Size_Z",
              "Grid_Size_X", "Grid_Size_Y", "Grid_Size_Z"]
PMC_COLS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
            "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
            "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]
COPY = "__amd_rocclr_copyBuffer"
QUANT = "void w4a8::(anonymous namespace)::quantize_rows_block<512, 4>(unsigned short const*, int, signed char*, float*)"


def gemm_name(args):
    return f"void w4a8::(anonymous namespace)::{args}(w4a8::SmallMArgs)"


def write_trace(path, kernels_us):
    """kernels_us: [(name, microseconds)] in launch order, back to back."""
    os.makedirs(path)
    t = 1_000_000
    with open(os.path.join(path, "p_kernel_trace.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, TRACE_COLS)
        w.writeheader()
        for i, (name, us) in enumerate(kernels_us):
            row = dict.fromkeys(TRACE_COLS, 0)
            row.update(Kernel_Name=name, Dispatch_Id=i + 1, Start_Timestamp=t, End_Timestamp=t + int(us * 1000))
            w.writerow(row)
            t += int(us * 1000) + 500


def write_pmc(path, dispatches):
    """dispatches: [(name, {counter: value})] in launch order."""
    os.makedirs(path)
    with open(os.path.join(path, "p_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, PMC_COLS)
        w.writeheader()
        for i, (name, vals) in enumerate(dispatches):
            for c, v in vals.items():
                row = dict.fromkeys(PMC_COLS, 0)
                row.update(Dispatch_Id=i + 1, Kernel_Name=name, Counter_Name=c, Counter_Value=v)
                w.writerow(row)


def test_short_kernel_names():
    assert bench._short_kernel(gemm_name("smallm<1, 6, false, 0, true, false>")) == "smallm<1, 6, false, 0, true, false>"
    assert bench._short_kernel("void w4a8::(anonymous namespace)::largem<2, 3, 2, 2, false, 4, false, 1>"
                               "(w4a8::(anonymous namespace)::LargeMArgs)") == "largem<2, 3, 2, 2, false, 4, false, 1>"
    assert bench._short_kernel(QUANT) == "quantize_rows_block<512, 4>"
    assert bench._short_kernel(COPY) == COPY


def values(text):
    out = {}
    for line in text.splitlines():
        if line and not line.startswith("#") and ":" in line:
            k, v = line.split(":", 1)
            out[k.strip()] = v.split("   (")[0].strip()  # without the trailing notes
    return out


def test_single_gemm_summary(tmp_path):
    d = str(tmp_path)
    name = "smallm_down_verify_m1"
    M, N, K = 1, 4096, 12288
    w_bytes = N * K // 2
    g = gemm_name("smallm<1, 1, false, 0, true, false>")
    write_trace(os.path.join(d, f"{name}_trace"), [(COPY, 3.0)] + [(QUANT, 2.0), (g, 6.0), (QUANT, 3.0), (g, 8.0)])
    # the counters read half of a copy's bytes (factor 2) and all of its writes
    copies = [(COPY, {"FETCH_SIZE": w_bytes / 2048}), (COPY, {"FETCH_SIZE": 10.0})]
    write_pmc(os.path.join(d, f"{name}_fetch"), copies + [(g, {"FETCH_SIZE": 12400.0})] * 3)
    write_pmc(os.path.join(d, f"{name}_write"),
              [(COPY, {"WRITE_SIZE": w_bytes / 1024})] + [(g, {"WRITE_SIZE": 8.0})] * 3)
    v = values(bench.summarize_profile(name, d))
    assert v["kernel"] == "smallm<1, 1, false, 0, true, false>"
    assert float(v["avg_us"]) == pytest.approx(7.0)
    assert float(v["min_us"]) == pytest.approx(6.0)
    assert v["calls"] == "2"
    assert float(v["quantize_avg_us"]) == pytest.approx(2.5)
    algo = w_bytes + 4 * N + M * K + 4 * M + 2 * M * N
    assert int(v["algorithmic_bytes_per_dispatch"]) == algo
    assert int(v["fetch_bytes_per_dispatch"]) == 12400 * 1024 * 2
    assert int(v["write_bytes_per_dispatch"]) == 8 * 1024
    assert float(v["traffic_over_algorithmic"]) == pytest.approx((12400 * 2048 + 8192) / algo, abs=1e-3)
    assert float(v["frac_of_8TBps_from_avg"]) == pytest.approx(algo / 7e-6 / 8e12, abs=1e-4)


def test_layer_summary_assigns_dispatches_in_order(tmp_path):
    d = str(tmp_path)
    name = "largem_group_layer_m256"
    us = {"qkv": 16.0, "o": 11.0, "gate_up": 44.0, "down": 25.0}
    names = {m: gemm_name(f"largem<{i}, 1, 2, 2, true, 4, false, 1>") for i, m in enumerate(us)}
    steps = [(n, t) for _ in range(3) for m, t in us.items() for n in (QUANT, names[m])]
    steps = [(n, t if n != QUANT else 4.0) for n, t in steps]
    write_trace(os.path.join(d, f"{name}_trace"), steps)
    big = 24576 * 4096 // 2  # the gate+up weight, the run's largest copy
    copies = [(COPY, {"FETCH_SIZE": big / 2048}), (COPY, {"FETCH_SIZE": big / 4096})]
    wcopies = [(COPY, {"WRITE_SIZE": big / 1024}), (COPY, {"WRITE_SIZE": big / 2048})]
    fetch = {"qkv": 100.0, "o": 200.0, "gate_up": 300.0, "down": 400.0}
    gemms = [(names[m], {"FETCH_SIZE": fetch[m]}) for _ in range(2) for m in us]
    write_pmc(os.path.join(d, f"{name}_fetch"), copies + gemms)
    write_pmc(os.path.join(d, f"{name}_write"), wcopies + [(names[m], {"WRITE_SIZE": 1.0}) for _ in range(2) for m in us])
    mf = {c: 1.0 for c in bench.MFMA_COUNTERS.split()}
    mf.update(SQ_INSTS_VALU_MFMA_MOPS_I8=2 * 256 * 6144 * 4096 / 512, SQ_INSTS_MFMA=100.0, SQ_INSTS_VALU=1000.0,
              SQ_VALU_MFMA_BUSY_CYCLES=1024 * 50.0, GRBM_GUI_ACTIVE=8 * 100.0)
    write_pmc(os.path.join(d, f"{name}_mfma"), [(names[m], mf) for m in us])
    v = values(bench.summarize_profile(name, d))
    for m, t in us.items():
        assert float(v[f"{m}.avg_us"]) == pytest.approx(t)
        assert v[f"{m}.calls"] == "3"
        assert int(v[f"{m}.hbm_bytes_per_dispatch"]) == int(fetch[m] * 2048 + 1024)
    assert float(v["gemm_sum_avg_us"]) == pytest.approx(sum(us.values()))
    assert float(v["quantize_avg_us"]) == pytest.approx(4.0)
    assert int(v["qkv.mfma_int8_ops_per_dispatch"]) == 2 * 256 * 6144 * 4096
    assert float(v["qkv.mfma_busy_over_gui_active_per_simd"]) == pytest.approx(0.5)
    assert float(v["qkv.valu_insts_per_mfma"]) == pytest.approx(10.0)
    assert v["source_hash"] == bench.kernel_source_hash()
