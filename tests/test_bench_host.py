"""Host logic of the benchmark (CPU): the rocprofv3 summarizers on small
synthetic CSV files of known values, the algorithmic work tables, and the
one-GPU refusal of ``--gpus N``."""
import csv
import json
import os
import subprocess
import sys

import pytest

import bench
import uad_workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _write_csv(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(header)
        w.writerows(rows)


def _agent(path, cus=256, simds=1024, xcc=8):
    _write_csv(path, ["Agent_Type", "Simd_Count", "Cu_Count", "Num_Xcc"],
               [["CPU", 0, 0, 0], ["GPU", simds, cus, xcc]])


def _step_kernels(layers):
    names = ["_ZN3uad11temb_kernelILi1EE", "void uad::gemm_kernel<0, 1, 4, false, true>(uad::GemmArgs)",
             "void uad::gemm_kernel<1, 1, 4, false, false>(uad::GemmArgs)"]
    for _ in range(layers):
        names += ["void uad::gemm_kernel<4, 1, 4, false, false>(uad::GemmArgs)",
                  "void uad::attn_kernel<256, 2, false, 4>(uad::AttnArgs)",
                  "void uad::attn_combine_kernel<16>(uad::AttnArgs, int)",
                  "void uad::gemm_kernel<1, 1, 4, false, true>(uad::GemmArgs)",
                  "void uad::gemm_kernel<3, 2, 4, false, false>(uad::GemmArgs)",
                  "void uad::gemm_kernel<1, 1, 4, false, true>(uad::GemmArgs)"]
    return names + ["void uad::final_kernel<4>(uad::FinalArgs)"]


def test_summarize_timeline_keeps_back_to_back_steps(tmp_path):
    """Three traced steps of the 18-layer batch-1 step (each kernel 1000 ns + 100 ns
    per position): one back to back, one with 100 ns gaps (11.1 us in all: kept), one
    with 5 us gaps (dropped)."""
    names = _step_kernels(W.get_workload("pi0_b1").shape.n_layers)
    rows, t = [], 1_000_000
    for gap in (0, 100, 5000):
        for i, n in enumerate(names):
            d = 1000 + 100 * (i % 7)
            rows.append([n, t, t + d])
            t += d + gap
        t += 1_000_000
    rows.append(["uad::stamp_kernel(unsigned long*)", t, t + 500])
    _write_csv(str(tmp_path / "run_kernel_trace.csv"), ["Kernel_Name", "Start_Timestamp", "End_Timestamp"], rows)
    s = bench.summarize_timeline(str(tmp_path), "pi0_b1")
    assert s["steps_in_trace"] == 3 and s["back_to_back_steps"] == 2
    assert s["gaps_total_us"] == pytest.approx(0.05 * (len(names) - 1)) and len(s["layers"]) == 18
    # layer 0 starts at position 3: durations 1000 + 100 * ((3 + j) % 7) ns
    assert s["layers"][0]["kernels_us"] == {r: (1000 + 100 * ((3 + j) % 7)) / 1e3
                                            for j, r in enumerate(bench.STEP_ROLES)}
    busy = sum(1000 + 100 * (i % 7) for i in range(len(names))) / 1e3
    assert s["step_busy_us"] == pytest.approx(busy)
    assert s["step_span_us"] == pytest.approx(busy + 0.05 * (len(names) - 1))


def test_summarize_lds_and_mfma_normalisation(tmp_path):
    """LDS counters per CU cycle of one XCC, MFMA busy per SIMD cycle, wave
    states per wave cycle, MFMA flops from the MOPS counters (x 512)."""
    k = "void uad::gemm_ring_kernel<3, 2>(uad::GemmArgs)"
    gui = 8 * 1000.0  # summed over 8 XCCs: 1000 cycles each
    lds = {"SQ_LDS_IDX_ACTIVE": 0.25 * 1000 * 256, "SQ_LDS_BANK_CONFLICT": 0.05 * 1000 * 256,
           "SQ_LDS_DATA_FIFO_FULL": 0.0, "SQ_VALU_MFMA_BUSY_CYCLES": 0.4 * 1000 * 1024,
           "SQ_ACTIVE_INST_VALU": 30.0, "SQ_ACTIVE_INST_LDS": 10.0, "SQ_WAIT_INST_LDS": 5.0,
           "SQ_WAVE_CYCLES": 100.0, "GRBM_GUI_ACTIVE": gui}
    rows = [[1, k, c, v / 2] for c, v in lds.items()] + [[2, k, c, v / 2] for c, v in lds.items()]
    _write_csv(str(tmp_path / "pmc_lds" / "run_counter_collection.csv"),
               ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"], rows)
    _agent(str(tmp_path / "pmc_lds" / "run_agent_info.csv"))
    s = bench.summarize_lds(str(tmp_path))["kernels"][k]
    assert s == {"launches": 2, "lds_active": 0.25, "lds_bank_conflict": 0.05, "lds_data_fifo_full": 0.0,
                 "mfma_busy": 0.4, "valu_active": 0.3, "lds_inst_active": 0.1, "wait_lds": 0.05}
    mf = {"SQ_VALU_MFMA_BUSY_CYCLES": 0.3 * 1000 * 1024, "SQ_WAVE_CYCLES": 200.0, "SQ_WAIT_ANY": 100.0,
          "SQ_WAIT_INST_ANY": 60.0, "SQ_ACTIVE_INST_ANY": 40.0, "SQ_INSTS_VALU_MFMA_MOPS_F16": 1e8,
          "SQ_INSTS_VALU_MFMA_MOPS_BF16": 0.0, "GRBM_GUI_ACTIVE": gui}
    _write_csv(str(tmp_path / "pmc_mfma" / "run_counter_collection.csv"),
               ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"], [[7, k, c, v] for c, v in mf.items()])
    _agent(str(tmp_path / "pmc_mfma" / "run_agent_info.csv"))
    m = bench.summarize_mfma(str(tmp_path))["kernels"][k]
    assert m == {"launches": 1, "mfma_busy": 0.3, "wait_any": 0.5, "wait_inst_any": 0.3, "active_inst_any": 0.2,
                 "mfma_gflop_per_launch": 51.2}


def test_summarize_counters_scales_by_the_copy(tmp_path):
    """FETCH_SIZE / WRITE_SIZE in KiB per dispatch, scaled so the 256 MiB copy
    reads 256 MiB; dispatches named by launch site, the merge added to its
    attention launch."""
    seq = ["void uad::gemm_kernel<0, 1, 4, false, true>(uad::GemmArgs)",
           "void uad::gemm_kernel<1, 1, 4, false, false>(uad::GemmArgs)",
           "void uad::gemm_kernel<4, 1, 4, false, false>(uad::GemmArgs)",
           "void uad::attn_kernel<256, 2, false, 4>(uad::AttnArgs)",
           "void uad::attn_combine_kernel<16>(uad::AttnArgs, int)",
           "void uad::gemm_kernel<1, 1, 4, false, true>(uad::GemmArgs)",
           "void uad::gemm_kernel<3, 2, 4, false, false>(uad::GemmArgs)",
           "void uad::gemm_kernel<1, 1, 4, false, true>(uad::GemmArgs)",
           "void uad::final_kernel<4>(uad::FinalArgs)"]
    for counter, copy_kib in (("FETCH_SIZE", 128 * 1024), ("WRITE_SIZE", 256 * 1024)):
        rows = [[i + 1, n, counter, 100.0 * (i + 1)] for i, n in enumerate(seq)]
        rows += [[100 + j, "__amd_rocclr_copyBuffer", counter, copy_kib] for j in range(3)]
        _write_csv(str(tmp_path / f"pmc_{counter}" / "run_counter_collection.csv"),
                   ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"], rows)
    s = bench.summarize_counters(str(tmp_path))
    assert s["calibration"]["FETCH_SIZE_scale"] == 2.0 and s["calibration"]["WRITE_SIZE_scale"] == 1.0
    c = s["classes"]
    assert set(c) == {"gemm_time_in", "gemm_time_out", "gemm_qkv", "attention", "gemm_o", "gemm_gateup",
                      "gemm_down", "final_euler"}
    assert c["gemm_qkv"]["read"] == 300 * 1024 * 2 and c["gemm_qkv"]["written"] == 300 * 1024
    assert c["attention"]["read"] == (400 + 500) * 1024 * 2  # attention + its merge
    assert c["gemm_o"]["read"] == 600 * 1024 * 2 and c["gemm_down"]["read"] == 800 * 1024 * 2
    assert s["source_hash"] == bench.kernel_source_hash()


def test_algorithmic_work_tables():
    """Per-launch bytes and flops of the batch-1 step against their definitions."""
    wl = W.get_workload("pi0_b1")
    s, M = wl.shape, wl.batch * wl.chunk
    kb, kf = bench.kernel_bytes(wl, M), bench.kernel_flops(wl, M)
    nqkv = (s.n_heads + 2 * s.n_kv_heads) * s.head_dim
    assert kb["gemm_qkv"] == nqkv * s.d_model * 2 + M * s.d_model * 2 + M * nqkv * 2
    assert kf["gemm_gateup"] == 2 * M * s.d_model * 2 * s.d_ff
    assert kb["attention"] == (wl.prefix + wl.chunk) * s.head_dim * 2 * 2 + M * s.n_heads * s.head_dim * 2 * 2
    # the step: every weight once plus the prefix K/V of every layer
    assert bench.step_bytes(wl) == W.weight_param_count(s) * 2 + s.n_layers * wl.prefix * s.head_dim * 2 * 2


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    out = json.loads(r.stdout.strip().splitlines()[-1])
    assert out["n_gpus"] == 2 and "one GPU" in out["error"]
