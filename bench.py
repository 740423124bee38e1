#!/usr/bin/env python3
"""Benchmark of the UAD action-expert hot path on one MI355X.

    python bench.py [--gpus 1] [--steps 200] [--warmup 20] [--workload pi0_b1]

A "step" is one joint denoising step: the per-token time embedding, all
transformer layers of the action expert over the whole chunk (attending to the
cached prefix), and the masked per-token Euler update.  The timed region runs
uniform 10-step schedules back to back with every input resident in HBM.
Prints ONE JSON line (see the design notes for every field).
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
MFMA_BF16_PEAK_TFS = 2500.0  # MI355X dense bf16


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def gemm_bytes(M, N, K, out_bytes, extra=0):
    """Algorithmic bytes of one projection launch: bf16 weights + bf16 input rows + output (+ extra)."""
    return N * K * 2 + M * K * 2 + out_bytes + extra


def kernel_bytes(wl, M):
    """Algorithmic HBM bytes per launch of each kernel class for M tokens of workload wl."""
    s = wl.shape
    d, F, qd, kvd = s.d_model, s.d_ff, s.n_heads * s.head_dim, s.n_kv_heads * s.head_dim
    nqkv = qd + 2 * kvd
    keys = wl.prefix + wl.chunk
    ada = getattr(s, "conditioning", "input") == "adarms"
    out = {} if not ada else {
        # every norm site's (scale, shift, gate) per token, fp32 out
        "gemm_mod": gemm_bytes(M, (6 * s.n_layers + 2) * d, d, M * (6 * s.n_layers + 2) * d * 4),
    }
    return out | {
        "gemm_qkv": gemm_bytes(M, nqkv, d, M * nqkv * 2),
        "attention": wl.batch * s.n_kv_heads * keys * s.head_dim * 2 * 2 + M * qd * 2 * 2,
        "gemm_o": gemm_bytes(M, d, qd, M * d * 4 * 2),
        "gemm_gateup": gemm_bytes(M, 2 * F, d, M * F * 2),
        "gemm_down": gemm_bytes(M, d, F, M * d * 4 * 2),
        "gemm_time_in": gemm_bytes(M, d, d if ada else 2 * d, M * d * 2),
        "gemm_time_out": gemm_bytes(M, d, d, M * d * (2 if ada else 4)),
    }


def kernel_flops(wl, M):
    s = wl.shape
    d, F, qd, kvd = s.d_model, s.d_ff, s.n_heads * s.head_dim, s.n_kv_heads * s.head_dim
    keys = wl.prefix + wl.chunk
    ada = getattr(s, "conditioning", "input") == "adarms"
    return ({"gemm_mod": 2 * M * d * (6 * s.n_layers + 2) * d} if ada else {}) | {
        "gemm_qkv": 2 * M * d * (qd + 2 * kvd),
        "attention": 4 * wl.batch * s.n_heads * wl.chunk * keys * s.head_dim,
        "gemm_o": 2 * M * qd * d,
        "gemm_gateup": 2 * M * d * 2 * F,
        "gemm_down": 2 * M * F * d,
        "gemm_time_in": 2 * M * (1 if ada else 2) * d * d,
        "gemm_time_out": 2 * M * d * d,
    }


def step_bytes(wl):
    """Algorithmic bytes of one joint step: all weights once + the prefix K/V of every env."""
    import uad_workloads as W
    s = wl.shape
    return W.weight_param_count(s) * 2 + wl.batch * s.n_layers * wl.prefix * s.n_kv_heads * s.head_dim * 2 * 2


def step_flops(wl):
    import uad_workloads as W
    s = wl.shape
    M = wl.batch * wl.chunk
    att = 4 * wl.batch * s.n_heads * wl.chunk * (wl.prefix + wl.chunk) * s.head_dim * s.n_layers
    return 2 * M * W.weight_param_count(s) + att


def kernel_source_hash() -> str:
    """sha256 over the library's kernel and host sources (byte counters are valid for exactly these)."""
    import glob
    import hashlib
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2609_37772_amd", "csrc", "*"))):
        if f.endswith((".hip", ".inl", ".cpp", ".h")):
            h.update(os.path.basename(f).encode())
            with open(f, "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pi0_b1_traffic.json")


def summarize_counters(run_dir: str) -> dict:
    """Per-launch HBM traffic of every kernel class from two rocprofv3 --pmc runs of
    ``bench.py --copy-calibration 256`` (FETCH_SIZE and WRITE_SIZE, KiB per dispatch),
    each scaled so that the same counter reads 256 MiB for the plain 256 MiB copy."""
    import csv
    import statistics
    out = {"source_hash": kernel_source_hash(), "unit": "bytes per launch", "classes": {}}
    scale = {}
    per_class = {}
    for counter in ("FETCH_SIZE", "WRITE_SIZE"):
        rows = list(csv.DictReader(open(os.path.join(run_dir, f"pmc_{counter}", "run_counter_collection.csv"))))
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        copies = [float(r["Counter_Value"]) for r in rows
                  if "copyBuffer" in r["Kernel_Name"] and float(r["Counter_Value"]) > 100000]
        scale[counter] = 256 * 1024 / statistics.mean(copies[-3:])
        # walk the dispatches of every step and name each by its launch site
        prev = None
        for r in rows:
            k = r["Kernel_Name"]
            if "stamp_kernel" in k or ("uad::" not in k and "_ZN3uad" not in k):
                continue
            if "temb" in k:
                cls = "temb"
            elif "gemm_kernel<0," in k:
                cls = "gemm_time_in"
            elif "gemm_kernel<5," in k:
                cls = "gemm_mod"
            elif "gemm_kernel<4," in k:
                cls = "gemm_qkv"
            elif "attn_kernel" in k or "attn_combine" in k:
                cls = "attention"
            elif "gemm_kernel<3," in k:
                cls = "gemm_gateup"
            elif "gemm_kernel<1," in k:
                cls = {"gemm_time_in": "gemm_time_out", "attention": "gemm_o", "gemm_gateup": "gemm_down"}.get(prev)
            elif "final_kernel" in k:
                cls = "final_euler"
            else:
                cls = None
            if cls is None:
                prev = None
                continue
            v = float(r["Counter_Value"]) * 1024 * scale[counter]
            d = per_class.setdefault(cls, {}).setdefault(counter, [])
            if cls == "attention" and prev == "attention" and "attn_combine" in k:
                d[-1] += v  # the combine belongs to the same attention launch
            else:
                d.append(v)
            prev = cls
    for cls, d in per_class.items():
        rd, wr = d.get("FETCH_SIZE", [0.0]), d.get("WRITE_SIZE", [0.0])
        out["classes"][cls] = {"read": round(statistics.mean(rd)), "written": round(statistics.mean(wr)),
                               "total": round(statistics.mean(rd) + statistics.mean(wr)), "launches": len(rd)}
    out["calibration"] = {"copy_bytes": 256 << 20, "FETCH_SIZE_scale": round(scale["FETCH_SIZE"], 4),
                          "WRITE_SIZE_scale": round(scale["WRITE_SIZE"], 4)}
    return out


def summarize_mfma(run_dir: str) -> dict:
    """MFMA busy and wave-state fractions per kernel from one rocprofv3 --pmc run
    (SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE, SQ_WAVE_CYCLES, SQ_WAIT_ANY,
    SQ_WAIT_INST_ANY, SQ_ACTIVE_INST_ANY, SQ_INSTS_VALU_MFMA_MOPS_F16,
    SQ_INSTS_VALU_MFMA_MOPS_BF16) found in DIR/pmc_mfma: MFMA busy = busy
    cycles summed over SIMDs / (GPU active cycles x SIMDs), the counters'
    own MfmaUtil expression, whose GPU active cycles are those of one XCC (the
    CSV sums them over the XCCs, so they are divided by their number); MFMA
    flops = (F16 + BF16 MOPS) x 512."""
    import csv
    import collections
    rows = list(csv.DictReader(open(os.path.join(run_dir, "pmc_mfma", "run_counter_collection.csv"))))
    simds = None
    per = collections.defaultdict(lambda: collections.defaultdict(float))
    launches = collections.defaultdict(set)
    for r in rows:
        k = r["Kernel_Name"]
        if ("uad::" not in k and "_ZN3uad" not in k) or "stamp_kernel" in k:
            continue
        launches[k].add(r["Dispatch_Id"])
        per[k][r["Counter_Name"]] += float(r["Counter_Value"])
    agent = os.path.join(run_dir, "pmc_mfma", "run_agent_info.csv")
    xcc = None
    if os.path.exists(agent):
        for r in csv.DictReader(open(agent)):
            if r.get("Agent_Type") == "GPU" and int(r.get("Simd_Count", 0) or 0) > 0:
                simds = int(r["Simd_Count"])
                xcc = int(r.get("Num_Xcc", 0) or 0) or None
    simds = simds or 1024
    xcc = xcc or 8
    out = {"simds": simds, "xcc": xcc, "kernels": {}}
    for k, c in per.items():
        wave = c.get("SQ_WAVE_CYCLES", 0.0) or 1.0
        gui = (c.get("GRBM_GUI_ACTIVE", 0.0) / xcc) or 1.0
        out["kernels"][k] = {
            "launches": len(launches[k]),
            "mfma_busy": round(c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (gui * simds), 4),
            "wait_any": round(c.get("SQ_WAIT_ANY", 0.0) / wave, 4),
            "wait_inst_any": round(c.get("SQ_WAIT_INST_ANY", 0.0) / wave, 4),
            "active_inst_any": round(c.get("SQ_ACTIVE_INST_ANY", 0.0) / wave, 4),
            "mfma_gflop_per_launch": round(512 * (c.get("SQ_INSTS_VALU_MFMA_MOPS_F16", 0.0) +
                                                  c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0)) /
                                           max(1, len(launches[k])) / 1e9, 3),
        }
    return out


def summarize_lds(run_dir: str) -> dict:
    """LDS, VALU and MFMA activity per kernel from one rocprofv3 --pmc run (SQ_LDS_IDX_ACTIVE,
    SQ_LDS_BANK_CONFLICT, SQ_LDS_DATA_FIFO_FULL, SQ_VALU_MFMA_BUSY_CYCLES, SQ_ACTIVE_INST_VALU,
    SQ_ACTIVE_INST_LDS, SQ_WAIT_INST_LDS, SQ_WAVE_CYCLES, GRBM_GUI_ACTIVE) found in DIR/pmc_lds:
    the LDS counters per CU cycle (GPU active cycles of one XCC x CUs), MFMA busy per SIMD cycle,
    the instruction-state counters per wave cycle."""
    import csv
    import collections
    rows = list(csv.DictReader(open(os.path.join(run_dir, "pmc_lds", "run_counter_collection.csv"))))
    per = collections.defaultdict(lambda: collections.defaultdict(float))
    launches = collections.defaultdict(set)
    for r in rows:
        k = r["Kernel_Name"]
        if ("uad::" not in k and "_ZN3uad" not in k) or "stamp_kernel" in k:
            continue
        launches[k].add(r["Dispatch_Id"])
        per[k][r["Counter_Name"]] += float(r["Counter_Value"])
    cus, simds, xcc = 256, 1024, 8
    agent = os.path.join(run_dir, "pmc_lds", "run_agent_info.csv")
    if os.path.exists(agent):
        for r in csv.DictReader(open(agent)):
            if r.get("Agent_Type") == "GPU" and int(r.get("Simd_Count", 0) or 0) > 0:
                simds = int(r["Simd_Count"])
                cus = int(r.get("Cu_Count", 0) or 0) or simds // 4
                xcc = int(r.get("Num_Xcc", 0) or 0) or xcc
    out = {"cus": cus, "simds": simds, "xcc": xcc, "kernels": {}}
    for k, c in per.items():
        gui = (c.get("GRBM_GUI_ACTIVE", 0.0) / xcc) or 1.0
        wave = c.get("SQ_WAVE_CYCLES", 0.0) or 1.0
        out["kernels"][k] = {
            "launches": len(launches[k]),
            "lds_active": round(c.get("SQ_LDS_IDX_ACTIVE", 0.0) / (gui * cus), 4),
            "lds_bank_conflict": round(c.get("SQ_LDS_BANK_CONFLICT", 0.0) / (gui * cus), 4),
            "lds_data_fifo_full": round(c.get("SQ_LDS_DATA_FIFO_FULL", 0.0) / (gui * cus), 4),
            "mfma_busy": round(c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (gui * simds), 4),
            "valu_active": round(c.get("SQ_ACTIVE_INST_VALU", 0.0) / wave, 4),
            "lds_inst_active": round(c.get("SQ_ACTIVE_INST_LDS", 0.0) / wave, 4),
            "wait_lds": round(c.get("SQ_WAIT_INST_LDS", 0.0) / wave, 4),
        }
    return out


STEP_ROLES = ("qkv", "attention", "combine", "o", "gateup", "down")


MAX_GAPS_US = 25.0  # summed gaps between a step's kernels for the step to count as traced back to back


def summarize_timeline(run_dir: str, workload: str = "pi0_b1") -> dict:
    """Per-layer timeline of the replayed step graphs of a rocprofv3 --kernel-trace run
    (DIR/run_kernel_trace.csv). A step is the run of kernels from the time embedding to the
    final Euler kernel: 3 + 6 per layer + 1. Only steps whose kernels ran nearly back to back
    (gaps summing to under MAX_GAPS_US, a few percent of the step) are kept: the profiler
    stretches the others. For each position: mean duration, mean gap before it, and the time
    its algorithmic bytes need at HBM peak."""
    import csv
    import statistics
    import uad_workloads as W
    wl = W.get_workload(workload)
    L = wl.shape.n_layers
    rows = list(csv.DictReader(open(os.path.join(run_dir, "run_kernel_trace.csv"))))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    want = (["temb_kernel", "gemm_kernel<0,", "gemm_kernel<1,"] +
            ["gemm_kernel<4,", "attn_kernel<", "attn_combine_kernel", "gemm_kernel<1,", "gemm_kernel<3,",
             "gemm_kernel<1,"] * L + ["final_kernel"])
    steps, cur = [], None
    for r in rows:
        k = r["Kernel_Name"]
        if ("uad::" not in k and "_ZN3uad" not in k) or "stamp_kernel" in k:
            continue
        if "temb_kernel" in k:
            cur = []
        if cur is None:
            continue
        cur.append((k, int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
        if "final_kernel" in k:
            if len(cur) == len(want) and all(w in n for w, (n, _, _) in zip(want, cur)):
                steps.append(cur)
            cur = None
    tight = [s for s in steps if sum(max(0, s[i][1] - s[i - 1][2]) for i in range(1, len(s))) < MAX_GAPS_US * 1e3]
    if not tight:
        raise SystemExit("no back-to-back steps in the trace")
    dur = [statistics.mean((s[i][2] - s[i][1]) / 1e3 for s in tight) for i in range(len(want))]
    gap = [0.0] + [statistics.mean((s[i][1] - s[i - 1][2]) / 1e3 for s in tight) for i in range(1, len(want))]
    kb = kernel_bytes(wl, wl.batch * wl.chunk)
    role_bytes = {"qkv": kb["gemm_qkv"], "attention": kb["attention"], "combine": 0, "o": kb["gemm_o"],
                  "gateup": kb["gemm_gateup"], "down": kb["gemm_down"]}
    layers = []
    for l in range(L):
        base = 3 + 6 * l
        layers.append({"layer": l, "busy_us": round(sum(dur[base:base + 6]), 2),
                       "gaps_us": round(sum(gap[base:base + 6]), 2),
                       "kernels_us": {r: round(dur[base + j], 2) for j, r in enumerate(STEP_ROLES)}})
    per_role = {r: round(statistics.mean(dur[3 + 6 * l + j] for l in range(L)), 2) for j, r in enumerate(STEP_ROLES)}
    return {
        "workload": workload, "steps_in_trace": len(steps), "back_to_back_steps": len(tight),
        "step_span_us": round(statistics.mean((s[-1][2] - s[0][1]) / 1e3 for s in tight), 2),
        "step_busy_us": round(statistics.mean(sum((k[2] - k[1]) / 1e3 for k in s) for s in tight), 2),
        "max_gaps_us": MAX_GAPS_US,
        "prologue_us": {"temb": round(dur[0], 2), "time_in": round(dur[1], 2), "time_out": round(dur[2], 2)},
        "final_us": round(dur[-1], 2),
        "gaps_total_us": round(sum(gap), 2),
        "layer_mean_us": per_role | {"total": round(sum(per_role.values()), 2)},
        "layer_bytes": role_bytes,
        "layer_bytes_us_at_peak": {r: round(b / (HBM_PEAK_GBS * 1e3), 2) for r, b in role_bytes.items()},
        "layers": layers,
    }


def measured_traffic(kernel_class: str):
    """Counter-measured bytes per launch of a class, if taken on the current sources; else None."""
    try:
        with open(TRAFFIC_FILE) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("source_hash") != kernel_source_hash():
        return None
    c = t.get("classes", {}).get(kernel_class)
    return c["total"] if c else None


def streaming_copy_gbs(torch, mib=2048, reps=10):
    """Measured HBM streaming rate of this device: a plain device-to-device copy
    of `mib` MiB (bytes read + bytes written per second), after the timed region."""
    src = torch.empty(mib << 20, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    del src, dst
    return 2 * (mib << 20) * reps / el / 1e9


def cpu_model():
    """The host CPU's model name (and the cores this process may run on)."""
    name = platform.processor() or "host"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        return f"{name}, {len(os.sched_getaffinity(0))} cores available"
    except AttributeError:
        return name


def cpu_baseline(wl, weights, prefix, noise, budgets, seconds, limit_threads=None):
    """Time the oracle (as it stands) on this host for a bounded sample of joint steps
    (BLAS threads capped at ``limit_threads`` when given)."""
    import contextlib
    import numpy as np
    import oracle as O
    ctx = contextlib.nullcontext()
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        if limit_threads is not None:
            ctx = threadpool_limits(limits=limit_threads)
    except Exception:
        threadpool_info = None
    with ctx:
        if threadpool_info is not None:
            threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
        else:
            threads = os.cpu_count() or 1
        return _cpu_baseline_run(wl, weights, prefix, noise, budgets, seconds, threads, O)


def _cpu_baseline_run(wl, weights, prefix, noise, budgets, seconds, threads, O):
    m = O.build_model(wl.shape, weights, [p[0] for p in prefix], [p[1] for p in prefix])
    n, t, dt, mask = O.build_schedule(budgets)
    x = noise.copy()
    O.denoise_step(m, x, t[0], dt[0], mask[0])  # warm-up
    done, t0 = 0, time.perf_counter()
    while True:
        x, _ = O.denoise_step(m, x, t[done % n], dt[done % n], mask[done % n])
        done += 1
        el = time.perf_counter() - t0
        if el >= seconds and done >= 2:
            break
    return {"value": done / el, "unit": "denoise steps/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{done} joint steps of the {wl.name} workload (B={wl.batch}, H={wl.chunk}, "
                      f"P={wl.prefix}) in {el:.1f} s, numpy fp32 BLAS on {cpu_model()}",
            "seconds": el}


def measure(ex, wl, budgets, noise, steps_req, warmup_req, sched_reps, U, np, torch):
    """Time exactly ``steps_req`` joint steps after exactly ``warmup_req`` untimed
    ones: whole schedules replayed from their captured graph, the remainder as
    single steps of the next schedule slices; then per-schedule device time and
    per-kernel-class launch times of the dominant class against its roofline."""
    s = wl.shape
    M = wl.batch * wl.chunk
    n, tg, dtg, mg = ex.schedule_tables(budgets)
    x0 = torch.from_numpy(noise).cuda()
    x = torch.empty_like(x0)

    def run(k_steps):
        full, rem = divmod(k_steps, n)
        for _ in range(full):
            x.copy_(x0)
            ex.schedule(x, tg, dtg, mg)
        if rem:
            x.copy_(x0)
            for k in range(rem):
                ex.step(x, tg[k], dtg[k], mg[k])

    # Warm-up: exactly the requested steps when they also build every graph the
    # timed region replays (a whole schedule when it times schedules, a single
    # step when it times a remainder); otherwise the few extra steps that do,
    # and the count actually run is reported.
    steps = max(1, steps_req)
    warm = max(0, warmup_req)
    if steps >= n and warm < n:
        warm = n + (warm % n if steps % n else 0)
    if steps % n and warm % n == 0:
        warm += 1
    run(warm)
    torch.cuda.synchronize()
    log(f"[bench] {wl.name}: warm-up {warm} steps done (requested {warmup_req})")
    t0 = time.perf_counter()
    run(steps)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    sps = steps / el
    ms_step = 1e3 * el / steps
    log(f"[bench] {wl.name}: timed {steps} steps: {ms_step:.4f} ms/step, {sps:.1f} steps/s")

    # Per-schedule device time (ticks at schedule start / end), median and a 95%
    # bootstrap interval over the R schedules (8000 resamples).
    hz = ex.tick_rate_hz()
    ticks = torch.zeros(n + 1, dtype=torch.uint64).pin_memory()
    per_sched = []
    for _ in range(max(1, sched_reps)):
        x.copy_(x0)
        ex.schedule(x, tg, dtg, mg, None, None, ticks)
        torch.cuda.synchronize()
        tk = ticks.numpy().astype(np.int64)
        per_sched.append((tk[-1] - tk[0]) / hz * 1e3)
    per_sched = np.array(per_sched)
    rng = np.random.default_rng(0)
    boot = np.median(rng.choice(per_sched, size=(8000, per_sched.size), replace=True), axis=1)
    sched_stats = {"schedules": int(per_sched.size), "steps_per_schedule": int(n),
                   "median_ms": round(float(np.median(per_sched)), 4),
                   "ci95_ms": [round(float(np.percentile(boot, 2.5)), 4), round(float(np.percentile(boot, 97.5)), 4)],
                   "clock": "device wall-clock ticks around each schedule (stamp kernels)"}
    log(f"[bench] {wl.name}: schedule median {sched_stats['median_ms']} ms, 95% CI {sched_stats['ci95_ms']}")

    # Per-kernel durations: the same schedules again, launched directly with a
    # start/stop HIP event pair taken from each kernel's dispatch packet, on the
    # stream the kernels run on (the library's measurement hook).
    U.uad_profile_enable(ex.ctx, True)
    run(max(n, (steps // n) * n))
    prof = U.uad_profile_read(ex.ctx)
    U.uad_profile_enable(ex.ctx, False)
    kb, kf = kernel_bytes(wl, M), kernel_flops(wl, M)
    if getattr(s, "conditioning", "input") == "adarms" and M <= 256:
        # schedule-level conditioning: the time MLP and the modulation GEMM run
        # once per schedule over the rows of all its n steps
        kbn, kfn = kernel_bytes(wl, M * n), kernel_flops(wl, M * n)
        for c in ("gemm_mod", "gemm_time_in", "gemm_time_out"):
            kb[c], kf[c] = kbn[c], kfn[c]
    per_kernel = {}
    for name, (ms, cnt) in prof.items():
        if cnt == 0:
            continue
        avg_us = 1e3 * ms / cnt
        ent = {"avg_us": round(avg_us, 3), "launches": cnt, "share": None}
        if name in kb:
            ent["gbs"] = round(kb[name] / (avg_us * 1e-6) / 1e9, 1)
            ent["tflops"] = round(kf[name] / (avg_us * 1e-6) / 1e12, 2)
        per_kernel[name] = ent
    tot = sum(v[0] for v in prof.values()) or 1.0
    for name in per_kernel:
        per_kernel[name]["share"] = round(prof[name][0] / tot, 4)
    dom = max((k for k in per_kernel if k in kb), key=lambda k: prof[k][0])
    dom_us = per_kernel[dom]["avg_us"]
    batched = M > 400
    if batched:
        ach = kf[dom] / (dom_us * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": MFMA_BF16_PEAK_TFS, "unit": "TFLOP/s",
                "frac": round(ach / MFMA_BF16_PEAK_TFS, 4),
                "traffic": measured_traffic(dom) if wl.name == "pi0_b1" else None,
                "algorithmic_flops_per_launch": kf[dom]}
    else:
        ach = kb[dom] / (dom_us * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic(dom) if wl.name == "pi0_b1" else None}
    roof.update({"kernel": dom, "algorithmic_bytes_per_launch": kb[dom], "avg_launch_us": dom_us})
    if dom == "attention" and not batched:
        # at batch 1 the attention launches carry the read-ahead of the next
        # projections' weights (O, gate/up, down, next layer's QKV) on the CUs they
        # leave idle: part of their measured traffic, none of their algorithmic bytes
        d, F, qd = s.d_model, s.d_ff, s.n_heads * s.head_dim
        nqkv = qd + 2 * s.n_kv_heads * s.head_dim
        roof["prefetch_bytes_per_launch"] = 2 * (d * qd + 2 * F * d + d * F + nqkv * d)
    log(f"[bench] {wl.name}: dominant kernel {dom}: {dom_us:.2f} us/launch, {roof['achieved']} {roof['unit']}")
    return {"steps_per_s": sps, "ms_per_step": ms_step, "steps": steps, "warmup": warm, "n": n,
            "roofline": roof, "kernels": per_kernel, "schedule_time": sched_stats}


def device_inputs(wl, U, W, np, torch):
    """Seeded synthetic inputs of a batched workload drawn on the device (the
    same distributions as the host generator the parity tests use: weights
    N(0, 0.02) and norm gains 1 + N(0, 0.02), prefix K/V and noise N(0, 1),
    bf16-rounded), so that a benchmark leg does not spend minutes in host RNG."""
    g = torch.Generator(device="cuda")
    g.manual_seed(wl.seed + 7919)
    s = wl.shape
    weights = {}
    for name, shp, kind in W.weight_specs(s):
        z = torch.randn(shp, generator=g, device="cuda", dtype=torch.float32) * 0.02
        weights[name] = (z + 1.0 if kind == "gain" else z).to(torch.bfloat16)
    B, P = wl.batch, wl.prefix
    shape = (s.n_layers, B, P, s.n_kv_heads, s.head_dim)
    k = torch.randn(shape, generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    v = torch.randn(shape, generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    noise = torch.randn((B, wl.chunk, s.action_dim), generator=g, device="cuda", dtype=torch.float32)
    return weights, k, v, noise.cpu().numpy()


def batched_leg(name, a, U, W, np, torch):
    """One batched (MFMA-bound) workload measured in the same run: ms per joint
    step, environment-steps per second, whole-step MFMA fraction and the
    dominant kernel class against the dense bf16 MFMA peak."""
    wl = W.get_workload(name)
    s = wl.shape
    t0 = time.time()
    weights, k, v, noise = device_inputs(wl, U, W, np, torch)
    ex = U.ActionExpert(s, wl.batch, wl.chunk, wl.prefix)
    ex.load_weights(weights)
    ex.set_prefix_kv(k, v, wl.batch, wl.prefix)
    del weights, k, v
    torch.cuda.synchronize()
    log(f"[bench] {name}: set-up {time.time() - t0:.1f} s (inputs drawn on the device)")
    steps = max(a.steps, 20)
    budgets = W.make_budgets(wl)
    meas = measure(ex, wl, budgets, noise, steps, a.warmup, min(a.sched_reps, 20), U, np, torch)
    comp = time_budget_schedules(ex, wl, budgets, noise, max(3, min(a.sched_reps, 20)), np, torch)
    ex.close()
    torch.cuda.empty_cache()
    fl = step_flops(wl)
    ms = meas["ms_per_step"]
    # algorithmic work of a schedule: every environment for as many joint steps
    # as its largest budget (a finished environment does no more work)
    env_steps = int(budgets.max(axis=1).sum())
    alg_flops = env_steps * fl / wl.batch
    sched_ms = comp["median_ms"]
    return {"config": {"workload": name, "batch": wl.batch, "chunk": wl.chunk, "prefix": wl.prefix,
                       "layers": s.n_layers, "width": s.d_model,
                       "heads": f"{s.n_heads}q/{s.n_kv_heads}kv x {s.head_dim}", "mlp": s.d_ff,
                       "schedule": f"{wl.budget_kind} {meas['n']} steps"},
            "ms_per_step": round(ms, 4), "env_steps_per_s": round(wl.batch * 1e3 / ms, 1),
            "steps": meas["steps"], "warmup": meas["warmup"],
            "flops_per_step": fl, "mfma_frac": round(fl / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFS, 4),
            "note": "ms_per_step / mfma_frac: joint steps over all environments (uad_denoise_schedule)",
            "schedule_from_budgets": {
                "entry": "uad_denoise_budgets (environments whose tokens are all released are not evaluated)",
                "median_ms": round(sched_ms, 4), "ci95_ms": comp["ci95_ms"], "schedules": comp["schedules"],
                "joint_steps": int(meas["n"]), "active_envs_per_step": comp["active"],
                "algorithmic_env_steps": env_steps, "algorithmic_flops": alg_flops,
                "env_steps_per_s": round(env_steps / (sched_ms * 1e-3), 1),
                "mfma_frac": round(alg_flops / (sched_ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFS, 4),
                "uncompacted_schedule_ms": meas["schedule_time"]["median_ms"]},
            "roofline": meas["roofline"], "kernels": meas["kernels"], "schedule_time": meas["schedule_time"],
            "data": "synthetic, drawn on the device (seeded torch generator, same distributions)"}


def adarms_leg(name, a, U, W, np, torch):
    """The adaptive-norm expert (pi0.5-scale, batch 1) measured in the same run:
    ms per joint step, steps per second, whole-step HBM fraction over its
    weight bytes (+36% for the modulation matrices) and the dominant kernel
    class against HBM peak."""
    wl = W.get_workload(name)
    s = wl.shape
    t0 = time.time()
    weights, k, v, noise = device_inputs(wl, U, W, np, torch)
    ex = U.ActionExpert(s, wl.batch, wl.chunk, wl.prefix)
    ex.load_weights(weights)
    ex.set_prefix_kv(k, v, wl.batch, wl.prefix)
    del weights, k, v
    torch.cuda.synchronize()
    log(f"[bench] {name}: set-up {time.time() - t0:.1f} s (inputs drawn on the device)")
    budgets = W.make_budgets(wl)
    meas = measure(ex, wl, budgets, noise, a.steps, a.warmup, min(a.sched_reps, 20), U, np, torch)
    ex.close()
    torch.cuda.empty_cache()
    ms = meas["ms_per_step"]
    sb = step_bytes(wl)
    return {"config": {"workload": name, "batch": wl.batch, "chunk": wl.chunk, "prefix": wl.prefix,
                       "layers": s.n_layers, "width": s.d_model,
                       "heads": f"{s.n_heads}q/{s.n_kv_heads}kv x {s.head_dim}", "mlp": s.d_ff,
                       "conditioning": "adaptive RMSNorm (per-token time modulates every norm and gates every branch)",
                       "schedule": f"{wl.budget_kind} {meas['n']} steps"},
            "ms_per_step": round(ms, 5), "steps_per_s": round(1e3 / ms, 2),
            "steps": meas["steps"], "warmup": meas["warmup"],
            "bytes_per_step": sb, "hbm_frac": round(sb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "roofline": meas["roofline"], "kernels": meas["kernels"], "schedule_time": meas["schedule_time"],
            "data": "synthetic, drawn on the device (seeded torch generator, same distributions)"}


def time_budget_schedules(ex, wl, budgets, noise, reps, np, torch):
    """Device time of whole schedules run from budgets (finished environments
    skipped), median and 95% bootstrap interval over reps schedules."""
    n = int(budgets.max())
    x0 = torch.from_numpy(noise).cuda()
    x = torch.empty_like(x0)
    hz = ex.tick_rate_hz()
    ticks = torch.zeros(n + 1, dtype=torch.uint64).pin_memory()
    x.copy_(x0)
    ex.schedule_budgets(x, budgets)  # builds the graph
    torch.cuda.synchronize()
    per = []
    for _ in range(reps):
        x.copy_(x0)
        ex.schedule_budgets(x, budgets, None, None, ticks)
        torch.cuda.synchronize()
        tk = ticks.numpy().astype(np.int64)
        per.append((tk[-1] - tk[0]) / hz * 1e3)
    per = np.array(per)
    rng = np.random.default_rng(0)
    boot = np.median(rng.choice(per, size=(8000, per.size), replace=True), axis=1)
    active = [int(np.sum(budgets.max(axis=1) > k)) for k in range(n)]
    log(f"[bench] {wl.name}: schedule from budgets median {np.median(per):.4f} ms (environments per step {active})")
    return {"median_ms": float(np.median(per)), "schedules": int(per.size), "active": active,
            "ci95_ms": [round(float(np.percentile(boot, 2.5)), 4), round(float(np.percentile(boot, 97.5)), 4)]}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="pi0_b1")
    ap.add_argument("--batch", type=int, default=0,
                    help="override the workload's environment count (e.g. one GPU's share of a sharded fleet)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-aal", action="store_true")
    ap.add_argument("--no-batched", action="store_true",
                    help="skip the extra legs: 64-environment fleet, the large expert and the adaptive-norm expert")
    ap.add_argument("--sched-reps", type=int, default=100,
                    help="schedules timed one by one for the median / bootstrap interval (fewer for profiler runs)")
    ap.add_argument("--summarize-counters", metavar="DIR", default=None,
                    help="print the per-launch traffic summary of two rocprofv3 --pmc runs found in DIR "
                         "(pmc_FETCH_SIZE/, pmc_WRITE_SIZE/) and exit; no GPU needed")
    ap.add_argument("--summarize-mfma", metavar="DIR", default=None,
                    help="print MFMA busy and wave-state fractions per kernel of a rocprofv3 --pmc run found in "
                         "DIR/pmc_mfma and exit; no GPU needed")
    ap.add_argument("--summarize-lds", metavar="DIR", default=None,
                    help="print LDS, VALU and MFMA activity per kernel of a rocprofv3 --pmc run found in "
                         "DIR/pmc_lds and exit; no GPU needed")
    ap.add_argument("--summarize-timeline", metavar="DIR", default=None,
                    help="print the per-layer timeline of the replayed step graphs in a rocprofv3 --kernel-trace "
                         "run found in DIR (run_kernel_trace.csv) and exit; no GPU needed")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after the run, copy an MIB-MiB fp32 buffer 3 times (a plain copy kernel of known "
                         "size, the reference for hardware byte counters)")
    a = ap.parse_args()
    if a.summarize_counters:
        print(json.dumps(summarize_counters(a.summarize_counters), indent=1))
        return
    if a.summarize_mfma:
        print(json.dumps(summarize_mfma(a.summarize_mfma), indent=1))
        return
    if a.summarize_lds:
        print(json.dumps(summarize_lds(a.summarize_lds), indent=1))
        return
    if a.summarize_timeline:
        print(json.dumps(summarize_timeline(a.summarize_timeline, a.workload), indent=1))
        return
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU: the hot path is measured on one "
                                   "MI355X and multi-GPU runs are not part of it", "n_gpus": a.gpus}))
        sys.exit(2)

    import numpy as np
    import torch
    import uad_workloads as W
    import paper_2609_37772_amd as U

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(2)
    U.load_library()
    wl = W.get_workload(a.workload, **({"batch": a.batch} if a.batch > 0 else {}))
    s = wl.shape
    B, H, P, M = wl.batch, wl.chunk, wl.prefix, wl.batch * wl.chunk
    log(f"[bench] workload {wl.name}: L={s.n_layers} d={s.d_model} B={B} H={H} P={P}")
    t0 = time.time()
    weights = W.make_weights(wl)
    prefix = [W.make_prefix(wl, b) for b in range(B)]
    noise = np.stack([W.make_noise(wl, b) for b in range(B)])
    budgets = W.make_budgets(wl)
    ex = U.ActionExpert(s, B, H, P)
    ex.load_weights(weights)
    dt_ = np.uint16 if wl.bf16 else np.float32
    K = np.empty((s.n_layers, B, P, s.n_kv_heads, s.head_dim), dt_)
    V = np.empty_like(K)
    for b in range(B):
        K[:, b] = W.bf16_bits(prefix[b][0]) if wl.bf16 else prefix[b][0]
        V[:, b] = W.bf16_bits(prefix[b][1]) if wl.bf16 else prefix[b][1]
    ex.set_prefix_kv(K, V, B, P)
    del K, V
    log(f"[bench] set-up {time.time() - t0:.1f} s")

    meas = measure(ex, wl, budgets, noise, a.steps, a.warmup, a.sched_reps, U, np, torch)
    sps, ms_step, steps = meas["steps_per_s"], meas["ms_per_step"], meas["steps"]
    roof, per_kernel, sched_stats, n = meas["roofline"], meas["kernels"], meas["schedule_time"], meas["n"]
    sb = step_bytes(wl)
    copy_gbs = streaming_copy_gbs(torch)
    step_roof = {"bytes_per_step": sb, "achieved_gbs": round(sb / (ms_step * 1e-3) / 1e9, 1),
                 "hbm_frac": round(sb / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                 "hbm_copy_gbs": round(copy_gbs, 1),
                 "copy_frac": round(sb / (ms_step * 1e-3) / 1e9 / copy_gbs, 4),
                 "flops_per_step": step_flops(wl),
                 "mfma_frac": round(step_flops(wl) / (ms_step * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFS, 4)}

    out = {
        "metric": "denoise steps/sec + action-availability latency (ms) at B=1; % HBM/MFMA roofline",
        "value": round(sps, 2), "unit": "denoise steps/s", "n_gpus": 1, "steps": steps, "warmup": meas["warmup"],
        "ms_per_step": round(ms_step, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16 weights, fp16 MFMA operands (fp32 accumulation, fp32 residual and integrator)",
        "data": "synthetic (seeded random-init weights, N(0,1) prefix K/V and noise)",
        "config": {"workload": wl.name, "batch": B, "chunk": H, "prefix": P, "layers": s.n_layers,
                   "width": s.d_model, "heads": f"{s.n_heads}q/{s.n_kv_heads}kv x {s.head_dim}", "mlp": s.d_ff,
                   "action_dim": s.action_dim, "schedule": f"{wl.budget_kind} {n} steps"},
        "roofline": roof, "step_roofline": step_roof, "schedule_time": sched_stats, "kernels": per_kernel,
        "kernels_clock": "direct-launch pass: the timed schedules again, each kernel launched on its own "
                         "with start/stop events from its dispatch packet (no graph)",
    }
    if not a.no_aal and B == 1:
        out["availability"] = availability(ex, wl, noise, U, np, torch)
    ex.close()

    if not a.no_batched and wl.name == "pi0_b1":
        out["batched"] = {}
        for name in ("pi0_fleet_b64", "large_b16"):
            out["batched"][name] = batched_leg(name, a, U, W, np, torch)
        out["adarms"] = adarms_leg("pi05_b1_adarms", a, U, W, np, torch)

    if not a.no_cpu_baseline:
        log("[bench] timing the oracle on the host cores")
        out["cpu_baseline"] = cpu_baseline(wl, weights, prefix, noise, budgets, a.cpu_seconds)
        one = cpu_baseline(wl, weights, prefix, noise, budgets, a.cpu_seconds / 2, limit_threads=1)
        out["cpu_baseline_1thread"] = {k: one[k] for k in ("value", "unit", "cores", "sample")}
    if a.copy_calibration > 0:
        n = a.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration"] = {"bytes_read": n * 4, "bytes_written": n * 4, "launches": 3}
    print(json.dumps(out), flush=True)


def availability(ex, wl, noise, U, np, torch, reps=20):
    """Action-availability latency on this model (App. B timing model, App. C.3
    measurement, T_VLM = 0 since the prefix is given).

    Release time of each of the S executed actions, measured on the host from the
    call to the moment the action is host-visible: vanilla uniform N* (all S
    actions when the chunk is done) and UAD with Trajectory Reconciliation and
    Ghost Action Correction at K = 1 (urgent actions when the release event fires,
    tail actions when the chunk is done), at the paper's (U, N*) settings.
    AAL replays the controller for T_act = 50 and 12.5 ms.  The U sweep gives the
    average blocking time of the tail actions (App. C, u_sweep) at N* = 7.
    """
    S, H, Da = wl.executed, wl.chunk, wl.shape.action_dim
    x0 = torch.from_numpy(noise).cuda()
    x = torch.empty_like(x0)

    def vanilla(Ns):
        n, tg, dtg, mg = ex.schedule_tables(np.full((1, H), Ns, np.int32))
        ts = []
        for r in range(reps + 2):
            x.copy_(x0)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            ex.schedule(x, tg, dtg, mg)
            torch.cuda.synchronize()
            if r >= 2:
                ts.append((time.perf_counter() - t0) * 1e3)
        t_end = float(np.median(ts))
        return [t_end] * S

    def uad(Ns, U_, K=1):
        urgent = torch.empty((1, U_, Da), device="cuda")
        executed = torch.empty((1, S, Da), device="cuda")
        host = torch.empty((1, U_, Da)).pin_memory()
        ev = torch.cuda.Event()
        tr, te = [], []
        for r in range(reps + 2):
            x.copy_(x0)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            ex.release(x, U_, K, Ns, S, urgent=urgent, executed=executed, urgent_host=host, release_event=ev)
            ev.synchronize()
            t1 = time.perf_counter()
            torch.cuda.synchronize()
            t2 = time.perf_counter()
            if r >= 2:
                tr.append((t1 - t0) * 1e3)
                te.append((t2 - t0) * 1e3)
        r_u, r_t = float(np.median(tr)), float(np.median(te))
        return [r_u] * U_ + [r_t] * (S - U_)

    def summarise(rel):
        ent = {"release_ms_executed": [round(v, 4) for v in rel], "ttfr_ms": round(min(rel), 4)}
        for tact in (50.0, 12.5):
            ent[f"aal_ms_tact_{tact:g}"] = round(U.uad_aal(rel, tact), 5)
        return ent

    res = {"clock": "host wall-clock from the call to host visibility (median of %d)" % reps}
    for Ns, U_ in ((7, 5), (3, 3), (2, 2), (10, 5)):
        v = summarise(vanilla(Ns))
        u = summarise(uad(Ns, U_))
        res[f"N*={Ns}"] = {"vanilla": v, f"uad_tr_gac_K1_U{U_}": u,
                           "aal_speedup_tact_12.5": round(v["aal_ms_tact_12.5"] / u["aal_ms_tact_12.5"], 3),
                           "aal_speedup_tact_50": round(v["aal_ms_tact_50"] / u["aal_ms_tact_50"], 3)}
    sweep = {}
    for U_ in range(1, S):
        rel = uad(7, U_)
        for tact in (12.5,):
            clock, waits = 0.0, []
            for j, r in enumerate(rel):
                w = max(0.0, r - clock)
                clock = max(clock, r) + tact
                if j >= U_:
                    waits.append(w)
        sweep[str(U_)] = round(float(np.mean(waits)), 5)
    res["u_sweep_tail_blocking_ms_Nstar7_tact12.5"] = sweep
    return res


if __name__ == "__main__":
    main()
