#!/usr/bin/env python3
"""Benchmark of the MI355X im2win path on one GPU.

One step is one pass of the whole hot path over the workload's input, which is
resident in device memory before timing starts:
  1. workspace size query (host),
  2. im2win transformation x -> window tensor,
  3. convolution from the window tensor -> y,
  4. fused convolution x -> y2 (window strips built on chip).
The step therefore computes the convolution twice; `value` is the total
convolution work of a step, 2 * (2*N*K*C*Ho*Wo*Fh*Fw) flops, divided by the
measured step time (host clock around the synchronised timed steps; the GPU
time between two events around them is reported beside it).  Per-kernel
launch durations, from which the roofline fractions are computed, come from a
second timed region per kernel: as many back-to-back launches as timed steps,
on the same stream, between two HIP events.

Prints one JSON line per workload (rank 0, N=1): the four others first, then
the headline workload (ResNet-style 3x3 fp32 layer) with the CPU baseline.
`--gpus N` with N > 1 exits: the library runs on one GPU.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "conv GFLOP/s + % of MFMA/HBM roofline; im2win workspace bytes vs im2col"
PEAK = {"f32": 157.3, "bf16": 2500.0}          # dense matrix-core TFLOP/s, MI355X
HBM_PEAK_GBS = 8000.0
KERNEL_SOURCES = {
    "transform": ["paper_2306_14320_amd/csrc/transform.hip", "paper_2306_14320_amd/csrc/common.h"],
    "conv": ["paper_2306_14320_amd/csrc/conv_f32.hip", "paper_2306_14320_amd/csrc/conv_bf16.hip",
             "paper_2306_14320_amd/csrc/conv_bf16_image.hip", "paper_2306_14320_amd/csrc/conv_f32_band.hip",
             "paper_2306_14320_amd/csrc/conv_plain.hip",
             "paper_2306_14320_amd/csrc/conv_common.h", "paper_2306_14320_amd/csrc/common.h"],
}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def source_hash(kind):
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[kind]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, kernel_kind):
    """HBM bytes per launch of a kernel ("transform", "conv" or "fused") from the
    committed counter summary, if it was taken on the current kernel source;
    otherwise None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    entry = t.get(workload, {}).get(kernel_kind)
    src = "transform" if kernel_kind == "transform" else "conv"
    if not entry or entry.get("source_hash") != source_hash(src):
        return None
    return entry.get("bytes_per_launch")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=None,
                    help="run only this workload (default: every workload, one line each, the "
                         "headline workload last with the CPU baseline)")
    ap.add_argument("--headline-only", action="store_true", help="run only the headline workload")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain device copy of known size (for counter scaling)")
    ap.add_argument("--profile-call", choices=["transform", "conv2d", "conv2d_fused"], default=None,
                    help="launch only this entry point (warmup + steps times) on the workload and "
                         "print its mean launch time: the program that counter runs profile")
    ap.add_argument("--traffic-summary", metavar="DIR", default=None,
                    help="turn the counter runs under DIR (see profiles/hbm_traffic_all_workloads.md) "
                         "into profiles/traffic.json and print the table")
    ap.add_argument("--table1", action="store_true",
                    help="time the paper's twelve benchmark layers (Table 1: batch 128, fp32, no "
                         "padding) instead: one line per layer, then a summary line")
    ap.add_argument("--baselines", action="store_true",
                    help="compare the im2win path with the paper's comparison systems on the GPU "
                         "(im2col = unfold + GEMM, and direct convolution) and the vendor library "
                         "convolution: times, speedups and peak device memory per workload (with "
                         "--table1: per Table 1 layer), then a summary line")
    ap.add_argument("--batch", type=int, default=None,
                    help="with --baselines: run every layer at this batch instead of its own")
    return ap.parse_args()


def copy_calibration():
    import torch
    nbytes = 256 << 20
    a = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda:0").fill_(1.0)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": nbytes, "copy_calibration_bytes_written": nbytes,
                      "launches": 5}), flush=True)


def run_workload(wl, steps, warmup, with_cpu):
    import torch
    import paper_2306_14320_amd as P
    import workloads

    dev = "cuda:0"
    d = P.desc_for((wl.n, wl.c, wl.h, wl.w), (wl.k, wl.c, wl.fh, wl.fw), (wl.sh, wl.sw),
                   (wl.ph, wl.pw), workloads.torch_dtype(wl.dtype))
    ho, wo = P.im2win_output_shape(d)
    ws_bytes = P.im2win_workspace_bytes(d)
    col_bytes = P.im2win_im2col_bytes(d)
    dt = P.desc_for((wl.n, wl.c, wl.h, wl.w), (wl.k, wl.c, wl.fh, wl.fw), (wl.sh, wl.sw),
                    (wl.ph, wl.pw), workloads.torch_dtype(wl.dtype), layout=P.IM2WIN_ROWS_TRIMMED)
    trimmed_bytes = P.im2win_workspace_bytes(dt)
    x = workloads.make_input(wl).to(dev)
    w = workloads.make_filter(wl).to(dev)
    ws = torch.empty(P.workspace_shape(d), dtype=x.dtype, device=dev)
    scratch_bytes = P.im2win_filter_scratch_bytes(d)
    scratch = torch.empty(max(scratch_bytes, 16), dtype=torch.uint8, device=dev)
    y = torch.empty((wl.n, wl.k, ho, wo), dtype=torch.float32, device=dev)
    y2 = torch.empty_like(y)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    xp, wp, wsp, yp, y2p = x.data_ptr(), w.data_ptr(), ws.data_ptr(), y.data_ptr(), y2.data_ptr()
    scp = scratch.data_ptr()

    launch = {
        "transform": lambda: P.im2win_transform(d, xp, wsp, ws_bytes, sp),
        "conv2d": lambda: P.im2win_conv2d(d, wsp, ws_bytes, wp, scp, scratch_bytes, yp, sp),
        "conv2d_fused": lambda: P.im2win_conv2d_fused(d, xp, wp, scp, scratch_bytes, y2p, sp),
    }

    def step():
        P.im2win_workspace_bytes(d)
        launch["transform"]()
        launch["conv2d"]()
        launch["conv2d_fused"]()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    # the timed steps: one event pair around all of them
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for i in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_step = e0.elapsed_time(e1) * 1e-3 / steps
    # per-kernel launch duration: the same number of launches of each kernel
    # back to back on the same stream, one event pair around them
    per = {}
    for name, fn in launch.items():
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for i in range(steps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        per[name] = a.elapsed_time(b) * 1e-3 / steps
    t_xf, t_cv, t_fu = per["transform"], per["conv2d"], per["conv2d_fused"]
    single = single_launch_times(launch, stream)

    conv_flops = 2 * wl.n * wl.k * wl.c * ho * wo * wl.fh * wl.fw
    e = x.element_size()
    x_bytes = wl.n * wl.c * wl.h * wl.w * e
    w_bytes = wl.k * wl.c * wl.fh * wl.fw * e
    y_bytes = wl.n * wl.k * ho * wo * 4
    xf_bytes = x_bytes + ws_bytes                 # read x once, write the window tensor
    cv_bytes = ws_bytes + w_bytes + y_bytes       # conv2d: window tensor and filter in, y out
    fu_bytes = x_bytes + w_bytes + y_bytes        # conv2d_fused: x and filter in, y out
    # HBM rates from the cold launches (each after a write that evicts the
    # 256 MB Infinity Cache); the back-to-back figures are warm
    t_xf_cold = single["transform"]["cold_median"] * 1e-3
    ms_per_step = wall / steps * 1e3
    value = 2 * conv_flops / (wall / steps) / 1e9   # host clock around the synchronised steps
    peak = PEAK[wl.dtype]
    dominant = max([("conv", t_cv), ("fused", t_fu), ("transform", t_xf)], key=lambda kv: kv[1])[0]
    if dominant == "transform":
        achieved = xf_bytes / t_xf_cold / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(wl.name, "transform"),
                "kernel": "transform", "timing": "cold median single launch"}
    else:
        t = t_cv if dominant == "conv" else t_fu
        achieved = conv_flops / t / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": measured_traffic(wl.name, dominant),
                "kernel": "conv2d" if dominant == "conv" else "conv2d_fused"}
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "GFLOP/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(ms_per_step, 4),
        "gpu_ms_per_step": round(gpu_step * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": wl.dtype, "data": "synthetic (seeded, distributions of the workload)",
        "config": {"workload": wl.label(), "global_batch": wl.n, "parallelism": "none (1 GPU)",
                   "step": "workspace query + transform + conv2d + conv2d_fused"},
        "roofline": roof,
        "kernels": {
            "transform": {"ms": round(t_xf * 1e3, 4), "cold_ms": round(t_xf_cold * 1e3, 4),
                          "GB_per_s": round(xf_bytes / t_xf_cold / 1e9, 1),
                          "hbm_frac": round(xf_bytes / t_xf_cold / 1e9 / HBM_PEAK_GBS, 4),
                          "warm_GB_per_s": round(xf_bytes / t_xf / 1e9, 1),
                          "warm_hbm_frac": round(xf_bytes / t_xf / 1e9 / HBM_PEAK_GBS, 4),
                          "algorithmic_bytes": xf_bytes,
                          "note": "GB_per_s and hbm_frac from the cold (Infinity Cache flushed) median "
                                  "single launch; warm_* from the back-to-back mean (ms)"},
            "conv2d": {"ms": round(t_cv * 1e3, 4), "GFLOP_per_s": round(conv_flops / t_cv / 1e9, 1),
                       "mfma_frac": round(conv_flops / t_cv / 1e12 / peak, 4),
                       "mfma_floor_ms": round(conv_flops / (peak * 1e12) * 1e3, 4),
                       "algorithmic_bytes": cv_bytes,
                       "hbm_floor_ms": round(cv_bytes / (HBM_PEAK_GBS * 1e9) * 1e3, 4),
                       "cold_hbm_frac": round(cv_bytes / (single["conv2d"]["cold_median"] * 1e-3) / 1e9
                                              / HBM_PEAK_GBS, 4)},
            "conv2d_fused": {"ms": round(t_fu * 1e3, 4), "GFLOP_per_s": round(conv_flops / t_fu / 1e9, 1),
                             "mfma_frac": round(conv_flops / t_fu / 1e12 / peak, 4),
                             "algorithmic_bytes": fu_bytes,
                             "hbm_floor_ms": round(fu_bytes / (HBM_PEAK_GBS * 1e9) * 1e3, 4),
                             "cold_hbm_frac": round(fu_bytes / (single["conv2d_fused"]["cold_median"] * 1e-3)
                                                    / 1e9 / HBM_PEAK_GBS, 4)},
            "transform_plus_conv2d_GFLOP_per_s": round(conv_flops / (t_xf + t_cv) / 1e9, 1),
            "single_launch_ms": single,
        },
        "workspace": {"im2win_bytes": ws_bytes, "im2col_bytes": col_bytes,
                      "im2win_over_im2col": round(ws_bytes / col_bytes, 4),
                      "im2win_trimmed_bytes": trimmed_bytes,
                      "im2win_trimmed_over_im2col": round(trimmed_bytes / col_bytes, 4)},
        "conv_flops": conv_flops,
    }
    if with_cpu:
        out["cpu_baseline"] = cpu_baseline(wl, conv_flops)
    return out


def single_launch_times(launch, stream, warm_reps=21, cold_reps=11):
    """Each kernel timed launch by launch (an event pair around every launch on
    its stream): the median over warm_reps warm launches and the best of the
    first five (the paper reports the best of five runs, Sec. IV-B), and the
    median over cold_reps launches that each follow a 1 GiB device write, which
    evicts the inputs from the 256 MB Infinity Cache."""
    import statistics
    import torch
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda:0")
    out = {}
    for name, fn in launch.items():
        times = {}
        for mode, reps in (("warm", warm_reps), ("cold", cold_reps)):
            evs = []
            for _ in range(reps):
                if mode == "cold":
                    flush.zero_()
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
                fn()
                b.record(stream)
                evs.append((a, b))
            torch.cuda.synchronize()
            times[mode] = [a.elapsed_time(b) for a, b in evs]
        out[name] = {"warm_median": round(statistics.median(times["warm"]), 4),
                     "warm_best_of_5": round(min(times["warm"][:5]), 4),
                     "cold_median": round(statistics.median(times["cold"]), 4)}
    del flush
    torch.cuda.empty_cache()
    return out


def cpu_baseline(wl, conv_flops):
    """The oracle (fp64 seven-loop direct convolution, OpenMP) on the host
    cores, repeated over the full workload until about 10 s have passed."""
    import oracle
    from oracle import Shape
    import workloads
    s = Shape(wl.n, wl.c, wl.h, wl.w, wl.k, wl.fh, wl.fw, wl.sh, wl.sw, wl.ph, wl.pw)
    x = workloads.make_input(wl).double().numpy()
    w = workloads.make_filter(wl).double().numpy()
    reps, total = 0, 0.0
    while total < 10.0 and reps < 30:
        t0 = time.perf_counter()
        oracle.direct_conv(s, x, w)
        total += time.perf_counter() - t0
        reps += 1
    # the oracle's transformation of the same input (bytes: x read once, the
    # window tensor written), one run
    xr = workloads.make_input(wl).numpy()
    t0 = time.perf_counter()
    win = oracle.im2win(s, xr)
    t_xf = time.perf_counter() - t0
    xf_bytes = xr.nbytes + win.nbytes
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), "")
    except OSError:
        pass
    return {"value": round(conv_flops * reps / total / 1e9, 3), "unit": "GFLOP/s",
            "cores": oracle.num_threads(), "kind": "oracle", "cpu_model": model,
            "transform_GB_per_s": round(xf_bytes / t_xf / 1e9, 2),
            "sample": f"full workload (N={wl.n}), {reps} run(s) of the convolution, {total:.1f} s; "
                      f"one run of the transformation, {t_xf:.2f} s"}


def profile_call(wl, call, steps, warmup):
    """warmup + steps launches of one entry point, nothing else on the GPU
    after the inputs are made (the transform runs once first for conv2d)."""
    import torch
    import paper_2306_14320_amd as P
    import workloads
    dev = "cuda:0"
    d = P.desc_for((wl.n, wl.c, wl.h, wl.w), (wl.k, wl.c, wl.fh, wl.fw), (wl.sh, wl.sw),
                   (wl.ph, wl.pw), workloads.torch_dtype(wl.dtype))
    ho, wo = P.im2win_output_shape(d)
    ws_bytes = P.im2win_workspace_bytes(d)
    x = workloads.make_input(wl).to(dev)
    w = workloads.make_filter(wl).to(dev)
    ws = torch.empty(P.workspace_shape(d), dtype=x.dtype, device=dev)
    sb = P.im2win_filter_scratch_bytes(d)
    scratch = torch.empty(max(sb, 16), dtype=torch.uint8, device=dev)
    y = torch.empty((wl.n, wl.k, ho, wo), dtype=torch.float32, device=dev)
    sp = torch.cuda.current_stream().cuda_stream
    fn = {"transform": lambda: P.im2win_transform(d, x.data_ptr(), ws.data_ptr(), ws_bytes, sp),
          "conv2d": lambda: P.im2win_conv2d(d, ws.data_ptr(), ws_bytes, w.data_ptr(), scratch.data_ptr(), sb,
                                            y.data_ptr(), sp),
          "conv2d_fused": lambda: P.im2win_conv2d_fused(d, x.data_ptr(), w.data_ptr(), scratch.data_ptr(), sb,
                                                        y.data_ptr(), sp)}[call]
    if call == "conv2d":
        P.im2win_transform(d, x.data_ptr(), ws.data_ptr(), ws_bytes, sp)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(warmup + steps):
        fn()
    torch.cuda.synchronize()
    print(json.dumps({"workload": wl.name, "call": call, "launches": warmup + steps,
                      "ms_per_launch": round((time.perf_counter() - t0) / (warmup + steps) * 1e3, 4)}),
          flush=True)


# Counter runs read by --traffic-summary, one rocprofv3 --pmc process each:
#   DIR/calib_<COUNTER>/        bench.py --copy-calibration
#   DIR/<workload>__<call>__<COUNTER>/   bench.py --workload <w> --profile-call <call>
# with COUNTER in FETCH_SIZE, WRITE_SIZE.
TRAFFIC_CALLS = {"transform": "transform", "conv2d": "conv", "conv2d_fused": "fused"}


def _counter_rows(path):
    import csv
    import glob
    files = glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {path}")
    with open(files[0]) as f:
        return list(csv.DictReader(f))


def _per_dispatch(rows, select):
    """Counter value summed per dispatch over the kernels `select` accepts:
    {dispatch id: (kernel name, KiB)}."""
    out = {}
    for r in rows:
        if select(r["Kernel_Name"]):
            name, v = out.get(r["Dispatch_Id"], (r["Kernel_Name"], 0.0))
            out[r["Dispatch_Id"]] = (name, v + float(r["Counter_Value"]))
    return out


def traffic_summary(root):
    import workloads
    copy = lambda n: "copyBuffer" in n
    ours = lambda n: "im2win::" in n
    factor = {}
    for ctr in ("FETCH_SIZE", "WRITE_SIZE"):
        disp = _per_dispatch(_counter_rows(os.path.join(root, "calib_" + ctr)), copy)
        kib = max(v for _, v in disp.values())   # the 256 MiB copy (torch may add small copies)
        factor[ctr] = (256 << 20) / (kib * 1024)
    out = {"_calibration": {"copy_bytes": 256 << 20, "fetch_factor": round(factor["FETCH_SIZE"], 4),
                            "write_factor": round(factor["WRITE_SIZE"], 4),
                            "note": "HBM bytes = counter KiB * 1024 * factor"}}
    print("| workload | call | kernels | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM read MB | HBM write MB |")
    print("|---|---|---|---|---|---|---|")
    for wl in workloads.WORKLOADS:
        for call, kind in TRAFFIC_CALLS.items():
            kib, names, calls = {}, set(), None
            for ctr in ("FETCH_SIZE", "WRITE_SIZE"):
                d = os.path.join(root, f"{wl.name}__{call}__{ctr}")
                if not os.path.isdir(d):
                    break
                disp = _per_dispatch(_counter_rows(d), ours)
                if call == "conv2d":   # the one transform launched before the timed calls
                    disp = {k: v for k, v in disp.items() if "transform" not in v[0]}
                main = [k for k, (n, _) in disp.items() if "pack_filter" not in n]
                calls = len(main)
                kib[ctr] = sum(v for _, v in disp.values()) / max(calls, 1)
                names |= {n.replace("void ", "").replace("im2win::(anonymous namespace)::", "").split("(")[0]
                          for n, _ in disp.values()}
            if len(kib) != 2:
                continue
            fetch = int(kib["FETCH_SIZE"] * 1024 * factor["FETCH_SIZE"])
            write = int(kib["WRITE_SIZE"] * 1024 * factor["WRITE_SIZE"])
            src = "transform" if kind == "transform" else "conv"
            out.setdefault(wl.name, {})[kind] = {
                "kernels": sorted(names), "fetch_bytes": fetch, "write_bytes": write,
                "bytes_per_launch": fetch + write, "launches": calls, "source_hash": source_hash(src)}
            print(f"| {wl.name} | {call} | {', '.join('`%s`' % n for n in sorted(names))} | "
                  f"{kib['FETCH_SIZE']:.1f} | {kib['WRITE_SIZE']:.1f} | {fetch / 1e6:.2f} | {write / 1e6:.2f} |")
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")


def table1_sweep(steps, warmup):
    """The paper's benchmark layers (Sec. IV-A, Table 1) at its batch of 128:
    each line as for a workload (no CPU baseline), then the workspace ratio
    im2col / im2win averaged over the layers (Sec. IV-C prints 2.93) and the
    sweep's aggregate rates."""
    import torch
    import workloads
    lines = []
    for wl in workloads.TABLE1:
        line = run_workload(wl, steps, warmup, False)
        line["sweep"] = "table1"
        print(json.dumps(line), flush=True)
        lines.append(line)
        torch.cuda.empty_cache()
    ratios = [l["workspace"]["im2col_bytes"] / l["workspace"]["im2win_bytes"] for l in lines]
    ratios_t = [l["workspace"]["im2col_bytes"] / l["workspace"]["im2win_trimmed_bytes"] for l in lines]
    flops = sum(l["conv_flops"] for l in lines)
    t = {k: sum(l["kernels"][k]["ms"] for l in lines) * 1e-3 for k in ("transform", "conv2d", "conv2d_fused")}
    print(json.dumps({
        "sweep": "table1", "layers": len(lines), "batch": workloads.TABLE1_BATCH, "dtype": "f32",
        "im2col_over_im2win_mean": round(sum(ratios) / len(ratios), 4),
        "im2col_over_im2win_trimmed_mean": round(sum(ratios_t) / len(ratios_t), 4),
        "conv2d_GFLOP_per_s": round(flops / t["conv2d"] / 1e9, 1),
        "conv2d_fused_GFLOP_per_s": round(flops / t["conv2d_fused"] / 1e9, 1),
        "transform_plus_conv2d_GFLOP_per_s": round(flops / (t["transform"] + t["conv2d"]) / 1e9, 1),
        "mfma_frac_conv2d": round(flops / t["conv2d"] / 1e12 / PEAK["f32"], 4),
        "mfma_frac_conv2d_fused": round(flops / t["conv2d_fused"] / 1e12 / PEAK["f32"], 4),
    }), flush=True)


# ---------------------------------------------------------------------------
# Comparison systems (Sec. IV-B, Fig. 4; Sec. IV-C, Fig. 6), on the GPU
# ---------------------------------------------------------------------------

def im2col_conv2d(x, w, stride, padding):
    """im2col-based convolution: the framework's unfold (the im2col matrix,
    N x C*Fh*Fw x Ho*Wo) and one batched GEMM with the filter as K x C*Fh*Fw
    (the filter operand is shared by the batch).  fp32 in and out; bf16 inputs
    give a bf16 GEMM result, returned widened to fp32."""
    import torch
    import torch.nn.functional as F
    n, k = x.shape[0], w.shape[0]
    fh, fw = w.shape[2], w.shape[3]
    cols = F.unfold(x, (fh, fw), padding=padding, stride=stride)
    a = w.reshape(k, -1).unsqueeze(0).expand(n, -1, -1)
    y = torch.bmm(a, cols)
    ho = (x.shape[2] + 2 * padding[0] - fh) // stride[0] + 1
    wo = (x.shape[3] + 2 * padding[1] - fw) // stride[1] + 1
    return y.view(n, k, ho, wo).float()


def _time_calls(fn, stream, budget_s=1.0, max_reps=50):
    """Mean duration of back-to-back calls between two events on `stream`
    (after two warm-up calls), with as many calls as fit in about budget_s."""
    import torch
    fn(); fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    fn()
    torch.cuda.synchronize()
    one = time.perf_counter() - t0
    reps = max(1, min(max_reps, int(budget_s / max(one, 1e-6))))
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(reps):
        fn()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1e-3 / reps, reps


def _peak_bytes(fn, resident_bytes):
    """Device bytes at the peak of one call: what the call allocates (work
    buffers, outputs) plus the inputs already resident (x and w)."""
    import torch
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    out = fn()
    torch.cuda.synchronize()
    peak = torch.cuda.max_memory_allocated() - base
    del out
    return peak + resident_bytes


def compare_baselines(wl, n=None):
    """One workload: the im2win path (transform + conv2d, as Alg. 2 / 3 call
    the transformation first; and the fused path) against im2col + GEMM, the
    direct convolution (no transformation) and the vendor library's conv2d,
    all on the same device inputs; times, speedups and peak device memory."""
    import dataclasses
    import torch
    import torch.nn.functional as F
    import paper_2306_14320_amd as P
    import workloads
    if n is not None and n != wl.n:
        wl = dataclasses.replace(wl, n=n)
    dev = "cuda:0"
    stride, pad = (wl.sh, wl.sw), (wl.ph, wl.pw)
    d = P.desc_for((wl.n, wl.c, wl.h, wl.w), (wl.k, wl.c, wl.fh, wl.fw), stride, pad,
                   workloads.torch_dtype(wl.dtype))
    ho, wo = P.im2win_output_shape(d)
    x = workloads.make_input(wl).to(dev)
    w = workloads.make_filter(wl).to(dev)
    stream = torch.cuda.current_stream()
    resident = x.numel() * x.element_size() + w.numel() * w.element_size()
    dt = P.desc_for((wl.n, wl.c, wl.h, wl.w), (wl.k, wl.c, wl.fh, wl.fw), stride, pad,
                    workloads.torch_dtype(wl.dtype), layout=P.IM2WIN_ROWS_TRIMMED)
    paths = {
        "im2win": lambda: P.conv2d(P.transform(x, d), w, d),
        "im2win_trimmed": lambda: P.conv2d(P.transform(x, dt), w, dt),
        "im2win_fused": lambda: P.conv2d_fused(x, w, d),
        "im2col_gemm": lambda: im2col_conv2d(x, w, stride, pad),
        "direct": lambda: P.direct_conv2d(x, w, d),
        "vendor_conv2d": lambda: F.conv2d(x, w, stride=stride, padding=pad),
    }
    conv_flops = 2 * wl.n * wl.k * wl.c * ho * wo * wl.fh * wl.fw
    res = {}
    for name, fn in paths.items():
        try:
            t, reps = _time_calls(fn, stream)
            mem = _peak_bytes(fn, resident)
            res[name] = {"ms": round(t * 1e3, 4), "GFLOP_per_s": round(conv_flops / t / 1e9, 1),
                         "peak_bytes": mem, "reps": reps}
        except Exception as e:   # a comparison system that cannot run this shape is reported, not fatal
            res[name] = {"error": f"{type(e).__name__}: {e}"[:200]}
        torch.cuda.empty_cache()
    ours = res["im2win"]
    line = {"workload": wl.label(), "dtype": wl.dtype, "conv_flops": conv_flops, "paths": res}
    if "ms" in ours:
        line["speedup_vs"] = {k: round(v["ms"] / ours["ms"], 3) for k, v in res.items()
                              if k != "im2win" and "ms" in v}
        line["im2col_peak_over_im2win"] = (round(res["im2col_gemm"]["peak_bytes"] / ours["peak_bytes"], 4)
                                           if "peak_bytes" in res["im2col_gemm"] else None)
    return line


def baselines_sweep(table1, batch):
    import torch
    import workloads
    wls = workloads.TABLE1 if table1 else workloads.WORKLOADS
    lines = []
    for wl in wls:
        line = compare_baselines(wl, batch)
        line["sweep"] = "baselines-table1" if table1 else "baselines"
        print(json.dumps(line), flush=True)
        lines.append(line)
        torch.cuda.empty_cache()
    ok = [l for l in lines if "speedup_vs" in l]

    def mean(key):
        v = [l["speedup_vs"][key] for l in ok if key in l["speedup_vs"]]
        return round(sum(v) / len(v), 3) if v else None
    mem = [l["im2col_peak_over_im2win"] for l in ok if l.get("im2col_peak_over_im2win")]
    print(json.dumps({
        "sweep": "baselines-table1" if table1 else "baselines", "layers": len(lines),
        "batch": batch or ("per layer" if not table1 else workloads.TABLE1_BATCH),
        "mean_speedup_vs_im2col_gemm": mean("im2col_gemm"),
        "mean_speedup_vs_direct": mean("direct"),
        "mean_speedup_vs_vendor_conv2d": mean("vendor_conv2d"),
        "mean_speedup_fused_vs_im2col_gemm": round(
            sum(l["paths"]["im2col_gemm"]["ms"] / l["paths"]["im2win_fused"]["ms"] for l in ok
                if "ms" in l["paths"]["im2col_gemm"] and "ms" in l["paths"]["im2win_fused"]) / max(len(ok), 1), 3),
        "im2col_peak_over_im2win_mean": round(sum(mem) / len(mem), 4) if mem else None,
        "im2col_peak_over_im2win_max": round(max(mem), 4) if mem else None,
        "memory_reduction_vs_im2col_mean": round(sum(1 - 1 / m for m in mem) / len(mem), 4) if mem else None,
    }), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the library has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.traffic_summary:
        traffic_summary(args.traffic_summary)
        return
    import workloads
    if args.profile_call:
        profile_call(workloads.BY_NAME[args.workload] if args.workload else workloads.HEADLINE,
                     args.profile_call, args.steps, args.warmup)
        return
    if args.baselines:
        baselines_sweep(args.table1, args.batch)
        return
    if args.table1:
        table1_sweep(args.steps, args.warmup)
        return
    if args.workload:
        print(json.dumps(run_workload(workloads.BY_NAME[args.workload], args.steps, args.warmup,
                                      not args.no_cpu_baseline)), flush=True)
        return
    # every workload, one line each; the headline workload last, with the
    # CPU baseline
    wl = workloads.HEADLINE
    if not args.headline_only:
        for other in workloads.WORKLOADS:
            if other.name != wl.name:
                line = run_workload(other, args.steps, args.warmup, False)
                line["headline"] = False
                print(json.dumps(line), flush=True)
    line = run_workload(wl, args.steps, args.warmup, not args.no_cpu_baseline)
    line["headline"] = True
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
