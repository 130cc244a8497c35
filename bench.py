#!/usr/bin/env python3
"""Throughput of the multipoint-quantization hot path on one MI355X.

One step = the whole path over one synthetic workload already resident in
HBM: for every layer, the greedy fit (mpq_fit_layer), the output error on
the layer's calibration batch (mpq_output_error) and the reconstruction
(mpq_reconstruct).  The default workload is the ResNet-18-shaped stack
(21 layers, 5,800 channels, 4 bits, up to 4 points, 256 candidate scales,
tol 1e-3, 1,024 calibration columns).

Prints one JSON line.  `value` is channel-points fitted per second over the
whole step (sum of the per-channel point counts of all layers / step time).
`roofline` describes the kernel with the most time in the timed region,
measured with HIP events on the stream the kernels run on.  `cpu_baseline`
times the fp64 CPU oracle on a sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
PEAK_MFMA_F32_TFLOPS = 157.3
PEAK_VALU_F32_TFLOPS = 157.3            # published (packed) FP32 vector peak
PEAK_VALU_F32_NONPACKED_TFLOPS = 78.6   # 256 CU x 64 lanes x 2 FLOP x 2.4 GHz
FLOP_PER_EVAL = 7                       # scale-mul, round, clamp, fma (2), square-acc fma (2)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="resnet18")
    ap.add_argument("--cpu-stride", type=int, default=1,
                    help="cpu_baseline fits every n-th channel of every layer")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--dense", action="store_true",
                    help="fit with mpq_fit_layer_dense (O(d G) search) instead of mpq_fit_layer")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print the HBM-traffic summary of two rocprofv3 --pmc runs "
                         "(FETCH_SIZE, WRITE_SIZE) of `bench.py --steps 1 --warmup 1 "
                         "--copy-calibration` and exit")
    ap.add_argument("--summarize-trace", metavar="TRACE_DIR",
                    help="print the per-kernel summary of a rocprofv3 --kernel-trace --stats run "
                         "of `bench.py --steps 5 --warmup 1 --no-cpu-baseline` and exit")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="before the steps, copy a 256 MiB device buffer once (a kernel of known "
                         "traffic, to scale the FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "resnet18_hbm_traffic.md")
COPY_BYTES = 256 << 20
KERNEL_KINDS = (("fit", ("fit_hist_kernel", "fit_dense_kernel")),
                ("output_error", ("form_dt_kernel", "gemm_err_kernel", "finish_err_kernel")),
                ("reconstruct", ("reconstruct_kernel",)))


def sources_digest():
    """sha256 of the HIP sources, to tell whether stored counters still apply."""
    import glob
    import hashlib
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2002_09049_amd", "csrc", "*"))):
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def summarize_pmc(fetch_dir, write_dir):
    """HBM bytes per step and stage from the FETCH_SIZE / WRITE_SIZE counters,
    each scaled so that the 256 MiB calibration copy reads / writes 256 MiB."""
    import csv
    import glob
    import re

    def per_kind(d):
        rows = []
        for f in glob.glob(os.path.join(d, "*counter_collection.csv")):
            rows += list(csv.DictReader(open(f)))
        cal = [r for r in rows if "copyBuffer" in r["Kernel_Name"] and int(r["Grid_Size"]) == 131072]
        if not cal:
            raise SystemExit(f"no calibration copy in {d}")
        factor = COPY_BYTES / 1024.0 / float(cal[0]["Counter_Value"])
        out = {k: 0.0 for k, _ in KERNEL_KINDS}
        steps = 0
        for r in rows:
            m = re.search(r"(\w+_kernel)", r["Kernel_Name"])
            name = m.group(1) if m else ""
            for kind, names in KERNEL_KINDS:
                if name in names:
                    out[kind] += float(r["Counter_Value"]) * factor * 1024.0
            if name == "gemm_err_kernel":
                steps += 1
        return factor, out, steps

    ff, fetch, steps = per_kind(fetch_dir)
    wf, write, _ = per_kind(write_dir)
    steps = max(steps, 1)
    lines = ["# HBM traffic per step: ResNet-18-shaped workload", "",
             "Two rocprofv3 counter runs (one counter each), from the repository root:", "",
             "```",
             "rocprofv3 --pmc FETCH_SIZE --output-format csv -d gpurun_out/pmc_FETCH_SIZE -o p -- \\",
             "    python3 bench.py --steps 1 --warmup 1 --no-cpu-baseline --copy-calibration",
             "rocprofv3 --pmc WRITE_SIZE --output-format csv -d gpurun_out/pmc_WRITE_SIZE -o p -- \\",
             "    python3 bench.py --steps 1 --warmup 1 --no-cpu-baseline --copy-calibration",
             "python3 bench.py --summarize-pmc gpurun_out/pmc_FETCH_SIZE gpurun_out/pmc_WRITE_SIZE",
             "```", "",
             f"Scale factors from a 256 MiB device copy: FETCH_SIZE x {ff:.4f}, WRITE_SIZE x {wf:.4f}.",
             f"Bytes per step (the run holds {steps} steps).", "",
             "| stage | fetch bytes | write bytes | total bytes |", "|---|---:|---:|---:|"]
    for kind, _ in KERNEL_KINDS:
        f_, w_ = fetch[kind] / steps, write[kind] / steps
        lines.append(f"| {kind} | {f_:.0f} | {w_:.0f} | {f_ + w_:.0f} |")
    lines += ["", f"sources: {sources_digest()}", ""]
    print("\n".join(lines))


def summarize_trace(trace_dir):
    """Per-kernel and per-stage time of a traced bench run, from the
    kernel_stats.csv that rocprofv3 --stats writes."""
    import csv
    import glob
    import re

    files = glob.glob(os.path.join(trace_dir, "*kernel_stats.csv"))
    if not files:
        raise SystemExit(f"no kernel_stats.csv in {trace_dir}")
    rows = list(csv.DictReader(open(files[0])))
    calls = max(int(r["Calls"]) for r in rows if "fit_" in r["Name"])
    lines = ["# rocprofv3 kernel summary: ResNet-18-shaped workload, one bench step", "",
             "Workload: 21 layers (5,800 channels, 11,678,912 weights), 4 bits, up to 4 points,",
             "256 candidate scales, tol 1e-3, calibration batches d x 1024.  One step = fit +",
             "output error + reconstruction of every layer through the batched C ABI calls.", "",
             "Command (one MI355X, from the repository root):", "", "```",
             "rocprofv3 --kernel-trace --stats --output-format csv -d gpurun_out/prof -o kt -- \\",
             "    python3 bench.py --steps 5 --warmup 1 --no-cpu-baseline",
             "python3 bench.py --summarize-trace gpurun_out/prof", "```", "",
             f"The traced process ran {calls} steps (warm-up + timed); `calls` counts all of them.",
             "Kernels of one stage may run concurrently on several streams, so a stage's",
             "kernel-time sum can exceed its wall time.", "",
             "| kernel | calls | total ms | avg us | % |", "|---|---:|---:|---:|---:|"]
    stage = {k: 0.0 for k, _ in KERNEL_KINDS}
    stage["other"] = 0.0
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        name = r["Name"]
        m = re.search(r"(\w+_kernel(<[^>]*>)?)", name)
        short = m.group(1) if m else name[:40]
        lines.append(f"| `{short}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.3f} | "
                     f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
        kind = "other"
        for k, names in KERNEL_KINDS:
            if any(n in name for n in names):
                kind = k
        stage[kind] += float(r["TotalDurationNs"]) / 1e6
    lines += ["", f"Kernel time per step (sum over the stage's kernels / {calls}):"]
    for k, v in stage.items():
        lines.append(f"- {k}: {v / calls:.3f} ms")
    lines += ["", f"sources: {sources_digest()}", ""]
    print("\n".join(lines))


def measured_traffic(kind):
    """HBM bytes per step of a stage from the stored counter summary, or None
    when the summary is missing or was taken on other kernel sources."""
    try:
        text = open(TRAFFIC_SUMMARY).read()
    except OSError:
        return None
    if f"sources: {sources_digest()}" not in text:
        return None
    for ln in text.splitlines():
        cells = [c.strip() for c in ln.strip("|").split("|")]
        if len(cells) == 4 and cells[0] == kind:
            return int(cells[3])
    return None


def main():
    args = parse()
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc)
        return 0
    if args.summarize_trace:
        summarize_trace(args.summarize_trace)
        return 0
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the fit has no cross-GPU step to measure)", file=sys.stderr, flush=True)
        return 2
    import numpy as np
    import torch

    from paper_2002_09049_amd import mpq, workloads as wl

    assert torch.cuda.is_available(), "bench.py needs a ROCm GPU"
    mpq.load()
    wk = wl.get(args.workload)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    # ---- inputs and outputs resident in HBM before the timed region
    Ws, Xs = [], []
    for li in range(len(wk.layers)):
        Ws.append(torch.from_numpy(wl.layer_weights(wk, li)).to(dev))
        Xs.append(torch.from_numpy(wl.layer_calib(wk, li)).to(dev))
    ls = mpq.LayerSet(Ws, wk.max_points, calib=Xs, with_fit_err=True)
    torch.cuda.synchronize()
    if args.copy_calibration:
        src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)            # reads and writes 256 MiB
        torch.cuda.synchronize()
        del src, dst

    def step(ev=None):
        if ev: ev[0].record(stream)
        if args.dense:
            for i, W in enumerate(Ws):
                mpq.fit_layer(W, wk.bits, wk.max_points, wk.n_grid, wk.tol, dense=True,
                              out=(ls.codes[i], ls.scales[i], ls.counts[i], ls.fit_err[i]))
        else:
            ls.fit(wk.bits, wk.n_grid, wk.tol)
        if ev: ev[1].record(stream)
        ls.output_error()
        if ev: ev[2].record(stream)
        ls.reconstruct()
        if ev: ev[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    nl = len(Ws)
    ev = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(4)) for _ in range(args.steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for s in range(args.steps):
        step(ev[s])
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_total = t_start.elapsed_time(t_end)
    ms_step = ms_total / args.steps

    # ---- per-kernel times (HIP events on the launch stream) and algorithmic work
    t_fit = sum(e[0].elapsed_time(e[1]) for e in ev)
    t_err = sum(e[1].elapsed_time(e[2]) for e in ev)
    t_rec = sum(e[2].elapsed_time(e[3]) for e in ev)
    points = evals = gemm_flop = rec_bytes = fit_bytes = 0
    for i, W in enumerate(Ws):
        C, d = W.shape
        counts = ls.counts[i].cpu().numpy().astype(np.int64)
        n = int(counts.sum())
        points += n
        evals += n * wk.n_grid * d
        gemm_flop += 2 * C * d * Xs[i].shape[1]
        # reconstruct: read the codes of the used points, write fp32
        rec_bytes += n * d + 4 * C * d
        # fit (algorithmic minimum): read W once, write the codes of every point
        fit_bytes += 4 * C * d + n * d
    steps = args.steps
    sec_fit = t_fit * 1e-3
    fit_gbs = fit_bytes * steps / sec_fit / 1e9
    fit_eff_tflops = FLOP_PER_EVAL * evals * steps / sec_fit / 1e12
    gemm_tflops = gemm_flop * steps / (t_err * 1e-3) / 1e12
    rec_gbs = rec_bytes * steps / (t_rec * 1e-3) / 1e9
    if args.dense:
        fit_k = {"search": "dense", "bound": "alu", "ms_per_step": t_fit / steps,
                 "achieved": fit_eff_tflops, "peak": PEAK_VALU_F32_TFLOPS, "unit": "TFLOP/s",
                 "frac": fit_eff_tflops / PEAK_VALU_F32_TFLOPS,
                 "frac_of_nonpacked_peak": fit_eff_tflops / PEAK_VALU_F32_NONPACKED_TFLOPS,
                 "candidate_evals_per_step": evals}
    else:
        # the histogram search does O(d M + G) work per channel-step instead of
        # O(d G): its bound is memory/latency, so it is priced against HBM with
        # the algorithmic bytes; the evaluation rate it delivers is reported apart
        fit_k = {"search": "histogram", "bound": "hbm", "ms_per_step": t_fit / steps,
                 "achieved": fit_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                 "frac": fit_gbs / PEAK_HBM_GBS, "algorithmic_bytes_per_step": fit_bytes,
                 "candidate_evals_per_step": evals,
                 "candidate_evals_per_s": evals * steps / sec_fit,
                 "dense_equivalent_tflops": fit_eff_tflops}
    kernels = {
        "fit": fit_k,
        "output_error": {"bound": "mfma", "ms_per_step": t_err / steps, "achieved": gemm_tflops,
                         "peak": PEAK_MFMA_F32_TFLOPS, "unit": "TFLOP/s",
                         "frac": gemm_tflops / PEAK_MFMA_F32_TFLOPS, "flop_per_step": gemm_flop},
        "reconstruct": {"bound": "hbm", "ms_per_step": t_rec / steps, "achieved": rec_gbs,
                        "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": rec_gbs / PEAK_HBM_GBS,
                        "bytes_per_step": rec_bytes},
    }
    dom = max(kernels, key=lambda k: kernels[k]["ms_per_step"])
    K = kernels[dom]
    for k in kernels:
        kernels[k]["hbm_bytes_per_step_measured"] = measured_traffic(k)
    roofline = {"kernel": dom, "bound": K["bound"], "achieved": round(K["achieved"], 4),
                "peak": K["peak"], "unit": K["unit"], "frac": round(K["frac"], 5),
                "traffic": kernels[dom]["hbm_bytes_per_step_measured"]}

    value = points * steps / (ms_total * 1e-3)
    res = {
        "metric": "channel-points fitted/sec (4-bit)",
        "value": round(value, 1),
        "unit": "channel-points/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wk.name, "layers": nl, "channels": wk.channels,
                   "weights": wk.weights, "bits": wk.bits, "max_points": wk.max_points,
                   "n_grid": wk.n_grid, "tol": wk.tol, "calib_columns": wk.n_calib,
                   "points_per_step": points, "parallelism": "none"},
        "roofline": roofline,
        "kernels": {k: {kk: (round(vv, 5) if isinstance(vv, float) else vv) for kk, vv in v.items()}
                    for k, v in kernels.items()},
        "wall_s_timed": round(wall, 3),
    }

    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wk, args.cpu_stride)
    print(json.dumps(res), flush=True)
    return 0


def cpu_baseline(wk, stride):
    """The fp64 oracle, as it stands, on every stride-th channel of every layer."""
    import numpy as np

    import oracle
    from paper_2002_09049_amd import workloads as wl
    orc = oracle.load()
    cores = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    pts = 0
    secs = 0.0
    for li in range(len(wk.layers)):
        W = np.ascontiguousarray(wl.layer_weights(wk, li)[::stride])
        t0 = time.perf_counter()
        _, _, counts, _ = orc.fit(W, wk.bits, wk.max_points, wk.n_grid, float(np.float32(wk.tol)),
                                  n_threads=cores)
        secs += time.perf_counter() - t0
        pts += int(counts.sum())
    return {"value": round(pts / secs, 2), "unit": "channel-points/s", "cores": cores,
            "kind": "oracle",
            "sample": f"every {stride}th channel of each of the {len(wk.layers)} layers of {wk.name} "
                      f"({pts} channel-points, {secs:.1f} s wall)"}


if __name__ == "__main__":
    sys.exit(main())
