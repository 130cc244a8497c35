#!/usr/bin/env python3
"""Throughput of the multipoint-quantization hot path on one MI355X.

One step = the whole path over one synthetic workload already resident in
HBM: for every layer, the greedy fit, the output error on the layer's
calibration batch and the reconstruction, in one mpq_quantize_layers call
(--separate: mpq_fit_layers, mpq_output_error_layers, mpq_reconstruct_layers
in turn, with the time of each stage).  The default workload is the largest
4-bit one, the ResNet-50-shaped stack (54 layers, 27,560 channels, 4 bits,
up to 8 points, 256 candidate scales, tol 1e-3, 1,024 calibration columns);
--workload names the others (conv64x576, resnet18, mobilenetv2, vgg16fc).

--rule calib times the path with Algorithm 2's stopping rule on the
calibration batch instead (mpq_fit_layers_calib, whose per-point output
errors are the scoring, then mpq_reconstruct_layers); tol is then the
relative threshold eps.

--deploy times the deployment arithmetic of Sec. 3.4 instead: after the fit
(untimed) and the integer scales A_i = [2^p a_i] (off-line, as the paper
does it), one step is the integer forward of every layer (Eq. (15): int8
MFMA point products, the A_i-weighted 64-bit sum, the shift) on a batch of
synthetic int8 activations of the layer's real size for --images 224 x 224
images (N = images x output positions); value is int8 OP/s (2 per
multiply-add of the points actually used).

Prints one JSON line.  `value` is channel-points fitted per second over the
whole step (sum of the per-channel point counts of all layers / step time).
An untimed profile step first times every kernel launch by HIP events that
the library records on the launch's own stream (mpq_timing_enable); the
timed steps then carry events around the error GEMM's launches only.
`roofline` is the error GEMM (the path's one dense contraction: fp32 products
of Eq. (12) from six bf16 piece products each, on bf16 MFMA), timed in the
timed steps, against the dense bf16 MFMA peak; `kernels` lists every kernel.  The fit kernels'
`dense_equivalent_tflops` prices their candidate search at 7 FLOP per
(element, candidate) pair, the work a dense evaluation of Eq. (9) does; the
histogram search does O(d M + G) per step instead, so that figure is not an
instruction rate and is kept out of any fraction of peak.  `search` carries
the rocprofv3 counter figures of the longest fit kernel (VALU FLOP rates,
VALU-busy and wait shares, HBM bytes) when a stored counter summary of this
workload matches the current kernel sources.  `cpu_baseline` times the fp64
CPU oracle on a sample of the same workload, on all host cores and on one.
"""
from __future__ import annotations

import argparse
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
PEAK_MFMA_BF16_TFLOPS = 2500.0          # dense bf16 MFMA
GEMM_PIECE_PRODUCTS = 6                 # bf16 products per fp32 product of the error GEMM
PEAK_VALU_F32_TFLOPS = 157.3            # published (packed) FP32 vector peak
PEAK_MFMA_I8_TOPS = 5000.0              # dense int8 MFMA
PEAK_VALU_F32_NONPACKED_TFLOPS = 78.6   # 256 CU x 64 lanes x 2 FLOP x 2.4 GHz
FLOP_PER_EVAL = 7                       # scale-mul, round, clamp, fma (2), square-acc fma (2)

PROFILES = os.path.join(ROOT, "profiles")
ROOFLINE_KERNEL = "gemm_err_kernel"
COPY_BYTES = 256 << 20
STAGES = (("fit", ("fit_hist_kernel", "fit_small_kernel", "fit_dense_kernel")),
          ("output_error", ("form_d_kernel", "gemm_err_kernel", "finish_err_kernel")),
          ("reconstruct", ("reconstruct_kernel",)),
          ("deploy", ("int_forward_kernel", "integer_scales_kernel")))


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="resnet50")
    ap.add_argument("--cpu-stride", type=int, default=1,
                    help="cpu_baseline fits every n-th channel of every layer")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--dense", action="store_true",
                    help="fit with mpq_fit_layer_dense (O(d G) search) instead of mpq_fit_layer "
                         "(implies --separate)")
    ap.add_argument("--rule", choices=("tol", "calib"), default="tol",
                    help="stopping rule: ||r||^2 <= tol ||w||^2 (default), or Algorithm 2's on the "
                         "calibration batch (output error <= tol x that of W)")
    ap.add_argument("--deploy", action="store_true",
                    help="time the integer forward of Sec. 3.4 (Eq. (15)) of every layer instead")
    ap.add_argument("--images", type=int, default=8,
                    help="--deploy: images of 224 x 224 in the activation batch")
    ap.add_argument("--shift", type=int, default=16, help="--deploy: p of Eq. (14)")
    ap.add_argument("--refit", action="store_true",
                    help="least-squares refit of each point's scale (mpq_fit_layers_ex; implies "
                         "--separate for the isotropic rule)")
    ap.add_argument("--clip", type=int, default=0, metavar="GC",
                    help="point 1 from the clipping of Eq. (13) with GC factors (the paper: 20; "
                         "mpq_fit_layers_ex; implies --separate for the isotropic rule)")
    ap.add_argument("--asym", action="store_true",
                    help="asymmetric per-channel codes (offset + points; mpq_fit_layers_ex; implies "
                         "--separate)")
    ap.add_argument("--paper-eta", type=float, default=0.0, metavar="ETA",
                    help="fit on the paper's own grid of Eq. (11) with maximal step ETA (the paper: "
                         "2^-10 = 0.0009765625; mpq_fit_layers_ex; implies --separate)")
    ap.add_argument("--separate", action="store_true",
                    help="the three batched calls in turn instead of mpq_quantize_layers")
    ap.add_argument("--summarize-counters", nargs="+", metavar="PMC_DIR",
                    help="print the per-kernel counter summary of rocprofv3 --pmc runs (one per "
                         "counter pass) of `bench.py --workload W --steps 1 --warmup 1 "
                         "--no-cpu-baseline --copy-calibration` and exit")
    ap.add_argument("--summarize-benches", nargs="+", metavar="BENCH_JSON",
                    help="print a markdown table of bench.py lines (one per workload)")
    ap.add_argument("--summarize-trace", metavar="TRACE_DIR",
                    help="print the per-kernel summary of a rocprofv3 --kernel-trace --stats run "
                         "and exit")
    ap.add_argument("--bench-json", metavar="FILE",
                    help="with --summarize-trace: the bench.py line of an untraced run of the "
                         "same build, compared kernel by kernel")
    ap.add_argument("--traced-steps", type=int, default=None,
                    help="with --summarize-*: steps the traced process ran (warm-up, profile "
                         "step and timed; default 3 for --summarize-counters; for --summarize-trace "
                         "those of the --bench-json line, which has no profile step with --deploy)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="before the steps, copy a 256 MiB device buffer once (a kernel of known "
                         "traffic, to scale the FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


def sources_digest():
    """sha256 of the HIP sources without their comments and blank space, to
    tell whether stored counters still apply to the kernels."""
    import glob
    import hashlib
    import re
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2002_09049_amd", "csrc", "*"))):
        with open(f, encoding="utf-8") as fh:
            code = re.sub(r"/\*.*?\*/", " ", fh.read(), flags=re.S)
        code = re.sub(r"//[^\n]*", " ", code)
        code = " ".join(code.split())
        h.update(os.path.basename(f).encode() + b"\0" + code.encode())
    return h.hexdigest()[:16]


def kernel_key(profiler_name):
    """The library's timing name of a kernel from the demangled name rocprofv3
    prints (fit_hist_kernel<T, EPT, kLinear, kLat, kGlobal> ->
    fit_hist_kernel<T,EPT,mode[,rebuilt]>; fit_small_kernel<d>)."""
    m = re.search(r"fit_hist_kernel<(\d+), (\d+), (true|false), (true|false), (true|false)>",
                  profiler_name)
    if m:
        mode = "lattice" if m.group(4) == "true" else "linear" if m.group(3) == "true" else "grid"
        rebuilt = ",rebuilt" if m.group(5) == "true" else ""
        return f"fit_hist_kernel<{m.group(1)},{m.group(2)},{mode}{rebuilt}>"
    m = re.search(r"fit_small_kernel<(\d+)>", profiler_name)
    if m:
        return f"fit_small_kernel<{m.group(1)}>"
    m = re.search(r"int_forward_kernel<(\d)(, \d+)?>", profiler_name)
    if m:
        return f"int_forward_kernel<{(16, 4, 1)[int(m.group(1))]}>"
    m = re.search(r"(\w+_kernel)\b", profiler_name)
    return m.group(1) if m else None


def stage_of(key):
    for stage, names in STAGES:
        if key and any(key.startswith(n) for n in names):
            return stage
    return None


COUNTER_PASSES = (
    ("SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_ACTIVE_INST_VALU", "SQ_INSTS_VALU",
     "SQ_INSTS_LDS", "SQ_WAIT_INST_LDS", "SQ_BUSY_CYCLES"),
    ("SQ_INSTS_VALU_FLOPS_FP32", "SQ_INSTS_VALU_FLOPS_FP32_TRANS", "SQ_INSTS_VALU_FLOPS_FP64",
     "SQ_INSTS_VALU_FLOPS_FP64_TRANS", "SQ_INSTS_VALU_IOPS", "SQ_VALU_MFMA_BUSY_CYCLES",
     "SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_BUSY_CU_CYCLES"),
    ("FETCH_SIZE",),
    ("WRITE_SIZE",),
)
PEAK_VALU_F64_TFLOPS = 78.6
CAL_MULS = 1 << 24   # multiplies of each known-FLOP calibration kernel


def counters_path(workload):
    return os.path.join(PROFILES, f"{workload}_counters.md")


def summarize_counters(dirs, workload, steps=3):
    """Per-kernel figures of rocprofv3 --pmc runs of `bench.py --workload W
    --steps 1 --warmup 1 --no-cpu-baseline --copy-calibration` (one run per
    pass of COUNTER_PASSES): counters averaged per dispatch, the dispatch's
    own duration (counter runs serialize the dispatches), and derived rates.
    FETCH_SIZE and WRITE_SIZE (KiB) are scaled so that the 256 MiB
    calibration copy reads and writes 256 MiB."""
    import csv
    import glob

    per = {}        # kernel -> counter -> [sum, n]
    dur = {}        # kernel -> [sum ns, n]
    launches = {}   # kernel -> dispatches in the run (largest over the passes)
    scale = {}
    for d in dirs:
        rows = []
        for f in glob.glob(os.path.join(d, "*counter_collection.csv")):
            rows += list(csv.DictReader(open(f)))
        if not rows:
            raise SystemExit(f"no counter_collection.csv in {d}")
        names = {r["Counter_Name"] for r in rows}
        for c in ("FETCH_SIZE", "WRITE_SIZE"):
            if c in names:
                cal = [r for r in rows if "copyBuffer" in r["Kernel_Name"] and r["Counter_Name"] == c
                       and int(r["Grid_Size"]) == 131072]
                if not cal:
                    raise SystemExit(f"no calibration copy in {d}")
                scale[c] = COPY_BYTES / 1024.0 / float(cal[0]["Counter_Value"])
        # the FLOP counters against the multiply kernels of known work
        for c, ty in (("SQ_INSTS_VALU_FLOPS_FP64", "double"), ("SQ_INSTS_VALU_FLOPS_FP32", "float")):
            if c in names:
                cal = [r for r in rows if r["Counter_Name"] == c and f"MulFunctor<{ty}>" in r["Kernel_Name"]]
                if cal and float(cal[0]["Counter_Value"]) > 0:
                    scale[c] = CAL_MULS / float(cal[0]["Counter_Value"])
        seen = {}
        for r in rows:
            k = kernel_key(r["Kernel_Name"])
            if not stage_of(k):
                continue
            c = r["Counter_Name"]
            a = per.setdefault(k, {}).setdefault(c, [0.0, 0])
            a[0] += float(r["Counter_Value"])
            a[1] += 1
            did = r["Dispatch_Id"]
            if (k, did) not in seen:
                seen[(k, did)] = 1
                t = dur.setdefault(k, [0.0, 0])
                t[0] += float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
                t[1] += 1
        cnt = {}
        for k, _ in seen:
            cnt[k] = cnt.get(k, 0) + 1
        for k, v in cnt.items():
            launches[k] = max(launches.get(k, 0), v)
    out = {}
    for k, cs in per.items():
        avg = {c: v[0] / v[1] for c, v in cs.items()}
        us = dur[k][0] / dur[k][1] / 1e3
        f = {"launches_per_step": launches[k] / steps, "avg_us_serialized": us}
        for c in ("FETCH_SIZE", "WRITE_SIZE"):
            if c in avg:
                f[c.lower() + "_bytes"] = avg[c] * scale[c] * 1024.0
        if "fetch_size_bytes" in f and "write_size_bytes" in f:
            f["hbm_bytes"] = f["fetch_size_bytes"] + f["write_size_bytes"]
            f["hbm_gbs"] = f["hbm_bytes"] / us / 1e3
        if "SQ_WAVE_CYCLES" in avg and avg["SQ_WAVE_CYCLES"] > 0:
            f["valu_active_share"] = avg.get("SQ_ACTIVE_INST_VALU", 0.0) / avg["SQ_WAVE_CYCLES"]
            f["wait_any_share"] = avg.get("SQ_WAIT_ANY", 0.0) / avg["SQ_WAVE_CYCLES"]
            f["lds_wait_share"] = avg.get("SQ_WAIT_INST_LDS", 0.0) / avg["SQ_WAVE_CYCLES"]
        if "SQ_INSTS_VALU_FLOPS_FP32" in avg:
            # counts scaled by what they read for the known-FLOP multiplies
            # (the fp64 factor also for fp32 when that one is missing)
            s64 = scale.get("SQ_INSTS_VALU_FLOPS_FP64", 1.0)
            s32 = scale.get("SQ_INSTS_VALU_FLOPS_FP32", s64)
            f32 = (avg["SQ_INSTS_VALU_FLOPS_FP32"] + avg.get("SQ_INSTS_VALU_FLOPS_FP32_TRANS", 0.0)) * s32
            f64 = (avg.get("SQ_INSTS_VALU_FLOPS_FP64", 0.0) + avg.get("SQ_INSTS_VALU_FLOPS_FP64_TRANS", 0.0)) * s64
            f["valu_fp32_tflops"] = f32 / us / 1e6
            f["valu_fp32_frac"] = f["valu_fp32_tflops"] / PEAK_VALU_F32_TFLOPS
            f["valu_fp64_tflops"] = f64 / us / 1e6
            f["valu_fp64_frac"] = f["valu_fp64_tflops"] / PEAK_VALU_F64_TFLOPS
            f["valu_iops_tops"] = avg.get("SQ_INSTS_VALU_IOPS", 0.0) / us / 1e6
        if "SQ_VALU_MFMA_BUSY_CYCLES" in avg and avg.get("SQ_BUSY_CU_CYCLES", 0) > 0:
            f["mfma_busy_per_cu_busy"] = avg["SQ_VALU_MFMA_BUSY_CYCLES"] / (4 * avg["SQ_BUSY_CU_CYCLES"])
        if "SQ_ACTIVE_INST_VALU" in avg and avg.get("SQ_BUSY_CU_CYCLES", 0) > 0:
            # each VALU wave-instruction holds its SIMD's VALU for 4 cycles
            # (SQ_ACTIVE_INST_VALU counts them in those 4-cycle units) and a
            # CU has 4 SIMDs: the SIMDs' VALU issue share of the busy cycles
            f["valu_busy_per_cu_busy"] = avg["SQ_ACTIVE_INST_VALU"] / avg["SQ_BUSY_CU_CYCLES"]
        f["counters"] = {c: round(v, 1) for c, v in sorted(avg.items())}
        out[k] = f

    def fmt(v, spec):
        return "" if v is None else format(v, spec)

    cmds = [f"rocprofv3 --pmc {' '.join(cs)} --output-format csv -d gpurun_out/pmc_{workload}_{i} -o p -- \\\n"
            f"    python3 bench.py --workload {workload} --steps 1 --warmup 1 --no-cpu-baseline --copy-calibration"
            for i, cs in enumerate(COUNTER_PASSES)]
    lines = [f"# Counters per kernel: {workload} workload, bench step", "",
             "One rocprofv3 counter run per pass (from the repository root; each run holds "
             f"{steps} steps: warm-up, profile and timed), then the summary:", "", "```", *cmds,
             f"python3 bench.py --workload {workload} --summarize-counters "
             + " ".join(f"gpurun_out/pmc_{workload}_{i}" for i in range(len(COUNTER_PASSES))),
             "```", "",
             "Per dispatch.  Counter runs serialize the dispatches, so `us` is the kernel alone.",
             "FETCH_SIZE / WRITE_SIZE are scaled by a 256 MiB device copy "
             f"(x {scale.get('FETCH_SIZE', float('nan')):.4f}, x {scale.get('WRITE_SIZE', float('nan')):.4f});",
             f"the FLOP counters by {CAL_MULS} fp64 and fp32 multiplies (torch) of the same run "
             f"(x {scale.get('SQ_INSTS_VALU_FLOPS_FP64', float('nan')):.4f} fp64, "
             f"x {scale.get('SQ_INSTS_VALU_FLOPS_FP32', float('nan')):.4f} fp32).",
             "VALU-active and wait shares are SQ_ACTIVE_INST_VALU and SQ_WAIT_ANY over SQ_WAVE_CYCLES",
             "(per wave); SIMD VALU busy is SQ_ACTIVE_INST_VALU (in 4-cycle issue units) over",
             "SQ_BUSY_CU_CYCLES (4 SIMDs per CU): the share of the SIMDs' VALU issue capacity used;",
             "FLOP rates are SQ_INSTS_VALU_FLOPS_FP32 (+ _TRANS) and _FP64 over the dispatch's duration,",
             f"against {PEAK_VALU_F32_TFLOPS} (FP32) and {PEAK_VALU_F64_TFLOPS} (FP64) TFLOP/s.", "",
             "| kernel | launches/step | us | HBM MB | HBM GB/s | SIMD VALU busy | VALU active | wait | FP32 TFLOP/s (frac) | FP64 TFLOP/s (frac) | INT TOP/s | MFMA busy |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for k in sorted(out, key=lambda k: -out[k]["avg_us_serialized"] * out[k]["launches_per_step"]):
        f = out[k]
        hb = f.get("hbm_bytes")
        lines.append(
            f"| `{k}` | {f['launches_per_step']:g} | {f['avg_us_serialized']:.1f} | "
            f"{fmt(None if hb is None else hb / 1e6, '.1f')} | {fmt(f.get('hbm_gbs'), '.0f')} | "
            f"{fmt(f.get('valu_busy_per_cu_busy'), '.1%')} | "
            f"{fmt(f.get('valu_active_share'), '.1%')} | {fmt(f.get('wait_any_share'), '.1%')} | "
            + ("" if "valu_fp32_tflops" not in f else
               f"{f['valu_fp32_tflops']:.2f} ({f['valu_fp32_frac']:.1%}) | "
               f"{f['valu_fp64_tflops']:.2f} ({f['valu_fp64_frac']:.1%}) | {f['valu_iops_tops']:.2f} | ")
            + ("| | | " if "valu_fp32_tflops" not in f else "")
            + f"{fmt(f.get('mfma_busy_per_cu_busy'), '.1%')} |")
    lines += ["", "counters-json: " + json.dumps(out, sort_keys=True), "",
              f"sources: {sources_digest()}", ""]
    print("\n".join(lines))


def stored_counters(workload):
    """The per-kernel counter figures of profiles/<workload>_counters.md, or
    None when it is missing or was taken on other kernel sources."""
    try:
        text = open(counters_path(workload)).read()
    except OSError:
        return None
    if f"sources: {sources_digest()}" not in text:
        return None
    for ln in text.splitlines():
        if ln.startswith("counters-json: "):
            return json.loads(ln[len("counters-json: "):])
    return None


def _stride_of(bench):
    """The CPU-sample stride of a bench line's cpu_baseline (from its sample text)."""
    sample = (bench.get("cpu_baseline") or {}).get("sample", "")
    if "every channel" in sample:
        return 1
    m = re.search(r"every (\d+)th channel", sample)
    return int(m.group(1)) if m else "-"


def summarize_benches(paths):
    """Markdown table of bench.py lines: rate, step time, the GEMM's roofline
    and HBM traffic, the longest fit, the search kernel's SIMD VALU busy
    share (from its stored counters) and the oracle's rate."""
    rows = [json.load(open(p)) for p in paths]
    lines = ["# Bench line per workload (one MI355X, one mpq_quantize_layers call per step)", "",
             "Commands (from the repository root), per workload W and CPU-sample stride S, then the table:",
             "", "```", "python3 bench.py --workload W --cpu-stride S > gpurun_out/wl/W.json",
             "python3 bench.py --summarize-benches " + " ".join(f"gpurun_out/wl/{b['config']['workload']}.json"
                                                                for b in rows),
             "```", "",
             "Strides: " + ", ".join(f"{b['config']['workload']} {_stride_of(b)}" for b in rows)
             + f"; {rows[0]['steps'] if rows else 0} timed steps after {rows[0]['warmup'] if rows else 0} "
               "warm-up steps.",
             "The roofline kernel is the error GEMM (6 x 2 C d n bf16 FLOP per layer against the dense bf16",
             "MFMA peak; fp32 equivalent: 2 C d n; event-timed in the timed steps);",
             "the other kernels are timed in the untimed profile step, where the fit launches share the",
             "device (so a fit's duration includes its neighbours).  `search` is the fit kernel with the",
             "most time per step; its SIMD VALU busy share (the share of the SIMDs' VALU issue capacity it",
             "used, SQ_ACTIVE_INST_VALU over SQ_BUSY_CU_CYCLES) and the GEMM's HBM traffic come from the",
             "stored counter summary `profiles/<workload>_counters.md` of the same sources.", "",
             "| workload | channel-points/s | ms/step | points/step | GEMM (roofline) | GEMM HBM traffic | "
             "longest fit | search SIMD VALU busy | oracle (cores) |",
             "|---|---:|---:|---:|---|---:|---|---:|---:|"]
    tops = []
    for b in rows:
        w = b["config"]["workload"]
        r = b["roofline"]
        fits = {k: v for k, v in b["kernels"].items() if v.get("stage") == "fit"}
        lf = max(fits.items(), key=lambda kv: kv[1]["us_per_step"])
        cb = b.get("cpu_baseline") or {}
        srch = b.get("search") or {}
        vb = (srch.get("counters") or {}).get("valu_busy_per_cu_busy")
        tr = r.get("traffic")
        lines.append(
            f"| {w} | {b['value'] / 1e6:.2f} M | {b['ms_per_step']:.3f} | {b['config']['points_per_step']} | "
            f"{r['achieved']:.1f} TFLOP/s ({100 * r['frac']:.0f}% of {r['peak']:g}), {r['avg_launch_us']:.1f} us | "
            + ("-" if tr is None else f"{tr / 1e6:.0f} MB") + " | "
            f"`{lf[0]}` {lf[1]['avg_us']:.1f} us | "
            + ("-" if vb is None else f"{100 * vb:.1f}%") + f" (`{srch.get('kernel')}`) | "
            f"{cb.get('value', 0) / 1e3:.2f} k ({cb.get('cores')}) |")
        tops.append((w, sorted(b["kernels"].items(), key=lambda kv: -kv[1]["us_per_step"])[:5]))
    lines += ["", "Top kernels per workload (microseconds per launch, launches per step):", ""]
    for w, ks in tops:
        lines.append(f"- **{w}**: " + "; ".join(f"`{k}` x{v['launches_per_step']:g} {v['avg_us']:.1f}"
                                                for k, v in ks))
    print("\n".join(lines))


def summarize_trace(trace_dir, bench_json=None, steps=None, rule="tol", workload="resnet50"):
    """Per-kernel average duration of a traced bench run (kernel_stats.csv of
    rocprofv3 --stats), beside the event-timed averages of a bench.py line
    whose --steps / --warmup the traced run used too (steps: the steps the
    traced run held, by default those of the bench line)."""
    import csv
    import glob

    files = glob.glob(os.path.join(trace_dir, "*kernel_stats.csv"))
    if not files:
        raise SystemExit(f"no kernel_stats.csv in {trace_dir}")
    rows = list(csv.DictReader(open(files[0])))
    agg = {}
    for r in rows:
        k = kernel_key(r["Name"])
        if not stage_of(k):
            continue
        if rule == "deploy" and not k.startswith("int_forward_kernel"):
            continue   # the fit and the scales are untimed set-up
        a = agg.setdefault(k, [0, 0.0])
        a[0] += int(r["Calls"])
        a[1] += float(r["TotalDurationNs"])
    bench = json.load(open(bench_json)) if bench_json else None
    K, W = (bench["steps"], bench["warmup"]) if bench else (5, 1)
    if steps is None:
        steps = W + K + (0 if rule == "deploy" else 1)   # deploy has no profile step
    calib = rule == "calib"
    r = {"calib": " --rule calib", "deploy": " --deploy"}.get(rule, "")
    what = {"calib": "the fit with Algorithm 2's stopping rule on each layer's calibration batch (one point\n"
                     "per step, each step scored on the batch; relative threshold 1e-3) and the\n"
                     "reconstruction, through mpq_fit_layers_calib and mpq_reconstruct_layers.",
            "deploy": "the integer forward of Eq. (15) of every layer (fitted codes, integer scales with\n"
                      "p = 16) on int8 activations of 8 images of 224 x 224 (N = 8 x output positions),\n"
                      "through mpq_integer_forward_layers; the fit and the scales are untimed set-up."
            }.get(rule, "fit + output error + reconstruction of every layer through the batched C ABI calls.")
    from paper_2002_09049_amd import workloads as wl
    wk = wl.get(workload)
    r = f" --workload {workload}" + r
    lines = [f"# rocprofv3 kernel summary: {workload} workload, bench step{r}", "",
             f"Workload: {len(wk.layers)} layers ({wk.channels:,} channels, {wk.weights:,} weights), "
             f"{wk.bits} bits, up to {wk.max_points} points,",
             f"{wk.n_grid} candidate scales, tol {wk.tol:g}, calibration batches d x {wk.n_calib}.  One step =",
             what, "",
             "Commands (one MI355X, from the repository root):", "", "```",
             "rocprofv3 --kernel-trace --stats --output-format csv -d gpurun_out/prof -o kt -- \\",
             f"    python3 bench.py{r} --steps {K} --warmup {W}" + ("" if rule == "deploy" else " --no-cpu-baseline"),
             f"python3 bench.py{r} --steps {K} --warmup {W} > gpurun_out/bench.json",
             f"python3 bench.py{r} --summarize-trace gpurun_out/prof --bench-json gpurun_out/bench.json",
             "```", "",
             f"The traced process ran {steps} steps ({W} warm-up" + ("" if rule == "deploy" else ", 1 profile")
             + f", {K} timed).  Kernels of one stage may",
             "run concurrently on several streams.  `bench avg us` is the untraced run's average",
             "per launch, timed by HIP events on the launch's own stream.", "",
             "| kernel | stage | launches/step | avg us (rocprofv3) | bench avg us | us/step |",
             "|---|---|---:|---:|---:|---:|"]
    bk = (bench or {}).get("kernels", {})
    for k in sorted(agg, key=lambda k: -agg[k][1]):
        calls, tot = agg[k]
        b = bk.get(k, {}).get("avg_us")
        lines.append(f"| `{k}` | {stage_of(k)} | {calls / steps:g} | {tot / calls / 1e3:.2f} | "
                     f"{'' if b is None else f'{b:.2f}'} | {tot / steps / 1e3:.2f} |")
    lines += ["", f"sources: {sources_digest()}", ""]
    if bench:
        lines += ["bench.py line of the same build (untraced run):", "", "```",
                  json.dumps({k: bench[k] for k in ("value", "unit", "ms_per_step", "roofline")}),
                  "```", ""]
    print("\n".join(lines))


def main():
    args = parse()
    if args.summarize_counters:
        summarize_counters(args.summarize_counters, args.workload, steps=args.traced_steps or 3)
        return 0
    if args.summarize_benches:
        summarize_benches(args.summarize_benches)
        return 0
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.bench_json, steps=args.traced_steps,
                        rule="deploy" if args.deploy else args.rule, workload=args.workload)
        return 0
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the fit has no cross-GPU step to measure)", file=sys.stderr, flush=True)
        return 2
    import numpy as np
    import torch

    from paper_2002_09049_amd import mpq, workloads as wl

    assert torch.cuda.is_available(), "bench.py needs a ROCm GPU"
    if args.deploy:
        return deploy_main(args)
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
        # kernels of known VALU work for the FLOP counters: 2^24 fp64 and
        # 2^24 fp32 multiplies (one FLOP each)
        x64 = torch.full((CAL_MULS,), 1.5, dtype=torch.float64, device=dev)
        y64 = x64 * x64
        x32 = torch.full((CAL_MULS,), 1.5, dtype=torch.float32, device=dev)
        y32 = x32 * x32
        torch.cuda.synchronize()
        del src, dst, x64, y64, x32, y32

    separate = (args.separate or args.dense or args.paper_eta > 0
                or ((args.refit or args.clip or args.asym) and args.rule != "calib"))
    calib = args.rule == "calib"
    if calib and separate:
        raise SystemExit("--rule calib has its own call sequence (no --separate / --dense)")

    def step(ev=None):
        if calib:
            if args.refit or args.clip or args.asym:
                ls.fit_ex(wk.bits, wk.n_grid, refit=args.refit, calib=True, eps=wk.tol, relative=True,
                          clip_grid=args.clip, asym=args.asym)
            else:
                ls.fit_calib(wk.bits, wk.n_grid, wk.tol, True)
            ls.reconstruct()
            return
        if not separate:
            ls.quantize(wk.bits, wk.n_grid, wk.tol)
            return
        if ev: ev[0].record(stream)
        if args.dense:
            for i, W in enumerate(Ws):
                mpq.fit_layer(W, wk.bits, wk.max_points, wk.n_grid, wk.tol, dense=True,
                              out=(ls.codes[i], ls.scales[i], ls.counts[i], ls.fit_err[i]))
        elif args.paper_eta > 0:
            ls.fit_ex(wk.bits, 1, wk.tol, paper_eta=args.paper_eta)
        elif args.refit or args.clip or args.asym:
            ls.fit_ex(wk.bits, wk.n_grid, wk.tol, refit=args.refit, clip_grid=args.clip, asym=args.asym)
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

    # ---- algorithmic work per kernel and step
    fit_kernel = {}
    work = {}   # kernel -> dict of per-step work figures

    def add(k, **kv):
        w = work.setdefault(k, {})
        for a, b in kv.items():
            w[a] = w.get(a, 0) + b

    points = 0
    count_hist = np.zeros(wk.max_points + 1, np.int64)
    for i, W in enumerate(Ws):
        C, d = W.shape
        cnt = ls.counts[i].cpu().numpy().astype(np.int64)
        count_hist += np.bincount(cnt, minlength=wk.max_points + 1)
        n = int(cnt.sum())
        N = Xs[i].shape[1]
        points += n
        fk = "fit_dense_kernel" if args.dense else fit_kernel.setdefault(
            d, mpq.fit_kernel_of(d, wk.bits, wk.n_grid, True))
        if args.paper_eta > 0:
            fk = "fit_paper_kernel"   # no algorithmic count: its candidates depend on the data
        if calib:
            # step s scores the channels that took point s + 1 (sum of counts
            # rows in all), plus W itself once for the relative threshold;
            # a fit step re-reads W and the codes of the points so far
            code_reads = int((cnt * (cnt - 1) // 2).sum())
            searched = n - int((cnt > 0).sum()) if args.clip else n
            add(fk, evals=searched * wk.n_grid * d, bytes=4 * n * d + code_reads * d + n * d)
            add("gemm_err_kernel", flop=2 * (n + C) * d * N)
            add("form_d_kernel", bytes=8 * (n + C) * d + (n + code_reads) * d)
        else:
            # fit: G candidate errors per (element, point); reads W once, writes the codes
            # (with --clip, point 1 comes from the clipping pass, not the search);
            # in the whole-path call the fit also writes the rows of D (fp32),
            # and no forming runs for them
            searched = n - int((cnt > 0).sum()) if args.clip else n
            fit_writes_d = not separate and not args.dense
            add(fk, evals=searched * wk.n_grid * d, bytes=4 * C * d + n * d + (4 * C * d if fit_writes_d else 0))
            add("gemm_err_kernel", flop=2 * C * d * N)
            # form: reads W and the codes of the used points, writes D
            if not fit_writes_d:
                add("form_d_kernel", bytes=4 * C * d + n * d + 4 * C * d)
        if args.clip:
            # the clipping pass: output errors of C * GC candidate rows
            add("gemm_err_kernel", flop=2 * C * args.clip * d * N)
            add("form_d_kernel", bytes=4 * C * d + 4 * C * args.clip * d)
        # reconstruct: reads the codes of the used points, writes fp32
        add("reconstruct_kernel", bytes=n * d + 4 * C * d)

    def kernel_table(launches, nsteps):
        per = {}
        for name, ms in launches:
            p = per.setdefault(name, [0, 0.0])
            p[0] += 1
            p[1] += ms
        kernels = {}
        for name, (cnt, tot) in per.items():
            avg_s = tot / cnt * 1e-3
            k = {"stage": stage_of(name), "launches_per_step": cnt / nsteps,
                 "avg_us": tot / cnt * 1e3, "us_per_step": tot / nsteps * 1e3}
            w = work.get(name, {})
            lps = cnt / nsteps
            if "evals" in w:
                # the histogram search does O(d M + G) per channel-step: the
                # dense-equivalent rate is what a dense evaluation of Eq. (9)
                # would have to sustain, not an instruction rate (no frac)
                ev_launch = w["evals"] / lps
                k.update({"unit": "TFLOP/s", "candidate_evals_per_launch": ev_launch,
                          "dense_equivalent_tflops": FLOP_PER_EVAL * ev_launch / avg_s / 1e12,
                          "bytes_per_launch": w["bytes"] / lps,
                          "hbm_gbs_algorithmic": w["bytes"] / lps / avg_s / 1e9,
                          "hbm_frac_algorithmic": w["bytes"] / lps / avg_s / 1e9 / PEAK_HBM_GBS})
            elif "flop" in w:
                # w["flop"]: 2 C d n, the fp32 products of Eq. (12); the GEMM
                # runs each as GEMM_PIECE_PRODUCTS bf16 products on the matrix cores
                bf = GEMM_PIECE_PRODUCTS * w["flop"] / lps
                k.update({"bound": "mfma", "unit": "TFLOP/s", "peak": PEAK_MFMA_BF16_TFLOPS,
                          "flop_per_launch": bf, "achieved": bf / avg_s / 1e12,
                          "fp32_equivalent_tflops": w["flop"] / lps / avg_s / 1e12})
            elif "bytes" in w:
                k.update({"bound": "hbm", "unit": "GB/s", "peak": PEAK_HBM_GBS,
                          "bytes_per_launch": w["bytes"] / lps, "achieved": w["bytes"] / lps / avg_s / 1e9})
            if "achieved" in k:
                k["frac"] = k["achieved"] / k["peak"]
            c = (counters or {}).get(name)
            if c:
                k["counters"] = {kk: c[kk] for kk in (
                    "hbm_bytes", "avg_us_serialized", "valu_busy_per_cu_busy", "valu_active_share",
                    "wait_any_share",
                    "valu_fp32_tflops", "valu_fp32_frac", "valu_fp64_tflops", "valu_fp64_frac",
                    "valu_iops_tops", "mfma_busy_per_cu_busy") if kk in c}
            kernels[name] = k
        return kernels

    counters = stored_counters(wk.name)

    # profile step (untimed): every launch between HIP events, to rank the
    # kernels; then the timed steps carry events around the dominant kernel
    # only, so the instrumentation barely touches the timed region
    mpq.timing_only(None)
    mpq.timing_enable(True)
    step()
    torch.cuda.synchronize()
    kernels = kernel_table(mpq.timing_read(), 1)
    mpq.timing_enable(False)
    for k in kernels.values():
        k["timed_in"] = "profile step"
    # the roofline kernel: the error GEMM (the path's one dense contraction);
    # a step without it (none here) would take the longest-running kernel
    dom = ROOFLINE_KERNEL if ROOFLINE_KERNEL in kernels else \
        max(kernels, key=lambda k: kernels[k]["us_per_step"])

    nl = len(Ws)
    ev = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(4)) for _ in range(args.steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    mpq.timing_only(dom)
    mpq.timing_enable(True)
    wall0 = time.perf_counter()
    t_start.record(stream)
    for s in range(args.steps):
        step(ev[s])
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    launches = mpq.timing_read()
    mpq.timing_enable(False)
    mpq.timing_only(None)
    ms_total = t_start.elapsed_time(t_end)
    ms_step = ms_total / args.steps
    steps = args.steps
    kernels[dom] = kernel_table(launches, steps)[dom]
    kernels[dom]["timed_in"] = "timed region"
    stages = {}
    if separate:
        for i, st in enumerate(("fit", "output_error", "reconstruct")):
            stages[st] = sum(e[i].elapsed_time(e[i + 1]) for e in ev) / steps
    K = kernels[dom]
    traffic = (counters or {}).get(dom, {}).get("hbm_bytes")
    roofline = {"kernel": dom, "bound": K.get("bound"), "achieved": round(K.get("achieved", 0.0), 4),
                "peak": K.get("peak"), "unit": K.get("unit"), "frac": round(K.get("frac", 0.0), 5),
                "traffic": None if traffic is None else int(traffic),
                "avg_launch_us": round(K["avg_us"], 3),
                "fp32_equivalent_tflops": round(K.get("fp32_equivalent_tflops", 0.0), 4),
                "achieved_is": "6 x 2 C d n bf16 FLOP per layer (six bf16 piece products for each of "
                               "Eq. (12)'s fp32 products) / event-timed launch duration, against the "
                               "dense bf16 MFMA peak"}
    # the candidate search: the fit kernel with the most time per step, with
    # the counter figures of the stored summary (FP32 / FP64 VALU rates
    # against their peaks, VALU-active and wait shares, HBM bytes)
    fits = [k for k in kernels if stage_of(k) == "fit"]
    search = None
    if fits:
        fk = max(fits, key=lambda k: kernels[k]["us_per_step"])
        F = kernels[fk]
        search = {"kernel": fk, "avg_launch_us": round(F["avg_us"], 3),
                  "dense_equivalent_tflops": round(F.get("dense_equivalent_tflops", 0.0), 3),
                  "counters": F.get("counters"),
                  "counters_from": (os.path.relpath(counters_path(wk.name), ROOT)
                                    if F.get("counters") else None)}

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
        "dtype": "f64+f32+bf16",
        "data": "synthetic",
        "config": {"workload": wk.name, "layers": nl, "channels": wk.channels,
                   "weights": wk.weights, "bits": wk.bits, "max_points": wk.max_points,
                   "n_grid": wk.n_grid, "tol": wk.tol, "calib_columns": wk.n_calib,
                   "points_per_step": points, "search": "dense" if args.dense else "histogram",
                   "refit": bool(args.refit), "clip_grid": args.clip, "paper_eta": args.paper_eta,
                   "asym": bool(args.asym),
                   "rule": ("Algorithm 2 on the calibration batch, relative" if calib
                            else "||r||^2 <= tol ||w||^2"),
                   "point_counts": count_hist.tolist(),
                   "calls": ("mpq_fit_layers_calib + mpq_reconstruct_layers" if calib else
                             "separate" if separate else "mpq_quantize_layers"),
                   "parallelism": "none"},
        "roofline": roofline,
        "search": search,
        "stages_ms_per_step": {k: round(v, 5) for k, v in stages.items()} or None,
        "kernels": {k: {kk: (round(vv, 5) if isinstance(vv, float) else vv) for kk, vv in v.items()}
                    for k, v in sorted(kernels.items(), key=lambda kv: -kv[1]["us_per_step"])},
        "wall_s_timed": round(wall, 3),
    }

    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wk, args.cpu_stride, calib)
    print(json.dumps(res), flush=True)
    return 0


def deploy_main(args):
    """--deploy: the integer forward of Sec. 3.4 of every layer."""
    import numpy as np
    import torch

    from paper_2002_09049_amd import accounting as ac, mpq, workloads as wl

    wk = wl.get(args.workload)
    hw = {"resnet18": wl.resnet18_out_hw, "resnet50": wl.resnet50_out_hw}.get(wk.name)
    if hw is None:
        raise SystemExit("--deploy knows the output sizes of resnet18 and resnet50")
    hw = hw()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    Ws = [torch.from_numpy(wl.layer_weights(wk, li)).to(dev) for li in range(len(wk.layers))]
    ls = mpq.LayerSet(Ws, wk.max_points)
    ls.fit(wk.bits, wk.n_grid, wk.tol)
    p = args.shift
    As = []
    for i in range(len(Ws)):
        A, cl = mpq.integer_scales(ls.scales[i], ls.counts[i], p)
        As.append(A)
        assert int(cl.item()) == 0, "integer scales clamped: lower --shift"
    gen = torch.Generator(device=dev)
    gen.manual_seed(wk.seed)
    layers, macs = [], 0
    kmacs = {}   # useful multiply-adds per kernel (layers go to a kernel by their load width)
    counts = [ls.counts[i].cpu().numpy().astype(np.int64) for i in range(len(Ws))]
    for i, (C, d) in enumerate(wk.layers):
        N = args.images * hw[i] * hw[i]
        X = torch.randint(-128, 128, (N, d), generator=gen, dtype=torch.int8, device=dev)
        Y = torch.empty((C, N), dtype=torch.int64, device=dev)
        layers.append((ls.codes[i], As[i], ls.counts[i], X, Y))
        m = int(counts[i].sum()) * d * N
        macs += m
        kname = f"int_forward_kernel<{16 if d % 16 == 0 else 4 if d % 4 == 0 else 1}>"
        kmacs[kname] = kmacs.get(kname, 0) + m
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        mpq.integer_forward_layers(layers, wk.max_points, p)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    mpq.timing_enable(True)
    t0.record(stream)
    for _ in range(args.steps):
        mpq.integer_forward_layers(layers, wk.max_points, p)
    t1.record(stream)
    torch.cuda.synchronize()
    launches = mpq.timing_read()
    mpq.timing_enable(False)
    ms = t0.elapsed_time(t1) / args.steps
    per = {}
    for name, t in launches:
        e = per.setdefault(name, [0, 0.0])
        e[0] += 1
        e[1] += t
    kernels = {}
    for name, (cnt, tot) in per.items():
        avg_s = tot / cnt * 1e-3
        lps = cnt / args.steps
        k = {"launches_per_step": lps, "avg_us": tot / cnt * 1e3, "us_per_step": tot / args.steps * 1e3}
        if name in kmacs:
            k.update({"bound": "mfma", "unit": "TOP/s", "peak": PEAK_MFMA_I8_TOPS,
                      "ops_per_launch": 2 * kmacs[name] / lps,
                      "achieved": 2 * kmacs[name] / lps / avg_s / 1e12})
            k["frac"] = k["achieved"] / k["peak"]
        kernels[name] = k
    dom = max(kernels, key=lambda k: kernels[k]["us_per_step"])
    K = kernels[dom]
    layers_acct = [(C, d, h * h) for (C, d), h in zip(wk.layers, hw)][1:-1]
    acct_mp = ac.network_cost(layers_acct, wk.bits, 8, counts[1:-1])
    acct_nv = ac.network_cost(layers_acct, wk.bits, 8)
    res = {
        "metric": "multipoint integer forward (Eq. 15), int8 OP/s",
        "value": round(2 * macs / (ms * 1e-3), 1),
        "unit": "OP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "i8", "data": "synthetic",
        "config": {"workload": f"{wk.name} integer forward, {args.images} images of 224 x 224",
                   "layers": len(wk.layers), "bits": wk.bits, "activation_bits": 8, "p": p,
                   "points": int(sum(c.sum() for c in counts)), "macs_per_step": macs,
                   "paper_ops_per_image_W4A8": {"multipoint": acct_mp["ops"], "naive": acct_nv["ops"]},
                   "parallelism": "none"},
        "roofline": {"kernel": dom, "bound": K.get("bound"), "achieved": round(K.get("achieved", 0.0), 3),
                     "peak": K.get("peak"), "unit": K.get("unit"), "frac": round(K.get("frac", 0.0), 5),
                     "traffic": None, "avg_launch_us": round(K["avg_us"], 3)},
        "kernels": kernels,
    }
    print(json.dumps(res), flush=True)
    return 0


def cpu_model():
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or None


def _oracle_rate(orc, wk, stride, threads, calib=False):
    """(channel-points, seconds) of the oracle's fit of every stride-th
    channel of every layer of wk on `threads` threads."""
    import numpy as np

    from paper_2002_09049_amd import workloads as wl
    pts, secs = 0, 0.0
    for li in range(len(wk.layers)):
        W = np.ascontiguousarray(wl.layer_weights(wk, li)[::stride])
        X = wl.layer_calib(wk, li) if calib else None
        t0 = time.perf_counter()
        if calib:
            counts = orc.fit_calib(W, wk.bits, wk.max_points, wk.n_grid, X, float(np.float32(wk.tol)),
                                   True, n_threads=threads)[2]
        else:
            counts = orc.fit(W, wk.bits, wk.max_points, wk.n_grid, float(np.float32(wk.tol)),
                             n_threads=threads)[2]
        secs += time.perf_counter() - t0
        pts += int(counts.sum())
    return pts, secs


def _every(st):
    return "every channel" if st == 1 else f"every {st}th channel"


def cpu_baseline(wk, stride, calib=False):
    """The fp64 oracle, as it stands, on every stride-th channel of every layer
    (calib: its fit with Algorithm 2's rule on the layer's batch), on all the
    host's cores; and on one thread on the single-conv and ResNet-18 shaped
    workloads (the latter every 8th channel)."""
    import oracle
    from paper_2002_09049_amd import workloads as wl
    orc = oracle.load()
    cores = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    pts, secs = _oracle_rate(orc, wk, stride, cores, calib)
    single = {}
    for name, st in (("conv64x576", 1), ("resnet18", 8)):
        p1, s1 = _oracle_rate(orc, wl.get(name), st, 1, calib)
        single[name] = {"value": round(p1 / s1, 2), "unit": "channel-points/s",
                        "sample": f"{_every(st)} ({p1} channel-points, {s1:.1f} s)"}
    return {"value": round(pts / secs, 2), "unit": "channel-points/s", "cores": cores,
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"{'calibration-rule fit, ' if calib else ''}"
                      f"{_every(stride)} of each of the {len(wk.layers)} layers of {wk.name} "
                      f"({pts} channel-points, {secs:.1f} s wall)",
            "single_thread": single}


if __name__ == "__main__":
    sys.exit(main())
