#!/usr/bin/env python3
"""Benchmark of the SGD-KV hot path on one MI355X.

One step is the whole path over one batch of synthetic, HBM-resident input:
  S0  per-KV-head budgets for every head of the stack (host, Eq. 2 + Algorithm 1)
  S1-S6  sgdkv_compress_layer for every layer (window scores, pooling, top-k,
         gather into the ragged per-head cache)
  S7-S8  sgdkv_decode_attention for every layer (one decode query per
         sequence and query head over that layer's compressed cache)
Layers are compressed first and decoded afterwards, so no decode reads a
cache still warm in the 256 MB last-level cache from its own compression.
Each layer's row gather but the last goes on a second stream (the
gather_stream option of sgdkv_compress_layer_ex) and runs beside the next
layer's window scoring, which is bound by instruction issue and leaves HBM
bandwidth unused; the decode waits for the gathers. The last layer's gather
(the only one of a one-layer workload) has nothing to overlap and runs on the
main stream with its full grid. --no-gather-stream keeps every kernel on one
stream, so that each kernel's measured duration is its own.

Default workload: the 28-layer Qwen2.5-7B-shaped stack (28 query / 4 KV
heads, head dim 128) at a 131072-token prompt, batch 8, bf16, 25 % budget,
observation window 64, pool kernel 7, sink/window 1024/1024.

Prints one JSON line: throughput in prompt tokens per second per layer for
the whole step, the decode HBM bandwidth, the roofline of the kernel that
takes the most time (per-kernel durations from HIP events recorded on the
launch stream during a timed run), and the CPU oracle timed on a bounded
sample of the same workload on this host.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
# published dense MFMA peaks of MI355X (TFLOP/s) for the score GEMM's operand type
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
# A second, composed figure for the score passes, reported beside the MFMA roofline as
# issue_peak / issue_frac: the chip-wide issue time of one logit when its MFMA share (2*d flops
# at the MFMA peak), its exp2 and its two plain vector ops (fma, add) are counted one after the
# other, at the vector-port costs the issue counters give on gfx950: 4 cycles for a 64-lane plain
# fp32 op (16 lanes per cycle) and 8 for a 64-lane exp2 (8 lanes per cycle), on 256 CUs x 4 SIMDs
# at 2.4 GHz. At d = 128 that is 16 + 16 cycles per 16x16x32 bf16 MFMA: half the MFMA peak.
VALU_OPS = 256 * 4 * 16 * 2.4e9
EXP2_OPS = 256 * 4 * 8 * 2.4e9


def score_logit_seconds(d, dtype):
    """Chip-wide issue time of one window-row x key logit of either score pass, serial model."""
    return 2.0 * d / (PEAK_TFLOPS[dtype] * 1e12) + 1.0 / EXP2_OPS + 2.0 / VALU_OPS


def compress_roof_seconds(B, C, Hq, Hkv, d, w, eb, T_layer, dtype):
    """Roofline time of one layer's compression at batch B from its algorithmic work: the window x
    key GEMM counted once (2*Hq*w*d flops per prompt token) at the MFMA peak, against the HBM
    bytes at 8 TB/s (read K once; read the kept K and V rows and write them; their positions;
    the window queries); the larger of the two."""
    flops = 2.0 * Hq * w * d * C * B
    hbm = B * (eb * (Hkv * C * d + 4.0 * T_layer * d) + 4.0 * T_layer + eb * Hq * w * d)
    t_mfma, t_hbm = flops / (PEAK_TFLOPS[dtype] * 1e12), hbm / (PEAK_HBM_GBS * 1e9)
    # with the window LSE computed by the library, the GEMM runs twice and K is read twice
    t_kread = B * eb * Hkv * C * d / (PEAK_HBM_GBS * 1e9)
    return max(t_mfma, t_hbm), max(2.0 * t_mfma, t_hbm + t_kread)


def percentile(xs, q):
    xs = sorted(xs)
    if not xs:
        return None
    k = (len(xs) - 1) * q
    lo, hi = int(math.floor(k)), int(math.ceil(k))
    return xs[lo] + (xs[hi] - xs[lo]) * (k - lo)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="qwen25_128k",
                    help="qwen25_128k (default), qwen25_32k, qwen3_256k, qwen25_1m, tiny")
    ap.add_argument("--ratio", type=float, default=0.25, help="budget as a fraction of all rows")
    ap.add_argument("--obs-window", type=int, default=0, metavar="W",
                    help="observation window in prompt tokens (default: the workload's, 64); the paper's "
                         "Query-Aware window is 128")
    ap.add_argument("--caller-lse", action="store_true",
                    help="hand each layer its window-row LSE (as prefill attention would), skipping pass 1")
    ap.add_argument("--alloc-variant", default="plain",
                    choices=["plain", "thr", "reverse", "mix", "binary", "binary_reverse"],
                    help="budget allocation variant of the head-configuration ablation (default plain)")
    ap.add_argument("--full-fraction", type=float, default=0.25,
                    help="fraction of heads with full KV for the binary variants")
    ap.add_argument("--group-agg", default="mean", choices=["mean", "ipt_max", "ipt_mean", "ipt_only"],
                    help="aggregation of a KV head's query heads: the plain mean (default) or an Ipt. variant; "
                         "the Ipt. runs draw per-query-head scores and allocate on their group maxima")
    ap.add_argument("--question-len", type=int, default=0,
                    help="Query-Unaware window: the window ends this many tokens before the prompt's end")
    ap.add_argument("--proxy-window", action="store_true",
                    help="Proxy-Query window: the window rows follow the prompt and see every cached key")
    ap.add_argument("--decode-new", type=int, default=0, metavar="N",
                    help="generation: each layer's decode also attends to N rows appended since compression, "
                         "and every step appends one row per KV head (sgdkv_append_kv) before decoding")
    ap.add_argument("--no-gather-stream", action="store_true",
                    help="run each layer's row gather on the main stream instead of a second stream beside "
                         "the next layer's scoring (then no kernel shares the GPU with another)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0, metavar="MIB",
                    help="first run three elementwise copies of MIB MiB (fp32 x 1.0), untimed: under "
                         "rocprofv3 --pmc they calibrate FETCH_SIZE / WRITE_SIZE")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="no GPU work: turn the counter CSVs of two rocprofv3 --pmc runs (FETCH_SIZE, "
                         "then WRITE_SIZE) of this script with --calibrate-copy-mib into "
                         "profiles/traffic_<workload>_w<window>_ratio<percent>.json")
    ap.add_argument("--summarize-counters", nargs="+", metavar="PMC_CSV",
                    help="no GPU work: turn the counter CSVs of rocprofv3 --pmc runs of this script (the "
                         "instruction-issue counters of COUNTER_PASSES) into profiles/counters_<...>.md")
    ap.add_argument("--summarize-kernel-trace", metavar="TRACE_CSV",
                    help="no GPU work: turn the kernel trace of a rocprofv3 --kernel-trace --stats run of "
                         "this script (same --steps/--warmup/--workload/...) into profiles/kernels_<...>.md")
    return ap.parse_args()


# ------------------------------------------------------------------ HBM traffic from counters
# the library's name for each kernel -> a pattern of its (demangled) name in rocprofv3's output
KERNEL_OF = {  # demangled ("sgdkv::name<...") or mangled ("_ZN5sgdkv<len>name...") in rocprofv3's output
    "score_lse": r"sgdkv(::|\d+)lse_kernel", "score_colsum": r"sgdkv(::|\d+)colsum_kernel",
    "lse_merge": r"sgdkv(::|\d+)lse_merge_kernel", "gather": r"sgdkv(::|\d+)copy_rows_kernel",
    "decode_split": r"sgdkv(::|\d+)decode_split_kernel", "decode_combine": r"sgdkv(::|\d+)decode_combine_kernel",
    "pool_radix_hist": r"sgdkv(::|\d+)radix_pass_kernel(<0, true, true|ILi0ELb1ELb1E)",
    "radix_hist": r"sgdkv(::|\d+)radix_pass_kernel(<[123], false, true|ILi[123]ELb0ELb1E)",
    "compact": r"sgdkv(::|\d+)compact_kernel"}
SOURCE_OF = {"score_lse": "score_kernels.hip", "score_colsum": "score_kernels.hip", "lse_merge": "score_kernels.hip",
             "gather": "select_kernels.hip", "pool_radix_hist": "select_kernels.hip", "radix_hist": "select_kernels.hip",
             "compact": "select_kernels.hip",
             "decode_split": "decode_kernels.hip", "decode_combine": "decode_kernels.hip"}
SHARED_SOURCES = ("device_common.h", "mfma_frag.h", "sgdkv_internal.h", "segment_init.h")


def source_sha(name):
    """Hash of the code a kernel is built from, comments and blank space left out: counters taken
    before a change to that code do not apply."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in (SOURCE_OF[name],) + SHARED_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_03235_amd", "csrc", f)) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def traffic_path(workload, ratio, w):
    return os.path.join(ROOT, "profiles", f"traffic_{workload}_w{w}_ratio{int(round(ratio * 100))}.json")


_TRAFFIC = {}


def traffic_of(name, workload=None, ratio=None, w=None):
    """HBM bytes per launch of a kernel from the committed counter summary, or None when there is
    none or the kernel's source changed since the counters were taken."""
    if workload is not None:
        _TRAFFIC.clear()
        try:
            with open(traffic_path(workload, ratio, w)) as fh:
                _TRAFFIC.update(json.load(fh))
        except (OSError, ValueError):
            pass
        return None
    rec = _TRAFFIC.get("kernels", {}).get(name)
    if not rec or rec.get("source_sha") != source_sha(name):
        return None
    return rec["hbm_bytes_per_launch"]


def summarize_traffic(fetch_csv, write_csv, args):
    import csv
    import statistics

    def per_kernel(path, counter):
        vals, calib = {}, []
        with open(path, newline="") as fh:
            for row in csv.DictReader(fh):
                if row["Counter_Name"] != counter:
                    continue
                name, v = row["Kernel_Name"], float(row["Counter_Value"])
                vals.setdefault(name, []).append(v)
                if "elementwise_kernel" in name and "MulFunctor" in name:
                    calib.append((int(row["Dispatch_Id"]), v))
        return vals, calib

    (fetch, fcal), (write, wcal) = per_kernel(fetch_csv, "FETCH_SIZE"), per_kernel(write_csv, "WRITE_SIZE")
    kib = args.calibrate_copy_mib * 1024.0

    def copy_median(calib):
        # the three calibration copies (torch.mul by 1.0) are the first multiplications the run makes
        xs = [v for _, v in sorted(calib)[:3]]
        return statistics.median(xs) if len(xs) == 3 and min(xs) > 0.25 * kib else None

    cf, cw = copy_median(fcal), copy_median(wcal)
    if not kib or cf is None or cw is None:
        sys.exit("no calibration copy found: run the counter passes with --calibrate-copy-mib")
    import workloads
    w = args.obs_window or workloads.WORKLOADS[args.workload].obs_window
    out = dict(workload=args.workload, ratio=args.ratio, obs_window=w, unit="KiB per dispatch",
               commands=[f"rocprofv3 --pmc {c} --output-format csv -d gpurun_out/pmc_{c.split('_')[0].lower()} "
                         f"-o pmc -- python3 bench.py --workload {args.workload} --ratio {args.ratio} "
                         f"--obs-window {w} --steps 1 --warmup 0 --no-cpu-baseline "
                         f"--calibrate-copy-mib {args.calibrate_copy_mib}"
                         for c in ("FETCH_SIZE", "WRITE_SIZE")],
               note="hbm_bytes_per_launch = 1024 * (fetch_kib * fetch_factor + write_kib * write_factor); "
                    "the factors make a plain elementwise copy of copy_kib read and write exactly copy_kib",
               calibration=dict(copy_kib=kib, fetch_kib=cf, write_kib=cw, fetch_factor=kib / cf,
                                write_factor=kib / cw),
               kernels={})
    import re
    for name, pat in KERNEL_OF.items():
        fv = [v for n, vs in fetch.items() if re.search(pat, n) for v in vs]
        wv = [v for n, vs in write.items() if re.search(pat, n) for v in vs]
        if not fv or not wv:
            continue
        f, w_ = statistics.mean(fv), statistics.mean(wv)
        out["kernels"][name] = dict(dispatches=len(fv), fetch_kib=f, write_kib=w_, source_sha=source_sha(name),
                                    hbm_bytes_per_launch=round(1024.0 * (f * kib / cf + w_ * kib / cw)))
    path = traffic_path(args.workload, args.ratio, w)
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1)
    print(f"wrote {path}")


# Counter passes for the instruction-issue summary: each within one rocprofv3 pass's limits
# (at most 8 SQ counters and 2 GRBM counters).
COUNTER_PASSES = (
    ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_VALU_MFMA_COEXEC_CYCLES", "SQ_BUSY_CYCLES", "SQ_ACTIVE_INST_VALU",
     "SQ_ACTIVE_INST_VALU2", "SQ_WAIT_INST_ANY", "SQ_INSTS_LDS", "SQ_CYCLES", "GRBM_GUI_ACTIVE"),
    ("SQ_INSTS_VALU", "SQ_INSTS_MFMA", "SQ_INSTS_VALU_TRANS_F32", "SQ_ACTIVE_INST_LDS", "SQ_WAVE_CYCLES",
     "SQ_ACTIVE_INST_ANY", "SQ_INSTS_SALU", "SQ_LDS_BANK_CONFLICT", "GRBM_GUI_ACTIVE"),
)
N_XCD, N_CU, N_SIMD = 8, 256, 1024  # MI355X


def _profile_tag(args):
    import workloads
    w = args.obs_window or workloads.WORKLOADS[args.workload].obs_window
    return f"{args.workload}_w{w}_ratio{int(round(args.ratio * 100))}", w


def _bench_flags(args, w):
    return f"--workload {args.workload} --ratio {args.ratio} --obs-window {w}"


def summarize_counters(paths, args):
    """Per library kernel, the mean per dispatch of each counter, and the derived issue figures."""
    import csv
    import re
    import statistics
    vals, dur = {}, {}
    for path in paths:
        with open(path, newline="") as fh:
            for row in csv.DictReader(fh):
                name = next((k for k, pat in KERNEL_OF.items() if re.search(pat, row["Kernel_Name"])), None)
                if name is None:
                    continue
                vals.setdefault(name, {}).setdefault(row["Counter_Name"], []).append(float(row["Counter_Value"]))
                d = (int(row["End_Timestamp"]) - int(row["Start_Timestamp"])) * 1e-9
                dur.setdefault(name, {}).setdefault((path, row["Dispatch_Id"]), d)
    tag, w = _profile_tag(args)
    cmds = [f"rocprofv3 --pmc {' '.join(p)} --output-format csv -d gpurun_out/pmc_issue{i} -o pmc -- "
            f"python3 bench.py {_bench_flags(args, w)} --steps 1 --warmup 0 --no-cpu-baseline"
            for i, p in enumerate(COUNTER_PASSES)]
    lines = [f"# Instruction-issue counters per kernel: {args.workload}, window {w}, {args.ratio:.0%} budget", "",
             "Commands (run from the repository root on one MI355X, gfx950), then "
             f"`python3 bench.py {_bench_flags(args, w)} --summarize-counters <the two pmc_counter_collection.csv>`:",
             "", "```", *cmds, "```", "",
             "Values are means per dispatch (rocprofv3 sums each counter over the XCDs and shader engines). "
             "Under counter collection the kernels run one at a time. Derived figures: clock = GRBM_GUI_ACTIVE "
             f"/ {N_XCD} XCDs / duration; MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / ({N_SIMD} SIMDs x GUI cycles "
             "per XCD); VALU issue = 4 x SQ_ACTIVE_INST_VALU / (SIMDs x cycles) (wave-cycles, so it can pass 1 "
             "with several waves per SIMD); dual issue = 4 x SQ_ACTIVE_INST_VALU2 / (SIMDs x cycles); "
             "co-execution = SQ_VALU_MFMA_COEXEC_CYCLES / SQ_VALU_MFMA_BUSY_CYCLES.", ""]
    for name in ("score_lse", "score_colsum", "pool_radix_hist", "radix_hist", "compact", "gather",
                 "decode_split", "decode_combine"):
        if name not in vals:
            continue
        v = {c: statistics.mean(x) for c, x in vals[name].items()}
        t = statistics.mean(dur[name].values())
        gui = v.get("GRBM_GUI_ACTIVE", 0.0) / N_XCD
        lines += [f"## `{name}`", "", f"dispatches per counter pass: {len(dur[name]) // max(1, len(paths))}, "
                  f"mean duration {t * 1e6:.2f} us", "", "| counter | per dispatch |", "|---|---:|"]
        lines += [f"| {c} | {v[c]:.6g} |" for c in sorted(v)]
        if gui > 0:
            der = [("clock (GHz)", gui / t / 1e9)]
            if "SQ_VALU_MFMA_BUSY_CYCLES" in v:
                der.append(("MFMA busy", v["SQ_VALU_MFMA_BUSY_CYCLES"] / (N_SIMD * gui)))
                if v["SQ_VALU_MFMA_BUSY_CYCLES"] > 0 and "SQ_VALU_MFMA_COEXEC_CYCLES" in v:
                    der.append(("co-execution / MFMA busy", v["SQ_VALU_MFMA_COEXEC_CYCLES"] / v["SQ_VALU_MFMA_BUSY_CYCLES"]))
            if "SQ_ACTIVE_INST_VALU" in v:
                der.append(("VALU issue (wave-cycles per SIMD cycle)", 4 * v["SQ_ACTIVE_INST_VALU"] / (N_SIMD * gui)))
            if "SQ_ACTIVE_INST_VALU2" in v:
                der.append(("dual VALU issue (per SIMD cycle)", 4 * v["SQ_ACTIVE_INST_VALU2"] / (N_SIMD * gui)))
            if "SQ_WAIT_INST_ANY" in v and "SQ_WAVE_CYCLES" in v and v["SQ_WAVE_CYCLES"] > 0:
                der.append(("waiting for issue / wave cycles", v["SQ_WAIT_INST_ANY"] / v["SQ_WAVE_CYCLES"]))
            for c in ("SQ_INSTS_MFMA", "SQ_INSTS_VALU", "SQ_INSTS_VALU_TRANS_F32", "SQ_INSTS_LDS", "SQ_INSTS_SALU"):
                if c in v:
                    der.append((f"{c} per SIMD", v[c] / N_SIMD))
            lines += ["", "| derived | value |", "|---|---:|"] + [f"| {k} | {x:.4g} |" for k, x in der]
        lines.append("")
    path = os.path.join(ROOT, "profiles", f"counters_{tag}.md")
    with open(path, "w") as fh:
        fh.write("\n".join(lines))
    print(f"wrote {path}")


def summarize_kernel_trace(path, args):
    """Mean kernel durations from a rocprofv3 kernel trace of this script: the timed steps (the timed
    region and the one with per-kernel events) and the untimed serial steps, separately."""
    import csv
    import statistics
    import workloads
    tag, w = _profile_tag(args)
    L = workloads.WORKLOADS[args.workload].layers
    per = {}
    with open(path, newline="") as fh:
        for row in csv.DictReader(fh):
            if "sgdkv" not in row["Kernel_Name"]:
                continue
            per.setdefault(row["Kernel_Name"], []).append(
                (int(row["Start_Timestamp"]), (int(row["End_Timestamp"]) - int(row["Start_Timestamp"])) * 1e-3))
    W, K = args.warmup, args.steps
    serial = L > 1 and not args.no_gather_stream
    rows = []
    for name, xs in per.items():
        xs.sort()
        n = len(xs)
        per_step = n // (W + (3 if serial else 2) * K)  # launches per step
        timed = [d for _, d in xs[W * per_step:(W + 2 * K) * per_step]]
        ser = [d for _, d in xs[(W + 2 * K) * per_step:]] if serial else []
        rows.append((statistics.mean(timed) * per_step * (2 * K) if timed else 0.0, name, n, timed, ser,
                     min(d for _, d in xs), max(d for _, d in xs)))
    rows.sort(reverse=True)
    cmd = (f"rocprofv3 --kernel-trace --stats --output-format csv -d gpurun_out/prof_{tag} -o run -- python3 bench.py "
           f"{_bench_flags(args, w)} --steps {K} --warmup {W} --no-cpu-baseline"
           + (" --no-gather-stream" if args.no_gather_stream else ""))
    lines = [f"# Kernel times: {args.workload}, window {w}, {args.ratio:.0%} budget", "",
             "Command (run from the repository root on one MI355X, gfx950), then "
             f"`python3 bench.py {_bench_flags(args, w)} --steps {K} --warmup {W} --summarize-kernel-trace "
             f"gpurun_out/prof_{tag}/run_kernel_trace.csv`:", "", "```", cmd, "```", "",
             f"Library kernels from rocprofv3's kernel trace. The run makes {W} warm-up steps, {K} timed steps, {K} "
             "timed steps with per-kernel events (the bench line's durations)"
             + (f" and {K} untimed steps with every kernel on one stream (`roofline_serial`)" if serial else "")
             + ". \"timed\" averages the launches of the timed steps" + (", \"serial\" those of the last ones" if serial
                                                                            else "") + ".", "",
             "| kernel | calls | avg us (timed) | avg us (serial) | min us | max us |", "|---|---:|---:|---:|---:|---:|"]
    for _, name, n, timed, ser, lo, hi in rows:
        ser_s = f"{statistics.mean(ser):.2f}" if ser else "—"  # no serial steps in this run
        lines.append(f"| `{name}` | {n} | {statistics.mean(timed):.2f} | {ser_s} | {lo:.2f} | {hi:.2f} |")
    out = os.path.join(ROOT, "profiles", f"kernels_{tag}.md")
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(f"wrote {out}")


def main():
    args = parse()
    if args.summarize_traffic:
        summarize_traffic(*args.summarize_traffic, args)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters, args)
        return
    if args.summarize_kernel_trace:
        summarize_kernel_trace(args.summarize_kernel_trace, args)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        log(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
            "this build has no multi-GPU path.")
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_03235_amd as sg
    import workloads

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(int(os.environ.get("LOCAL_RANK", "0")))
    dev = torch.device("cuda")
    wl = workloads.WORKLOADS[args.workload]
    if args.obs_window:
        import dataclasses
        wl = dataclasses.replace(wl, obs_window=args.obs_window)
    L, B, Hq, Hkv, d = wl.layers, wl.batch, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    C, w, s, W, kp = wl.seq_len, wl.obs_window, wl.b_sink, wl.b_window, wl.pool_kernel
    eb = 2 if wl.dtype == "bf16" else 4
    win0 = C if args.proxy_window else C - w - args.question_len  # position of the first window row
    n_scored = win0
    stream = torch.cuda.current_stream()
    traffic_of(None, args.workload, args.ratio, w)
    if args.calibrate_copy_mib:
        src = torch.ones(args.calibrate_copy_mib << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst

    # ------------------------------------------------------------ inputs (HBM-resident)
    t0 = time.perf_counter()
    scores = workloads.head_scores(wl)
    agg = ["mean", "ipt_max", "ipt_mean", "ipt_only"].index(args.group_agg)
    qscores = [None] * L
    if agg:
        # per-attention-head scores (Beta(0.5, 2), the workload's distribution); the allocation uses
        # their maximum over each group, as the paper does for GQA models
        qs = np.random.Generator(np.random.PCG64(wl.seed + 200)).beta(0.5, 2.0, size=(L, Hq))
        scores = sg.reduce_query_head_scores(qs, Hkv).reshape(-1)
        qscores = [qs[l] for l in range(L)]
    total = sg.total_from_ratio(args.ratio, L, Hkv, C, s, W)
    variant = ["plain", "thr", "reverse", "mix", "binary", "binary_reverse"].index(args.alloc_variant)
    # the mix variant's second score vector stands in for retrieval-head scores the paper mixes in
    scores2 = np.random.Generator(np.random.PCG64(wl.seed + 100)).beta(0.5, 2.0, size=scores.size)

    def allocate():
        return sg.allocate_budgets_variant(scores, L, Hkv, C, s, W, total, variant, scores2=scores2,
                                           full_fraction=args.full_fraction)

    budgets = allocate().reshape(L, Hkv)
    n_new = args.decode_new

    def make_set(r):
        """One copy of every layer's inputs and outputs (copy r draws its inputs as layers L*r ..)."""
        layers = [workloads.torch_layer_tensors(wl, l + L * r, dev) for l in range(L)]
        lse_in = [None] * L
        if args.caller_lse:
            # Stand-in for the LSE prefill attention already produced: fp32 logits of each window
            # row over its causal keys, one (sequence, KV head) block at a time, outside the timed region.
            G = Hq // Hkv
            scale = 1.0 / math.sqrt(d)
            pos = torch.arange(win0, win0 + w, device=dev)[:, None]
            for l in range(L):
                out = torch.empty((B, Hq, w), dtype=torch.float32, device=dev)
                for b in range(B):
                    for h in range(Hkv):
                        qg = layers[l]["q_win"][b, h * G:(h + 1) * G].float().reshape(G * w, d)
                        kt = layers[l]["k"][b, h].float().t().contiguous()
                        lg = (qg @ kt) * scale
                        lg = lg.reshape(G, w, C).masked_fill(torch.arange(C, device=dev)[None, :] > pos,
                                                             float("-inf"))
                        out[b, h * G:(h + 1) * G] = torch.logsumexp(lg, dim=-1)
                        del lg, kt
                lse_in[l] = out
        outs = []
        for l in range(L):
            T = int(budgets[l].sum())
            outs.append(dict(k_c=torch.empty((B * T, d), dtype=layers[l]["k"].dtype, device=dev),
                             v_c=torch.empty((B * T, d), dtype=layers[l]["k"].dtype, device=dev),
                             kept_pos=torch.empty(B * T, dtype=torch.int32, device=dev),
                             offsets=torch.empty(B * Hkv + 1, dtype=torch.int64, device=dev),
                             scores=torch.empty((B, Hkv, n_scored), dtype=torch.float32, device=dev)))
        tails = [None] * L
        if n_new > 0:
            # rows appended since compression (one generated token per row), drawn like the cache
            gen = torch.Generator(device=dev)
            gen.manual_seed(wl.seed + 300 + r)
            for l in range(L):
                kn = torch.randn((B, Hkv, n_new, d), generator=gen, device=dev).to(layers[l]["k"].dtype)
                vn = torch.randn((B, Hkv, n_new, d), generator=gen, device=dev).to(layers[l]["k"].dtype)
                step_kv = torch.randn((2, B, Hkv, d), generator=gen, device=dev).to(layers[l]["k"].dtype)
                tails[l] = (kn, vn, step_kv)
        return dict(layers=layers, lse_in=lse_in, outs=outs, tails=tails,
                    dec_out=[torch.empty((B, Hq, d), dtype=torch.float32, device=dev) for _ in range(L)],
                    dec_lse=[torch.empty((B, Hq), dtype=torch.float32, device=dev) for _ in range(L)])

    # A step whose inputs and outputs fit the last-level caches would time cached reads: below
    # 1 GiB per step, the steps rotate over enough distinct copies to make 1 GiB.
    def tensor_bytes(x):
        if isinstance(x, torch.Tensor):
            return x.numel() * x.element_size()
        if isinstance(x, dict):
            return sum(tensor_bytes(v) for v in x.values())
        if isinstance(x, (list, tuple)):
            return sum(tensor_bytes(v) for v in x)
        return 0

    sets = [make_set(0)]
    step_bytes = tensor_bytes(sets[0])
    n_copies = max(1, -(-(1 << 30) // max(step_bytes, 1)))
    sets += [make_set(r) for r in range(1, n_copies)]
    layers, tails = sets[0]["layers"], sets[0]["tails"]
    step_count = [0]
    cdesc = sg.compress_desc(layers[0]["q_win"], layers[0]["k"], pool_kernel=kp, b_sink=s, b_window=W)
    # the gathers' stream keeps torch's default priority; the gather does not use the workspace
    gstream = None if args.no_gather_stream else torch.cuda.Stream(device=dev)
    ws_c = sg.alloc_workspace(sg.compress_workspace_size(cdesc), dev)
    offsets_host = [sg.segment_offsets(budgets[l], B) for l in range(L)]
    ddesc = sg.decode_desc(layers[0]["q"], Hkv, torch.float32)
    ws_d = sg.alloc_workspace(max(sg.decode_workspace_size(ddesc, oh, n_new) for oh in offsets_host), dev)
    torch.cuda.synchronize()
    log(f"[bench] inputs ready in {time.perf_counter() - t0:.1f}s: {wl.name}, total budget {total} rows "
        f"({args.ratio:.0%}), {L} layers x {B} sequences")

    def step(gs=gstream, dec_ev=None):
        # S0 on the host, then every layer's compression, then every layer's decode; dec_ev (a pair
        # of events) brackets the decode phase on the launch stream
        cur = sets[step_count[0] % n_copies]
        step_count[0] += 1
        layers, lse_in, outs, tails = cur["layers"], cur["lse_in"], cur["outs"], cur["tails"]
        dec_out, dec_lse = cur["dec_out"], cur["dec_lse"]
        allocate()
        for l in range(L):
            t = layers[l]
            sg.compress_layer(t["q_win"], t["k"], t["v"], budgets[l], pool_kernel=kp, b_sink=s, b_window=W,
                              window_lse=lse_in[l], group_agg=agg, qhead_scores=qscores[l], window_pos=win0,
                              out=outs[l], workspace=ws_c, stream=stream,
                              gather_stream=gs if l < L - 1 else None)  # nothing follows the last
        if gs is not None and L > 1:
            stream.wait_stream(gs)  # every layer's compressed cache is complete before decode
        if dec_ev is not None:
            dec_ev[0].record(stream)
        for l in range(L):
            o = outs[l]
            kn = vn = None
            if tails[l] is not None:
                # this step's token goes into the last slot, then decode attends to all n_new rows
                kn, vn, step_kv = tails[l]
                sg.append_kv(layers[l]["q"], step_kv[0], step_kv[1], kn, vn, n_new - 1, stream=stream)
            sg.decode_attention(layers[l]["q"], o["k_c"], o["v_c"], o["offsets"], offsets_host[l], Hkv,
                                out_dtype=torch.float32, k_new=kn, v_new=vn, n_new=n_new, workspace=ws_d,
                                out=dec_out[l], lse=dec_lse[l], stream=stream)
        if dec_ev is not None:
            dec_ev[1].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # ------------------------------------------------------------ timed region (headline)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # an event after every step on the launch stream gives the spread of the step times (recording
    # an event adds no synchronisation)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    # two more per step bracket its decode phase (all layers' decode kernels, launch gaps included)
    dec_evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    ev0.record(stream)
    t_wall0 = time.perf_counter()
    for i in range(args.steps):
        step(dec_ev=dec_evs[i])
        evs[i].record(stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_wall0) * 1e3 / args.steps
    ms_per_step = ev0.elapsed_time(ev1) / args.steps
    step_ms = [ev0.elapsed_time(evs[0])] + [evs[i - 1].elapsed_time(evs[i]) for i in range(1, args.steps)]
    dec_phase_ms = statistics.mean(a.elapsed_time(b) for a, b in dec_evs)

    # ------------------------------------------------------------ timed region with kernel events
    sg.profile_reset()
    sg.profile_enable(True)
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    sg.profile_enable(False)
    prof_ms_per_step = ev0.elapsed_time(ev1) / args.steps
    kern = sg.profile_read()

    # ------------------------------------------------------------ untimed: every kernel on one stream
    # (only with a gather stream: the same kernels without overlap, for the serial roofline)
    kern_serial = None
    if gstream is not None and L > 1:
        sg.profile_reset()
        sg.profile_enable(True)
        for _ in range(args.steps):
            step(gs=None)
        torch.cuda.synchronize()
        sg.profile_enable(False)
        kern_serial = sg.profile_read()

    # ------------------------------------------------------------ algorithmic work per launch
    T_layers = budgets.sum(axis=1)
    T_mean = float(T_layers.mean())
    flops_tok = 2.0 * Hq * w * d                      # window x key GEMM, counted once
    lse_keys = min(C, win0 + w)                       # keys some window row sees
    work = {
        # MFMA flops of the logits: the bf16 (or fp32) MFMA roofline; issue_frac beside it is the
        # fraction of the serial MFMA + exp2 + fma + add issue model (score_logit_seconds)
        "score_lse": ("mfma", flops_tok * B * lse_keys, "TFLOP/s"),
        "score_colsum": ("mfma", flops_tok * B * n_scored, "TFLOP/s"),
        # read the kept K and V rows and their positions, write the rows
        "gather": ("hbm", B * T_mean * (4 * d * eb + 4), "GB/s"),
        # read every kept K and V row once (and the rows appended since), plus the queries and outputs
        "decode_split": ("hbm", B * (T_mean + Hkv * n_new) * 2 * d * eb + B * Hq * d * (eb + 4.0), "GB/s"),
        # pooling + digit-0 histogram: read the column sums (one per row split), write the pooled scores
        "pool_radix_hist": ("hbm", B * Hkv * n_scored * 4.0 * (-(-(Hq // Hkv * w) // 512) + 1), "GB/s"),
    }
    kernels = {}
    for name, (count, ms) in sorted(kern.items(), key=lambda kv: -kv[1][1]):
        kernels[name] = dict(launches_per_step=count / args.steps, ms_per_step=ms / args.steps,
                             avg_us=1e3 * ms / count, share=ms / max(1e-9, sum(v[1] for v in kern.values())))
    dominant = max(kern.items(), key=lambda kv: kv[1][1])[0]

    def roof(name, kern=kern):
        count, ms = kern[name]
        bound, amount, unit = work[name]
        avg_s = ms / count / 1e3
        extra = {}
        if bound == "mfma":
            achieved, peak = amount / avg_s / 1e12, PEAK_TFLOPS[wl.dtype]
            issue_peak = 2.0 * d / score_logit_seconds(d, wl.dtype) / 1e12
            extra = dict(issue_peak=round(issue_peak, 1), issue_frac=round(achieved / issue_peak, 4))
        else:
            achieved, peak = amount / avg_s / 1e9, PEAK_HBM_GBS
        return dict(kernel=name, bound=bound, achieved=round(achieved, 2), peak=round(peak, 1), unit=unit,
                    frac=round(achieved / peak, 4), traffic=traffic_of(name), avg_us=round(avg_s * 1e6, 2),
                    work_per_launch=amount, **extra)

    roofline = roof(dominant) if dominant in work else None
    roofline_serial = None
    if kern_serial is not None and dominant in work and dominant in kern_serial:
        roofline_serial = dict(roof(dominant, kern_serial),
                               note="same kernel, every kernel on one stream (an extra untimed run); "
                                    "roofline above is the timed run, where the gathers overlap the scoring")
    decode = roof("decode_split") if "decode_split" in kern else None
    other_roofs = {n: roof(n) for n in ("score_lse", "score_colsum", "gather", "pool_radix_hist")
                   if n in kern and n != dominant}
    # decode time: the decode phase of the timed steps (two events around it on the launch stream:
    # every layer's split and combine kernels with the launch gaps between them, and no per-kernel
    # events); the per-kernel event durations of the profiled run are kept beside it
    dec_ms = dec_phase_ms
    dec_kernel_ms = sum(kern.get(n, (0, 0))[1] for n in ("decode_split", "decode_combine", "append")) / args.steps
    dec_bytes = work["decode_split"][1] * L
    # compression time: the step minus its decode phase (the gathers overlap other kernels, so a
    # sum of kernel durations would count them twice)
    comp_ms = ms_per_step - dec_ms
    roofs = [compress_roof_seconds(B, C, Hq, Hkv, d, w, eb, float(T_layers[l]), wl.dtype) for l in range(L)]
    roof_s, roof2_s = sum(r[0] for r in roofs), sum(r[1] for r in roofs)
    compress_roof = dict(
        frac=round(roof_s * 1e3 / comp_ms, 4) if comp_ms > 0 else None,
        roof_us_per_layer=round(roof_s * 1e6 / L, 2), measured_us_per_layer=round(comp_ms * 1e3 / L, 2),
        two_pass_cap=None if args.caller_lse else round(roof_s / roof2_s, 4),
        note="roof = max(GEMM counted once at the MFMA peak, algorithmic HBM bytes at 8 TB/s) per layer; "
             "two_pass_cap = the best fraction when the library computes the window LSE itself (the GEMM "
             "twice, K read twice)")

    tokens = float(B) * C * L  # prompt tokens per step, over all layers
    value = tokens / (ms_per_step / 1e3)

    # ------------------------------------------------------------ CPU oracle on a bounded sample
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        threads = oracle.num_threads()
        # (1) the tiny fp32 workload (one layer, 4/2 heads, C 2048), median of 3, with all host
        # threads and with one
        tw = workloads.WORKLOADS["tiny"]
        tt = {k: x.astype(np.float64) for k, x in workloads.numpy_tensors(tw).items()}
        ttot = oracle.total_from_ratio(0.25, 1, tw.num_kv_heads, tw.seq_len, tw.b_sink, tw.b_window)
        tbud = oracle.allocate_budgets(workloads.head_scores(tw), 1, tw.num_kv_heads, tw.seq_len, tw.b_sink,
                                       tw.b_window, ttot)

        def tiny_once():
            t0 = time.perf_counter()
            r = oracle.compress(tt["q_win"], tt["k"], tt["v"], tbud, w=tw.obs_window, kp=tw.pool_kernel,
                                s=tw.b_sink, W=tw.b_window)
            oracle.decode(tt["q"], r["k_c"], r["v_c"], r["offsets"], tw.num_kv_heads)
            return time.perf_counter() - t0
        tiny_all = statistics.median(tiny_once() for _ in range(3))
        oracle.set_num_threads(1)
        tiny_one = statistics.median(tiny_once() for _ in range(3))
        oracle.set_num_threads(threads)
        # (2) sequences of layer 0 of this workload, one after another, until about 8 s of the
        # oracle's work (at most 4): compression and decode timed apart
        t = layers[0]
        nb, comp_s, dec_s, dec_b = 0, 0.0, 0.0, 0.0
        for b in range(min(B, 4)):
            if comp_s + dec_s > 8.0:
                break
            nb += 1
            q_win = t["q_win"][b:b + 1].cpu().double().numpy()
            kk = t["k"][b:b + 1].cpu().double().numpy()
            vv = t["v"][b:b + 1].cpu().double().numpy()
            qq = t["q"][b:b + 1].cpu().double().numpy()
            tc0 = time.perf_counter()
            res = oracle.compress(q_win, kk, vv, budgets[0], w=w, kp=kp, s=s, W=W, agg=agg,
                                  qhead_scores=qscores[0], win0=win0)
            tc1 = time.perf_counter()
            if n_new > 0:
                kn, vn, _ = tails[0]
                oracle.decode_append(qq, res["k_c"], res["v_c"], res["offsets"], kn[b:b + 1].cpu().double().numpy(),
                                     vn[b:b + 1].cpu().double().numpy(), n_new, Hkv)
            else:
                oracle.decode(qq, res["k_c"], res["v_c"], res["offsets"], Hkv)
            tc2 = time.perf_counter()
            comp_s += tc1 - tc0
            dec_s += tc2 - tc1
            dec_b += (float(T_layers[0]) + Hkv * n_new) * 2 * d * eb
            del res
        cpu = dict(value=round(nb * C / (comp_s + dec_s), 1), unit="tokens/s per layer", cores=threads,
                   kind="oracle",
                   sample=f"sequences 0-{nb - 1} of layer 0 ({Hkv} KV heads, C={C}): compress + decode, "
                          f"{comp_s + dec_s:.1f} s",
                   cpu_model=cpu_model(),
                   compress_tokens_per_s=round(nb * C / comp_s, 1),
                   decode_gbps=round(dec_b / dec_s / 1e9, 3),
                   decode_bytes_note="the compressed cache's K and V rows at the workload's element size, "
                                     "as for the GPU's decode GB/s",
                   tiny_workload=dict(workload=tw.name, seconds_all_threads=round(tiny_all, 4),
                                      seconds_one_thread=round(tiny_one, 4),
                                      tokens_per_s_all_threads=round(tw.seq_len / tiny_all, 1),
                                      tokens_per_s_one_thread=round(tw.seq_len / tiny_one, 1),
                                      note="compress + decode, median of 3"))

    line = dict(
        metric="compressed K/V tokens/s per layer + ragged decode-attn HBM GB/s (% of peak), 1 GPU",
        value=round(value, 1), unit="tokens/s per layer", n_gpus=1, steps=args.steps, warmup=args.warmup,
        ms_per_step=round(ms_per_step, 4), higher_is_better=True, scaling="weak", vs_baseline=None,
        dtype=wl.dtype, data="synthetic",
        config=dict(workload=wl.name, layers=L, batch=B, prompt=C, q_heads=Hq, kv_heads=Hkv, head_dim=d,
                    obs_window=w, pool_kernel=kp, b_sink=s, b_window=W, budget_ratio=args.ratio,
                    total_budget_rows=int(budgets.sum()), window_lse="caller" if args.caller_lse else "computed",
                    alloc_variant=args.alloc_variant, group_agg=args.group_agg, window_start=win0,
                    decode_appended_rows=n_new, gather_stream=not args.no_gather_stream,
                    input_copies=n_copies),
        step_ms=dict(median=round(statistics.median(step_ms), 4), p10=round(percentile(step_ms, 0.1), 4),
                     p90=round(percentile(step_ms, 0.9), 4), mean=round(ms_per_step, 4)),
        compress_tokens_per_s=round(tokens / (comp_ms / 1e3), 1) if comp_ms > 0 else None,
        compress_roof=compress_roof,
        decode=dict(gbps=round(dec_bytes / (dec_ms / 1e3) / 1e9, 1) if dec_ms > 0 else None,
                    frac_of_peak=round(dec_bytes / (dec_ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4) if dec_ms > 0 else None,
                    ms_per_step=round(dec_ms, 4), kernel_events_ms_per_step=round(dec_kernel_ms, 4),
                    note="ms_per_step: the decode phase of the timed steps (events around it); "
                         "kernel_events_ms_per_step: the sum of its kernels' own event durations in the "
                         "profiled run (each bracketed by two events)",
                    split_kernel=decode),
        roofline=roofline, roofline_serial=roofline_serial, other_rooflines=other_roofs, kernels=kernels,
        profiled_ms_per_step=round(prof_ms_per_step, 4),
        wall_ms_per_step=round(wall_ms, 4), cpu_baseline=cpu,
    )
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
