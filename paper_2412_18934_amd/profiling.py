"""Summaries of rocprofv3 output for libdv kernels (text, for profiles/).

    python -m paper_2412_18934_amd.profiling stats <kernel_stats.csv> <kernel_trace.csv> <out.md> <command>
    python -m paper_2412_18934_amd.profiling hbm <fetch counter_collection.csv> <write counter_collection.csv> <out.txt> <command> <ref bytes>
    python -m paper_2412_18934_amd.profiling mfma <counter_collection.csv> <out.txt> <command>

``stats`` writes a per-kernel table (calls, average, share) plus the average
duration of the projection kernels (k_proj, k_gemm_valu), the figure bench.py's roofline
uses.  ``hbm`` turns FETCH_SIZE / WRITE_SIZE (KiB per dispatch) into bytes per
dispatch, scaled by what the same counters read for a plain copy of known
size: the weight-packing kernel k_pack_blocks, which at init reads every
projection matrix once and writes its packed copy once (<ref bytes> in total
each way, over all its dispatches).  It records a hash of the kernel source
so that a reader can tell whether the numbers still describe the current
kernels.  ``mfma`` reads SQ_VALU_MFMA_BUSY_CYCLES and
SQ_INSTS_VALU_MFMA_MOPS_BF16 per dispatch and reports, per kernel that issues
bf16 MFMAs, the MFMA busy fraction (busy cycles over duration x 2.4 GHz x
1024 SIMDs) and the executed MFMA rate (512 flops per MOP over the dispatch
duration) against the 2.5 PFLOP/s dense bf16 peak.
"""
from __future__ import annotations

import collections
import csv
import hashlib
import os
import statistics
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCES = ("csrc/dv_kernels.hip", "csrc/dv_engine.cpp", "csrc/dv_internal.h")
PROJ_PREFIXES = ("k_proj", "k_gemm")
REF_KERNEL = "k_pack_blocks"
CLOCK_HZ = 2.4e9      # peak engine clock
N_SIMD = 256 * 4      # compute units x SIMDs
BF16_PEAK = 2.5e15    # dense bf16 MFMA flop/s


def is_projection(name: str) -> bool:
    return name.startswith(PROJ_PREFIXES)


def source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(PKG, rel), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _short(name: str) -> str:
    return name.replace("void ", "").split("(")[0]


def summarize_stats(stats_csv, trace_csv, out_path, command):
    rows = list(csv.DictReader(open(stats_csv)))
    lines = ["# rocprofv3 kernel statistics", "", "Command:", "", "    " + command, "",
             "Source hash of the kernels: `%s`" % source_hash(), "",
             "| kernel | calls | average (us) | share |", "|---|---|---|---|"]
    gemm_ns, gemm_n = 0.0, 0
    for r in rows:
        name = _short(r["Name"])
        n = int(r["Calls"])
        avg = float(r["AverageNs"]) / 1e3
        lines.append("| `%s` | %d | %.2f | %.1f%% |" % (name, n, avg, float(r["Percentage"])))
        if is_projection(name):
            gemm_ns += float(r["TotalDurationNs"])
            gemm_n += n
    lines += ["", "Projection kernels (k_proj, k_gemm_valu): %d launches, average %.2f us."
              % (gemm_n, gemm_ns / max(gemm_n, 1) / 1e3)]
    # one full greedy step from the trace: the span between two k_accept
    # dispatches (the sampled leg that follows ends in k_accept_sampled)
    trace = list(csv.DictReader(open(trace_csv)))
    trace.sort(key=lambda r: int(r["Start_Timestamp"]))
    acc = [i for i, r in enumerate(trace) if _short(r["Kernel_Name"]) == "k_accept"]
    if len(acc) >= 2:
        step = trace[acc[-2] + 1: acc[-1] + 1]
        span = (int(step[-1]["End_Timestamp"]) - int(step[0]["Start_Timestamp"])) / 1e3
        busy = sum(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in step) / 1e3
        per = collections.defaultdict(list)
        for r in step:
            per[_short(r["Kernel_Name"])].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
        lines += ["", "Last full step in the trace: %d dispatches, GPU span %.1f us, kernels busy %.1f us."
                  % (len(step), span, busy), "", "| kernel (last step) | calls | average (us) | total (us) |",
                  "|---|---|---|---|"]
        for k, v in sorted(per.items(), key=lambda kv: -sum(kv[1])):
            lines.append("| `%s` | %d | %.2f | %.1f |" % (k, len(v), statistics.mean(v), sum(v)))
    with open(out_path, "w") as fh:
        fh.write("\n".join(lines) + "\n")


def summarize_hbm(fetch_csv, write_csv, out_path, command, ref_bytes):
    def per_kernel(path):
        agg = collections.defaultdict(list)
        for r in csv.DictReader(open(path)):
            agg[_short(r["Kernel_Name"])].append(float(r["Counter_Value"]))
        return agg
    f, w = per_kernel(fetch_csv), per_kernel(write_csv)
    ref_bytes = float(ref_bytes)
    f_ref, w_ref = sum(f.get(REF_KERNEL, [])), sum(w.get(REF_KERNEL, []))
    fs = ref_bytes / (f_ref * 1024) if f_ref else float("nan")
    ws = ref_bytes / (w_ref * 1024) if w_ref else float("nan")
    lines = ["# HBM bytes per dispatch (rocprofv3 FETCH_SIZE / WRITE_SIZE)", "",
             "command: " + command,
             "source_hash: %s" % source_hash(),
             "reference: %s, %d dispatches reading and writing %.0f bytes in total; FETCH_SIZE reads "
             "%.1f KiB -> scale %.4f; WRITE_SIZE reads %.1f KiB -> scale %.4f"
             % (REF_KERNEL, len(f.get(REF_KERNEL, [])), ref_bytes, f_ref, fs, w_ref, ws), ""]
    for k in sorted(set(f) & set(w)):
        if not k.startswith("k_"):
            continue
        fb = statistics.mean(f[k]) * 1024 * fs
        wb = statistics.mean(w[k]) * 1024 * ws
        lines.append("kernel %s: dispatches %d, fetch_bytes %.0f, write_bytes %.0f"
                     % (k, len(f[k]), fb, wb))
    with open(out_path, "w") as fh:
        fh.write("\n".join(lines) + "\n")


def summarize_mfma(counter_csv, out_path, command):
    per = collections.defaultdict(lambda: collections.defaultdict(dict))
    for r in csv.DictReader(open(counter_csv)):
        k = _short(r["Kernel_Name"])
        d = per[k][r["Dispatch_Id"]]
        d[r["Counter_Name"]] = float(r["Counter_Value"])
        d["dur"] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e9
    lines = ["# MFMA utilisation per dispatch (rocprofv3 SQ_VALU_MFMA_BUSY_CYCLES, SQ_INSTS_VALU_MFMA_MOPS_BF16)",
             "", "command: " + command, "source_hash: %s" % source_hash(),
             "busy = busy cycles / (duration x %.1f GHz x %d SIMDs); rate = 512 x MOPS / duration, "
             "against %.1f PFLOP/s dense bf16; durations are those of the counter run" %
             (CLOCK_HZ / 1e9, N_SIMD, BF16_PEAK / 1e15), "",
             "| kernel | dispatches | avg us | MFMA busy | executed TFLOP/s | of bf16 peak |",
             "|---|---|---|---|---|---|"]
    for k, ds in sorted(per.items()):
        vals = [d for d in ds.values() if d.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0) > 0 and d["dur"] > 0]
        if not vals:
            continue
        dur = statistics.mean(d["dur"] for d in vals)
        busy = statistics.mean(d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (d["dur"] * CLOCK_HZ * N_SIMD)
                               for d in vals)
        rate = statistics.mean(512 * d["SQ_INSTS_VALU_MFMA_MOPS_BF16"] / d["dur"] for d in vals)
        lines.append("| `%s` | %d | %.1f | %.1f%% | %.1f | %.1f%% |"
                     % (k[:90], len(vals), dur * 1e6, 100 * busy, rate / 1e12, 100 * rate / BF16_PEAK))
    with open(out_path, "w") as fh:
        fh.write("\n".join(lines) + "\n")


def read_hbm_summary(path):
    """(source_hash, {kernel: (dispatches, fetch_bytes, write_bytes)})."""
    out, sh = {}, None
    with open(path) as fh:
        for ln in fh:
            if ln.startswith("source_hash:"):
                sh = ln.split(":", 1)[1].strip()
            elif ln.startswith("kernel "):
                name, rest = ln[len("kernel "):].rsplit(":", 1)
                kv = dict(p.strip().split(" ", 1) for p in rest.split(","))
                out[name.strip()] = (int(kv["dispatches"]), float(kv["fetch_bytes"]),
                                     float(kv["write_bytes"]))
    return sh, out


def gemm_traffic_per_launch(path):
    """Average HBM bytes (fetch + write) over all projection dispatches of a
    summary, or None when the summary is missing or the kernel sources have
    changed since it was taken."""
    if not os.path.exists(path):
        return None
    sh, per = read_hbm_summary(path)
    if sh != source_hash():
        return None
    n = sum(d for k, (d, f, w) in per.items() if is_projection(k))
    if not n:
        return None
    return sum(d * (f + w) for k, (d, f, w) in per.items() if is_projection(k)) / n


if __name__ == "__main__":
    if sys.argv[1] == "stats":
        summarize_stats(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5])
    elif sys.argv[1] == "hbm":
        summarize_hbm(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5], sys.argv[6])
    elif sys.argv[1] == "mfma":
        summarize_mfma(sys.argv[2], sys.argv[3], sys.argv[4])
    else:
        raise SystemExit(__doc__)
