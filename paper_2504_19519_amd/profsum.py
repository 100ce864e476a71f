"""Summaries of rocprofv3 runs of bench.py, and the HBM traffic they give.

`python -m paper_2504_19519_amd.profsum OUT WORKLOAD PHASE GROUPS SUMMARY.md COPY_BYTES [LIVE_US]`
reads
the CSV output of the rocprofv3 runs listed in `commands()` (a kernel trace
with --stats of the bench phase; one --pmc FETCH_SIZE and one --pmc
WRITE_SIZE run of the same signalling GEMM launched alone, since rocprofv3
runs kernels one at a time while it collects counters and the consumers'
waits could then not overlap the GEMM; and the same two counters over a
plain copy of known size) and writes a short markdown summary. The summary ends with a
block of `key: value` lines that bench.py reads back (`read_traffic`):
FETCH_SIZE and WRITE_SIZE count in KiB per dispatch and are scaled by what
they read for the plain copy, whose bytes are known.

The GEMM figures are tied to the sources the kernel is built from (their
SHA-256): once those change, the figures no longer describe the kernel and
read_traffic returns None.
"""
from __future__ import annotations

import collections
import csv
import hashlib
import os
import re
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
GEMM_SOURCES = ["csrc/gemm.hip", "csrc/gemm.h", "csrc/fo_device.h", "csrc/fo_internal.h"]


def gemm_sources_sha256() -> str:
    h = hashlib.sha256()
    for rel in GEMM_SOURCES:
        with open(os.path.join(PKG, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def commands(workload: str, phase: str, sizes: str, steps: int = 20, warmup: int = 5):
    run = (f"python3 R/bench.py --workload {workload} --phase {phase} --sizes {sizes} --steps {steps} "
           f"--warmup {warmup} --skip-cpu")
    copy = f"python3 R/bench.py --workload {workload} --phase copy --steps {steps} --warmup {warmup} --skip-cpu"
    gemm = f"python3 R/bench.py --workload {workload} --phase gemm --steps {steps} --warmup {warmup} --skip-cpu"
    out = [f"rocprofv3 --kernel-trace --stats --output-format csv -d OUT/trace -o trace -- {run}"]
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        out.append(f"rocprofv3 --pmc {c} --output-format csv -d OUT/step_{c} -o step_{c} -- {gemm}")
        out.append(f"rocprofv3 --pmc {c} --output-format csv -d OUT/copy_{c} -o copy_{c} -- {copy}")
    return out


def _short(name: str) -> str:
    m = re.search(r"(\w+_kernel)<([^>]*)>", name) or re.search(r"(\w+kernel\w*)", name)
    return m.group(0) if m else name[:48]


def _counter_means(path: str):
    agg = collections.defaultdict(list)
    with open(path) as f:
        for r in csv.DictReader(f):
            agg[_short(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in agg.items()}


def summarize(out_dir: str, workload: str, phase: str, sizes: str, summary: str, copy_bytes: int,
              live_gemm_us: float | None = None) -> str:
    lines = [f"# rocprofv3: GEMM in the {phase} phase of bench.py, {workload}", ""]
    lines.append("Commands (from /tmp with TMPDIR=/tmp; R = repository root, OUT = output folder):")
    lines.append("```")
    lines += commands(workload, phase, sizes)
    lines.append("```")
    lines.append("")
    lines.append("## Kernel trace (--stats)")
    lines.append("")
    lines.append("| kernel | calls | avg us | min us | max us |")
    lines.append("|---|---|---|---|---|")
    gemm_avg = None
    gemm_name = None
    with open(os.path.join(out_dir, "trace", "trace_kernel_stats.csv")) as f:
        for r in csv.DictReader(f):
            k = _short(r["Name"])
            avg = float(r["AverageNs"]) / 1e3
            lines.append(f"| {k} | {r['Calls']} | {avg:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                         f"{float(r['MaxNs']) / 1e3:.2f} |")
            if "gemm_signal_kernel" in k or "gemm_w4_kernel" in k:
                gemm_avg, gemm_name = avg, k
    # The step phase runs warmup + timed + instrumented passes; bench.py's
    # live GEMM figure is the average over the instrumented pass, so the
    # trace is also averaged over the same (last) launches.
    last_avg, last_n = None, 20
    tpath = os.path.join(out_dir, "trace", "trace_kernel_trace.csv")
    if gemm_name is not None and os.path.exists(tpath):
        with open(tpath) as f:
            d = sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for r in csv.DictReader(f)
                       if _short(r["Kernel_Name"]) == gemm_name)
        if len(d) >= last_n:
            last_avg = sum(e - b for b, e in d[-last_n:]) / last_n / 1e3
    if live_gemm_us is not None and gemm_avg is not None:
        lines.append("")
        lines.append(f"GEMM launch average measured by bench.py with HIP events in the same phase "
                     f"(its instrumented pass, {last_n} launches): {live_gemm_us:.2f} us; trace over the same "
                     f"{last_n} launches: " + (f"{last_avg:.2f} us" if last_avg is not None else "n/a") +
                     f" (all {gemm_avg:.2f} us above include warm-up).")
    vals = {p: _counter_means(os.path.join(out_dir, p, f"{p}_counter_collection.csv"))
            for p in ("step_FETCH_SIZE", "step_WRITE_SIZE", "copy_FETCH_SIZE", "copy_WRITE_SIZE")}
    copy_k = [k for k in vals["copy_FETCH_SIZE"] if "consume" in k][0]
    lines.append("")
    lines.append("## HBM-side byte counters (KiB per dispatch, averages; GEMM launched alone)")
    lines.append("")
    lines.append("| kernel | FETCH_SIZE | WRITE_SIZE |")
    lines.append("|---|---|---|")
    for k in vals["step_FETCH_SIZE"]:
        lines.append(f"| {k} | {vals['step_FETCH_SIZE'][k]:.1f} | {vals['step_WRITE_SIZE'].get(k, 0.0):.1f} |")
    cf, cw = vals["copy_FETCH_SIZE"][copy_k], vals["copy_WRITE_SIZE"][copy_k]
    lines.append(f"| plain copy of {copy_bytes} bytes ({copy_k}) | {cf:.1f} | {cw:.1f} |")
    fscale, wscale = copy_bytes / (cf * 1024.0), copy_bytes / (cw * 1024.0)
    gf = vals["step_FETCH_SIZE"][gemm_name]
    gw = vals["step_WRITE_SIZE"][gemm_name]
    traffic = gf * 1024.0 * fscale + gw * 1024.0 * wscale
    lines.append("")
    lines.append(f"Scale from the plain copy: FETCH_SIZE x {fscale:.3f}, WRITE_SIZE x {wscale:.3f}. "
                 f"GEMM HBM traffic per launch: {traffic / 1e6:.1f} MB "
                 f"(read {gf * 1024.0 * fscale / 1e6:.1f} MB, written {gw * 1024.0 * wscale / 1e6:.1f} MB).")
    lines.append("")
    lines.append("## Figures read by bench.py")
    lines.append("")
    lines.append("```")
    lines.append(f"workload: {workload}")
    lines.append(f"phase: {phase}")
    lines.append(f"groups: {sizes}")
    lines.append(f"kernel: {gemm_name}")
    lines.append(f"gemm_sources_sha256: {gemm_sources_sha256()}")
    lines.append(f"gemm_trace_avg_us: {gemm_avg:.3f}")
    lines.append(f"gemm_fetch_kib: {gf:.1f}")
    lines.append(f"gemm_write_kib: {gw:.1f}")
    lines.append(f"fetch_scale: {fscale:.4f}")
    lines.append(f"write_scale: {wscale:.4f}")
    lines.append(f"traffic_bytes_per_launch: {traffic:.0f}")
    lines.append("```")
    text = "\n".join(lines) + "\n"
    with open(summary, "w") as f:
        f.write(text)
    return text


def read_traffic(summary: str, workload: str):
    """HBM bytes per GEMM launch from a committed summary, or None when the
    summary is missing, is for another workload, or the GEMM sources have
    changed since the counters were taken."""
    if not os.path.exists(summary):
        return None
    kv = {}
    with open(summary) as f:
        for line in f:
            m = re.match(r"^(\w+): (\S+)$", line.strip())
            if m:
                kv[m.group(1)] = m.group(2)
    if kv.get("workload") != workload or kv.get("gemm_sources_sha256") != gemm_sources_sha256():
        return None
    try:
        return float(kv["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


if __name__ == "__main__":
    out_dir, workload, phase, sizes, summary, copy_bytes = sys.argv[1:7]
    live = float(sys.argv[7]) if len(sys.argv) > 7 else None
    print(summarize(out_dir, workload, phase, sizes, summary, int(copy_bytes), live))
