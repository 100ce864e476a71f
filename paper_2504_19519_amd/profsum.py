"""Summaries of rocprofv3 runs of bench.py, and the HBM traffic they give.

`python -m paper_2504_19519_amd.profsum OUT WORKLOAD PHASE GROUPS SUMMARY.md COPY_BYTES [LIVE_US]`
(and `... profsum counters OUT WORKLOAD GROUPS SUMMARY.md STEP_SUMMARY.md FLOPS` for the serialized
step's bytes and the GEMM's MFMA / L2 counters, runs listed in `counter_commands()`)
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
    if gemm_avg is not None:
        lines.append("")
        lines.append(f"GEMM launch average over the {last_n} launches of the instrumented pass (after the "
                     f"warm-up and the timed steps): " + (f"{last_avg:.2f} us" if last_avg is not None else "n/a") +
                     (f"; bench.py's HIP events on the same launches: {live_gemm_us:.2f} us"
                      if live_gemm_us is not None else "") +
                     f" (the {gemm_avg:.2f} us of the table include the warm-up launches).")
    gemm_timed = last_avg if last_avg is not None else gemm_avg
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
    lines.append(f"gemm_trace_avg_us: {gemm_timed:.3f}")
    lines.append(f"gemm_trace_all_launches_avg_us: {gemm_avg:.3f}")
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


def counter_commands(workload: str, sizes: str, steps: int = 20, warmup: int = 5):
    base = f"python3 R/bench.py --workload {workload}"
    ser = f"{base} --phase step --serial --sizes {sizes} --steps {steps} --warmup {warmup} --skip-cpu"
    gemm = f"{base} --phase gemm --steps {steps} --warmup {warmup} --skip-cpu"
    return [f"rocprofv3 --kernel-trace --stats --output-format csv -d OUT/sertrace -o sertrace -- {ser}",
            f"rocprofv3 --pmc FETCH_SIZE --output-format csv -d OUT/ser_FETCH_SIZE -o ser_FETCH_SIZE -- {ser}",
            f"rocprofv3 --pmc WRITE_SIZE --output-format csv -d OUT/ser_WRITE_SIZE -o ser_WRITE_SIZE -- {ser}",
            f"rocprofv3 --kernel-trace --stats --output-format csv -d OUT/gtrace -o gtrace -- {gemm}",
            "rocprofv3 --pmc " + " ".join(MFMA_COUNTERS) + f" --output-format csv -d OUT/mfma -o mfma -- {gemm}",
            f"rocprofv3 --pmc TCC_HIT_sum TCC_MISS_sum --output-format csv -d OUT/l2 -o l2 -- {gemm}"]


MFMA_COUNTERS = ["SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CYCLES", "GRBM_GUI_ACTIVE", "SQ_WAVE_CYCLES", "SQ_INSTS_MFMA",
                 "SQ_WAIT_ANY", "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT"]


def _stats(path):
    out = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            out[_short(r["Name"])] = (int(r["Calls"]), float(r["AverageNs"]) / 1e3)
    return out


def _counters(path):
    """Per kernel: each counter's mean per dispatch (the dimensions of one
    dispatch summed) and the dispatches' mean duration (_dur_us)."""
    per = collections.defaultdict(lambda: collections.defaultdict(float))
    dur = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            key = (_short(r["Kernel_Name"]), r["Dispatch_Id"])
            per[key][r["Counter_Name"]] += float(r["Counter_Value"])
            dur[key] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    for (k, d), cs in per.items():
        for c, v in cs.items():
            agg[k][c].append(v)
        agg[k]["_dur_us"].append(dur[(k, d)])
    return {k: {c: sum(v) / len(v) for c, v in cs.items()} for k, cs in agg.items()}


def summarize_counters(out_dir: str, workload: str, sizes: str, summary: str, fetch_scale: float,
                       write_scale: float, flops: float, peak_tflops: float = 2516.6) -> str:
    """The serialized step's kernels (trace and HBM bytes) and the GEMM
    alone's MFMA and L2 counters."""
    ser = _stats(os.path.join(out_dir, "sertrace", "sertrace_kernel_stats.csv"))
    sf = _counters(os.path.join(out_dir, "ser_FETCH_SIZE", "ser_FETCH_SIZE_counter_collection.csv"))
    sw = _counters(os.path.join(out_dir, "ser_WRITE_SIZE", "ser_WRITE_SIZE_counter_collection.csv"))
    gt = _stats(os.path.join(out_dir, "gtrace", "gtrace_kernel_stats.csv"))
    mf = _counters(os.path.join(out_dir, "mfma", "mfma_counter_collection.csv"))
    l2 = _counters(os.path.join(out_dir, "l2", "l2_counter_collection.csv"))
    lines = [f"# rocprofv3: serialized step and the signalling GEMM alone, {workload}", "",
             "Commands (from /tmp with TMPDIR=/tmp; R = repository root, OUT = output folder):", "```"]
    lines += counter_commands(workload, sizes)
    lines += ["```", "", "## Serialized step (consumers and post-reorder on the GEMM stream): trace and HBM-side bytes",
              "", f"FETCH_SIZE x {fetch_scale:.4f} and WRITE_SIZE x {write_scale:.4f} (the plain-copy calibration of "
              f"gemm_step_{workload}.md).", "",
              "| kernel | calls | avg us | bytes read / launch | bytes written / launch | GB/s |", "|---|---|---|---|---|---|"]
    for k, (calls, us) in sorted(ser.items(), key=lambda kv: -kv[1][1]):
        rd = sf.get(k, {}).get("FETCH_SIZE", 0.0) * 1024 * fetch_scale
        wr = sw.get(k, {}).get("WRITE_SIZE", 0.0) * 1024 * write_scale
        lines.append(f"| {k} | {calls} | {us:.2f} | {rd / 1e6:.1f} MB | {wr / 1e6:.1f} MB | {(rd + wr) / us / 1e3:.0f} |")
    gk = [k for k in mf if "gemm_signal_kernel" in k or "gemm_w4_kernel" in k][0]
    m, h = mf[gk], l2[gk]
    gus = m["_dur_us"]
    cycles = m["GRBM_GUI_ACTIVE"] / 8            # the counter sums the 8 chiplets
    busy = m["SQ_VALU_MFMA_BUSY_CYCLES"]
    lines += ["", "## Signalling GEMM alone: MFMA and L2 counters (per launch, averages)", "",
              "| counter | value |", "|---|---|"]
    for c in MFMA_COUNTERS + ["TCC_HIT_sum", "TCC_MISS_sum"]:
        lines.append(f"| {c} | {(m if c in m else h)[c]:.0f} |")
    lines += ["",
              f"- GEMM launch ({gk}): {gt[gk][1]:.1f} us trace average over {gt[gk][0]} launches; {gus:.1f} us "
              f"in the counter run.",
              f"- MFMA busy cycles per MFMA instruction: {busy / m['SQ_INSTS_MFMA']:.1f}.",
              f"- GRBM_GUI_ACTIVE / 8 chiplets = {cycles:.0f} cycles in {gus:.1f} us: {cycles / gus / 1e3:.2f} GHz.",
              f"- MFMA utilisation at that clock: {busy:.0f} / (1024 SIMDs x {cycles:.0f}) = "
              f"{busy / (1024 * cycles) * 100:.1f} %.",
              f"- Against the published peak (2.4 GHz, {peak_tflops} TFLOP/s): {flops / gus / 1e6:.0f} TFLOP/s = "
              f"{flops / gus / 1e6 / peak_tflops * 100:.1f} %.",
              f"- Wave-cycles waiting (SQ_WAIT_ANY / SQ_WAVE_CYCLES): {m['SQ_WAIT_ANY'] / m['SQ_WAVE_CYCLES'] * 100:.1f} %.",
              f"- L2 hit rate: {h['TCC_HIT_sum'] / (h['TCC_HIT_sum'] + h['TCC_MISS_sum']) * 100:.1f} %; LDS bank "
              f"conflicts: {m['SQ_LDS_BANK_CONFLICT'] / m['SQ_INSTS_LDS'] * 100:.1f} per 100 LDS instructions."]
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
    if sys.argv[1] == "counters":
        # counters OUT WORKLOAD GROUPS SUMMARY.md STEP_SUMMARY.md FLOPS
        out_dir, workload, sizes, summary, step_summary, flops = sys.argv[2:8]
        kv = {}
        with open(step_summary) as f:
            for line in f:
                mm = re.match(r"^(\w+): (\S+)$", line.strip())
                if mm:
                    kv[mm.group(1)] = mm.group(2)
        print(summarize_counters(out_dir, workload, sizes, summary, float(kv["fetch_scale"]),
                                 float(kv["write_scale"]), float(flops)))
    else:
        out_dir, workload, phase, sizes, summary, copy_bytes = sys.argv[1:7]
        live = float(sys.argv[7]) if len(sys.argv) > 7 else None
        print(summarize(out_dir, workload, phase, sizes, summary, int(copy_bytes), live))
