#!/usr/bin/env python3
"""Benchmark of the signaled + reordered GEMM path on one MI355X.

A step is one pass of the whole path over one batch of synthetic input:
counter reset -> signalling, reordering GEMM on stream 1 || per-group
consumers on stream 2 -> post-reorder (fused bias / RMSNorm when the workload
has them). Inputs are resident in HBM before the timed region starts.

Headline workload: fp16 GEMM M=8192, N=8192, K=3584 (MLP down-projection
shard), 256x256 tiles (4 waves on 256 CUs), ReduceScatter stand-in (R=4)
with the group partition chosen by the planner's predictive search from the
measured GEMM time and consumer latency curve.

Prints one JSON line. `value` is whole-step throughput (GEMM flops / time of
the whole step: GEMM, consumers and post-reorder); `roofline` is the GEMM
kernel itself (its launches timed with HIP events on the GEMM's stream inside
overlapped steps). Further keys: the GEMM alone with the plain row-major
epilogue (static schedule, and the same position dispensers, coherent stores
and counters as the signalling runs), the overhead of each reorder pattern
(Section 6.6, Table 5: GEMM epilogue and fused post-reorder + RMSNorm), the
consumer's and the post-reorder's HBM bandwidth, overlapped vs serialized
steps, the fraction of the theoretical speedup (Section 6.4), Algorithm 1's
estimate against measurement, the group-size sweep at two tile shapes, every
other workload's summary, and `cpu_baseline` (the oracle's whole path on a
bounded sample).
"""
from __future__ import annotations

import argparse
import ctypes
import dataclasses
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2504_19519_amd as fo  # noqa: E402
import workloads  # noqa: E402

METRIC = "signaled+reordered fp16 GEMM TFLOP/s (% MFMA peak); overlap speedup vs serial"
PEAK_TFLOPS = 256 * 2.4e9 * 4096 / 1e12      # dense fp16/bf16 MFMA: 2516.6 TFLOP/s
PEAK_HBM_GBS = 8000.0
HEADLINE = "rs_8192x8192x3584"
OTHER_WORKLOADS = ("tiny", "ar_2048x4096x4096", "ar_rmsnorm_16384x4096x3584_bf16", "a2a_4096x7168x2048")

# Options of every library call of this run (None: the process defaults); the
# slow-link phase sets a consumer launch cap here.
OPTS = None


# The run's streams, created once: the GEMM stream, the consumer stream and
# one more for a GEMM that a consumer measurement runs beside. HIP maps
# streams onto a few hardware queues per device (GPU_MAX_HW_QUEUES, 4 by
# default); each new pair of streams in a process risks sharing a queue
# with another stream, and kernels of one queue do not overlap (measured:
# a second stream pair in the process took a2a_4096x7168x2048 from 147 to
# 164 us per step), so every phase reuses these.
_STREAMS = None


def streams(torch):
    global _STREAMS
    if _STREAMS is None:
        _STREAMS = tuple(torch.cuda.Stream() for _ in range(3))
    return _STREAMS


class Ev:
    """A HIP event of the process's HIP runtime (the one torch loaded). For
    timing marks it is created with hipEventDisableSystemFence: recording it
    then does not write back and invalidate the caches, which would add to
    the interval it brackets (a GEMM bracketed by torch's events measured ~8
    us longer than its kernel trace). fence=True: a default event, for one
    that another stream waits on."""
    _hip = None

    @classmethod
    def _lib(cls):
        if cls._hip is None:
            with open("/proc/self/maps") as f:
                paths = sorted({ln.split()[-1] for ln in f if ln.rstrip().endswith(".so") and
                                os.path.basename(ln.split()[-1]).startswith("libamdhip64")})
            assert paths, "the HIP runtime is not loaded"
            h = ctypes.CDLL(paths[0])
            vp = ctypes.c_void_p
            h.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(vp), ctypes.c_uint]
            h.hipEventRecord.argtypes = [vp, vp]
            h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
            h.hipEventDestroy.argtypes = [vp]
            h.hipStreamWaitEvent.argtypes = [vp, vp, ctypes.c_uint]
            cls._hip = h
        return cls._hip

    def __init__(self, fence=False):
        h = ctypes.c_void_p()
        rc = self._lib().hipEventCreateWithFlags(ctypes.byref(h), 0 if fence else 0x20000000)
        assert rc == 0, f"hipEventCreateWithFlags: {rc}"
        self.cuda_event = h.value

    def record(self, stream):
        rc = self._lib().hipEventRecord(self.cuda_event, stream.cuda_stream)
        assert rc == 0, f"hipEventRecord: {rc}"

    def elapsed_time(self, end):
        ms = ctypes.c_float()
        rc = self._lib().hipEventElapsedTime(ctypes.byref(ms), self.cuda_event, end.cuda_event)
        assert rc == 0, f"hipEventElapsedTime: {rc}"
        return ms.value

    def wait(self, stream):
        rc = self._lib().hipStreamWaitEvent(stream.cuda_stream, self.cuda_event, 0)
        assert rc == 0, f"hipStreamWaitEvent: {rc}"

    def __del__(self):
        try:
            if self.cuda_event and Ev._hip is not None:
                Ev._hip.hipEventDestroy(self.cuda_event)
        except Exception:      # interpreter shutdown
            pass


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=HEADLINE, choices=list(workloads.WORKLOADS))
    ap.add_argument("--phase", default="all",
                    choices=["all", "step", "gemm", "copy", "predict", "trace", "slowlink", "sync"],
                    help="step/gemm/copy run only that loop (for profiler runs); predict: Algorithm 1's "
                         "estimate vs the measured GEMM+consume time of every partition, at the workload's "
                         "size and at M/4, M/2 and 2M; trace: tile timeline; slowlink: consumer launch caps; "
                         "sync: the producer/consumer publication modes")
    ap.add_argument("--sizes", default=None, help="explicit partition in waves, e.g. 1,1,2,4")
    ap.add_argument("--tile", default=None, help="override the workload's output tile, e.g. 256x128")
    ap.add_argument("--consumer-grid", default=None,
                    help="grid of the consumers beside the GEMM: BLOCKSxTHREADS, e.g. 256x64")
    ap.add_argument("--serial", action="store_true", help="step phase: run the consumers on the GEMM stream")
    ap.add_argument("--skip-cpu", action="store_true")
    ap.add_argument("--skip-workloads", action="store_true", help="headline workload only")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    return ap.parse_args()


class Bufs:
    def __init__(self, torch, w, inp, dest_elems):
        dev = "cuda"

        def d(bits):
            return torch.from_numpy(np.ascontiguousarray(bits).reshape(-1).view(np.int16)).to(dev)

        self.A, self.W = d(inp.A), d(inp.W)
        self.peer = d(inp.peer) if w.pattern != "subtoken" else None
        self.bias = d(inp.bias) if inp.bias is not None else None
        self.gamma = d(inp.gamma) if inp.gamma is not None else None
        n = w.M * w.N
        self.C = torch.empty(n, dtype=torch.int16, device=dev)
        self.dst = torch.empty(max(dest_elems, n), dtype=torch.int16, device=dev)
        self.out = torch.empty(n, dtype=torch.int16, device=dev)
        self.counters = torch.zeros(1024, dtype=torch.int32, device=dev)   # >= fo_plan_num_counters of any plan here
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)


def dev_plan(torch, plan):
    buf = torch.empty(plan.device_bytes // 4 + 4, dtype=torch.int32, device="cuda")
    plan.to_device(buf)
    return buf


def check_status(b, what):
    if int(b.status.cpu()[0]) != 0:
        raise RuntimeError(f"a device-side wait timed out during {what}")


def time_loop(torch, fn, iters, warmup, stream):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0, e1 = Ev(), Ev()
    e0.record(stream)
    for _ in range(iters):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1000.0 / iters      # us per iteration


def time_gemm(torch, plan, dp, b, stream, iters, warmup, signal=True, opts=None):
    """Mean time of one GEMM launch (us), each bracketed by its own event
    pair; with signal=True the group counters are zeroed before every launch
    (outside the events) and the GEMM signals them, taking its positions from
    the dispensers; signal=False: no counters (static schedule, plain
    stores)."""
    ev = [(Ev(), Ev()) for _ in range(iters)]

    def one(pair=None):
        if signal:
            fo.reset_counters(b.counters, plan.num_counters, stream)
        if pair:
            pair[0].record(stream)
        fo.gemm_signal_reorder(plan, dp, b.A, b.W, b.C, b.counters if signal else None, stream,
                               opts=opts if opts is not None else OPTS)
        if pair:
            pair[1].record(stream)

    for _ in range(warmup):
        one()
    torch.cuda.synchronize()
    for k in range(iters):
        one(ev[k])
    torch.cuda.synchronize()
    return float(np.mean([a.elapsed_time(c) * 1000.0 for a, c in ev]))


# The All-to-All stand-in moves every destination's piece of a group through
# this one device, so Algorithm 1's estimate counts all of them (on several
# GPUs the largest piece, the slowest link, would set the time).
DEST_BYTES = "all"


def make_plan(w, inp, num_cus, sizes=None, pattern=None, gemm_us=0.0, curve=None, bucket=None):
    """The plan of workload w (or of another reorder pattern on its shape:
    R = 4 identity destinations for subtile, B = 8 buckets from `bucket` for
    subtoken)."""
    pattern = pattern or w.pattern
    if pattern == w.pattern:
        nd = w.num_dest if pattern in ("subtile", "subtoken") else 0
        sigma = inp.sigma if pattern == "subtile" else None
        bucket = inp.bucket if pattern == "subtoken" and bucket is None else bucket
    else:
        nd = {"subtile": 4, "subtoken": 8}.get(pattern, 0)
        sigma = None
    kw = dict(dtype=w.dtype, tile_m=w.tile_m, tile_n=w.tile_n, order=w.order, num_cus=num_cus,
              pattern=pattern, num_dest=nd, dest_perm=sigma,
              row_bucket=bucket if pattern == "subtoken" else None, dest_bytes=DEST_BYTES)
    if sizes is not None:
        if curve is not None:      # given partition + Algorithm 1's estimate of it
            return fo.plan_groups(w.M, w.N, w.K, sizes=list(sizes), gemm_us=gemm_us, **curve_kw(curve), **kw)
        return fo.plan_groups(w.M, w.N, w.K, sizes=list(sizes), **kw)
    if curve is None:
        tiles = (w.M // w.tile_m) * (w.N // w.tile_n)
        return fo.plan_groups(w.M, w.N, w.K, sizes=[-(-tiles // num_cus)], **kw)
    return fo.plan_groups(w.M, w.N, w.K, sizes=None, gemm_us=gemm_us, s_first=2, s_last=4, **curve_kw(curve),
                          **kw)


def curve_kw(curve):
    """Planner keywords of a curve: (bytes, us) of the groups beside the
    GEMM, optionally followed by (bytes, us) of the last group's."""
    kw = dict(curve_bytes=curve[0], curve_us=curve[1])
    if len(curve) > 2:
        kw.update(last_curve_bytes=curve[2], last_curve_us=curve[3])
    return kw


def run_step(torch, w, plan, dp, b, s1, s2, ev=None):
    fo.run_overlapped(plan, dp, b.A, b.W, b.C, b.peer, b.dst, b.out, b.bias, b.gamma, w.eps,
                      w.rmsnorm, b.counters, b.status, s1, s2,
                      ev[0] if ev else None, ev[1] if ev else None, opts=OPTS)


def timed_steps(torch, w, plan, dp, b, s1, s2, steps, warmup):
    """Warmup, then exactly `steps` steps between a device-wide sync and two
    events on s1 (s1 joins s2 before the post-reorder of every step). A
    second, untimed pass of the same steps brackets each GEMM launch with an
    event pair for the GEMM's duration inside the step; those events stay out
    of the timed pass, as recording them would add to its time."""
    ev = [(Ev(), Ev()) for _ in range(steps)]
    for a, c in ev:          # create the events
        a.record(s1)
        c.record(s1)
    for _ in range(warmup):
        run_step(torch, w, plan, dp, b, s1, s2)
    torch.cuda.synchronize()
    t0, t1 = Ev(), Ev()
    wall0 = time.perf_counter()
    t0.record(s1)
    for k in range(steps):
        run_step(torch, w, plan, dp, b, s1, s2)
    t1.record(s1)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    step_us = t0.elapsed_time(t1) * 1000.0 / steps
    check_status(b, "the timed steps")
    for k in range(steps):
        run_step(torch, w, plan, dp, b, s1, s2, ev[k])
    torch.cuda.synchronize()
    gemm = [a.elapsed_time(c) * 1000.0 for a, c in ev]
    check_status(b, "the instrumented steps")
    return step_us, float(np.mean(gemm)), float(np.median(gemm)), wall


def traffic_bytes(w):
    """HBM bytes per GEMM launch (FETCH_SIZE + WRITE_SIZE, scaled by a plain
    copy of known size) from the committed rocprofv3 summary of this
    workload's overlapped steps; None if there is none or the GEMM has
    changed since it was taken."""
    from paper_2504_19519_amd import profsum
    t = profsum.read_traffic(os.path.join(ROOT, "profiles", f"gemm_step_{w.name}.md"), w.name)
    return None if t is None else round(t)


def consume_all(torch, w, b, stream, n, iters, warmup):
    """The consumer over the whole buffer in one launch on the full grid (how
    the last group of an overlapped run streams)."""
    full = fo.options(consumer_blocks=256, consumer_threads=256)
    if OPTS is not None:
        full.consumer_limit = OPTS.consumer_limit
    return time_loop(torch, lambda: fo.consume_group(b.C, b.peer, b.dst, n, w.dtype, None, 0, None, stream,
                                                     opts=full), iters, warmup, stream)


def consumer_curve(torch, w, b, stream, total_elems, beside=None):
    """Consumer latency vs bytes (one launch, no wait, the grid the consumers
    beside the GEMM use): the 1-GPU stand-in for the communication bandwidth
    curve the search interpolates. With beside = (plan, dev_plan) each
    launch is timed while that GEMM runs on another stream (every group but
    the last streams beside the GEMM, and there the stand-in is slower than
    alone); without, alone."""
    sizes = []
    n = 1 << 15
    while n <= total_elems:
        sizes.append(n)
        if n == total_elems:
            break
        n = min(n * 2, total_elems)
    launch = lambda n: fo.consume_group(b.C, b.peer, b.dst, n, w.dtype, None, 0, None, stream, opts=OPTS)
    if beside is None:
        return [2.0 * n for n in sizes], [time_loop(torch, lambda: launch(n), 20, 3, stream) for n in sizes]
    plan, dp = beside
    sg = streams(torch)[2]
    ys = []
    for n in sizes:
        vals = []
        for r in range(6):
            eg, e0, e1 = Ev(fence=True), Ev(), Ev()
            eg.record(sg)
            for _ in range(2):        # about 700 us of GEMM for the consumer to run beside
                fo.gemm_signal_reorder(plan, dp, b.A, b.W, b.C, None, sg)
            eg.wait(stream)
            e0.record(stream)
            launch(n)
            e1.record(stream)
            torch.cuda.synchronize()
            if r > 0:
                vals.append(e0.elapsed_time(e1) * 1000.0)
        ys.append(float(np.median(vals)))
    return [2.0 * n for n in sizes], ys


def consumer_curve_after(torch, w, b, inp, num_cus, s1, s2, total_elems):
    """The last group's latency vs bytes: a consumer on the full grid, on the
    communication stream, waiting for the GEMM's one group counter (a plan of
    one group), timed from the GEMM's end to its own end -- the part of an
    overlapped run that follows the GEMM."""
    tiles = (w.M // w.tile_m) * (w.N // w.tile_n)
    one = make_plan(w, inp, num_cus, sizes=[-(-tiles // num_cus)])
    dp = dev_plan(torch, one)
    full = fo.options(consumer_blocks=256, consumer_threads=256)
    if OPTS is not None:
        full.consumer_limit = OPTS.consumer_limit
    sizes = []
    n = 1 << 15
    while n <= total_elems:
        sizes.append(n)
        if n == total_elems:
            break
        n = min(n * 2, total_elems)
    ys = []
    for n in sizes:
        vals = []
        for r in range(5):
            er, eg, e1 = Ev(fence=True), Ev(), Ev()
            fo.reset_counters(b.counters, one.num_counters, s1)
            er.record(s1)
            fo.gemm_signal_reorder(one, dp, b.A, b.W, b.C, b.counters, s1)
            eg.record(s1)
            er.wait(s2)
            fo.consume_group(b.C, b.peer, b.dst, n, w.dtype, b.counters, int(one.targets[0]), b.status, s2,
                             opts=full)
            e1.record(s2)
            torch.cuda.synchronize()
            if r > 0:
                vals.append(eg.elapsed_time(e1) * 1000.0)
        ys.append(float(np.median(vals)))
    check_status(b, "the last group's latency curve")
    return [2.0 * n for n in sizes], ys


def gemm_comm_times(torch, w, plan, dp, b, s1, s2, steps, with_gemm=False):
    """GEMM + consume time of overlapped runs without the post-reorder: from
    the GEMM's start (event on the GEMM stream) to the end of the last
    consumer (event on the stream it ran on: the communication stream, or
    the GEMM stream for a plan of one group, which runs serialized)."""
    ev = [(Ev(), Ev(), Ev()) for _ in range(steps)]
    last = s2 if plan.P > 1 else s1
    for a, g, c in ev:       # create the events
        a.record(s1)
        g.record(s1)
        c.record(last)
    for a, g, c in ev:
        fo.run_overlapped(plan, dp, b.A, b.W, b.C, b.peer, b.dst, None, None, None, w.eps, False,
                          b.counters, b.status, s1, s2, a, g, opts=OPTS)
        c.record(last)
    torch.cuda.synchronize()
    check_status(b, "GEMM + consume runs")
    if with_gemm:
        return [a.elapsed_time(c) * 1000.0 for a, g, c in ev], [a.elapsed_time(g) * 1000.0 for a, g, c in ev]
    return [a.elapsed_time(c) * 1000.0 for a, g, c in ev]


def theoretical(plan, sig_us, cons_all_us, post_us):
    """Lower bound of an overlapped step (Section 6.4: the communication of
    the last group cannot be hidden, nor that of the first group before its
    compute is done): the GEMM plus the last group's share of the consumer,
    or the first group's compute plus the whole consumer, plus the
    post-reorder."""
    tiles = int(sum(plan.targets))
    last_share = plan.targets[-1] / tiles
    first = sig_us * plan.targets[0] / tiles
    return max(sig_us + cons_all_us * last_share, first + cons_all_us) + post_us


def overlap_rounds(torch, w, plan, dp, base_plan, dp_base, b, s1, s2, rounds, per):
    """Overlapped and serialized steps, GEMM + consume of the overlapped run,
    the GEMM alone and the consumer alone (whole buffer, full grid), in
    alternating rounds so that all see the same device state (clock,
    temperature)."""
    ov, se, ov_g, se_g, gc, ga, ca = [], [], [], [], [], [], []
    n_all = w.M * w.N
    for _ in range(rounds):
        us, gm, _, _ = timed_steps(torch, w, plan, dp, b, s1, s2, per, 2)
        ov.append(us)
        ov_g.append(gm)
        us, gm, _, _ = timed_steps(torch, w, plan, dp, b, s1, s1, per, 2)
        se.append(us)
        se_g.append(gm)
        gc.append(float(np.median(gemm_comm_times(torch, w, plan, dp, b, s1, s2, per))))
        ga.append(time_gemm(torch, base_plan, dp_base, b, s1, per, 1))
        ca.append(consume_all(torch, w, b, s1, n_all, per, 1))
    med = lambda v: float(np.median(v))  # noqa: E731
    return {"overlapped_step_us": med(ov), "serial_step_us": med(se), "overlapped_rounds_us": ov,
            "serial_rounds_us": se, "gemm_in_overlapped_us": med(ov_g), "gemm_in_serial_us": med(se_g),
            "gemm_consume_overlapped_us": med(gc), "gemm_alone_us": med(ga), "consume_alone_us": med(ca)}


def overlap_fields(r, bound_us):
    """Derived overlap figures: speedup over the serialized step, GEMM +
    consume against max(GEMM, consume), and the fractions of the theoretical
    bound (Section 6.4: achieved over theoretical speedup, and bound over
    achieved time)."""
    ov, se = r["overlapped_step_us"], r["serial_step_us"]
    th_speedup = se / bound_us
    return {
        "overlapped_step_us": round(ov, 2), "serial_step_us": round(se, 2),
        "speedup_vs_serial": round(se / ov, 4),
        "gemm_consume_overlapped_us": round(r["gemm_consume_overlapped_us"], 2),
        "gemm_alone_us": round(r["gemm_alone_us"], 2), "consume_alone_us": round(r["consume_alone_us"], 2),
        "overlapped_gemm_consume_over_max": round(r["gemm_consume_overlapped_us"] /
                                                  max(r["gemm_alone_us"], r["consume_alone_us"]), 4),
        "gemm_in_overlapped_us": round(r["gemm_in_overlapped_us"], 2),
        "gemm_in_serial_us": round(r["gemm_in_serial_us"], 2),
        "theoretical_bound_us": round(bound_us, 2), "theoretical_speedup": round(th_speedup, 4),
        "fraction_of_theoretical_speedup": round((se / ov - 1) / (th_speedup - 1), 4) if th_speedup > 1 else None,
        "fraction_of_theoretical_performance": round(bound_us / ov, 4),
    }


def with_bucket_seed(w):
    """A seeded row-to-bucket map for the subtoken pattern on a workload that
    has none (the Table 5 analogue on the headline shape)."""
    return np.random.default_rng(w.seed + 5).integers(0, 8, w.M).astype(np.int32)


def table5(torch, w, inp, b, num_cus, T, s1, rounds=3, iters=30):
    """Section 6.6, Table 5 analogue on this workload's shape: the GEMM with
    each reorder pattern's epilogue against the row-major epilogue, all
    signalling counters under the same position dispensers and coherent
    stores (interleaved rounds), and the fused post-reorder + RMSNorm of each
    pattern against the same kernel on the identity map; the plain gather
    (no norm) beside it."""
    bucket = with_bucket_seed(w)
    plans = {p: make_plan(w, inp, num_cus, sizes=[1] * T, pattern=p, bucket=bucket)
             for p in ("rowmajor", "tile", "subtile", "subtoken")}
    dps = {p: dev_plan(torch, q) for p, q in plans.items()}
    torch.cuda.synchronize()
    gemm = {p: [] for p in plans}
    static = []
    for _ in range(rounds):
        static.append(time_gemm(torch, plans["rowmajor"], dps["rowmajor"], b, s1, iters, 3, signal=False))
        for p in plans:
            gemm[p].append(time_gemm(torch, plans[p], dps[p], b, s1, iters, 3))
    g = {p: float(np.median(v)) for p, v in gemm.items()}
    st = float(np.median(static))
    n = w.M * w.N
    b.dst[:n].copy_(b.C[:n])        # finite values to normalise
    post = {}
    for norm in (False, True):
        ident = time_loop(torch, lambda: fo.post_reorder(plans["rowmajor"], None, b.dst, b.out, None, None, w.eps,
                                                         norm, s1), iters, 5, s1)
        post[norm] = {"identity_us": round(ident, 2)}
        for p in ("tile", "subtile", "subtoken"):
            us = time_loop(torch, lambda: fo.post_reorder(plans[p], dps[p], b.dst, b.out, None, None, w.eps, norm,
                                                          s1), iters, 5, s1)
            post[norm][p] = {"us": round(us, 2), "overhead_pct": round((us / ident - 1) * 100, 2)}
    rows = {p: {"us": round(g[p], 2), "overhead_pct": round((g[p] / g["rowmajor"] - 1) * 100, 2)}
            for p in ("tile", "subtile", "subtoken")}
    return {"shape": [w.M, w.N, w.K], "tile": [w.tile_m, w.tile_n],
            "gemm_rowmajor_signalled_us": round(g["rowmajor"], 2), "gemm_rowmajor_static_us": round(st, 2),
            "gemm_epilogue": rows,
            "post_reorder_rmsnorm": post[True], "post_reorder_gather": post[False],
            "paper_context": "A800 / RTX 4090: GEMM +0.07-0.68 %, fused RMSNorm +7.46-9.63 % (Table 5)"}


def sweep(torch, w, inp, num_cus, b, s1, s2, steps):
    """Group-size sweep (waves per group, Section 6.5) on the workload's tile
    and on 256x128 tiles (twice the waves), overlapped steps; sizes above the
    wave count are listed as skipped."""
    res = {}
    for tm, tn in sorted({(w.tile_m, w.tile_n), (256, 128)}, reverse=True):
        wt = dataclasses.replace(w, tile_m=tm, tile_n=tn)
        T = -(-((w.M // tm) * (w.N // tn)) // num_cus)
        rows, skipped = {}, []
        base = make_plan(wt, inp, num_cus, sizes=[1] * T)
        dbase = dev_plan(torch, base)
        torch.cuda.synchronize()
        alone = time_gemm(torch, base, dbase, b, s1, 20, 3)
        for g in (w.sweep or (1, 2, 4, 8)):
            if g > T:
                skipped.append(g)
                continue
            sizes = [g] * (T // g) + ([T % g] if T % g else [])
            p = make_plan(wt, inp, num_cus, sizes=sizes)
            d = dev_plan(torch, p)
            torch.cuda.synchronize()
            us, gm, _, _ = timed_steps(torch, wt, p, d, b, s1, s2, steps, 3)
            rows[str(g)] = {"groups": sizes, "step_us": round(us, 2), "gemm_us": round(gm, 2)}
        res[f"{tm}x{tn}"] = {"waves": T, "gemm_alone_us": round(alone, 2), "waves_per_group": rows,
                             "skipped_waves_per_group": skipped}
    return res


def workload_summary(torch, name, num_cus, steps):
    """One workload end to end: GEMM alone, consumer and post-reorder
    bandwidth, the Algorithm 1 plan, overlapped vs serialized steps and the
    overlap fractions."""
    w = workloads.WORKLOADS[name]
    log(f"workload {name}")
    inp = workloads.make_inputs(w)
    tiles = (w.M // w.tile_m) * (w.N // w.tile_n)
    T = -(-tiles // num_cus)
    s1, s2, _ = streams(torch)
    if w.groups is not None:
        base_plan = make_plan(w, inp, num_cus, sizes=list(w.groups)) if w.group_unit == "waves" else \
            fo.plan_groups(w.M, w.N, w.K, dtype=w.dtype, tile_m=w.tile_m, tile_n=w.tile_n, order=w.order,
                           num_cus=num_cus, pattern=w.pattern, sizes=list(w.groups), unit=w.group_unit)
    else:
        base_plan = make_plan(w, inp, num_cus, sizes=[1] * T)
    b = Bufs(torch, w, inp, base_plan.dest_elems)
    dp_base = dev_plan(torch, base_plan)
    torch.cuda.synchronize()
    sig_us = time_gemm(torch, base_plan, dp_base, b, s1, 30, 20)
    xs, ys = consumer_curve(torch, w, b, s1, w.M * w.N, beside=(base_plan, dp_base))
    lx, ly = consumer_curve_after(torch, w, b, inp, num_cus, s1, s2, w.M * w.N)
    if w.groups is not None:
        plan, dp = base_plan, dp_base
    else:
        plan = make_plan(w, inp, num_cus, gemm_us=sig_us, curve=(xs, ys, lx, ly))
        dp = dev_plan(torch, plan)
    torch.cuda.synchronize()
    r = overlap_rounds(torch, w, plan, dp, base_plan, dp_base, b, s1, s2, 3, max(6, steps // 4))
    post_us = time_loop(torch, lambda: fo.post_reorder(plan, dp, b.dst, b.out, b.bias, b.gamma, w.eps, w.rmsnorm,
                                                       s1), 30, 5, s1)
    n = w.M * w.N
    cons_bytes = (6 if b.peer is not None else 4) * n
    post_bytes = 4.0 * n + (2.0 * w.N * (int(w.bias) + int(w.gamma)))
    bound = theoretical(plan, r["gemm_alone_us"], r["consume_alone_us"], post_us)
    g_in = r["gemm_in_overlapped_us"]
    # the GEMM alone as measured in the interleaved rounds (the first
    # measurement above, right after the inputs were made, sees a colder
    # clock; it only feeds the search)
    ga = r["gemm_alone_us"]
    return {"M": w.M, "N": w.N, "K": w.K, "dtype": w.dtype, "pattern": w.pattern, "tile": [w.tile_m, w.tile_n],
            "waves": T, "groups": [int(x) for x in plan.sizes], "unit": w.group_unit,
            "gemm_alone_us": round(ga, 2), "gemm_tflops": round(w.flops / ga / 1e6, 2),
            "gemm_frac_peak": round(w.flops / ga / 1e6 / PEAK_TFLOPS, 4),
            "gemm_in_step_tflops": round(w.flops / g_in / 1e6, 2),
            "consumer_GBps": round(cons_bytes / r["consume_alone_us"] / 1e3, 1),
            "consumer_frac_hbm": round(cons_bytes / r["consume_alone_us"] / 1e3 / PEAK_HBM_GBS, 4),
            "post_reorder_us": round(post_us, 2), "post_reorder_GBps": round(post_bytes / post_us / 1e3, 1),
            "post_reorder_frac_hbm": round(post_bytes / post_us / 1e3 / PEAK_HBM_GBS, 4),
            "step_tflops": round(w.flops / r["overlapped_step_us"] / 1e6, 2),
            "overlap": overlap_fields(r, bound)}

def planner_report(w, inp, num_cus, gemm_us, curve):
    """Host cost of the planner's online stage (Section 4.2): Algorithm 1 on
    this workload vs. a lookup in a plan cache filled ahead of time for
    representative sizes of the same family (M/4, M/2, 2M; the GEMM time
    scaled with M), and the estimated latency of the cached partitions at
    unseen sizes against the search's own optimum there."""
    ckw = curve_kw(curve)
    kw = dict(dtype=w.dtype, tile_m=w.tile_m, tile_n=w.tile_n, order=w.order, num_cus=num_cus,
              pattern=w.pattern, num_dest=w.num_dest if w.pattern in ("subtile", "subtoken") else 0,
              dest_perm=inp.sigma if w.pattern == "subtile" else None, dest_bytes=DEST_BYTES)
    rng = np.random.default_rng(w.seed + 11)

    def bucket(M):
        return rng.integers(0, w.num_dest, M) if w.pattern == "subtoken" else None

    def search(M, b):
        return fo.plan_groups(M, w.N, w.K, row_bucket=b, sizes=None, gemm_us=gemm_us * M / w.M,
                              s_first=2, s_last=4, **ckw, **kw)

    b = bucket(w.M)
    reps = 20
    t0 = time.perf_counter()
    for _ in range(reps):
        search(w.M, b)
    search_us = (time.perf_counter() - t0) / reps * 1e6
    cache = fo.PlanCache()
    reps_m = [m for m in (w.M // 4, w.M // 2, 2 * w.M) if m % w.tile_m == 0 and m > 0]
    for m in reps_m:
        cache.add(m, w.N, w.K, row_bucket=bucket(m), sizes=None, gemm_us=gemm_us * m / w.M,
                  s_first=2, s_last=4, **ckw, **kw)
    t0 = time.perf_counter()
    for _ in range(reps):
        cache.lookup(w.M, w.N, w.K, row_bucket=b, **kw)
    lookup_us = (time.perf_counter() - t0) / reps * 1e6
    unseen = []
    for frac in (3, 5, 6, 7):          # M * frac / 4: between and beyond the cached sizes
        m = w.M * frac // 4
        if m % w.tile_m:
            continue
        bm = bucket(m)
        plan, matched = cache.lookup(m, w.N, w.K, row_bucket=bm, **kw)
        est = fo.plan_groups(m, w.N, w.K, row_bucket=bm, sizes=list(plan.sizes), gemm_us=gemm_us * m / w.M,
                             **ckw, **kw).predicted_us
        best = search(m, bm)
        unseen.append({"M": m, "matched_M": matched, "cached_groups": [int(x) for x in plan.sizes],
                       "searched_groups": [int(x) for x in best.sizes],
                       "estimate_cached_over_searched": round(est / best.predicted_us, 4)})
    return {"search_us": round(search_us, 1), "cache_lookup_us": round(lookup_us, 1),
            "cached_sizes_M": reps_m, "unseen": unseen}


def partitions(T):
    """Every composition of T waves, by cut vector (bit i = cut after wave i+1)."""
    out = []
    for x in range(1 << (T - 1)):
        sizes, run = [], 0
        for wv in range(1, T + 1):
            run += 1
            if wv == T or (x >> (wv - 1)) & 1:
                sizes.append(run)
                run = 0
        out.append(tuple(sizes))
    return out


def predictor_accuracy(torch, w, inp, b, base_plan, dp_base, num_cus, T, flops, s1, s2, args):
    """Algorithm 1's estimate against the measured GEMM+consume time for every
    partition of the waves (interleaved rounds), and the searched partition's
    measured time against the best measured one."""
    log("predictor: GEMM alone and consumer curve")
    sig_us = time_gemm(torch, base_plan, dp_base, b, s1, 50, 10)
    xs, ys = consumer_curve(torch, w, b, s1, w.M * w.N, beside=(base_plan, dp_base))
    lx, ly = consumer_curve_after(torch, w, b, inp, num_cus, s1, s2, w.M * w.N)
    cands = partitions(T)
    plans = {}
    for c in cands:
        p = make_plan(w, inp, num_cus, sizes=c, gemm_us=sig_us, curve=(xs, ys, lx, ly))
        plans[c] = (p, dev_plan(torch, p))
    searched = make_plan(w, inp, num_cus, gemm_us=sig_us, curve=(xs, ys, lx, ly))
    torch.cuda.synchronize()
    meas = {c: [] for c in cands}
    gemm_in = []
    for c in cands:                      # warm-up
        gemm_comm_times(torch, w, plans[c][0], plans[c][1], b, s1, s2, 2)
    for _ in range(5):
        for c in cands:
            t, g = gemm_comm_times(torch, w, plans[c][0], plans[c][1], b, s1, s2, 4, with_gemm=True)
            meas[c] += t
            if plans[c][0].P > 1:
                gemm_in += g
    # the same estimate fed with the GEMM's duration inside the overlapped
    # runs (slower than alone: the consumer's traffic), not modelled by the
    # GEMM-alone input
    gemm_ov = float(np.median(gemm_in)) if gemm_in else sig_us
    rows = []
    for c in cands:
        m = float(np.median(meas[c]))
        pr = plans[c][0].predicted_us
        pr_ov = make_plan(w, inp, num_cus, sizes=c, gemm_us=gemm_ov, curve=(xs, ys, lx, ly)).predicted_us
        rows.append({"groups": list(c), "predicted_us": round(pr, 2), "measured_us": round(m, 2),
                     "error_pct": round((pr - m) / m * 100, 2),
                     "predicted_overlap_gemm_us": round(pr_ov, 2),
                     "error_overlap_gemm_pct": round((pr_ov - m) / m * 100, 2)})
    best = min(rows, key=lambda r: r["measured_us"])
    pick = next(r for r in rows if tuple(r["groups"]) == tuple(int(x) for x in searched.sizes))
    pred_best = min(rows, key=lambda r: r["predicted_us"])
    return {"phase": "predict", "workload": w.name, "waves": T, "gemm_alone_us": round(sig_us, 2),
            "mean_abs_error_pct": round(float(np.mean([abs(r["error_pct"]) for r in rows])), 2),
            "gemm_in_overlap_us": round(gemm_ov, 2),
            "mean_abs_error_overlap_gemm_pct":
                round(float(np.mean([abs(r["error_overlap_gemm_pct"]) for r in rows])), 2),
            "searched_groups": pick["groups"], "searched_measured_us": pick["measured_us"],
            "best_measured_groups": best["groups"], "best_measured_us": best["measured_us"],
            "searched_over_best": round(best["measured_us"] / pick["measured_us"], 4),
            "unpruned_predicted_best": pred_best["groups"], "partitions": rows}


def tile_timeline(torch, w, plan, dp, b, stream):
    """Wave pattern of the signalling GEMM (Section 2.1.1, Figure 3): one
    traced launch after warm-up; per wave of W positions, how far apart its
    tiles start and finish against the wave's length, and whether position p
    ran on chiplet p mod 8 as the XCD dispatch order assumes."""
    tiles = plan.tiles
    trace = torch.zeros(4 * tiles, dtype=torch.int64, device="cuda")
    time_gemm(torch, plan, dp, b, stream, 10, 5)
    time_gemm(torch, plan, dp, b, stream, 1, 0,
              opts=fo.options(tile_trace=trace, tile_trace_capacity=tiles))
    khz = fo.device_wall_clock_khz()
    t = trace.cpu().numpy().reshape(-1, 4)
    us = 1000.0 / khz
    t0 = t[:, 0].min()
    start, end = (t[:, 0] - t0) * us, (t[:, 1] - t0) * us
    chip = (t[:, 2] >> 32) & 0xF
    W, T = plan.W, plan.T
    waves = []
    prev_end = 0.0
    for j in range(T):
        sl = slice(j * W, min((j + 1) * W, tiles))
        e_mean = float(end[sl].mean())
        waves.append({"wave": j, "tiles": int(end[sl].size),
                      "start_us": [round(float(start[sl].min()), 2), round(float(start[sl].max()), 2)],
                      "end_us": [round(float(end[sl].min()), 2), round(float(end[sl].max()), 2)],
                      "end_spread_over_wave_len": round(float(end[sl].max() - end[sl].min()) /
                                                        max(e_mean - prev_end, 1e-9), 4)})
        prev_end = e_mean
    pos = np.arange(tiles)
    dur = end - start
    per_chip = [{"chiplet": int(c), "tiles": int((chip == c).sum()),
                 "mean_tile_us": round(float(dur[chip == c].mean()), 2),
                 "last_end_us": round(float(end[chip == c].max()), 2)} for c in sorted(set(chip.tolist()))]
    return {"phase": "trace", "workload": w.name, "tiles": int(tiles), "wave_width": int(W), "waves": waves,
            "per_chiplet": per_chip,
            "kernel_us": round(float(end.max()), 2),
            "chiplets_seen": int(len(set(chip.tolist()))),
            "position_on_chiplet_p_mod_8": round(float(np.mean(chip == pos % 8)), 4)}


def vendor_gemm(torch, w, plan, dp, b, stream, iters, rounds=3):
    """Context for the GEMM's roofline fraction: the vendor library's GEMM of
    the same operands (torch.nn.functional.linear, A x W^T, hipBLASLt on
    ROCm; a plain 2-D product, no reorder or signal) timed in rounds that
    alternate with the signalled, reordered GEMM alone on the same box."""
    import torch.nn.functional as F
    dt = torch.float16 if w.dtype == "fp16" else torch.bfloat16
    A = b.A.view(dt).reshape(w.M, w.K)
    W = b.W.view(dt).reshape(w.N, w.K)
    ours, theirs = [], []
    for _ in range(rounds):
        ours.append(time_gemm(torch, plan, dp, b, stream, iters, 3))
        with torch.cuda.stream(stream):
            for _ in range(3):
                F.linear(A, W)
            ev = [(Ev(), Ev()) for _ in range(iters)]
            for e0, e1 in ev:
                e0.record(stream)
                F.linear(A, W)
                e1.record(stream)
        torch.cuda.synchronize()
        theirs.append(float(np.mean([e0.elapsed_time(e1) * 1000.0 for e0, e1 in ev])))
    flops = 2.0 * w.M * w.N * w.K
    o, t = float(np.median(ours)), float(np.median(theirs))
    return {"op": "torch.nn.functional.linear (A x W^T; hipBLASLt), same operands, alternating rounds",
            "us": round(t, 2), "tflops": round(flops / t / 1e6, 2),
            "signalled_us_same_rounds": round(o, 2), "signalled_tflops_same_rounds": round(flops / o / 1e6, 2),
            "signalled_over_vendor_time": round(o / t, 4)}


def cpu_baseline(w, inp, seconds, sizes, num_cus):
    """The oracle's whole path on the host: the fp64 GEMM on a seeded sample
    of output rows (sized to about `seconds`, scaled to all rows), then the
    plan, pre-communication reorder, consumer and post-reorder (+ bias /
    RMSNorm) at full size on a GEMM output of the workload's shape (their
    cost does not depend on the values). value = GEMM flops / total time."""
    import oracle
    threads = oracle.num_threads()
    rng = np.random.default_rng(w.seed + 7)
    # calibrate time(n) = fixed (operand decode) + n * per_row on 8 and 40
    # rows, then size the sample to about `seconds`
    times = []
    for n in (8, 40):
        rows = np.sort(rng.choice(w.M, n, replace=False))
        t = time.perf_counter()
        oracle.gemm_exact(inp.A, inp.W, w.dtype, rows=rows)
        times.append(time.perf_counter() - t)
    per_row = max((times[1] - times[0]) / 32, 1e-6)
    fixed = max(times[0] - 8 * per_row, 0.0)
    nrows = int(min(w.M, max(8, (seconds - fixed) / per_row)))
    rows = np.sort(rng.choice(w.M, nrows, replace=False))
    t = time.perf_counter()
    oracle.gemm_exact(inp.A, inp.W, w.dtype, rows=rows)
    dt = time.perf_counter() - t
    gemm_full = dt * w.M / nrows
    stages = {"gemm_sampled_s": round(dt, 3), "gemm_all_rows_est_s": round(gemm_full, 3)}
    t = time.perf_counter()
    o = oracle.make_plan(w.M, w.N, w.tile_m, w.tile_n, num_cus=num_cus, order=w.order, pattern=w.pattern,
                         num_dest=w.num_dest if w.pattern in ("subtile", "subtoken") else 0,
                         sigma=inp.sigma, bucket=inp.bucket, sizes=tuple(int(x) for x in sizes))
    stages["plan_s"] = time.perf_counter() - t
    C = workloads.uniform_bits(w.M * w.N, w.seed + 8, w.dtype)
    t = time.perf_counter()
    Cr = C[oracle.reorder_index(o)]
    stages["reorder_s"] = time.perf_counter() - t
    t = time.perf_counter()
    dst = oracle.apply_consumer(o, Cr, inp.peer if w.pattern != "subtoken" else None, w.dtype)
    stages["consume_s"] = time.perf_counter() - t
    t = time.perf_counter()
    x = dst[oracle.post_index(o)].reshape(w.M, w.N)
    if w.rmsnorm or inp.bias is not None:
        x = oracle.rmsnorm(x, w.dtype, bias=inp.bias, gamma=inp.gamma, eps=w.eps, do_norm=w.rmsnorm)
    stages["post_s"] = time.perf_counter() - t
    total = gemm_full + stages["plan_s"] + stages["reorder_s"] + stages["consume_s"] + stages["post_s"]
    for k in ("plan_s", "reorder_s", "consume_s", "post_s"):
        stages[k] = round(stages[k], 3)
    return {"value": w.flops / total / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"fp64 oracle GEMM on {nrows} of {w.M} output rows (all {w.N} columns, K={w.K}, "
                      f"operand decode included, {dt:.1f} s, scaled to all rows), then the oracle's plan, "
                      f"reorder, consumer and post-reorder at full size; {total:.1f} s per step",
            "stages": stages}


def slow_link(torch, w, inp, b, base_plan, dp_base, num_cus, s1, s2):
    """The overlap as the communication side gets slower: every consumer
    launch capped at a few workgroups (the consumer_limit option) stands in
    for a slower interconnect. For each cap: the consumer's latency curve, the
    partition Algorithm 1 picks on it, and overlapped vs serialized steps in
    alternating rounds."""
    global OPTS
    rows = []
    sig_us = time_gemm(torch, base_plan, dp_base, b, s1, 30, 5)
    try:
        for cap in (0, 64, 32, 16, 8):
            OPTS = fo.options(consumer_limit=cap)
            xs, ys = consumer_curve(torch, w, b, s1, w.M * w.N, beside=(base_plan, dp_base))
            lx, ly = consumer_curve_after(torch, w, b, inp, num_cus, s1, s2, w.M * w.N)
            p = make_plan(w, inp, num_cus, gemm_us=sig_us, curve=(xs, ys, lx, ly))
            d = dev_plan(torch, p)
            torch.cuda.synchronize()
            ov, se = [], []
            for _ in range(3):
                ov.append(timed_steps(torch, w, p, d, b, s1, s2, 6, 2)[0])
                se.append(timed_steps(torch, w, p, d, b, s1, s1, 6, 2)[0])
            o, r = float(np.median(ov)), float(np.median(se))
            rows.append({"consumer_limit": cap, "consume_beside_gemm_us": round(ys[-1], 2),
                         "consume_over_gemm": round(ys[-1] / sig_us, 3),
                         "groups": [int(x) for x in p.sizes], "predicted_us": round(p.predicted_us, 2),
                         "overlapped_step_us": round(o, 2), "serial_step_us": round(r, 2),
                         "speedup_vs_serial": round(r / o, 4)})
    finally:
        OPTS = None
    return rows


def sync_modes(torch, w, inp, b, base_plan, dp_base, num_cus, s1, s2):
    """The three publication schemes of a finished tile (producer, consumer
    modes), the GEMM alone and the overlapped step with each."""
    global OPTS
    sig_us = time_gemm(torch, base_plan, dp_base, b, s1, 30, 5)
    xs, ys = consumer_curve(torch, w, b, s1, w.M * w.N, beside=(base_plan, dp_base))
    lx, ly = consumer_curve_after(torch, w, b, inp, num_cus, s1, s2, w.M * w.N)
    plan = make_plan(w, inp, num_cus, gemm_us=sig_us, curve=(xs, ys, lx, ly))
    dp = dev_plan(torch, plan)
    torch.cuda.synchronize()
    rows = {}
    try:
        for pm, cm in ((0, 0), (1, 1), (2, 2)):
            OPTS = fo.options(sync_producer=pm, sync_consumer=cm)
            sg = time_gemm(torch, base_plan, dp_base, b, s1, 30, 5)
            us, gm, _, _ = timed_steps(torch, w, plan, dp, b, s1, s2, 20, 3)
            rows[f"{pm}{cm}"] = {"signaled_alone_us": round(sg, 2), "overlapped_step_us": round(us, 2),
                                 "overlapped_gemm_us": round(gm, 2)}
    finally:
        OPTS = None
    return rows


def predictor_breadth(torch, w, num_cus, steps):
    """Algorithm 1's estimate against measurement over every partition at the
    workload's size and at M/4, M/2 and 2M (the sizes a plan cache of the
    family would hold; Section 6.5, Fig. 14 analogue)."""
    rows, per_size = [], []
    for frac in (1, 2, 4, 8):
        M = w.M * frac // 4
        if M % w.tile_m or M <= 0:
            continue
        ws = w.with_shape(M, w.N, w.K)
        inp = workloads.make_inputs(ws)
        tiles = (ws.M // ws.tile_m) * (ws.N // ws.tile_n)
        T = -(-tiles // num_cus)
        s1, s2, _ = streams(torch)
        base_plan = make_plan(ws, inp, num_cus, sizes=[1] * T)
        b = Bufs(torch, ws, inp, base_plan.dest_elems)
        dp_base = dev_plan(torch, base_plan)
        torch.cuda.synchronize()
        log(f"predict {ws.name}: T={T}")
        r = predictor_accuracy(torch, ws, inp, b, base_plan, dp_base, num_cus, T, ws.flops, s1, s2, None)
        per_size.append({k: v for k, v in r.items() if k not in ("phase", "partitions")})
        rows += [dict(p, M=M) for p in r["partitions"]]
        del b
        torch.cuda.empty_cache()
    errs = [abs(p["error_pct"]) for p in rows]
    errs_ov = [abs(p["error_overlap_gemm_pct"]) for p in rows]
    return {"phase": "predict", "workload": w.name, "combinations": len(rows),
            "mean_abs_error_pct": round(float(np.mean(errs)), 2),
            "mean_abs_error_overlap_gemm_pct": round(float(np.mean(errs_ov)), 2),
            "searched_over_best_min": round(min(s["searched_over_best"] for s in per_size), 4),
            "searched_over_best_mean": round(float(np.mean([s["searched_over_best"] for s in per_size])), 4),
            "sizes": per_size, "partitions": rows}


def main():
    global OPTS
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    fo.lib()
    w = workloads.WORKLOADS[args.workload]
    if args.tile:
        tm, tn = (int(x) for x in args.tile.lower().split("x"))
        w = dataclasses.replace(w, tile_m=tm, tile_n=tn)
    log(f"workload {w.name}: M={w.M} N={w.N} K={w.K} {w.dtype} pattern={w.pattern}")
    if args.consumer_grid:
        fo.set_consumer_grid(*(int(x) for x in args.consumer_grid.lower().split("x")))
    num_cus = fo.device_num_cus(0)
    if args.phase == "predict":
        print(json.dumps(predictor_breadth(torch, w, num_cus, args.steps)), flush=True)
        return
    inp = workloads.make_inputs(w)
    tiles = (w.M // w.tile_m) * (w.N // w.tile_n)
    T = -(-tiles // num_cus)
    flops = w.flops
    s1, s2, _ = streams(torch)

    plan_rm = make_plan(w, inp, num_cus, sizes=[1] * T, pattern="rowmajor")
    base_plan = make_plan(w, inp, num_cus, sizes=[1] * T)
    b = Bufs(torch, w, inp, base_plan.dest_elems)
    dp_rm = dev_plan(torch, plan_rm)
    dp_base = dev_plan(torch, base_plan)
    torch.cuda.synchronize()

    if args.phase == "copy":
        # plain copy of a known size: calibration run for the HBM byte counters
        n = w.M * w.N
        us = time_loop(torch, lambda: fo.consume_group(b.C, None, b.dst, n, w.dtype, None, 0, None, s1,
                                                       opts={"consumer_blocks": 256, "consumer_threads": 256}),
                       args.steps, args.warmup, s1)
        print(json.dumps({"phase": "copy", "bytes_read": 2 * n, "bytes_written": 2 * n, "us": us}))
        return
    if args.phase == "trace":
        print(json.dumps(tile_timeline(torch, w, base_plan, dp_base, b, s1)), flush=True)
        return
    if args.phase == "gemm":
        us = time_gemm(torch, base_plan, dp_base, b, s1, args.steps, args.warmup)
        print(json.dumps({"phase": "gemm", "us": us, "tflops": flops / us / 1e6}))
        return
    if args.phase == "step":
        # profiler run: only identical overlapped steps (one group per wave
        # unless --sizes), so per-kernel averages match the live timing
        sizes = [int(x) for x in args.sizes.split(",")] if args.sizes else [1] * T
        plan = make_plan(w, inp, num_cus, sizes=sizes)
        dp = dev_plan(torch, plan)
        torch.cuda.synchronize()
        step_us, gemm_mean_us, gemm_med_us, wall = timed_steps(torch, w, plan, dp, b, s1,
                                                               s1 if args.serial else s2, args.steps,
                                                               args.warmup)
        print(json.dumps({"phase": "step", "groups": sizes, "serial": args.serial,
                          "consumer_grid": list(fo.get_consumer_grid()), "step_us": round(step_us, 2),
                          "gemm_us": round(gemm_mean_us, 2), "gemm_tflops": round(flops / gemm_mean_us / 1e6, 2)}))
        return
    if args.phase == "slowlink":
        print(json.dumps({"phase": "slowlink", "rows": slow_link(torch, w, inp, b, base_plan, dp_base, num_cus,
                                                                  s1, s2)}), flush=True)
        return
    if args.phase == "sync":
        print(json.dumps({"phase": "sync", "rows": sync_modes(torch, w, inp, b, base_plan, dp_base, num_cus, s1,
                                                              s2)}), flush=True)
        return

    # ---- GEMM alone: plain (static schedule / signalled) vs reordered ------
    log("GEMM alone: row-major static, row-major signalled, reordered signalled")
    plain_static, plain_sig, sig = [], [], []
    for _ in range(3):
        plain_static.append(time_gemm(torch, plan_rm, dp_rm, b, s1, 30, 5, signal=False))
        plain_sig.append(time_gemm(torch, plan_rm, dp_rm, b, s1, 30, 5))
        sig.append(time_gemm(torch, base_plan, dp_base, b, s1, 30, 5))
    plain_static_us, plain_sig_us, sig_us = (float(np.median(v)) for v in (plain_static, plain_sig, sig))
    log("consumer curve")
    n_all = w.M * w.N
    xs, ys = consumer_curve(torch, w, b, s1, n_all, beside=(base_plan, dp_base))
    lx, ly = consumer_curve_after(torch, w, b, inp, num_cus, s1, s2, n_all)
    cons_bytes_per_elem = 6 if b.peer is not None else 4
    cons_all_us = consume_all(torch, w, b, s1, n_all, 20, 3)

    # ---- the plan: explicit, or Algorithm 1 on the measured inputs ---------
    if args.sizes:
        plan = make_plan(w, inp, num_cus, sizes=[int(x) for x in args.sizes.split(",")])
    else:
        plan = make_plan(w, inp, num_cus, gemm_us=sig_us, curve=(xs, ys, lx, ly))
    dp = dev_plan(torch, plan)
    torch.cuda.synchronize()
    log(f"plan: T={plan.T} groups={list(plan.sizes)} predicted {plan.predicted_us:.1f} us")
    planner = planner_report(w, inp, num_cus, sig_us, (xs, ys, lx, ly)) if not args.sizes else None

    # ---- overlapped vs serialized, alternating rounds ----------------------
    log("overlapped vs serialized rounds")
    per = max(4, args.steps // 5)
    rounds = overlap_rounds(torch, w, plan, dp, base_plan, dp_base, b, s1, s2, 5, per)

    # ---- the timed region: exactly `steps` overlapped steps after `warmup` --
    log(f"timed steps: warmup {args.warmup}, steps {args.steps}")
    step_us, gemm_mean_us, gemm_med_us, wall = timed_steps(torch, w, plan, dp, b, s1, s2, args.steps,
                                                           args.warmup)

    # ---- consistency at full size: overlapped vs serialized output bits ----
    # (every buffer the step writes is poisoned first; 0xFFFF is a NaN)
    for buf in (b.C, b.dst, b.out):
        buf.fill_(-1)
    run_step(torch, w, plan, dp, b, s1, s1)
    torch.cuda.synchronize()
    ref_C, ref_dst, ref_out = b.C.clone(), b.dst.clone(), b.out.clone()
    for buf in (b.C, b.dst, b.out):
        buf.fill_(-1)
    run_step(torch, w, plan, dp, b, s1, s2)
    torch.cuda.synchronize()
    check_status(b, "the consistency runs")
    consistent = bool(torch.equal(ref_out, b.out) and torch.equal(ref_dst, b.dst) and torch.equal(ref_C, b.C))
    if not consistent:
        raise RuntimeError("overlapped and serialized runs disagree: C' %d, dst %d, out %d differing elements" % (
            int((ref_C != b.C).sum()), int((ref_dst != b.dst).sum()), int((ref_out != b.out).sum())))
    del ref_C, ref_dst, ref_out

    # ---- post-reorder vs the same kernel on an identity map -----------------
    post_us = time_loop(torch, lambda: fo.post_reorder(plan, dp, b.dst, b.out, b.bias, b.gamma, w.eps,
                                                       w.rmsnorm, s1), 50, 5, s1)
    post_id_us = time_loop(torch, lambda: fo.post_reorder(plan_rm, None, b.C, b.out, b.bias, b.gamma, w.eps,
                                                          w.rmsnorm, s1), 50, 5, s1)
    post_bytes = 4.0 * w.M * w.N + (2.0 * w.N * (int(w.bias) + int(w.gamma)))

    # ---- Algorithm 1's estimate vs measurement, every partition ------------
    pred = predictor_accuracy(torch, w, inp, b, base_plan, dp_base, num_cus, T, flops, s1, s2, args) \
        if 1 < T <= 8 else None

    # ---- Table 5 analogue, group-size sweep ---------------------------------
    log("Table 5 analogue")
    t5 = table5(torch, w, inp, b, num_cus, T, s1)
    log("group-size sweep")
    sw = sweep(torch, w, inp, num_cus, b, s1, s2, max(10, args.steps // 2))
    log("vendor GEMM")
    vendor = vendor_gemm(torch, w, base_plan, dp_base, b, s1, max(10, args.steps // 2))

    # ---- every other workload -------------------------------------------------
    others = {}
    if not args.skip_workloads and w.name == HEADLINE:
        del b
        torch.cuda.empty_cache()
        for name in OTHER_WORKLOADS:
            others[name] = workload_summary(torch, name, num_cus, args.steps)
            torch.cuda.empty_cache()

    # ---- CPU baseline ----------------------------------------------------
    cpu = None
    if not args.skip_cpu:
        log("CPU oracle baseline")
        cpu = cpu_baseline(w, inp, args.cpu_seconds, plan.sizes, num_cus)

    gemm_tflops = flops / gemm_mean_us / 1e6
    value = flops / step_us / 1e6
    bound_us = theoretical(plan, rounds["gemm_alone_us"], rounds["consume_alone_us"], post_us)
    ov = overlap_fields(rounds, bound_us)
    ov.update({"timed_steps_us": round(step_us, 2), "rounds": 5, "steps_per_round": per,
               "overlapped_rounds_us": [round(x, 1) for x in rounds["overlapped_rounds_us"]],
               "serial_rounds_us": [round(x, 1) for x in rounds["serial_rounds_us"]],
               "predicted_us": round(plan.predicted_us, 2),
               "paper_context": "up to 1.65x overlap speedup on 4x RTX 4090 over PCIe (multi-GPU collectives; "
                                "not comparable to this 1-GPU stand-in)"})
    headline = {"gemm_alone_us": round(sig_us, 2), "gemm_tflops": round(flops / sig_us / 1e6, 2),
                "gemm_frac_peak": round(flops / sig_us / 1e6 / PEAK_TFLOPS, 4),
                "gemm_in_step_tflops": round(gemm_tflops, 2),
                "consumer_GBps": round(cons_bytes_per_elem * n_all / cons_all_us / 1e3, 1),
                "post_reorder_GBps": round(post_bytes / post_us / 1e3, 1), "step_tflops": round(value, 2),
                "overlap": {k: ov[k] for k in ("speedup_vs_serial", "overlapped_gemm_consume_over_max",
                                               "fraction_of_theoretical_speedup")}}
    line = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "value_is": "GEMM flops / time of the whole overlapped step (GEMM, consumers, post-reorder)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_us / 1000.0, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded U[-1,1] / N(0,1) operands, see workloads/)",
        "config": {"workload": w.name, "M": w.M, "N": w.N, "K": w.K, "tile": [w.tile_m, w.tile_n],
                   "pattern": w.pattern, "num_dest": w.num_dest, "waves": T,
                   "groups": [int(x) for x in plan.sizes], "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "achieved": round(gemm_tflops, 2), "peak": round(PEAK_TFLOPS, 1),
                     "unit": "TFLOP/s", "frac": round(gemm_tflops / PEAK_TFLOPS, 4),
                     "traffic": traffic_bytes(w)},
        "gemm": {"signaled_overlapped_us": round(gemm_mean_us, 2),
                 "signaled_overlapped_median_us": round(gemm_med_us, 2),
                 "signaled_alone_us": round(sig_us, 2),
                 "plain_signalled_alone_us": round(plain_sig_us, 2),
                 "plain_static_alone_us": round(plain_static_us, 2),
                 "signaled_tflops": round(flops / sig_us / 1e6, 2),
                 "plain_signalled_tflops": round(flops / plain_sig_us / 1e6, 2),
                 "plain_static_tflops": round(flops / plain_static_us / 1e6, 2),
                 "interference_pct": round((sig_us / plain_sig_us - 1) * 100, 2),
                 "interference_vs_static_pct": round((sig_us / plain_static_us - 1) * 100, 2),
                 "pct_peak_signaled": round(flops / sig_us / 1e6 / PEAK_TFLOPS * 100, 2),
                 "vendor": vendor},
        "consumer": {"whole_buffer_us": round(cons_all_us, 2),
                     "GBps": round(cons_bytes_per_elem * n_all / cons_all_us / 1e3, 1),
                     "frac_hbm": round(cons_bytes_per_elem * n_all / cons_all_us / 1e3 / PEAK_HBM_GBS, 4),
                     "whole_buffer_beside_running_gemm_us": round(ys[-1], 2),
                     "whole_buffer_after_gemm_us": round(ly[-1], 2),
                     "beside_gemm_grid": "%dx%d" % fo.get_consumer_grid()},
        "post_reorder": {"us": round(post_us, 2), "identity_map_us": round(post_id_us, 2),
                         "GBps": round(post_bytes / post_us / 1e3, 1),
                         "frac_hbm": round(post_bytes / post_us / 1e3 / PEAK_HBM_GBS, 4),
                         "overhead_pct": round((post_us / post_id_us - 1) * 100, 2)},
        "overlap": ov,
        "overlapped_equals_serial_bits": consistent,
        "table5": t5,
        "sweep_waves_per_group": sw,
        "predictor": None if pred is None else {k: v for k, v in pred.items() if k != "phase"},
        "planner": planner,
        "workloads": dict({w.name: headline}, **others),
        "cpu_baseline": cpu,
        "wall_s_timed": round(wall, 3),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
