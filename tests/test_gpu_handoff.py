"""The two device-side handoffs of an overlapped run, on the GPU.

fo_run_overlapped orders its two streams without events: the reset kernel on
the GEMM stream writes the run's tag into a gate word that a one-wave kernel
on the consumer stream waits for (so the consumers of a run start only after
the counters are zero and the previous run's post-reorder has read the
destination buffer), and the final consumer launch counts its finished
workgroups into done words that a one-wave wait on the GEMM stream checks
before the post-reorder (so the post-reorder reads complete groups and the
next GEMM does not overwrite what a consumer still reads). These tests run
back-to-back runs that share every buffer but their outputs, runs of two
workloads on shared and on separate stream pairs, hold either stream back
before a run, and force the bounded waits to time out from the
host (a tiny wall-clock limit), which must end in the status bit and not in
a hang.
"""
import time

import numpy as np
import pytest

import oracle
import paper_2504_19519_amd as fo
import workloads
from gpu_util import assert_close_bits, dev_plan, empty16, from_dev, plan_for, say, to_dev, torch_mod, zeros_u32

pytestmark = pytest.mark.gpu

# workload: (M, N, K, modelled CUs, partition in waves); no RMSNorm, so every
# output is compared bit for bit
CASES = {
    "rs_8192x8192x3584": (1024, 1280, 512, 8, (2, 1)),
    "a2a_4096x7168x2048": (1024, 1280, 512, 8, (1, 2)),          # 256x256 tiles: 20 tiles, T = 3
}


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = torch_mod()
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    fo.lib()


class Setup:
    """One small workload, its plan, two A operands and the expected output
    of the whole path for each (the oracle's consumer and post-reorder
    applied to the GPU's plain GEMM of that A)."""

    def __init__(self, name):
        torch = torch_mod()
        M, N, K, cus, sizes = CASES[name]
        w = workloads.WORKLOADS[name].with_shape(M, N, K)
        inp = workloads.make_inputs(w)
        self.w, self.inp = w, inp
        self.plan, self.o = plan_for(w, inp, num_cus=cus, sizes=list(sizes))
        self.dp = dev_plan(self.plan)
        a0 = np.asarray(inp.A).reshape(M, K)
        a1 = np.ascontiguousarray(a0[::-1])          # same values, other rows
        self.A = [to_dev(a0), to_dev(a1)]
        self.W = to_dev(inp.W)
        self.peer = to_dev(inp.peer) if w.pattern != "subtoken" else None
        plan_rm = fo.plan_groups(M, N, K, dtype=w.dtype, tile_m=w.tile_m, tile_n=w.tile_n,
                                 order=w.order, num_cus=256, pattern="rowmajor", sizes=None,
                                 curve_bytes=[1.0], curve_us=[0.0])
        self.expected = []
        for A in self.A:
            C = empty16(M * N)
            fo.gemm_signal_reorder(plan_rm, None, A, self.W, C, None)
            torch.cuda.synchronize()
            Cr = from_dev(C)[:M * N][oracle.reorder_index(self.o)]
            dst = oracle.apply_consumer(self.o, Cr, inp.peer if w.pattern != "subtoken" else None, w.dtype)
            self.expected.append(dst[oracle.post_index(self.o)])
        self.C = empty16(M * N)
        self.dst = empty16(self.plan.dest_elems)
        self.counters = zeros_u32(self.plan.num_counters)
        self.status = zeros_u32(1)

    def run(self, k, out, s1, s2, opts=None):
        fo.run_overlapped(self.plan, self.dp, self.A[k % 2], self.W, self.C, self.peer, self.dst, out,
                          counters=self.counters, status_word=self.status, gemm_stream=s1, comm_stream=s2,
                          opts=opts)

    def check(self, k, out):
        n = self.w.M * self.w.N
        np.testing.assert_array_equal(from_dev(out)[:n], self.expected[k % 2], err_msg=f"run {k}")


@pytest.mark.parametrize("name", list(CASES))
def test_back_to_back_runs_share_buffers(name):
    # six runs with no host synchronisation between them, alternating two A
    # operands, share C, dst, counters and status; each writes its own out
    torch = torch_mod()
    say(f"[handoff back-to-back] {name}")
    st = Setup(name)
    outs = [empty16(st.w.M * st.w.N, st.w.dtype) for _ in range(6)]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for k, out in enumerate(outs):
        st.run(k, out, s1, s2)
    torch.cuda.synchronize()
    assert int(st.status.cpu()[0]) == 0
    for k, out in enumerate(outs):
        st.check(k, out)
    np.testing.assert_array_equal(st.counters.cpu().numpy()[:st.plan.P], np.array(st.o.targets))


@pytest.mark.parametrize("held", ["gemm_stream", "comm_stream"])
def test_a_held_stream_is_waited_for(held):
    # a ~20 ms spin kernel on one stream ahead of the run: with the GEMM
    # stream held, the gate holds the consumers back (they would otherwise
    # see the previous run's counters at their targets); with the consumer
    # stream held, the done wait holds the post-reorder back
    torch = torch_mod()
    say(f"[handoff held] {held}")
    st = Setup("rs_8192x8192x3584")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    out0 = empty16(st.w.M * st.w.N, st.w.dtype)
    st.run(0, out0, s1, s2)                 # leaves every counter at its target
    out1 = empty16(st.w.M * st.w.N, st.w.dtype)
    with torch.cuda.stream(s1 if held == "gemm_stream" else s2):
        torch.cuda._sleep(50_000_000)
    st.run(1, out1, s1, s2)
    torch.cuda.synchronize()
    assert int(st.status.cpu()[0]) == 0
    st.check(0, out0)
    st.check(1, out1)


def test_timed_out_handoffs_raise_the_status_bit():
    # the wall-clock limit of every wait of one run is cut to 1 ms (a
    # per-call option) and the GEMM stream is held ~20 ms: the gate times out
    # (marking the gate word), so do the consumers and the done wait; the
    # run must end, with bit 0 of the status word set (by the reset kernel
    # finding the mark, as the reset runs after the gate gave up). The bit
    # stays set (the library never clears it); once the caller clears it, a
    # run with the normal limit works again on the same counters.
    torch = torch_mod()
    say("[handoff timeout]")
    st = Setup("rs_8192x8192x3584")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    out0 = empty16(st.w.M * st.w.N, st.w.dtype)
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        torch.cuda._sleep(50_000_000)
    st.run(0, out0, s1, s2, opts={"poll_timeout_us": 1000})
    torch.cuda.synchronize()
    assert int(st.status.cpu()[0]) & 1 == 1
    out1 = empty16(st.w.M * st.w.N, st.w.dtype)
    st.run(1, out1, s1, s2)
    torch.cuda.synchronize()
    assert int(st.status.cpu()[0]) & 1 == 1, "the status bit is sticky"
    st.check(1, out1)
    st.status.zero_()
    out2 = empty16(st.w.M * st.w.N, st.w.dtype)
    st.run(2, out2, s1, s2)
    torch.cuda.synchronize()
    assert int(st.status.cpu()[0]) == 0
    st.check(2, out2)


def test_a_timed_out_run_does_not_count_for_the_next():
    # run N waits at most 1 ms, run N+1 the normal limit; both are queued
    # back to back while the consumer stream is held ~20 ms. Run N's done
    # wait and gate time out (its output is unspecified, the status bit
    # records it and stays set); run N+1's reset tags the done word before
    # run N's late consumers finish, so they do not count for run N+1, and
    # run N's gate, finding the later run's tag, leaves it in place: run N+1
    # waits for its own consumers and its output is exact.
    torch = torch_mod()
    say("[handoff timeout back-to-back]")
    st = Setup("rs_8192x8192x3584")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    out0 = empty16(st.w.M * st.w.N, st.w.dtype)
    out1 = empty16(st.w.M * st.w.N, st.w.dtype)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    with torch.cuda.stream(s2):
        torch.cuda._sleep(50_000_000)
    st.run(0, out0, s1, s2, opts={"poll_timeout_us": 1000})
    st.run(1, out1, s1, s2)
    torch.cuda.synchronize()
    # run N+1's gate (2 s limit) found its tag: it did not sit out its limit
    assert time.perf_counter() - t0 < 1.0
    assert int(st.status.cpu()[0]) & 1 == 1
    st.check(1, out1)
    np.testing.assert_array_equal(st.counters.cpu().numpy()[:st.plan.P], np.array(st.o.targets))


def test_stale_counter_words_do_not_reach_a_run():
    # group and position counters left dirty by some earlier user of the
    # array (values below, at and far past every class's positions): an
    # overlapped run zeroes them on its GEMM stream before the GEMM and the
    # consumers use them, so its output is whole; a standalone GEMM launch
    # after fo_reset_counters is whole as well
    torch = torch_mod()
    say("[handoff stale counters] rs_8192x8192x3584 small")
    st = Setup("rs_8192x8192x3584")
    P = st.plan.P
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for k, junk in enumerate([3, 1 << 20, 0x7FFFFFF0]):
        st.counters[:P + fo.DISPENSER_WORDS] = junk
        torch.cuda.synchronize()
        out = empty16(st.w.M * st.w.N, st.w.dtype)
        st.run(k, out, s1, s2)
        torch.cuda.synchronize()
        assert int(st.status.cpu()[0]) == 0, f"junk {junk}"
        st.check(k, out)
        np.testing.assert_array_equal(st.counters.cpu().numpy()[:P], np.array(st.o.targets))
        np.testing.assert_array_equal(st.counters.cpu().numpy()[P:P + fo.DISPENSER_WORDS], 0)
    # standalone: fo_reset_counters clears what a dirty array holds
    st.counters[:P + fo.DISPENSER_WORDS] = 5
    fo.reset_counters(st.counters, P + fo.DISPENSER_WORDS)
    C = empty16(st.w.M * st.w.N)
    fo.gemm_signal_reorder(st.plan, st.dp, st.A[0], st.W, C, st.counters)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(st.counters.cpu().numpy()[:P], np.array(st.o.targets))
    np.testing.assert_array_equal(st.counters.cpu().numpy()[P:P + fo.DISPENSER_WORDS], 0)


def test_back_to_back_runs_at_full_size():
    # the bench's configuration: rs 8192x8192x3584, 256 CUs, waves [1, 2, 1];
    # three runs without host synchronisation, alternating two A operands,
    # sharing C, dst, counters and status, each output checked bit for bit
    # (the GPU's plain GEMM of each A is first checked against the exact
    # product, every output)
    torch = torch_mod()
    w = workloads.WORKLOADS["rs_8192x8192x3584"]
    say("[handoff back-to-back full size] rs_8192x8192x3584 [1, 2, 1]")
    inp = workloads.make_inputs(w)
    plan, o = plan_for(w, inp, num_cus=256, sizes=[1, 2, 1])
    dp = dev_plan(plan)
    a0 = np.asarray(inp.A).reshape(w.M, w.K)
    As = [to_dev(a0), to_dev(np.ascontiguousarray(a0[::-1]))]
    Wd, peer = to_dev(inp.W), to_dev(inp.peer)
    plan_rm = fo.plan_groups(w.M, w.N, w.K, dtype=w.dtype, tile_m=w.tile_m, tile_n=w.tile_n,
                             order=w.order, num_cus=256, pattern="rowmajor", sizes=None,
                             curve_bytes=[1.0], curve_us=[0.0])
    expected = []
    for k, A in enumerate(As):
        C = empty16(w.M * w.N)
        fo.gemm_signal_reorder(plan_rm, None, A, Wd, C, None)
        torch.cuda.synchronize()
        Cp = from_dev(C)[:w.M * w.N]
        ak = a0 if k == 0 else np.ascontiguousarray(a0[::-1])
        ref = oracle.gemm_ref(ak, inp.W, w.dtype).reshape(-1)
        assert_close_bits(Cp, ref, w.dtype, f"plain GEMM of A[{k}]")
        del ref
        dst = oracle.apply_consumer(o, Cp[oracle.reorder_index(o)], inp.peer, w.dtype)
        expected.append(dst[oracle.post_index(o)])
        del C
    C = empty16(w.M * w.N)
    dst = empty16(plan.dest_elems)
    counters = zeros_u32(plan.num_counters)
    status = zeros_u32(1)
    outs = [empty16(w.M * w.N, w.dtype) for _ in range(3)]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for k, out in enumerate(outs):
        fo.run_overlapped(plan, dp, As[k % 2], Wd, C, peer, dst, out, counters=counters,
                          status_word=status, gemm_stream=s1, comm_stream=s2)
    torch.cuda.synchronize()
    assert int(status.cpu()[0]) == 0
    for k, out in enumerate(outs):
        np.testing.assert_array_equal(from_dev(out)[:w.M * w.N], expected[k % 2], err_msg=f"run {k}")


def test_two_plans_alternate_on_the_same_streams():
    # two workloads (ReduceScatter and All-to-All shapes), each with its own
    # buffers and counters, run alternately on one pair of streams without
    # host synchronisation, as consecutive layers would: every output is the
    # one its own plan expects
    torch = torch_mod()
    say("[handoff two plans alternating]")
    a, b = Setup("rs_8192x8192x3584"), Setup("a2a_4096x7168x2048")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    torch.cuda.synchronize()
    for k in range(6):
        st = a if k % 2 == 0 else b
        out = empty16(st.w.M * st.w.N, st.w.dtype)
        st.run(k // 2, out, s1, s2)
        outs.append((st, k // 2, out))
    torch.cuda.synchronize()
    assert int(a.status.cpu()[0]) == 0 and int(b.status.cpu()[0]) == 0
    for st, k, out in outs:
        st.check(k, out)


def test_two_runs_at_once_on_their_own_streams():
    # the same two workloads, each on a stream pair of its own, submitted
    # interleaved without host synchronisation, so that their GEMMs,
    # consumers and handoff waits run at the same time (and, with more
    # streams than hardware queues, may share a queue with the other run's
    # kernels): each run's handoffs see only its own counters and tags
    torch = torch_mod()
    say("[handoff two runs at once]")
    a, b = Setup("rs_8192x8192x3584"), Setup("a2a_4096x7168x2048")
    streams = {id(a): (torch.cuda.Stream(), torch.cuda.Stream()), id(b): (torch.cuda.Stream(), torch.cuda.Stream())}
    outs = []
    torch.cuda.synchronize()
    for k in range(8):
        st = a if k % 2 == 0 else b
        out = empty16(st.w.M * st.w.N, st.w.dtype)
        st.run(k // 2, out, *streams[id(st)])
        outs.append((st, k // 2, out))
    torch.cuda.synchronize()
    assert int(a.status.cpu()[0]) == 0 and int(b.status.cpu()[0]) == 0
    for st, k, out in outs:
        st.check(k, out)
    for st in (a, b):
        np.testing.assert_array_equal(st.counters.cpu().numpy()[:st.plan.P], np.array(st.o.targets))
