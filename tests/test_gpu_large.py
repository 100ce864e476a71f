"""Sizes past the 31-bit byte offsets the fast paths use, on the GPU.

The GEMM epilogue writes a signalled tile with 16-byte buffer stores when the
whole output fits a 31-bit byte range, and with 8-byte device-coherent
stores addressed in 64 bits otherwise; the consumer reads a segment with
16-byte buffer loads when it fits 31 bits, and with 8-byte coherent loads
otherwise. These tests run the second kind of each: a 32768 x 32768 output
(2 GiB) and a segment of 2^30 + 37 elements. GEMM values are checked on
seeded rows on both sides of the 2 GiB boundary against the exact product
(and every element for having been written);
the consumer input repeats one seeded block, so the whole output is
compared (on the GPU) with the oracle's sum of that block, repeated.
"""
import numpy as np
import pytest

import oracle
import paper_2504_19519_amd as fo
import workloads
from gpu_util import assert_close_bits, dev_plan, from_dev, say, to_dev, torch_mod, zeros_u32

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = torch_mod()
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    fo.lib()


def test_signalled_gemm_output_past_2_gib():
    torch = torch_mod()
    M = N = 32768
    K = 64
    say(f"[large GEMM] {M}x{N}x{K} row-major, signalled (8-byte coherent stores)")
    assert M * N * 2 > 2**31 - 1
    A = workloads.uniform_bits((M, K), 41)
    W = workloads.uniform_bits((N, K), 42, lo=-0.125, hi=0.125)
    plan = fo.plan_groups(M, N, K, dtype="fp16", tile_m=256, tile_n=256, order="xcd", num_cus=256,
                          pattern="rowmajor", sizes=[32, 32])
    dp = dev_plan(plan)
    C = torch.empty(M * N, dtype=torch.int16, device="cuda")
    C.fill_(0x7E00)                              # NaN: rows left unwritten would show
    counters = zeros_u32(plan.num_counters)
    fo.gemm_signal_reorder(plan, dp, to_dev(A), to_dev(W), C, counters)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(counters.cpu().numpy()[:plan.P], plan.targets)
    # every element was written: no NaN fill is left on either side of 2 GiB
    assert not bool(torch.isnan(C.view(torch.float16)).any()), "unwritten output elements"
    rng = np.random.default_rng(43)
    rows = np.sort(np.concatenate([rng.choice(M // 2, 8, replace=False),
                                   M // 2 + rng.choice(M // 2, 8, replace=False), [M - 1]]))
    got = from_dev(C.view(M, N)[torch.as_tensor(rows, device="cuda")].reshape(-1))
    ref = oracle.encode(oracle.gemm_exact(A, W, "fp16", rows=rows), "fp16")
    assert_close_bits(got, ref.reshape(-1), "fp16", "GEMM rows past 2 GiB")


@pytest.mark.parametrize("mode", ["sum", "copy"])
def test_consumer_segment_past_2_gib(mode):
    torch = torch_mod()
    block = 1 << 16
    n = (1 << 30) + 37
    say(f"[large consume] {n} elements, {mode} (8-byte coherent loads)")
    sb = workloads.uniform_bits(block, 44, "bf16", -4, 4)
    pb = workloads.uniform_bits(block, 45, "bf16", -4, 4)
    reps = -(-n // block)
    src = to_dev(sb).repeat(reps)[:n].contiguous()
    peer = to_dev(pb).repeat(reps)[:n].contiguous() if mode == "sum" else None
    dst = torch.empty(n, dtype=torch.int16, device="cuda")
    dst.fill_(0x7FC0)
    ctr = zeros_u32(1)
    ctr.fill_(1)
    fo.consume_group(src, peer, dst, n, "bf16", ctr, 1)
    torch.cuda.synchronize()
    eb = oracle.add_rne(sb, pb, "bf16") if mode == "sum" else sb
    expect = to_dev(eb).repeat(reps)[:n]
    assert torch.equal(dst, expect)
