"""GPU parity of each kernel against the oracle, through the C ABI.

GEMM values: within |err| <= 2e-3 + 1e-2 |ref| of the exact product rounded
once. Everything that only moves or rounds sums of two stored values is
bit-exact: the reordered output against the oracle's permutation of the GPU's
own plain GEMM output, the counters against the group tile counts, the
consumer sum, the post-reorder gather and the bias add.
"""
import numpy as np
import pytest

import oracle
import paper_2504_19519_amd as fo
import workloads
from gpu_util import (assert_close_bits, dev_plan, empty16, from_dev, say, to_dev, zeros_u32,
                      torch_mod)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = torch_mod()
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    fo.lib()
    yield
    torch.cuda.synchronize()


def _operands(M, N, K, dtype, seed):
    rng = np.random.default_rng(seed)
    A = workloads.to_bits(rng.uniform(-1, 1, (M, K)), dtype)
    W = workloads.to_bits(rng.uniform(-1, 1, (N, K)) / np.sqrt(max(K, 1)), dtype)
    return A, W


def _gemm(plan, A, W, counters=None, poison=None):
    torch = torch_mod()
    dA, dW = to_dev(A), to_dev(W)
    C = empty16(plan.M * plan.N, poison)
    dp = dev_plan(plan)
    fo.gemm_signal_reorder(plan, dp, dA, dW, C, counters)
    torch.cuda.synchronize()
    return from_dev(C)[:plan.M * plan.N]


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
@pytest.mark.parametrize("tile,shape", [((256, 128), (512, 384, 320)),
                                        ((256, 128), (1024, 640, 192)),
                                        ((256, 256), (768, 512, 320)),
                                        ((256, 256), (512, 768, 3584)),
                                        ((64, 64), (256, 256, 256)),
                                        ((64, 64), (192, 320, 128))])
def test_plain_gemm_matches_oracle(dtype, tile, shape):
    M, N, K = shape
    say(f"[gemm rowmajor] dtype={dtype} tile={tile} M={M} N={N} K={K}")
    A, W = _operands(M, N, K, dtype, 11)
    plan = fo.plan_groups(M, N, K, dtype=dtype, tile_m=tile[0], tile_n=tile[1], order="xcd",
                          num_cus=4, pattern="rowmajor", sizes=None, curve_bytes=[1.0], curve_us=[0.0])
    C = _gemm(plan, A, W, poison=dtype)
    assert_close_bits(C, oracle.gemm_ref(A, W, dtype).reshape(-1), dtype, "plain GEMM")


@pytest.mark.parametrize("K", [64 * kt for kt in range(1, 10)] + [64 * 56])
@pytest.mark.parametrize("tile", [(256, 128), (256, 256), (64, 64)])
def test_gemm_every_k_step_count(K, tile):
    # the main loop runs k steps in groups of three; cover every remainder
    M, N = 2 * tile[0], 3 * tile[1]
    say(f"[gemm k sweep] tile={tile} K={K}")
    A, W = _operands(M, N, K, "fp16", 15 + K)
    plan = fo.plan_groups(M, N, K, tile_m=tile[0], tile_n=tile[1], order="xcd", num_cus=4,
                          pattern="rowmajor", sizes=[2])
    C = _gemm(plan, A, W, poison="fp16")
    assert_close_bits(C, oracle.gemm_ref(A, W, "fp16").reshape(-1), "fp16", f"GEMM K={K}")


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
@pytest.mark.parametrize("tile", [(256, 128), (256, 256), (64, 64)])
def test_identity_operand_is_exact(dtype, tile):
    # A = I: every output is one product by 1 plus sums of zeros, so C = B
    # exactly, whatever the accumulation order (pins the epilogue layout).
    K = N = M = 256
    say(f"[gemm identity] dtype={dtype} tile={tile}")
    A = workloads.to_bits(np.eye(K), dtype)
    _, W = _operands(M, N, K, dtype, 12)
    plan = fo.plan_groups(M, N, K, dtype=dtype, tile_m=tile[0], tile_n=tile[1], num_cus=4,
                          pattern="rowmajor", sizes=[-(-((M // tile[0]) * (N // tile[1])) // 4)])
    C = _gemm(plan, A, W, poison=dtype).reshape(M, N)
    np.testing.assert_array_equal(C, W.T)


def test_k_zero_gives_zeros():
    M, N = 256, 128
    say("[gemm K=0]")
    plan = fo.plan_groups(M, N, 0, pattern="rowmajor", num_cus=4, sizes=[1])
    A = np.zeros(8, np.uint16)
    C = _gemm(plan, A, A, poison="fp16")
    assert np.all(C == 0)


@pytest.mark.parametrize("pattern,nd", [("tile", 0), ("subtile", 4), ("subtoken", 8), ("rowmajor", 0)])
@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
@pytest.mark.parametrize("sizes", [(1, 2), (3,), (1, 1, 1)])
@pytest.mark.parametrize("tile", [(256, 128), (256, 256)])
def test_reordered_output_is_permuted_plain_output(pattern, nd, dtype, sizes, tile):
    # 4 x 5 tiles on a modelled 8-CU device: W = 8, T = 3 with a 4-tile last
    # wave; the XCD order with 8 chiplets on 20 tiles is ragged.
    M, N, K = 4 * tile[0], 5 * tile[1], 256
    say(f"[reorder] pattern={pattern} dtype={dtype} sizes={sizes} tile={tile}")
    rng = np.random.default_rng(13)
    A, W = _operands(M, N, K, dtype, 14)
    sigma = rng.permutation(nd) if pattern == "subtile" else None
    bucket = rng.integers(0, nd, M) if pattern == "subtoken" else None
    common = dict(dtype=dtype, tile_m=tile[0], tile_n=tile[1], order="xcd", num_cus=8, num_dest=nd,
                  dest_perm=sigma, row_bucket=bucket)
    plain = fo.plan_groups(M, N, K, pattern="rowmajor", sizes=list(sizes), **common)
    C = _gemm(plain, A, W, poison=dtype)
    plan = fo.plan_groups(M, N, K, pattern=pattern, sizes=list(sizes), **common)
    o = oracle.make_plan(M, N, tile[0], tile[1], num_cus=8, order="xcd", pattern=pattern, num_dest=nd,
                         sigma=sigma, bucket=bucket, sizes=sizes)
    counters = zeros_u32(plan.num_counters)
    Cr = _gemm(plan, A, W, counters=counters, poison=dtype)
    np.testing.assert_array_equal(Cr, C[oracle.reorder_index(o)])
    np.testing.assert_array_equal(counters.cpu().numpy()[:plan.P], np.array(o.targets))


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
@pytest.mark.parametrize("length", [1, 7, 8, 4096 + 3, 1_000_003, 8 * 1024 * 1024 + 5])
@pytest.mark.parametrize("offset", [0, 1])
@pytest.mark.parametrize("mode", ["sum", "copy"])
def test_consumer_bit_exact(dtype, length, offset, mode):
    torch = torch_mod()
    say(f"[consume] dtype={dtype} len={length} offset={offset} mode={mode}")
    src = workloads.uniform_bits(length + 8, 21, dtype, -4, 4)
    peer = workloads.uniform_bits(length + 8, 22, dtype, -4, 4)
    dS, dP = to_dev(src), to_dev(peer)
    dD = empty16(length + 8, dtype)
    ctr = zeros_u32(1)
    ctr.fill_(5)
    el = 2
    fo.consume_group(dS.data_ptr() + el * offset, dP.data_ptr() + el * offset if mode == "sum" else None,
                     dD.data_ptr() + el * offset, length, dtype, ctr, 5)
    torch.cuda.synchronize()
    got = from_dev(dD)[offset:offset + length]
    s, p = src[offset:offset + length], peer[offset:offset + length]
    ref = oracle.add_rne(s, p, dtype) if mode == "sum" else s
    np.testing.assert_array_equal(got, ref)


SPECIAL_BITS = {
    # +0, -0, smallest and largest subnormal, smallest normal, 1, -1.5, largest
    # finite (both signs), +inf, -inf, NaN
    "fp16": [0x0000, 0x8000, 0x0001, 0x03FF, 0x0400, 0x3C00, 0xBE00, 0x7BFF, 0xFBFF, 0x7C00, 0xFC00, 0x7E00],
    "bf16": [0x0000, 0x8000, 0x0001, 0x007F, 0x0080, 0x3F80, 0xBFC0, 0x7F7F, 0xFF7F, 0x7F80, 0xFF80, 0x7FC0],
}


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
def test_consumer_sum_special_values(dtype):
    # every pair of special values (signed zeros, subnormals, overflow of the
    # largest finite to infinity, inf - inf): the sum is the correctly
    # rounded one, bit for bit; a NaN result only has to be a NaN
    torch = torch_mod()
    say(f"[consume special values] dtype={dtype}")
    v = np.array(SPECIAL_BITS[dtype], dtype=np.uint16)
    src, peer = np.repeat(v, v.size), np.tile(v, v.size)       # 144 pairs: 18 vector chunks
    n = src.size
    dD = empty16(n, dtype)
    fo.consume_group(to_dev(src), to_dev(peer), dD, n, dtype)
    torch.cuda.synchronize()
    got = from_dev(dD)[:n]
    ref = oracle.add_rne(src, peer, dtype)
    exp_mask, man_mask = (0x7C00, 0x03FF) if dtype == "fp16" else (0x7F80, 0x007F)
    nan_ref = ((ref & exp_mask) == exp_mask) & ((ref & man_mask) != 0)
    nan_got = ((got & exp_mask) == exp_mask) & ((got & man_mask) != 0)
    np.testing.assert_array_equal(nan_got, nan_ref)
    np.testing.assert_array_equal(got[~nan_ref], ref[~nan_ref])


def test_consumer_timeout_reports_and_skips():
    torch = torch_mod()
    say("[consume timeout] counter never reaches the target; 2 ms limit")
    old = fo.get_poll_timeout_us()
    fo.set_poll_timeout_us(2000)
    try:
        n = 4096
        src = workloads.uniform_bits(n, 23)
        dS = to_dev(src)
        dD = empty16(n, "fp16")
        ctr = zeros_u32(1)
        status = zeros_u32(1)
        fo.consume_group(dS, None, dD, n, "fp16", ctr, 1, status)
        torch.cuda.synchronize()
        assert int(status.cpu()[0]) & 1
        assert np.all(from_dev(dD)[:n] == 0x7E00)
    finally:
        fo.set_poll_timeout_us(old)


def _post_case(pattern, nd, M, N, BM, BN, dtype, seed):
    rng = np.random.default_rng(seed)
    sigma = rng.permutation(nd) if pattern == "subtile" else None
    bucket = rng.integers(0, nd, M) if pattern == "subtoken" else None
    tiles = (M // BM) * (N // BN)
    plan = fo.plan_groups(M, N, 64, dtype=dtype, tile_m=BM, tile_n=BN, order="xcd", num_cus=16,
                          pattern=pattern, num_dest=nd, dest_perm=sigma, row_bucket=bucket,
                          sizes=[-(-tiles // 16)])
    o = oracle.make_plan(M, N, BM, BN, num_cus=16, order="xcd", pattern=pattern, num_dest=nd,
                         sigma=sigma, bucket=bucket, sizes=(-(-tiles // 16),))
    return plan, o


@pytest.mark.parametrize("pattern,nd", [("tile", 0), ("subtile", 4), ("subtoken", 8), ("rowmajor", 0)])
@pytest.mark.parametrize("N", [256, 4096, 7168, 16384])
@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
def test_post_reorder(pattern, nd, N, dtype):
    torch = torch_mod()
    M, BM, BN = 512, 256, 128
    say(f"[post] pattern={pattern} N={N} dtype={dtype}")
    plan, o = _post_case(pattern, nd, M, N, BM, BN, dtype, 31)
    dst = workloads.uniform_bits(plan.dest_elems, 32, dtype, -3, 3)
    bias = workloads.uniform_bits(N, 33, dtype, -0.1, 0.1)
    gamma = workloads.uniform_bits(N, 34, dtype, 0.5, 1.5)
    dD, dB, dG = to_dev(dst), to_dev(bias), to_dev(gamma)
    dp = dev_plan(plan)
    x_ref = dst[oracle.post_index(o)].reshape(M, N)
    out = empty16(M * N, dtype)
    fo.post_reorder(plan, dp, dD, out)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(from_dev(out)[:M * N].reshape(M, N), x_ref)
    fo.post_reorder(plan, dp, dD, out, bias=dB)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(from_dev(out)[:M * N].reshape(M, N),
                                  oracle.rmsnorm(x_ref, dtype, bias=bias, do_norm=False))
    fo.post_reorder(plan, dp, dD, out, bias=dB, gamma=dG, eps=1e-6, do_rmsnorm=True)
    torch.cuda.synchronize()
    assert_close_bits(from_dev(out)[:M * N], oracle.rmsnorm(x_ref, dtype, bias=bias, gamma=gamma, eps=1e-6),
                      dtype, "post + bias + RMSNorm")
    fo.post_reorder(plan, dp, dD, out, eps=1e-6, do_rmsnorm=True)
    torch.cuda.synchronize()
    assert_close_bits(from_dev(out)[:M * N], oracle.rmsnorm(x_ref, dtype, eps=1e-6), dtype, "post + RMSNorm")
    # every combination of bias and gamma around the norm is a kernel of its own
    fo.post_reorder(plan, dp, dD, out, bias=dB, eps=1e-6, do_rmsnorm=True)
    torch.cuda.synchronize()
    assert_close_bits(from_dev(out)[:M * N], oracle.rmsnorm(x_ref, dtype, bias=bias, eps=1e-6), dtype,
                      "post + bias + RMSNorm without gamma")
    fo.post_reorder(plan, dp, dD, out, gamma=dG, eps=1e-6, do_rmsnorm=True)
    torch.cuda.synchronize()
    assert_close_bits(from_dev(out)[:M * N], oracle.rmsnorm(x_ref, dtype, gamma=gamma, eps=1e-6), dtype,
                      "post + RMSNorm with gamma, no bias")
    # gamma without the norm is ignored: a bias-only run
    fo.post_reorder(plan, dp, dD, out, bias=dB, gamma=dG)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(from_dev(out)[:M * N].reshape(M, N),
                                  oracle.rmsnorm(x_ref, dtype, bias=bias, do_norm=False))


@pytest.mark.parametrize("BN", [192, 96])
def test_post_rowmajor_any_tile_width(BN):
    # a row-major source is read as one piece per row, whatever tile_n / 8 is
    torch = torch_mod()
    M, N, BM = 512, 8 * BN, 256
    say(f"[post rowmajor] tile_n={BN} N={N}")
    plan = fo.plan_groups(M, N, 64, dtype="fp16", tile_m=BM, tile_n=BN, num_cus=16, pattern="rowmajor",
                          sizes=[1])
    src = workloads.uniform_bits(M * N, 35, "fp16", -3, 3)
    bias = workloads.uniform_bits(N, 36, "fp16", -0.1, 0.1)
    out = empty16(M * N, "fp16")
    fo.post_reorder(plan, None, to_dev(src), out)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(from_dev(out)[:M * N], src)
    fo.post_reorder(plan, None, to_dev(src), out, bias=to_dev(bias))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(from_dev(out)[:M * N].reshape(M, N),
                                  oracle.rmsnorm(src.reshape(M, N), "fp16", bias=bias, do_norm=False))


def test_bad_arguments_are_rejected_before_launch():
    plan = fo.plan_groups(512, 256, 100, num_cus=4, pattern="rowmajor", sizes=[1])
    with pytest.raises(fo.FoError) as e:
        fo.gemm_signal_reorder(plan, None, 256, 256, 256)
    assert e.value.status == -2           # K % 64
    plan = fo.plan_groups(512, 256, 64, num_cus=4, pattern="tile", sizes=[1])
    with pytest.raises(fo.FoError):
        fo.gemm_signal_reorder(plan, None, 256, 256, 256)     # tile pattern needs dev_plan
    with pytest.raises(fo.FoError):
        fo.consume_group(0, None, 0, 10, "fp16")
    with pytest.raises(fo.FoError):
        fo.consume_group(256, None, 256, -1, "fp16")


def test_tile_trace():
    # the tile timeline: one record per dispatch position, start <= end, the
    # workgroup that ran it within the grid; outputs are unchanged by tracing
    torch = torch_mod()
    M, N, K = 1024, 1280, 256
    say("[tile trace] 1024x1280x256 tiles 256x256")
    A, W = _operands(M, N, K, "fp16", 21)
    plan = fo.plan_groups(M, N, K, dtype="fp16", tile_m=256, tile_n=256, order="xcd", num_cus=8,
                          pattern="tile", sizes=[3])
    dA, dW = to_dev(A), to_dev(W)
    dp = dev_plan(plan)
    ref = empty16(M * N, "fp16")
    ctr = zeros_u32(plan.num_counters)
    fo.gemm_signal_reorder(plan, dp, dA, dW, ref, ctr)
    trace = torch.zeros(4 * plan.tiles, dtype=torch.int64, device="cuda")
    C = empty16(M * N, "fp16")
    ctr = zeros_u32(plan.num_counters)
    fo.gemm_signal_reorder(plan, dp, dA, dW, C, ctr, opts={"tile_trace": trace, "tile_trace_capacity": plan.tiles})
    torch.cuda.synchronize()
    np.testing.assert_array_equal(from_dev(C)[:M * N], from_dev(ref)[:M * N])
    t = trace.cpu().numpy().reshape(-1, 4)
    assert np.all(t[:, 0] > 0) and np.all(t[:, 1] >= t[:, 0])
    assert np.all((t[:, 3] >= 0) & (t[:, 3] < min(plan.tiles, plan.W)))
    assert fo.device_wall_clock_khz() > 0


@pytest.mark.parametrize("order,tile,shape,cus", [("xcd", (256, 256), (1024, 1280, 512), 8),
                                                  ("xcd", (256, 128), (1024, 1024, 256), 8),
                                                  ("rowmajor", (64, 64), (256, 256, 128), 4)])
def test_back_to_back_launches_need_no_dispenser_reset(order, tile, shape, cus):
    # launches on one counters array whose position words are never cleared
    # in between (only the group counters are): each launch must leave them
    # zero (the last workgroup of each position class clears its word), so
    # every launch computes every tile
    torch = torch_mod()
    M, N, K = shape
    say(f"[gemm dispensers] order={order} tile={tile} M={M} N={N} K={K} cus={cus}")
    A, W = _operands(M, N, K, "fp16", 31)
    plan = fo.plan_groups(M, N, K, dtype="fp16", tile_m=tile[0], tile_n=tile[1], order=order, num_cus=cus,
                          pattern="tile", sizes=[plan_T(M, N, tile, cus)])
    dA, dW = to_dev(A), to_dev(W)
    dp = dev_plan(plan)
    ref = empty16(M * N, "fp16")
    ctr = zeros_u32(plan.num_counters)
    fo.gemm_signal_reorder(plan, dp, dA, dW, ref, ctr)
    torch.cuda.synchronize()
    assert not ctr.cpu().numpy()[plan.P:plan.P + fo.DISPENSER_WORDS].any(), "position words left non-zero"
    for k in range(3):
        C = empty16(M * N, "fp16")
        ctr[:plan.P].zero_()
        fo.gemm_signal_reorder(plan, dp, dA, dW, C, ctr)
        torch.cuda.synchronize()
        c = ctr.cpu().numpy()
        np.testing.assert_array_equal(c[:plan.P], np.array(plan.targets), err_msg=f"launch {k}")
        assert not c[plan.P:plan.P + fo.DISPENSER_WORDS].any(), f"launch {k}: position words left non-zero"
        np.testing.assert_array_equal(from_dev(C)[:M * N], from_dev(ref)[:M * N], err_msg=f"launch {k}")


def plan_T(M, N, tile, cus):
    return -(-((M // tile[0]) * (N // tile[1])) // cus)
