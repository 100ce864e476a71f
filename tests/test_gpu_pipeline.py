"""The whole path on the GPU (plan -> signalling GEMM on one stream ||
consumers on a second stream -> post-reorder), against the oracle.

For every workload: the reordered GEMM output is the oracle's permutation of
the GPU's plain GEMM output (bit-exact), the consumer output is the oracle's
consumer applied to it (bit-exact), the restored output is the oracle's
post-reorder of that (bit-exact, or within the fp16/bf16 tolerance when
RMSNorm runs), every counter ends at its group's tile count, and the GEMM
values match the exact product (every output, at the reduced and at the full
sizes). Destination buffers are filled with NaN before each
run, so a consumer that read a group early would leave NaNs behind.
"""
import numpy as np
import pytest

import oracle
import paper_2504_19519_amd as fo
import workloads
from gpu_util import (assert_close_bits, dev_plan, empty16, from_dev, plan_for, say, to_dev,
                      torch_mod, zeros_u32)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = torch_mod()
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    fo.lib()


class Dev:
    """Device copies of one workload's inputs."""

    def __init__(self, w, inp, plan):
        self.A, self.W = to_dev(inp.A), to_dev(inp.W)
        self.peer = to_dev(inp.peer) if w.pattern != "subtoken" else None
        self.bias = to_dev(inp.bias) if inp.bias is not None else None
        self.gamma = to_dev(inp.gamma) if inp.gamma is not None else None
        self.dp = dev_plan(plan)


def run(w, plan, d: Dev, *, overlap=True, opts=None):
    torch = torch_mod()
    C = empty16(w.M * w.N, w.dtype)
    dst = empty16(plan.dest_elems, w.dtype)
    out = empty16(w.M * w.N, w.dtype)
    counters = zeros_u32(plan.num_counters)
    status = zeros_u32(1)
    s1 = torch.cuda.Stream()
    s2 = torch.cuda.Stream() if overlap else s1
    torch.cuda.synchronize()
    fo.run_overlapped(plan, d.dp, d.A, d.W, C, d.peer, dst, out, d.bias, d.gamma, w.eps,
                      w.rmsnorm, counters, status, s1, s2, opts=opts)
    torch.cuda.synchronize()
    n = w.M * w.N
    return (from_dev(C)[:n], from_dev(dst)[:plan.dest_elems], from_dev(out)[:n],
            counters.cpu().numpy()[:plan.P], int(status.cpu()[0]))


def plain_gemm(w, d: Dev, plan_rm):
    torch = torch_mod()
    C = empty16(w.M * w.N, w.dtype)
    fo.gemm_signal_reorder(plan_rm, None, d.A, d.W, C, None)
    torch.cuda.synchronize()
    return from_dev(C)[:w.M * w.N]


# exact products of the full-size workloads, computed once per module
_EXACT = {}


def exact_product(w, inp):
    key = (w.name, w.M, w.N, w.K)
    if key not in _EXACT:
        _EXACT[key] = oracle.gemm_ref(inp.A, inp.W, w.dtype).reshape(-1)
    return _EXACT[key]


def check(w, inp, plan, o, sample_rows=None, opts=None):
    d = Dev(w, inp, plan)
    plan_rm = fo.plan_groups(w.M, w.N, w.K, dtype=w.dtype, tile_m=w.tile_m, tile_n=w.tile_n,
                             order=w.order, num_cus=256, pattern="rowmajor",
                             sizes=None, curve_bytes=[1.0], curve_us=[0.0])
    C_plain = plain_gemm(w, d, plan_rm)
    # GEMM values against the exact product
    if sample_rows is None:
        assert_close_bits(C_plain, exact_product(w, inp), w.dtype, "GEMM")
    else:
        rows = np.sort(np.random.default_rng(w.seed + 1000).choice(w.M, sample_rows, replace=False))
        ref = oracle.encode(oracle.gemm_exact(inp.A, inp.W, w.dtype, rows=rows), w.dtype)
        assert_close_bits(C_plain.reshape(w.M, w.N)[rows], ref, w.dtype, "GEMM (sampled rows)")
    Cr, dst, out, counters, status = run(w, plan, d, overlap=True)
    assert status == 0
    # a plan of one group runs serialized and leaves the counters alone
    np.testing.assert_array_equal(counters, np.array(o.targets) if plan.P > 1 else np.zeros(plan.P, np.int64))
    np.testing.assert_array_equal(Cr, C_plain[oracle.reorder_index(o)])
    dst_ref = oracle.apply_consumer(o, Cr, inp.peer if w.pattern != "subtoken" else None, w.dtype)
    np.testing.assert_array_equal(dst, dst_ref)
    x = dst_ref[oracle.post_index(o)].reshape(w.M, w.N)
    if w.rmsnorm:
        ref = oracle.rmsnorm(x, w.dtype, bias=inp.bias, gamma=inp.gamma, eps=w.eps)
        assert_close_bits(out, ref, w.dtype, "post + RMSNorm")
    elif inp.bias is not None:
        np.testing.assert_array_equal(out.reshape(w.M, w.N), oracle.rmsnorm(x, w.dtype, bias=inp.bias, do_norm=False))
    else:
        np.testing.assert_array_equal(out.reshape(w.M, w.N), x)
    # the same work serialized on one stream gives the same bits
    Cr2, dst2, out2, counters2, status2 = run(w, plan, d, overlap=False)
    assert status2 == 0
    np.testing.assert_array_equal(Cr2, Cr)
    np.testing.assert_array_equal(dst2, dst)
    np.testing.assert_array_equal(out2, out)
    return C_plain, out


SMALL = {
    # workload: (M, N, K, modelled CUs, partition in waves)
    "tiny": None,
    "ar_2048x4096x4096": (1024, 1024, 512, 8, (1, 2, 1)),
    "rs_8192x8192x3584": (1024, 1280, 512, 8, (2, 1)),          # 256x256 tiles: 20 tiles, T = 3
    "ar_rmsnorm_16384x4096x3584_bf16": (1024, 1280, 512, 8, (1, 2)),
    "a2a_4096x7168x2048": (1024, 1280, 512, 8, (1, 2)),          # 256x256 tiles: 20 tiles, T = 3
}


@pytest.mark.parametrize("name", list(SMALL))
def test_small_workloads(name):
    w = workloads.WORKLOADS[name]
    cus, sizes = 256, None
    if SMALL[name] is not None:
        M, N, K, cus, sizes = SMALL[name]
        w = w.with_shape(M, N, K)
    say(f"[pipeline small] {w.name} cus={cus} sizes={sizes}")
    inp = workloads.make_inputs(w)
    plan, o = plan_for(w, inp, num_cus=cus, sizes=list(sizes) if sizes else None)
    C_plain, out = check(w, inp, plan, o)
    # end to end against the oracle's own chain from the exact GEMM
    C_ref = oracle.gemm_ref(inp.A, inp.W, w.dtype)
    _, dst_ref, out_ref = oracle.run_path(o, C_ref, inp.peer if w.pattern != "subtoken" else None,
                                          w.dtype, bias=inp.bias, gamma=inp.gamma, eps=w.eps,
                                          do_norm=w.rmsnorm)
    if w.dtype == "fp16":
        assert_close_bits(out, out_ref, w.dtype, "end to end")
    else:
        # bf16 keeps 8 significant bits: the GEMM output may legitimately sit
        # one ulp (<= 2^-7 |C|) from the exactly rounded product, and the sum
        # with the peer can cancel most of C, so that one ulp is carried
        # through the sum and scaled by the row's 1/rms and gamma.
        y = oracle.decode(out.reshape(-1), w.dtype)
        r = oracle.decode(out_ref.reshape(-1), w.dtype)
        c_mag = np.abs(oracle.decode(C_ref.reshape(-1), w.dtype))
        scale = np.ones(w.M * w.N)
        if w.rmsnorm:
            h = oracle.decode(dst_ref[oracle.post_index(o)], w.dtype).reshape(w.M, w.N)
            if inp.bias is not None:
                h = h + oracle.decode(inp.bias, w.dtype)[None, :]
            inv = 1.0 / np.sqrt((h * h).mean(axis=1) + w.eps)
            g = np.abs(oracle.decode(inp.gamma, w.dtype)) if inp.gamma is not None else np.ones(w.N)
            scale = (inv[:, None] * g[None, :]).reshape(-1)
        # C and the output are in the same (row, column) order for these patterns
        bound = 2e-3 + 1e-2 * np.abs(r) + 1.1 * 2.0 ** -7 * c_mag * scale
        assert np.all(np.abs(y - r) <= bound), "end to end (bf16 bound)"


def _composition(rng, total, parts):
    cuts = sorted(rng.choice(np.arange(1, total), size=parts - 1, replace=False)) if parts > 1 else []
    b = [0] + [int(c) for c in cuts] + [total]
    return [b[i + 1] - b[i] for i in range(parts)]


def random_cases(n, seed=2504):
    """Seeded random small paths: tile shape, M / N / K, dtype, dispatch order,
    pattern and destination count, bias / RMSNorm / gamma, modelled CU count
    and a partition in waves or in tiles (mostly several groups)."""
    rng = np.random.default_rng(seed)
    out = []
    for k in range(n):
        tm, tn = [(256, 128), (256, 256), (64, 64)][int(rng.integers(3))]
        M, N, K = tm * int(rng.integers(1, 7)), tn * int(rng.integers(1, 7)), 64 * int(rng.integers(1, 9))
        pattern = ["tile", "subtile", "subtoken"][int(rng.integers(3))]
        nd = (int(rng.choice([2, 4, 8])) if pattern == "subtile" else
              int(rng.integers(2, 9)) if pattern == "subtoken" else 2)
        rms, bias = bool(rng.integers(2)), bool(rng.integers(2))
        gamma = rms and bool(rng.integers(2))
        w = workloads.Workload(name=f"random{k}", M=M, N=N, K=K, dtype=["fp16", "bf16"][int(rng.integers(2))],
                               tile_m=tm, tile_n=tn, order=["xcd", "rowmajor"][int(rng.integers(2))],
                               pattern=pattern, seed=100 + k, dist="uniform", num_dest=nd,
                               bias=bias, rmsnorm=rms, gamma=gamma)
        cus = int(rng.choice([2, 3, 5, 8]))
        tiles = (M // tm) * (N // tn)
        T = -(-tiles // cus)
        if rng.integers(3) == 0 and tiles > 1:
            unit, sizes = "tiles", _composition(rng, tiles, int(rng.integers(min(2, tiles), min(5, tiles) + 1)))
        else:
            unit = "waves"
            sizes = _composition(rng, T, int(rng.integers(2, min(5, T) + 1))) if T > 1 else [1]
        out.append((w, cus, sizes, unit))
    return out


@pytest.mark.parametrize("case", range(40))
def test_random_paths(case):
    # the whole path on seeded random small shapes: every check of
    # test_small_workloads' first part (GEMM against the exact product,
    # reorder, consumer and post-reorder against the oracle, serialized run
    # equal to the overlapped one)
    w, cus, sizes, unit = random_cases(40)[case]
    say(f"[pipeline random] {w.name} {w.M}x{w.N}x{w.K} {w.dtype} tile {w.tile_m}x{w.tile_n} {w.order} "
        f"{w.pattern}/{w.num_dest} bias={w.bias} rms={w.rmsnorm} gamma={w.gamma} cus={cus} {unit} {sizes}")
    inp = workloads.make_inputs(w)
    plan, o = plan_for(w, inp, num_cus=cus, sizes=sizes, unit=unit)
    check(w, inp, plan, o)


def dispatch_cases(n, seed=2505):
    """Seeded random small paths over the dispatch-order parameters that the
    GEMM evaluates per position: the grouped and XCD orders with band heights
    1..6 (bands that do and do not divide the tile rows, one band taller than
    the grid) and 1..12 chiplets (more than the position counters, or more
    than the workgroups of the grid), on 2..12 modelled compute units."""
    rng = np.random.default_rng(seed)
    out = []
    for k in range(n):
        tm, tn = [(256, 128), (256, 256), (64, 64)][int(rng.integers(3))]
        M, N, K = tm * int(rng.integers(1, 9)), tn * int(rng.integers(1, 6)), 64 * int(rng.integers(1, 5))
        pattern = ["tile", "subtile"][int(rng.integers(2))]
        nd = int(rng.choice([2, 4, 8])) if pattern == "subtile" else 2
        w = workloads.Workload(name=f"dispatch{k}", M=M, N=N, K=K, dtype=["fp16", "bf16"][int(rng.integers(2))],
                               tile_m=tm, tile_n=tn, order=["grouped", "xcd"][int(rng.integers(2))],
                               pattern=pattern, seed=300 + k, dist="uniform", num_dest=nd,
                               bias=bool(rng.integers(2)), rmsnorm=False, gamma=False)
        group_m, num_xcds = int(rng.integers(1, 7)), int(rng.integers(1, 13))
        cus = int(rng.integers(2, 13))
        T = -(-((M // tm) * (N // tn)) // cus)
        sizes = _composition(rng, T, int(rng.integers(2, min(4, T) + 1))) if T > 1 else [1]
        out.append((w, cus, sizes, group_m, num_xcds))
    return out


@pytest.mark.parametrize("case", range(24))
def test_dispatch_orders(case):
    # the whole path (checks of test_random_paths) with the grouped and XCD
    # dispatch orders at random band heights and chiplet counts: the GEMM
    # computes the tile of each position itself, and must still run every
    # tile exactly once (a tile missed leaves NaNs, a group short of its
    # target leaves the consumer waiting) whatever the position classes
    w, cus, sizes, group_m, num_xcds = dispatch_cases(24)[case]
    say(f"[pipeline dispatch] {w.name} {w.M}x{w.N}x{w.K} {w.dtype} tile {w.tile_m}x{w.tile_n} {w.order} "
        f"group_m={group_m} num_xcds={num_xcds} {w.pattern}/{w.num_dest} bias={w.bias} cus={cus} {sizes}")
    inp = workloads.make_inputs(w)
    plan, o = plan_for(w, inp, num_cus=cus, sizes=sizes, unit="waves", group_m=group_m, num_xcds=num_xcds)
    np.testing.assert_array_equal(plan.order, np.array(o.order))
    check(w, inp, plan, o)


FULL = {
    "ar_2048x4096x4096": [(1,)],
    "rs_8192x8192x3584": [(1,) * 4, (2, 2), (1, 3)],
    "ar_rmsnorm_16384x4096x3584_bf16": [(1,) * 4],
    "a2a_4096x7168x2048": [(1, 1)],
}


@pytest.mark.parametrize("name,sizes", [(n, s) for n, ss in FULL.items() for s in ss])
def test_full_size_workloads(name, sizes):
    w = workloads.WORKLOADS[name]
    say(f"[pipeline full] {w.name} sizes={sizes}")
    inp = workloads.make_inputs(w)
    plan, o = plan_for(w, inp, num_cus=256, sizes=list(sizes))
    check(w, inp, plan, o)      # every GEMM output against the exact product


def test_consumers_wait_for_a_delayed_gemm():
    # the consumers are enqueued and start polling before the GEMM is even
    # launched (the GEMM stream first runs a ~20 ms spin kernel)
    torch = torch_mod()
    w = workloads.WORKLOADS["ar_2048x4096x4096"].with_shape(1024, 1024, 512)
    say("[pipeline delayed GEMM]")
    inp = workloads.make_inputs(w)
    plan, o = plan_for(w, inp, num_cus=8, sizes=[1, 1, 1, 1])
    d = Dev(w, inp, plan)
    C = empty16(w.M * w.N, w.dtype)
    dst = empty16(plan.dest_elems, w.dtype)
    counters = zeros_u32(plan.num_counters)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for (j, _, so, do, ln) in plan.segments:
        fo.consume_group(C.data_ptr() + 2 * so, d.peer.data_ptr() + 2 * so, dst.data_ptr() + 2 * do,
                         ln, w.dtype, counters.data_ptr() + 4 * j, int(plan.targets[j]), None, s2)
    with torch.cuda.stream(s1):
        torch.cuda._sleep(50_000_000)
    fo.gemm_signal_reorder(plan, d.dp, d.A, d.W, C, counters, s1)
    torch.cuda.synchronize()
    Cr = from_dev(C)[:w.M * w.N]
    ref = oracle.apply_consumer(o, Cr, inp.peer, w.dtype)
    np.testing.assert_array_equal(from_dev(dst)[:plan.dest_elems], ref)


@pytest.mark.parametrize("producer", [0, 1, 2])
@pytest.mark.parametrize("consumer", [0, 1, 2])
@pytest.mark.parametrize("name", ["ar_2048x4096x4096", "rs_8192x8192x3584", "a2a_4096x7168x2048"])
def test_sync_modes(producer, consumer, name):
    # every producer x consumer publication scheme gives the same bits
    old = fo.get_sync_mode()
    fo.set_sync_mode(producer, consumer)
    try:
        M, N, K, cus, sizes = SMALL[name]
        w = workloads.WORKLOADS[name].with_shape(M, N, K)
        say(f"[sync modes] producer={producer} consumer={consumer} {w.name}")
        inp = workloads.make_inputs(w)
        plan, o = plan_for(w, inp, num_cus=cus, sizes=list(sizes))
        check(w, inp, plan, o)
    finally:
        fo.set_sync_mode(*old)


@pytest.mark.parametrize("grid", [(1, 64), (3, 256), (64, 128), (256, 64)])
@pytest.mark.parametrize("name", ["ar_2048x4096x4096", "rs_8192x8192x3584", "a2a_4096x7168x2048"])
def test_consumer_grid(grid, name):
    # any consumer grid (grid-stride over every piece of the group) gives the
    # same bits
    old = fo.get_consumer_grid()
    fo.set_consumer_grid(*grid)
    try:
        M, N, K, cus, sizes = SMALL[name]
        w = workloads.WORKLOADS[name].with_shape(M, N, K)
        say(f"[consumer grid] grid={grid} {w.name}")
        inp = workloads.make_inputs(w)
        plan, o = plan_for(w, inp, num_cus=cus, sizes=list(sizes))
        check(w, inp, plan, o)
    finally:
        fo.set_consumer_grid(*old)


@pytest.mark.parametrize("name", ["rs_8192x8192x3584", "a2a_4096x7168x2048"])
def test_plan_from_cache_runs_the_path(name):
    # a size seen only at run time takes the partition cached for its nearest
    # neighbour (Section 4.2); the plan built from it runs the whole path
    M, N, K, cus, _ = SMALL[name]
    w = workloads.WORKLOADS[name].with_shape(M, N, K)
    say(f"[pipeline plan cache] {w.name}")
    inp = workloads.make_inputs(w)
    nd = w.num_dest
    kw = dict(dtype=w.dtype, tile_m=w.tile_m, tile_n=w.tile_n, order=w.order, num_cus=cus,
              pattern=w.pattern, num_dest=nd, dest_perm=inp.sigma if w.pattern == "subtile" else None)
    rng = np.random.default_rng(7)
    cache = fo.PlanCache()
    waves = lambda m: -(-(m // w.tile_m) * (N // w.tile_n) // cus)
    cached = {512: oracle.rescale_partition((1, 1), waves(512)),
              2048: oracle.rescale_partition((1, 2, 2), waves(2048))}
    for m, sizes in cached.items():
        bucket = rng.integers(0, nd, m) if w.pattern == "subtoken" else None
        cache.add(m, N, K, sizes=list(sizes), row_bucket=bucket, **kw)
    plan, matched = cache.lookup(M, N, K, row_bucket=inp.bucket if w.pattern == "subtoken" else None, **kw)
    assert matched == oracle.nearest_size(list(cached), M)
    sizes = oracle.rescale_partition(cached[matched], plan.T)
    assert tuple(plan.sizes) == sizes
    o = oracle.make_plan(w.M, w.N, w.tile_m, w.tile_n, num_cus=cus, order=w.order, pattern=w.pattern,
                         num_dest=nd, sigma=inp.sigma, bucket=inp.bucket, sizes=sizes, unit="waves")
    check(w, inp, plan, o)


@pytest.mark.parametrize("limit", [8, 1])
@pytest.mark.parametrize("name", ["rs_8192x8192x3584", "a2a_4096x7168x2048"])
def test_capped_consumers_give_the_same_bits(name, limit):
    # a consumer launch cap (the slower-link stand-in, a per-call option)
    # changes grids and the consumer variant of every launch, not the result
    M, N, K, cus, sizes = SMALL[name]
    w = workloads.WORKLOADS[name].with_shape(M, N, K)
    say(f"[capped consumers] limit={limit} {w.name}")
    inp = workloads.make_inputs(w)
    plan, o = plan_for(w, inp, num_cus=cus, sizes=list(sizes))
    check(w, inp, plan, o, opts={"consumer_limit": limit})
