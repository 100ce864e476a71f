"""Host planner (libfo's fo_plan_groups) against the oracle's plan, bit for
bit: dispatch order, reorder map, groups, counter targets, segments, pools,
and the Algorithm 1 choice. Runs on the CPU (no GPU call is made)."""
import math
import re
import os

import numpy as np
import pytest

import oracle
import paper_2504_19519_amd as fo
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _both(M, N, BM, BN, *, cus, order="xcd", group_m=4, num_xcds=8, pattern="tile", nd=0,
          sigma=None, bucket=None, sizes=None, unit="waves", wg_per_cu=1, reserved=0):
    p = fo.plan_groups(M, N, 64, tile_m=BM, tile_n=BN, order=order, group_m=group_m,
                       num_xcds=num_xcds, num_cus=cus, wg_per_cu=wg_per_cu, reserved_cus=reserved,
                       pattern=pattern, num_dest=nd, dest_perm=sigma, row_bucket=bucket,
                       sizes=sizes, unit=unit)
    o = oracle.make_plan(M, N, BM, BN, num_cus=cus, wg_per_cu=wg_per_cu, reserved_cus=reserved,
                         order=order, group_m=group_m, num_xcds=num_xcds, pattern=pattern,
                         num_dest=nd, sigma=sigma, bucket=bucket, sizes=sizes, unit=unit)
    return p, o


def _compare(p, o):
    assert p.tiles == o.tiles and p.W == o.W and p.T == o.T and p.P == o.P
    np.testing.assert_array_equal(p.order, np.array(o.order))
    np.testing.assert_array_equal(p.tile_to_slot, o.tile_to_slot)
    np.testing.assert_array_equal(p.group_first, np.array(o.first))
    np.testing.assert_array_equal(p.targets, np.array(o.targets))
    np.testing.assert_array_equal(p.segments, np.array(oracle.segments(o), dtype=np.int64).reshape(-1, 5))
    assert p.dest_elems == oracle.dest_buffer_elems(o)
    if o.pattern == "subtoken":
        np.testing.assert_array_equal(p.pool_base, o.pool_base)
        np.testing.assert_array_equal(p.pool_off, o.pool_off)


def _workload_plan_args(w: workloads.Workload, inp=None):
    kw = dict(cus=256, order=w.order, pattern=w.pattern, nd=w.num_dest if w.pattern in ("subtile", "subtoken") else 0)
    if w.pattern == "subtile":
        kw["sigma"] = np.random.default_rng(w.seed).permutation(w.num_dest)
    if w.pattern == "subtoken":
        kw["bucket"] = np.random.default_rng(w.seed).integers(0, w.num_dest, w.M)
    return kw


@pytest.mark.parametrize("name", list(workloads.WORKLOADS))
def test_workload_plans_match_oracle(name):
    w = workloads.WORKLOADS[name]
    kw = _workload_plan_args(w)
    tiles = (w.M // w.tile_m) * (w.N // w.tile_n)
    T = -(-tiles // 256)
    if w.groups is not None:
        sizes, unit = list(w.groups), w.group_unit
    else:
        sizes, unit = [1] * T, "waves"
    p, o = _both(w.M, w.N, w.tile_m, w.tile_n, sizes=sizes, unit=unit, **kw)
    _compare(p, o)


@pytest.mark.parametrize("pattern,nd", [("tile", 0), ("subtile", 4), ("subtoken", 8), ("rowmajor", 0)])
@pytest.mark.parametrize("order", ["rowmajor", "grouped", "xcd"])
@pytest.mark.parametrize("shape", [(1024, 640, 256, 128, 8, (1, 2)),     # 20 tiles, W=8, T=3
                                   (768, 384, 64, 64, 5, (2, 1, 3, 1)),   # 72 tiles, W=5, T=15 -> sizes sum 7? fixed below
                                   (512, 1024, 256, 128, 3, None)])
def test_small_plans_match_oracle(pattern, nd, order, shape):
    M, N, BM, BN, cus, sizes = shape
    rng = np.random.default_rng(7)
    tiles = (M // BM) * (N // BN)
    T = -(-tiles // cus)
    if sizes is None or sum(sizes) != T:
        # a deterministic irregular partition of T waves
        sizes, left = [], T
        while left:
            s = min(left, int(rng.integers(1, 4)))
            sizes.append(s)
            left -= s
    kw = dict(cus=cus, order=order, group_m=3, num_xcds=8 if order == "xcd" else 1,
              pattern=pattern, nd=nd, sizes=sizes)
    if pattern == "subtile":
        kw["sigma"] = rng.permutation(nd)
    if pattern == "subtoken":
        kw["bucket"] = rng.integers(0, nd, M)
    p, o = _both(M, N, BM, BN, **kw)
    _compare(p, o)


@pytest.mark.parametrize("order", ["grouped", "xcd"])
@pytest.mark.parametrize("group_m,num_xcds", [(1, 1), (2, 3), (5, 11), (6, 12), (40, 8)])
def test_dispatch_parameters_match_oracle(order, group_m, num_xcds):
    # band heights that do not divide the 13 tile rows (and one taller than
    # the grid) and chiplet counts above the GEMM's 8 position counters
    p, o = _both(13 * 64, 9 * 64, 64, 64, cus=10, order=order, group_m=group_m, num_xcds=num_xcds,
                 sizes=[3, 4, 5])
    _compare(p, o)


def test_tile_unit_and_reserved_cus():
    p, o = _both(2048, 1024, 256, 128, cus=16, reserved=3, wg_per_cu=2, sizes=[5, 20, 39], unit="tiles")
    _compare(p, o)
    assert p.W == (16 - 3) * 2


def _curve(seed):
    rng = np.random.default_rng(seed)
    xs = np.sort(rng.uniform(1e4, 5e8, 12))
    bw = rng.uniform(0.5e3, 6e3, 12)            # bytes per us
    ys = np.maximum.accumulate(xs / bw + rng.uniform(2, 10))
    return xs, ys


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("pattern,nd", [("tile", 0), ("subtoken", 8), ("subtile", 4)])
@pytest.mark.parametrize("dest_bytes", ["largest", "all"])
def test_predictive_search_matches_oracle(seed, pattern, nd, dest_bytes):
    rng = np.random.default_rng(100 + seed)
    M, N, BM, BN = 4096, 7168, 256, 128      # 896 tiles, 3.5 waves at 256 CUs
    cus = int(rng.choice([64, 128, 256]))
    xs, ys = _curve(seed)
    gemm_us = float(rng.uniform(20, 400))
    bucket = rng.integers(0, nd, M) if pattern == "subtoken" else None
    sigma = rng.permutation(nd) if pattern == "subtile" else None
    p = fo.plan_groups(M, N, 2048, num_cus=cus, pattern=pattern, num_dest=nd, row_bucket=bucket,
                       dest_perm=sigma, sizes=None, gemm_us=gemm_us, curve_bytes=xs, curve_us=ys,
                       s_first=2, s_last=4, dest_bytes=dest_bytes)
    o = oracle.make_plan(M, N, BM, BN, num_cus=cus, order="xcd", pattern=pattern, num_dest=nd,
                         bucket=bucket, sigma=sigma, sizes=(-(-896 // cus),))
    best, t = oracle.search_partition(o, gemm_us, xs, ys, 2, 4, all_dest=dest_bytes == "all")
    assert tuple(p.sizes) == best
    assert p.predicted_us == pytest.approx(t, rel=1e-12)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("pattern,nd", [("tile", 0), ("subtoken", 8), ("subtile", 4)])
def test_search_and_estimate_with_last_group_curve_match_oracle(seed, pattern, nd):
    # a second curve for the last group (its communication after the GEMM):
    # the search and the estimate of a given partition against the oracle
    rng = np.random.default_rng(300 + seed)
    M, N, BM, BN = 4096, 7168, 256, 128
    cus = int(rng.choice([64, 128, 256]))
    xs, ys = _curve(seed + 20)
    lx, ly = _curve(seed + 40)
    gemm_us = float(rng.uniform(20, 400))
    bucket = rng.integers(0, nd, M) if pattern == "subtoken" else None
    sigma = rng.permutation(nd) if pattern == "subtile" else None
    kw = dict(num_cus=cus, pattern=pattern, num_dest=nd, row_bucket=bucket, dest_perm=sigma, gemm_us=gemm_us,
              curve_bytes=xs, curve_us=ys, last_curve_bytes=lx, last_curve_us=ly)
    p = fo.plan_groups(M, N, 2048, sizes=None, s_first=2, s_last=4, **kw)
    o = oracle.make_plan(M, N, BM, BN, num_cus=cus, order="xcd", pattern=pattern, num_dest=nd,
                         bucket=bucket, sigma=sigma, sizes=(-(-896 // cus),))
    best, t = oracle.search_partition(o, gemm_us, xs, ys, 2, 4, last_curve=(lx, ly))
    assert tuple(p.sizes) == best
    assert p.predicted_us == pytest.approx(t, rel=1e-12)
    T = -(-896 // cus)
    cuts = sorted(rng.choice(np.arange(1, T), size=int(rng.integers(0, T)), replace=False)) if T > 1 else []
    sizes = tuple(int(b - a) for a, b in zip([0] + list(cuts), list(cuts) + [T]))
    q = fo.plan_groups(M, N, 2048, sizes=list(sizes), **kw)
    first = oracle.group_first_slots(sizes, "waves", o.W, o.tiles)
    lat = [oracle.interp_latency(*((lx, ly) if j == len(sizes) - 1 else (xs, ys)),
                                 oracle.slot_range_bytes(o, first[j], first[j + 1], 2)) for j in range(len(sizes))]
    assert q.predicted_us == pytest.approx(oracle.predicted_latency(sizes, T, gemm_us, lambda j: lat[j]), rel=1e-12)


def test_last_group_curve_is_checked():
    with pytest.raises(fo.FoError):
        fo.plan_groups(4096, 7168, 2048, sizes=None, gemm_us=100.0, curve_bytes=[1e6, 1e8], curve_us=[5.0, 20.0],
                       last_curve_bytes=[1e8, 1e6], last_curve_us=[5.0, 20.0])


def test_search_single_wave_gives_one_group():
    # 2048 x 4096 in 256x128 tiles is 256 tiles: one wave on 256 CUs
    p = fo.plan_groups(2048, 4096, 4096, num_cus=256, sizes=None, gemm_us=40.0,
                       curve_bytes=[1e6, 1e8], curve_us=[5.0, 20.0])
    assert p.T == 1 and list(p.sizes) == [1] and list(p.targets) == [256]


@pytest.mark.parametrize("kwargs,status", [
    (dict(M=1000, N=1024, K=64), -2),                          # M % tile_m
    (dict(M=1024, N=1024, K=64, sizes=[1, 1, 1]), -1),         # sizes do not sum to T
    (dict(M=1024, N=1024, K=64, pattern="subtile", num_dest=3, sizes=[1]), -2),   # 256 % 3
    (dict(M=1024, N=1024, K=64, pattern="subtoken", num_dest=4, sizes=[1]), -1),  # no row_bucket
    (dict(M=1024, N=1024, K=64, pattern="subtile", num_dest=4, dest_perm=[0, 0, 1, 2], sizes=[1]), -1),
    (dict(M=1024, N=1024, K=64, sizes=None), -1),              # search without a curve
    (dict(M=1024, N=1024, K=64, num_cus=0, sizes=[1]), -1),
    (dict(M=1024, N=1024, K=64, order="grouped", group_m=0, sizes=[1]), -1),
    (dict(M=1024, N=1024, K=64, order="xcd", group_m=-2, sizes=[1]), -1),
    (dict(M=1024, N=1024, K=64, order="xcd", num_xcds=0, sizes=[1]), -1),
    (dict(M=256 * 64, N=128 * 64, K=64, num_cus=16, sizes=None, curve_bytes=[1.0], curve_us=[1.0]), -3),
])
def test_plan_errors(kwargs, status):
    with pytest.raises(fo.FoError) as e:
        fo.plan_groups(**kwargs)
    assert e.value.status == status


def test_rowmajor_order_ignores_band_and_chiplet_fields():
    # the band height and chiplet count are read by the grouped and XCD
    # orders only
    p = fo.plan_groups(1024, 1024, 64, order="rowmajor", group_m=0, num_xcds=0, sizes=[1])
    np.testing.assert_array_equal(p.order, np.arange(p.tiles))


def test_empty_problem():
    p = fo.plan_groups(0, 1024, 64, sizes=None, curve_bytes=[1.0], curve_us=[1.0])
    assert p.tiles == 0 and p.T == 0 and p.P == 0 and p.segments.shape == (0, 5)
    # an empty problem launches nothing: the calls return before any device
    # work (the pointers are never used)
    fake = 1 << 20
    fo.gemm_signal_reorder(p, fake, fake, fake, fake)
    fo.post_reorder(p, fake, fake, fake)
    fo.run_overlapped(p, fake, fake, fake, fake, fake, fake, fake, counters=fake, gemm_stream=fake,
                      comm_stream=fake + 64)


def test_header_symbols_are_exported():
    with open(os.path.join(ROOT, "include", "fo.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = set(re.findall(r"\b(fo_[a-z0-9_]+)\s*\(", text))
    assert len(names) >= 25
    L = fo.lib()
    missing = [n for n in sorted(names) if not hasattr(L, n)]
    assert not missing, missing


def test_process_wide_settings_validate_and_round_trip():
    # host-side setters only: no device work
    old_modes, old_grid = fo.get_sync_mode(), fo.get_consumer_grid()
    try:
        for bad in ((0, 64), (257, 64), (-3, 64), (16, 32), (16, 96), (16, 512)):
            with pytest.raises(fo.FoError) as e:
                fo.set_consumer_grid(*bad)
            assert e.value.status == -1
        assert fo.get_consumer_grid() == old_grid
        fo.set_consumer_grid(7, 128)
        assert fo.get_consumer_grid() == (7, 128)
        with pytest.raises(fo.FoError):
            fo.set_sync_mode(3, 0)
        fo.set_sync_mode(1, 0)
        assert fo.get_sync_mode() == (1, 0)
        # per-call options start from the process defaults as they stand
        o = fo.options()
        assert (o.sync_producer, o.sync_consumer) == (1, 0)
        assert (o.consumer_blocks, o.consumer_threads) == (7, 128)
        assert o.poll_timeout_us == fo.get_poll_timeout_us() and o.consumer_limit == 0
        assert o.tile_trace is None and o.tile_trace_capacity == 0
    finally:
        fo.set_consumer_grid(*old_grid)
        fo.set_sync_mode(*old_modes)


@pytest.mark.parametrize("bad", [dict(sync_producer=3), dict(sync_consumer=-1), dict(consumer_blocks=0),
                                 dict(consumer_blocks=257), dict(consumer_threads=96),
                                 dict(poll_timeout_us=0), dict(consumer_limit=-1), dict(consumer_limit=257),
                                 dict(reserved0=1), dict(tile_trace=8, tile_trace_capacity=0),
                                 dict(tile_trace=12, tile_trace_capacity=4)])
def test_per_call_options_are_checked(bad):
    # checked before any device work: an empty consumer call (no counter, no
    # elements) with bad options fails, with good ones launches nothing
    fo.consume_group(None, None, None, 0, "fp16", opts={})
    with pytest.raises(fo.FoError) as e:
        fo.consume_group(None, None, None, 0, "fp16", opts=bad)
    assert e.value.status == -1


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("pattern,nd", [("tile", 0), ("subtoken", 8), ("subtile", 4)])
def test_given_partition_estimate_matches_oracle(seed, pattern, nd):
    # a partition given in waves together with a curve carries Algorithm 1's
    # estimate of that partition: the oracle's latency recurrence on it
    rng = np.random.default_rng(200 + seed)
    M, N, BM, BN = 4096, 7168, 256, 128      # 896 tiles
    cus = int(rng.choice([64, 128, 256]))
    xs, ys = _curve(seed + 10)
    gemm_us = float(rng.uniform(20, 400))
    T = -(-896 // cus)
    cuts = sorted(rng.choice(np.arange(1, T), size=int(rng.integers(0, T)), replace=False)) if T > 1 else []
    sizes = tuple(int(b - a) for a, b in zip([0] + list(cuts), list(cuts) + [T]))
    bucket = rng.integers(0, nd, M) if pattern == "subtoken" else None
    sigma = rng.permutation(nd) if pattern == "subtile" else None
    p = fo.plan_groups(M, N, 2048, num_cus=cus, pattern=pattern, num_dest=nd, row_bucket=bucket,
                       dest_perm=sigma, sizes=list(sizes), gemm_us=gemm_us, curve_bytes=xs, curve_us=ys)
    o = oracle.make_plan(M, N, BM, BN, num_cus=cus, order="xcd", pattern=pattern, num_dest=nd,
                         bucket=bucket, sigma=sigma, sizes=sizes)
    first = oracle.group_first_slots(sizes, "waves", o.W, o.tiles)
    lat = [oracle.interp_latency(xs, ys, oracle.slot_range_bytes(o, first[j], first[j + 1], 2))
           for j in range(len(sizes))]
    t = oracle.predicted_latency(sizes, T, gemm_us, lambda j: lat[j])
    assert tuple(p.sizes) == sizes
    assert p.predicted_us == pytest.approx(t, rel=1e-12)
    # without a curve there is no estimate
    q = fo.plan_groups(M, N, 2048, num_cus=cus, pattern=pattern, num_dest=nd, row_bucket=bucket,
                       dest_perm=sigma, sizes=list(sizes))
    assert q.predicted_us == 0.0


def test_counters_and_overlapped_argument_checks():
    # host-side checks only: these calls return before any device work
    p = fo.plan_groups(1024, 1024, 64, sizes=[2, 2], num_cus=8, tile_m=256, tile_n=128)   # 32 tiles, 4 waves
    assert p.num_counters == p.P + 8 + 226        # groups, positions, handoff words
    fake = 1 << 20                                # never dereferenced
    for kw in (dict(counters=None, gemm_stream=fake, comm_stream=fake + 64),   # no counters
               dict(counters=fake, gemm_stream=None, comm_stream=fake + 64)):  # null GEMM stream
        with pytest.raises(fo.FoError) as e:
            fo.run_overlapped(p, fake, fake, fake, fake, fake, fake, None, **kw)
        assert e.value.status == -1


def test_binding_rejects_short_tensors_before_the_call():
    # the binding checks tensor sizes against the plan (host-side only: the
    # tensors here are CPU tensors and the calls never reach the library)
    import torch
    with open(os.path.join(ROOT, "include", "fo.h")) as f:
        m = re.search(r"#define FO_DISPENSER_WORDS (\d+)", f.read())
    assert m and int(m.group(1)) == fo.DISPENSER_WORDS
    p = fo.plan_groups(1024, 1024, 64, sizes=[2, 2], num_cus=8, tile_m=256, tile_n=128)
    short = torch.zeros(p.num_counters - 1, dtype=torch.int32)
    with pytest.raises(ValueError, match="counters"):
        fo.run_overlapped(p, 1, 1, 1, 1, 1, 1, counters=short, gemm_stream=1, comm_stream=2)
    with pytest.raises(ValueError, match="C_out"):
        fo.gemm_signal_reorder(p, 1, 1, 1, torch.zeros(1024 * 1024 - 1, dtype=torch.int16))
    with pytest.raises(ValueError, match="dst"):
        fo.consume_group(1, None, torch.zeros(7, dtype=torch.int16), 8, "fp16")
    with pytest.raises(ValueError, match="gamma"):
        fo.post_reorder(p, 1, 1, 1, gamma=torch.zeros(1023, dtype=torch.int16))


def test_noalloc_rejects_plans_beyond_its_static_array():
    # 1024 groups of one 64x64 tile need 1024 + 10 counter words: refused
    # before any device work, with the limit in the message
    plan = fo.plan_groups(2048, 2048, 64, dtype="fp16", tile_m=64, tile_n=64, order="rowmajor", num_cus=256,
                          pattern="tile", sizes=[1] * 1024, unit="tiles")
    assert plan.num_counters > fo.NOALLOC_MAX_COUNTERS
    with pytest.raises(fo.FoError) as e:
        fo.run_overlapped_noalloc(plan, 16, 16, 16, 16, None, 16, None)
    assert e.value.status == -1 and str(fo.NOALLOC_MAX_COUNTERS) in str(e.value)
