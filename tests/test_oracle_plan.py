"""Pins for the oracle's plan: dispatch order, waves, groups, counters and the
Algorithm 1 predictive search.

Pinned against the paper's worked examples (tests/golden/, each citing its
passage), closed-form counts of the design space, closed-form pipeline
latencies, and exhaustive search.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


# ---- worked examples from the paper -----------------------------------------

def test_counting_example():
    g = _gold("paper_counting_example.json")
    BM = BN = 16
    plan = oracle.make_plan(g["tiles_m"] * BM, g["tiles_n"] * BN, BM, BN,
                            num_cus=g["num_cus"], order=g["order"],
                            sizes=g["partition_waves"])
    assert plan.T == g["expect_waves"]
    assert plan.targets == g["expect_targets"]
    g0 = sorted(plan.order[s] for s in range(plan.first[0], plan.first[1]))
    assert g0 == g["expect_group0_tiles"]


def test_swizzle_example():
    g = _gold("paper_swizzle_example.json")
    order = oracle.dispatch_order(g["tiles_m"], g["tiles_n"], g["order"], g["group_m"])
    W = oracle.wave_width(g["num_cus"])
    assert sorted(order[:W]) == g["expect_first_wave_tiles"]


def test_reorder_example():
    g = _gold("paper_reorder_example.json")
    BM = BN = 8
    plan = oracle.make_plan(g["tiles_m"] * BM, g["tiles_n"] * BN, BM, BN,
                            num_cus=g["num_cus"], order=g["order"], group_m=g["group_m"],
                            sizes=(3,))
    for t, s in g["expect_slot_of_tile"].items():
        assert plan.tile_to_slot[int(t)] == s


def test_design_space_example():
    g = _gold("paper_design_space.json")
    T = g["T"]
    assert len(oracle.all_partitions(T)) == g["expect_space_size"]
    for ex in g["examples"]:
        cuts = [1 if w in ex["comm_after_waves"] else 0 for w in range(1, T)]
        assert oracle.cuts_to_partition(cuts) == tuple(ex["partition"])
        assert oracle.partition_to_cuts(ex["partition"]) == tuple(cuts)


def test_tuning_space_example():
    g = _gold("paper_tuning_space.json")
    assert len(oracle.all_partitions(g["T"])) == g["expect_unpruned"]


def test_wave_count_example():
    g = _gold("paper_wave_count.json")
    tiles = (g["M"] // g["tile_m"]) * (g["N"] // g["tile_n"])
    assert tiles == g["expect_tiles"]
    assert oracle.num_waves(tiles, oracle.wave_width(g["num_cus"])) == g["expect_waves"]


# ---- dispatch order -----------------------------------------------------------

@pytest.mark.parametrize("order", ["rowmajor", "grouped", "xcd"])
@pytest.mark.parametrize("grid", [(1, 1), (3, 2), (5, 7), (8, 32), (16, 56), (13, 9)])
@pytest.mark.parametrize("group_m,num_xcds", [(4, 8), (2, 3), (1, 1)])
def test_dispatch_order_is_bijection(order, grid, group_m, num_xcds):
    tm, tn = grid
    o = oracle.dispatch_order(tm, tn, order, group_m, num_xcds)
    assert sorted(o) == list(range(tm * tn))


def test_xcd_order_gives_compact_blocks_per_chiplet():
    # 8192x8192 output in 256x128 tiles: 32 x 64 tiles, 256 per wave. Each
    # chiplet (positions p = x mod 8) runs 32 tiles per wave; with bands of 4
    # tile rows they form a 4 x 8 block of the tile grid.
    tiles_m, tiles_n = 32, 64
    o = oracle.dispatch_order(tiles_m, tiles_n, "xcd", 4, 8)
    for wave in range(8):
        for x in range(8):
            ts = [o[p] for p in range(wave * 256, (wave + 1) * 256) if p % 8 == x]
            rows = {t // tiles_n for t in ts}
            cols = {t % tiles_n for t in ts}
            assert len(ts) == 32 and len(rows) == 4 and len(cols) == 8
            assert max(rows) - min(rows) == 3 and max(cols) - min(cols) == 7


def test_grouped_order_closed_form():
    # bands of group_m rows, column-major inside a band
    o = oracle.dispatch_order(4, 3, "grouped", 2)
    assert o == [0, 3, 1, 4, 2, 5, 6, 9, 7, 10, 8, 11]
    # a short last band (5 rows, bands of 2: the last band has 1 row)
    o = oracle.dispatch_order(5, 2, "grouped", 2)
    assert o[8:] == [8, 9]


@pytest.mark.parametrize("grid", [(1, 1), (3, 2), (5, 7), (8, 32), (13, 9), (7, 1), (1, 9)])
def test_dispatch_orders_reduce_to_plain_walks(grid):
    # special cases with a definition of their own: bands of one row are the
    # row-major walk; one band covering every row is the column-major walk;
    # one chiplet is the grouped order; and for any chiplet count the
    # positions of chiplet 0, then of chiplet 1, ... (p = x, x + X, ...) walk
    # the grouped order from its start, each chiplet a contiguous share
    tm, tn = grid
    T = tm * tn
    assert oracle.dispatch_order(tm, tn, "grouped", 1) == list(range(T))
    for g in (tm, tm + 3):
        assert oracle.dispatch_order(tm, tn, "grouped", g) == [(q % tm) * tn + q // tm for q in range(T)]
    for g in (1, 2, 3, 5):
        grouped = oracle.dispatch_order(tm, tn, "grouped", g)
        assert oracle.dispatch_order(tm, tn, "xcd", g, 1) == grouped
        for X in (2, 3, 8, 11, T + 2):
            o = oracle.dispatch_order(tm, tn, "xcd", g, X)
            assert [o[p] for x in range(X) for p in range(x, T, X)] == grouped, (g, X)


# ---- groups and counters ----------------------------------------------------------

@pytest.mark.parametrize("tiles_m,tiles_n,cus,sizes", [
    (4, 5, 8, (1, 1, 1)),       # 20 tiles, W=8, T=3, last wave holds 4 tiles
    (4, 5, 8, (2, 1)),
    (4, 5, 8, (3,)),
    (16, 56, 256, (1, 2, 1)),   # 896 tiles, 3.5 waves
    (1, 1, 256, (1,)),
])
def test_groups_cover_slots_and_targets_sum(tiles_m, tiles_n, cus, sizes):
    plan = oracle.make_plan(tiles_m * 8, tiles_n * 8, 8, 8, num_cus=cus, order="xcd", sizes=sizes)
    tiles = tiles_m * tiles_n
    assert sum(plan.targets) == tiles
    assert plan.first[0] == 0 and plan.first[-1] == tiles
    for j, g in enumerate(sizes):
        # every group but a partial last one is a union of whole waves
        f0, f1 = plan.first[j], plan.first[j + 1]
        assert f0 % plan.W == 0
        assert f1 % plan.W == 0 or f1 == tiles
        assert plan.targets[j] == min(g * plan.W, tiles - f0)
    # the slot of a tile is its dispatch position, so a slot's wave is p // W
    for s in range(tiles):
        assert plan.tile_to_slot[plan.order[s]] == s


def test_tile_unit_partition():
    plan = oracle.make_plan(256, 256, 64, 64, num_cus=256, order="rowmajor",
                            sizes=(4, 4, 4, 4), unit="tiles")
    assert plan.T == 1
    assert plan.targets == [4, 4, 4, 4]
    assert list(plan.tile_to_slot) == list(range(16))
    assert [list(plan.slot_group[4 * j:4 * j + 4]) for j in range(4)] == [[j] * 4 for j in range(4)]


# ---- design space and Algorithm 1 -------------------------------------------------------

def _compositions(n):
    return 1 if n == 0 else 2 ** (n - 1)


@pytest.mark.parametrize("T", range(1, 11))
@pytest.mark.parametrize("s1,sp", [(2, 4), (1, 1), (3, 2), (20, 20)])
def test_pruned_candidate_count_closed_form(T, s1, sp):
    # one group: its size is T (it is both first and last); P >= 2: a first
    # group a <= s1, a last group b <= sp and any composition of the middle.
    count = 1 if T <= min(s1, sp) else 0
    for a in range(1, s1 + 1):
        for b in range(1, sp + 1):
            if a + b <= T:
                count += _compositions(T - a - b)
    assert len(oracle.candidates(T, s1, sp)) == count


def test_candidate_order_is_cut_vector_order():
    c = oracle.all_partitions(3)
    assert c == [(3,), (1, 2), (2, 1), (1, 1, 1)]


def _linear(us_per_byte):
    return [1.0, 1e12], [us_per_byte, us_per_byte * 1e12]


def test_alg1_closed_form_linear_comm():
    # T = 2, GEMM 2 us, communication of one wave costs 1 us (proportional):
    # (1,1) -> wave 1 computes 0..1, its communication 1..2, wave 2 computes
    # 1..2, its communication 2..3: 3 us. (2) -> 2 + 2 = 4 us.
    W, BM, BN = 4, 8, 8
    wave_bytes = W * BM * BN * 2
    comm = lambda sizes: (lambda j: sizes[j] * 1.0)
    assert oracle.predicted_latency((1, 1), 2, 2.0, comm((1, 1))) == pytest.approx(3.0)
    assert oracle.predicted_latency((2,), 2, 2.0, comm((2,))) == pytest.approx(4.0)
    plan = oracle.make_plan(2 * BM, 4 * BN, BM, BN, num_cus=W, sizes=(2,))
    best, t = oracle.search_partition(plan, 2.0, [wave_bytes], [1.0])
    assert best == (1, 1) and t == pytest.approx(3.0)


def test_alg1_last_group_curve_closed_form():
    # T = 2, GEMM 2 us. Groups before the last: 2 us per wave of bytes; the
    # last group (after the GEMM): 0.5 us per wave. (1,1) -> wave 1's
    # communication 1..3, wave 2's 3..3.5: 3.5 us; (2) -> 2 + 2 * 0.5 = 3 us.
    # With the slow curve for both, (1,1) -> 5 us beats (2) -> 6 us.
    W, BM, BN = 4, 8, 8
    wave_bytes = W * BM * BN * 2
    plan = oracle.make_plan(2 * BM, 4 * BN, BM, BN, num_cus=W, sizes=(2,))
    slow, fast = ([wave_bytes], [2.0]), ([wave_bytes], [0.5])
    best, t = oracle.search_partition(plan, 2.0, *slow, last_curve=fast)
    assert best == (2,) and t == pytest.approx(3.0)
    best, t = oracle.search_partition(plan, 2.0, *slow)
    assert best == (1, 1) and t == pytest.approx(5.0)
    # the same curve given as the last group's changes nothing
    assert oracle.search_partition(plan, 2.0, *slow, last_curve=slow) == (best, t)


def test_alg1_closed_form_fixed_cost():
    # fixed 2 us per call plus 1 us per wave: (1,1) -> 7 us, (2) -> 6 us
    comm = lambda sizes: (lambda j: 2.0 + sizes[j])
    assert oracle.predicted_latency((1, 1), 2, 2.0, comm((1, 1))) == pytest.approx(7.0)
    assert oracle.predicted_latency((2,), 2, 2.0, comm((2,))) == pytest.approx(6.0)
    best, _ = oracle.predictive_search(2, 2.0, comm, 2, 4)
    assert best == (2,)


@pytest.mark.parametrize("P,tp,c", [(4, 10.0, 3.0), (4, 10.0, 25.0), (8, 5.0, 5.0), (1, 7.0, 2.0)])
def test_alg1_equal_groups_closed_form(P, tp, c):
    # P equal groups of one wave each, compute tp per wave, communication c
    # per group: a two-stage pipeline finishes at P*tp + c if c <= tp, else
    # at tp + P*c.
    sizes = (1,) * P
    t = oracle.predicted_latency(sizes, P, P * tp, lambda j: c)
    assert t == pytest.approx(P * tp + c if c <= tp else tp + P * c)


def test_alg1_zero_comm_picks_first_candidate():
    comm = lambda sizes: (lambda j: 0.0)
    best, t = oracle.predictive_search(6, 12.0, comm, 2, 4)
    assert t == pytest.approx(12.0)
    assert best == oracle.candidates(6, 2, 4)[0]


@pytest.mark.parametrize("T", [3, 5, 7])
@pytest.mark.parametrize("fixed", [0.0, 1.5, 6.0])
def test_pruned_search_matches_exhaustive_when_optimum_is_in_bounds(T, fixed):
    per_wave = 2.0
    comm = lambda sizes: (lambda j: fixed + per_wave * sizes[j])
    gemm = 3.0 * T
    ex_best, ex_t = oracle.predictive_search(T, gemm, comm, 99, 99, cands=oracle.all_partitions(T))
    pr_best, pr_t = oracle.predictive_search(T, gemm, comm, 2, 4)
    assert pr_t >= ex_t - 1e-9
    if ex_best[0] <= 2 and ex_best[-1] <= 4:
        assert pr_t == pytest.approx(ex_t)


def test_interp_latency():
    xs, ys = [100.0, 200.0, 400.0], [1.0, 1.5, 2.0]
    assert oracle.interp_latency(xs, ys, 150.0) == pytest.approx(1.25)
    assert oracle.interp_latency(xs, ys, 400.0) == pytest.approx(2.0)
    assert oracle.interp_latency(xs, ys, 800.0) == pytest.approx(4.0)   # end-point bandwidth
    assert oracle.interp_latency(xs, ys, 50.0) == pytest.approx(0.5)
    assert oracle.interp_latency(xs, ys, 0.0) == 0.0


@pytest.mark.parametrize("B", [1, 3, 8])
def test_all_to_all_group_bytes(B):
    # every tile row goes to exactly one destination pool, so a group's pieces
    # add up to its tiles' bytes; the largest piece is at most that, equal
    # with one destination, and at least the average over destinations
    rng = np.random.default_rng(60 + B)
    M, N, BM, BN = 1024, 512, 256, 128                      # 16 tiles
    bucket = rng.integers(0, B, M)
    o = oracle.make_plan(M, N, BM, BN, num_cus=4, order="xcd", pattern="subtoken", num_dest=B,
                         bucket=bucket, sizes=(1, 2, 1))
    first = o.first
    for j in range(len(first) - 1):
        f0, f1 = first[j], first[j + 1]
        total = oracle.slot_range_bytes(o, f0, f1, 2, all_dest=True)
        largest = oracle.slot_range_bytes(o, f0, f1, 2)
        assert total == (f1 - f0) * BM * BN * 2
        assert largest <= total and largest * B >= total
        if B == 1:
            assert largest == total
