"""Reuse of searched partitions for sizes seen only at run time (Section 4.2,
online stage: the search runs ahead of time for representative GEMM sizes,
an unseen size takes the partition of its nearest neighbour).

Oracle pins (no library): the rescaling of a partition to another wave
count reduces to the identity on equal counts and to exact scaling on
integer multiples, keeps every group non-empty and the total equal to the
new wave count, and matches hand-worked cases; the nearest size agrees with
brute force over the distance and the tie rule. Library parity (CPU only):
fo_plan_cache_lookup builds the same partition as the oracle, on given and
on searched (Algorithm 1) entries, for every pattern."""
import numpy as np
import pytest

import oracle
import paper_2504_19519_amd as fo


# ---- oracle pins ----------------------------------------------------------

@pytest.mark.parametrize("T", range(1, 9))
def test_rescale_identity_on_equal_wave_counts(T):
    for sizes in oracle.all_partitions(T):
        assert oracle.rescale_partition(sizes, T) == sizes


@pytest.mark.parametrize("T,k", [(3, 2), (4, 2), (4, 3), (5, 4)])
def test_rescale_integer_multiple_scales_every_group(T, k):
    # boundaries b -> k*b land exactly, so every group grows k-fold
    for sizes in oracle.all_partitions(T):
        assert oracle.rescale_partition(sizes, k * T) == tuple(k * s for s in sizes)


@pytest.mark.parametrize("sizes,T,want", [
    ((1, 2, 1), 8, (2, 4, 2)),      # boundaries 1, 3 of 4 -> 2, 6 of 8
    ((1, 2, 1), 6, (2, 3, 1)),      # 1.5 -> 2, 4.5 -> 5 (halves up)
    ((1, 2, 1), 2, (1, 1)),         # 0.5 -> 1; 1.5 -> 2 = T is dropped
    ((1, 2, 1), 1, (1,)),           # everything collapses into one group
    ((2, 2, 4), 10, (3, 2, 5)),     # 2.5 -> 3, 5 -> 5
    ((1, 1, 1, 1), 3, (1, 1, 1)),   # 0.75 -> 1, 1.5 -> 2, 2.25 -> 2 (not after 2: dropped)
    ((4,), 7, (7,)),
])
def test_rescale_hand_cases(sizes, T, want):
    assert oracle.rescale_partition(sizes, T) == want


def test_rescale_properties_random():
    rng = np.random.default_rng(0)
    for _ in range(300):
        T_ref = int(rng.integers(1, 12))
        parts = oracle.all_partitions(T_ref)
        sizes = parts[int(rng.integers(0, len(parts)))]
        T = int(rng.integers(1, 30))
        got = oracle.rescale_partition(sizes, T)
        assert sum(got) == T and min(got) >= 1 and len(got) <= len(sizes)


def test_nearest_size_brute_force_and_ties():
    rng = np.random.default_rng(1)
    for _ in range(200):
        ms = sorted(set(int(x) for x in rng.integers(1, 64, int(rng.integers(1, 6))) * 256))
        M = int(rng.integers(1, 80)) * 256
        best = min(ms, key=lambda m: (abs(M - m), m))
        assert oracle.nearest_size(ms, M) == best
    assert oracle.nearest_size([1024, 3072], 2048) == 1024       # tie: the smaller size
    assert oracle.nearest_size([3072, 1024], 2048) == 1024
    with pytest.raises(KeyError):
        oracle.nearest_size([], 1024)


# ---- library against the oracle --------------------------------------------

def _family(pattern, nd, rng):
    kw = dict(dtype="fp16", tile_m=256, tile_n=128, order="xcd", num_cus=int(rng.choice([64, 128, 256])),
              pattern=pattern, num_dest=nd)
    if pattern == "subtile":
        kw["dest_perm"] = list(rng.permutation(nd))
    return kw


def _bucket(pattern, nd, M, rng):
    return list(rng.integers(0, nd, M)) if pattern == "subtoken" else None


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("pattern,nd", [("tile", 0), ("subtile", 4), ("subtoken", 8)])
def test_lookup_matches_oracle_on_given_partitions(seed, pattern, nd):
    rng = np.random.default_rng(10 * seed + nd)
    N, K = 7168, 2048
    kw = _family(pattern, nd, rng)
    cache = fo.PlanCache()
    ref = {}
    for M in sorted(set(int(x) * 256 for x in rng.integers(1, 40, 4))):
        T = -(-(M // 256) * (N // 128) // kw["num_cus"])
        parts = oracle.all_partitions(T) if T <= 10 else [oracle.rescale_partition((1, 2, 1), T)]
        sizes = parts[int(rng.integers(0, len(parts)))]
        cache.add(M, N, K, sizes=list(sizes), row_bucket=_bucket(pattern, nd, M, rng), **kw)
        ref[M] = sizes
    assert len(cache) == len(ref) and dict((m, tuple(s)) for m, s in cache.entries()) == ref
    for _ in range(6):
        M = int(rng.integers(1, 48)) * 256
        plan, matched = cache.lookup(M, N, K, row_bucket=_bucket(pattern, nd, M, rng), **kw)
        m_ref = oracle.nearest_size(list(ref), M)
        T = -(-(M // 256) * (N // 128) // kw["num_cus"])
        assert matched == m_ref
        assert tuple(plan.sizes) == oracle.rescale_partition(ref[m_ref], T)
        assert plan.T == T and int(plan.targets.sum()) == plan.tiles


@pytest.mark.parametrize("seed", range(4))
def test_lookup_of_searched_entries_matches_oracle(seed):
    rng = np.random.default_rng(50 + seed)
    N, K, cus = 8192, 3584, 256
    xs = np.sort(rng.uniform(1e5, 5e8, 10))
    ys = np.maximum.accumulate(xs / rng.uniform(1e3, 6e3, 10) + rng.uniform(2, 10))
    kw = dict(tile_m=256, tile_n=256, num_cus=cus, pattern="tile")
    cache = fo.PlanCache()
    searched = {}
    for M in (4096, 8192, 16384):
        gemm_us = 48.0 * M / 1024
        cache.add(M, N, K, sizes=None, gemm_us=gemm_us, curve_bytes=xs, curve_us=ys, s_first=2, s_last=4, **kw)
        o = oracle.make_plan(M, N, 256, 256, num_cus=cus, order="xcd", pattern="tile",
                             sizes=(-(-(M // 256) * (N // 256) // cus),))
        searched[M], _ = oracle.search_partition(o, gemm_us, xs, ys, 2, 4)
    assert dict((m, tuple(s)) for m, s in cache.entries()) == searched
    for M in (2048, 6144, 10240, 12288, 24576):
        plan, matched = cache.lookup(M, N, K, **kw)
        T = -(-(M // 256) * (N // 256) // cus)
        assert matched == oracle.nearest_size(list(searched), M)
        assert tuple(plan.sizes) == oracle.rescale_partition(searched[matched], T)


def test_add_replaces_same_size_and_families_are_separate():
    kw = dict(tile_m=256, tile_n=256, num_cus=256, pattern="tile")
    cache = fo.PlanCache()
    cache.add(8192, 8192, 3584, sizes=[1, 2, 1], **kw)
    cache.add(8192, 8192, 3584, sizes=[2, 2], **kw)              # same family and M: replaced
    cache.add(8192, 4096, 3584, sizes=[1, 1], **kw)              # other N: another family
    assert cache.entries() == [(8192, [2, 2]), (8192, [1, 1])]
    plan, m = cache.lookup(8192, 4096, 3584, **kw)
    assert m == 8192 and list(plan.sizes) == [1, 1]
    with pytest.raises(fo.FoError) as e:
        cache.lookup(8192, 8192, 7168, **kw)                      # other K: no entry
    assert e.value.status == -1
    with pytest.raises(fo.FoError):
        cache.add(1024, 1024, 64, sizes=[4], unit="tiles", tile_m=256, tile_n=256, num_cus=256)
    s = dict(kw, pattern="subtile", num_dest=4)
    cache.add(8192, 8192, 3584, sizes=[4], dest_perm=[1, 0, 2, 3], **s)
    with pytest.raises(fo.FoError):
        cache.lookup(8192, 8192, 3584, dest_perm=[0, 1, 2, 3], **s)    # other sigma: other family
    plan, _ = cache.lookup(4096, 8192, 3584, dest_perm=[1, 0, 2, 3], **s)
    assert list(plan.sizes) == [2]


def test_lookup_of_an_empty_problem():
    cache = fo.PlanCache()
    cache.add(1024, 1024, 64, sizes=[1], tile_m=256, tile_n=256, num_cus=256)
    plan, m = cache.lookup(0, 1024, 64, tile_m=256, tile_n=256, num_cus=256)
    assert m == 1024 and plan.tiles == 0 and plan.P == 0
