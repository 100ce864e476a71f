"""Pins for the oracle's reorder permutations, consumer segments and the
post-communication gather (Section 3.3).

The forward permutation (what the epilogue writes where), the segment list
(what each group hands to the communication) and the post gather (where the
element-wise kernel loads from) are built independently from the layout
definitions; composing them must give the identity. Brute force on a 2x2 tile
grid checks every slot order and every group partition against dense
permutation matrices.
"""
import itertools

import numpy as np
import pytest

import oracle
import workloads


def _bits(n, seed, dtype="fp16"):
    return workloads.uniform_bits(n, seed, dtype)


def _plans():
    rng = np.random.default_rng(0)
    out = []
    # (M, N, BM, BN, cus, order, pattern, num_dest, sizes)
    for pattern, nd in [("tile", 0), ("subtile", 4), ("subtoken", 8), ("rowmajor", 0)]:
        for (M, N, BM, BN, cus, sizes) in [
            (128, 96, 32, 16, 5, (1, 2, 2)),     # 24 tiles, W=5, T=5, last wave 4 tiles
            (64, 64, 16, 16, 16, (1,)),
            (96, 48, 32, 16, 2, (2, 1, 1, 1)),   # 9 tiles, W=2, T=5
        ]:
            kw = dict(num_cus=cus, order="xcd", group_m=2, num_xcds=3, pattern=pattern,
                      num_dest=nd, sizes=sizes)
            if pattern == "subtile":
                kw["sigma"] = rng.permutation(nd)
            if pattern == "subtoken":
                kw["bucket"] = rng.integers(0, nd, M)
            out.append(oracle.make_plan(M, N, BM, BN, **kw))
    return out


PLANS = _plans()


@pytest.mark.parametrize("plan", PLANS, ids=lambda p: f"{p.pattern}-{p.M}x{p.N}-{p.sizes}")
def test_reorder_is_permutation(plan):
    perm = oracle.reorder_index(plan)
    assert np.array_equal(np.sort(perm), np.arange(plan.M * plan.N))


@pytest.mark.parametrize("plan", PLANS, ids=lambda p: f"{p.pattern}-{p.M}x{p.N}-{p.sizes}")
def test_post_after_copy_consumer_after_reorder_is_identity(plan):
    C = _bits(plan.M * plan.N, 1)
    _, _, out = oracle.run_path(plan, C, None, "fp16")
    np.testing.assert_array_equal(out.reshape(-1), C)


@pytest.mark.parametrize("plan", PLANS, ids=lambda p: f"{p.pattern}-{p.M}x{p.N}-{p.sizes}")
def test_segments_are_contiguous_disjoint_and_cover(plan):
    segs = oracle.segments(plan)
    n_src = plan.M * plan.N
    covered = np.zeros(n_src, dtype=np.int32)
    dcovered = np.zeros(oracle.dest_buffer_elems(plan), dtype=np.int32)
    for (j, d, so, do, ln) in segs:
        covered[so:so + ln] += 1
        dcovered[do:do + ln] += 1
    assert np.all(covered == 1)
    assert np.all(dcovered == 1)
    if plan.pattern == "rowmajor":
        return
    # per group, the pieces add up to the group's tiles
    for j in range(plan.P):
        assert sum(s[4] for s in segs if s[0] == j) == plan.targets[j] * plan.BM * plan.BN
    # a group's data is exactly the output of the group's tiles
    perm = oracle.reorder_index(plan)
    for j in range(plan.P):
        elems = np.concatenate([perm[so:so + ln] for (jj, d, so, do, ln) in segs if jj == j])
        tiles = {plan.order[s] for s in range(plan.first[j], plan.first[j + 1])}
        rows, cols = elems // plan.N, elems % plan.N
        got = {(r // plan.BM) * plan.tiles_n + c // plan.BN for r, c in zip(rows, cols)}
        assert got == tiles


@pytest.mark.parametrize("plan", [p for p in PLANS if p.pattern == "subtile"],
                         ids=lambda p: f"{p.M}x{p.N}-{p.sizes}")
def test_subtile_rows_complete_on_one_destination(plan):
    # Section 3.3 Insight (2): each row must end up entirely on one GPU
    idx = oracle.post_index(plan).reshape(plan.M, plan.N)
    per_dest = plan.tiles * (plan.BM // plan.num_dest) * plan.BN
    dest = idx // per_dest
    assert np.all(dest == dest[:, :1])
    # and destination sigma(k) receives slice k of every tile
    h = plan.BM // plan.num_dest
    for i in range(plan.M):
        assert dest[i, 0] == plan.sigma[(i % plan.BM) // h]


@pytest.mark.parametrize("plan", [p for p in PLANS if p.pattern == "subtoken"],
                         ids=lambda p: f"{p.M}x{p.N}-{p.sizes}")
def test_subtoken_rows_land_in_their_bucket_pool(plan):
    # Section 3.3 Approach (3): pool b holds exactly the rows bound for b
    idx = oracle.post_index(plan).reshape(plan.M, plan.N)
    subtok = idx // plan.BN
    pool = np.searchsorted(plan.pool_off, subtok, side="right") - 1
    np.testing.assert_array_equal(pool, np.repeat(plan.bucket[:, None], plan.N, axis=1))
    # every subtoken appears once: each pool has (rows of b) * tiles_n subtokens
    for b in range(plan.num_dest):
        assert plan.pool_off[b + 1] - plan.pool_off[b] == (plan.bucket == b).sum() * plan.tiles_n
    # inside a pool, subtokens follow slot order
    for b in range(plan.num_dest):
        assert np.all(np.diff(plan.pool_base[:, b]) >= 0)


def test_tile_reorder_identity_order_layout():
    # Section 3.3 Approach (1): with row-major dispatch the reordered buffer is
    # the column of tiles in tile order
    plan = oracle.make_plan(256, 256, 64, 64, num_cus=256, order="rowmajor",
                            sizes=(4, 4, 4, 4), unit="tiles")
    C = np.arange(256 * 256, dtype=np.int64).reshape(256, 256)
    perm = oracle.reorder_index(plan)
    Cr = C.reshape(-1)[perm].reshape(16, 64, 64)
    for t in range(16):
        tm, tn = divmod(t, 4)
        np.testing.assert_array_equal(Cr[t], C[tm * 64:(tm + 1) * 64, tn * 64:(tn + 1) * 64])


def _dense_perm(perm):
    n = perm.size
    P = np.zeros((n, n), dtype=np.int8)
    P[np.arange(n), perm] = 1
    return P


@pytest.mark.parametrize("pattern,nd", [("tile", 0), ("subtile", 2), ("subtoken", 3)])
def test_bruteforce_2x2_tiles(pattern, nd):
    # M = N = 16 in 8x8 tiles (4 tiles), one tile per wave: every slot order
    # (24) x every partition of the 4 waves (8).
    M = N = 16
    BM = BN = 8
    rng = np.random.default_rng(3)
    C = _bits(M * N, 4)
    peer = _bits(M * N, 5)
    bucket = rng.integers(0, 3, M) if pattern == "subtoken" else None
    sigma = np.array([1, 0]) if pattern == "subtile" else None
    count = 0
    for order in itertools.permutations(range(4)):
        for sizes in oracle.all_partitions(4):
            plan = oracle.make_plan(M, N, BM, BN, num_cus=1, pattern=pattern, num_dest=nd,
                                    sigma=sigma, bucket=bucket, sizes=sizes, exec_order=order)
            perm = oracle.reorder_index(plan)
            Pm = _dense_perm(perm)
            assert np.all(Pm.sum(0) == 1) and np.all(Pm.sum(1) == 1)
            Cr = (Pm.astype(np.int64) @ C.astype(np.int64)).astype(np.uint16)
            np.testing.assert_array_equal(Cr, C[perm])
            assert plan.targets == [s for s in sizes]           # one tile per wave
            if pattern == "subtoken":
                _, _, out = oracle.run_path(plan, C, None, "fp16")
                np.testing.assert_array_equal(out.reshape(-1), C)
            else:
                # peer partial laid out by the same reorder (the peer's own
                # epilogue): the restored output is RNE(C + P) element-wise
                peer_r = peer[perm]
                _, _, out = oracle.run_path(plan, C, peer_r, "fp16")
                np.testing.assert_array_equal(out.reshape(-1), oracle.add_rne(C, peer, "fp16"))
            count += 1
    assert count == 24 * 8
