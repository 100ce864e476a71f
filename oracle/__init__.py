"""CPU oracle for the signaled + reordered GEMM path -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The GPU path (the HIP library and its
Python binding) never imports it, and this package imports nothing from the
GPU path: the two share no kernels, tables, helpers or constants. Inputs come
from ``workloads`` (random draws only).

What it computes, each part citing the passage it follows:

* GEMM  C = A x B  (Section 2.1.1), fp64 sums of exact products, one
  round-to-nearest-even to the storage dtype (C library ``fo_oracle.c``).
* Tile dispatch order, waves and wave groups (Sections 2.1.1-2.1.2, 3.2,
  3.4): position p of the dispatch order runs in wave p // W, and a wave
  group is a run of consecutive waves.
* Group-wise tile counting (Section 3.2, Approach): group j is signalled when
  its counter reaches the number of tiles in G_j.
* Execution-order-aware reordering (Section 3.3, Approach): an explicit
  permutation from the row-major output C to the reordered buffer for the
  tile (AllReduce), subtile (ReduceScatter) and subtoken (All-to-All)
  patterns, the contiguous (offset, length) segment each group hands to the
  communication, and the post-communication gather back to row-major order.
* Predictive search over wave-group partitions (Section 4.1, Algorithm 1), and
  the reuse of searched partitions by nearest size (Section 4.2).

Readings of points the paper leaves open are listed in the module-level
constants' comments and in the function docstrings; they match the readings
the GPU path documents in its public header.
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
from typing import Callable, List, Optional, Sequence, Tuple

import numpy as np

FP16, BF16 = "fp16", "bf16"
_DT = {FP16: 0, BF16: 1}
TILE, SUBTILE, SUBTOKEN, ROWMAJOR = "tile", "subtile", "subtoken", "rowmajor"

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libfo_oracle.so")
_lib = None


def lib():
    """Load the C part of the oracle (built by ``oracle/build.py``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        L = ctypes.CDLL(_LIB_PATH)
        u16p = np.ctypeslib.ndpointer(np.uint16, flags="C_CONTIGUOUS")
        f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
        i64p = np.ctypeslib.ndpointer(np.int64, flags="C_CONTIGUOUS")
        i64, c_int, c_double = ctypes.c_int64, ctypes.c_int, ctypes.c_double
        L.fo_orc_half_to_f64.argtypes = [ctypes.c_uint16]
        L.fo_orc_half_to_f64.restype = c_double
        L.fo_orc_bf16_to_f64.argtypes = [ctypes.c_uint16]
        L.fo_orc_bf16_to_f64.restype = c_double
        L.fo_orc_f64_to_half.argtypes = [c_double]
        L.fo_orc_f64_to_half.restype = ctypes.c_uint16
        L.fo_orc_f64_to_bf16.argtypes = [c_double]
        L.fo_orc_f64_to_bf16.restype = ctypes.c_uint16
        L.fo_orc_decode.argtypes = [u16p, i64, c_int, f64p]
        L.fo_orc_encode.argtypes = [f64p, i64, c_int, u16p]
        L.fo_orc_gemm_rows.argtypes = [u16p, u16p, c_int, i64, i64p, i64, i64, i64, f64p, i64]
        L.fo_orc_gemm_f64.argtypes = [f64p, f64p, i64, i64, i64, i64p, i64, i64, i64, f64p, i64]
        L.fo_orc_add.argtypes = [u16p, u16p, i64, c_int, u16p]
        L.fo_orc_rmsnorm.argtypes = [u16p, i64, i64, ctypes.c_void_p, ctypes.c_void_p,
                                     c_double, c_int, c_int, u16p]
        L.fo_orc_num_threads.restype = c_int
        _lib = L
    return _lib


def num_threads() -> int:
    return int(lib().fo_orc_num_threads())


# --------------------------------------------------------------------------
# Storage formats
# --------------------------------------------------------------------------

def decode(bits: np.ndarray, dtype: str) -> np.ndarray:
    """fp16/bf16 bits -> exact float64 values."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).reshape(-1)
    out = np.empty(b.size, dtype=np.float64)
    lib().fo_orc_decode(b, b.size, _DT[dtype], out)
    return out.reshape(np.shape(bits))


def encode(x: np.ndarray, dtype: str) -> np.ndarray:
    """float64 -> fp16/bf16 bits, round to nearest, ties to even."""
    v = np.ascontiguousarray(x, dtype=np.float64).reshape(-1)
    out = np.empty(v.size, dtype=np.uint16)
    lib().fo_orc_encode(v, v.size, _DT[dtype], out)
    return out.reshape(np.shape(x))


# --------------------------------------------------------------------------
# GEMM (Section 2.1.1): C = A x B, B given as W = B^T [N, K]
# --------------------------------------------------------------------------

def gemm_exact(A: np.ndarray, W: np.ndarray, dtype: str,
               rows: Optional[np.ndarray] = None,
               cols: Optional[Tuple[int, int]] = None) -> np.ndarray:
    """fp64 product of the stored operands (exact products, k-order sums).

    ``rows``/``cols`` select a sub-block (for sampled checks of large
    shapes); the result has shape [len(rows), n1 - n0].
    """
    M, K = A.shape
    N = W.shape[0]
    assert W.shape[1] == K
    rows = np.arange(M, dtype=np.int64) if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    n0, n1 = (0, N) if cols is None else cols
    C = np.empty((rows.size, n1 - n0), dtype=np.float64)
    if rows.size == 0 or n1 == n0:
        return C
    Af = decode(A, dtype)
    Wf = decode(W, dtype)
    lib().fo_orc_gemm_f64(np.ascontiguousarray(Af), np.ascontiguousarray(Wf), M, N, K,
                          rows, rows.size, n0, n1, C, n1 - n0)
    return C


def gemm_exact_bits_path(A: np.ndarray, W: np.ndarray, dtype: str) -> np.ndarray:
    """Same product, decoding every operand inside the loop (slow, tiny sizes)."""
    M, K = A.shape
    N = W.shape[0]
    rows = np.arange(M, dtype=np.int64)
    C = np.empty((M, N), dtype=np.float64)
    lib().fo_orc_gemm_rows(np.ascontiguousarray(A), np.ascontiguousarray(W), _DT[dtype], K,
                           rows, M, 0, N, C, N)
    return C


def gemm_ref(A: np.ndarray, W: np.ndarray, dtype: str) -> np.ndarray:
    """Reference GEMM output: the exact product rounded once (bits, [M, N])."""
    return encode(gemm_exact(A, W, dtype), dtype)


# --------------------------------------------------------------------------
# Consumer stand-in and RMSNorm
# --------------------------------------------------------------------------

def add_rne(a: np.ndarray, b: np.ndarray, dtype: str) -> np.ndarray:
    """Correctly rounded sum of two partials (the AllReduce of two ranks)."""
    x = np.ascontiguousarray(a, dtype=np.uint16).reshape(-1)
    y = np.ascontiguousarray(b, dtype=np.uint16).reshape(-1)
    assert x.size == y.size
    out = np.empty_like(x)
    lib().fo_orc_add(x, y, x.size, _DT[dtype], out)
    return out.reshape(np.shape(a))


def rmsnorm(x: np.ndarray, dtype: str, bias: Optional[np.ndarray] = None,
            gamma: Optional[np.ndarray] = None, eps: float = 1e-6,
            do_norm: bool = True) -> np.ndarray:
    """Row-wise y = (x + bias) / sqrt(mean((x + bias)^2) + eps) * gamma."""
    x = np.ascontiguousarray(x, dtype=np.uint16)
    rows, n = x.shape
    out = np.empty_like(x)
    bp = None if bias is None else np.ascontiguousarray(bias, dtype=np.uint16)
    gp = None if gamma is None else np.ascontiguousarray(gamma, dtype=np.uint16)
    lib().fo_orc_rmsnorm(x, rows, n,
                         None if bp is None else bp.ctypes.data,
                         None if gp is None else gp.ctypes.data,
                         float(eps), int(do_norm), _DT[dtype], out)
    return out


# --------------------------------------------------------------------------
# Dispatch order of tiles (Section 2.1.2, block swizzling)
# --------------------------------------------------------------------------

def dispatch_order(tiles_m: int, tiles_n: int, order: str,
                   group_m: int = 4, num_xcds: int = 8) -> List[int]:
    """Tile index (row-major over the tile grid) run at each dispatch position.

    ``rowmajor``: position p runs tile p.
    ``grouped``: block swizzling over bands of ``group_m`` tile rows; inside a
      band, positions walk down a column of the band before moving to the next
      column (with group_m = 2 on a 3x2 grid the first two positions are tiles
      0 and 2, the Section 3.3 challenge example).
    ``xcd``: positions are first dealt round-robin to ``num_xcds`` chiplets
      (position p runs on chiplet p mod num_xcds); each chiplet's positions
      are given a contiguous share of the grouped order, so tiles that run
      together on one chiplet share rows of A and columns of B.
    """
    tiles = tiles_m * tiles_n
    out = []
    for p in range(tiles):
        if order == "rowmajor":
            out.append(p)
            continue
        q = p
        if order == "xcd":
            per = -(-tiles // num_xcds)          # positions of a full chiplet
            full = tiles % num_xcds or num_xcds  # chiplets that get `per`
            x, local = p % num_xcds, p // num_xcds
            if x < full:
                q = x * per + local
            else:
                q = full * per + (x - full) * (per - 1) + local
        elif order != "grouped":
            raise ValueError(order)
        band_tiles = group_m * tiles_n
        band = q // band_tiles
        first_m = band * group_m
        rows_in_band = min(tiles_m - first_m, group_m)
        r = q % band_tiles
        tm = first_m + r % rows_in_band
        tn = r // rows_in_band
        out.append(tm * tiles_n + tn)
    return out


# --------------------------------------------------------------------------
# Waves and wave groups (Sections 2.1.1, 3.2, 3.4; Algorithm 1 wave count)
# --------------------------------------------------------------------------

def wave_width(num_cus: int, wg_per_cu: int = 1, reserved_cus: int = 0) -> int:
    """Tiles that run concurrently: the compute units left to the GEMM times
    the workgroups each holds (Algorithm 1 divides the tile count by the SMs
    not taken by communication)."""
    return (num_cus - reserved_cus) * wg_per_cu


def num_waves(tiles: int, W: int) -> int:
    """T = number of waves; a partial last wave counts as a wave."""
    return -(-tiles // W) if tiles else 0


def group_first_slots(sizes: Sequence[int], unit: str, W: int, tiles: int) -> List[int]:
    """First slot of every group plus the end: group j owns slots
    [first[j], first[j+1]). Sizes are in waves (a group is a run of whole
    waves, Section 3.2 Insight) or in tiles (tile-wise signalling)."""
    first = [0]
    acc = 0
    for s in sizes:
        acc += s
        first.append(min(acc * W, tiles) if unit == "waves" else acc)
    return first


def cuts_to_partition(cuts: Sequence[int]) -> Tuple[int, ...]:
    """Section 3.4: a binary decision after each of the first T-1 waves
    (1 = communicate the accumulated waves); the last wave always closes a
    group. ``cuts`` has T-1 entries."""
    sizes, run = [], 0
    for c in list(cuts) + [1]:
        run += 1
        if c:
            sizes.append(run)
            run = 0
    return tuple(sizes)


def partition_to_cuts(sizes: Sequence[int]) -> Tuple[int, ...]:
    T = sum(sizes)
    ends = set()
    acc = 0
    for s in sizes:
        acc += s
        ends.add(acc)
    return tuple(1 if w in ends else 0 for w in range(1, T))


def all_partitions(T: int) -> List[Tuple[int, ...]]:
    """The whole design space, 2^(T-1) partitions, in cut-vector order:
    candidate x has a cut after wave i+1 when bit i of x is set."""
    if T <= 0:
        return []
    out = []
    for x in range(1 << (T - 1)):
        out.append(cuts_to_partition([(x >> i) & 1 for i in range(T - 1)]))
    return out


def candidates(T: int, s_first: int, s_last: int) -> List[Tuple[int, ...]]:
    """Algorithm 1 candidate generation with the Section 4.1 pruning |G_1| <= S_1 and
    |G_P| <= S_P."""
    return [g for g in all_partitions(T) if g[0] <= s_first and g[-1] <= s_last]


def interp_latency(curve_bytes: Sequence[float], curve_us: Sequence[float], nbytes: float) -> float:
    """Communication latency for ``nbytes`` from the sampled curve
    (Section 4.2 offline stage: dense samples, interpolated). Reading:
    piecewise linear between samples; outside the sampled range the latency
    scales with size at the nearest end point's bandwidth; zero bytes cost
    nothing."""
    if nbytes <= 0:
        return 0.0
    xs, ys = list(curve_bytes), list(curve_us)
    if nbytes <= xs[0]:
        return ys[0] * nbytes / xs[0]
    if nbytes >= xs[-1]:
        return ys[-1] * nbytes / xs[-1]
    for i in range(1, len(xs)):
        if nbytes <= xs[i]:
            x0, x1, y0, y1 = xs[i - 1], xs[i], ys[i - 1], ys[i]
            return y0 + (y1 - y0) * (nbytes - x0) / (x1 - x0)
    raise AssertionError


def predicted_latency(sizes: Sequence[int], T: int, gemm_us: float,
                      comm_us_of_group: Callable[[int], float]) -> float:
    """Algorithm 1 latency prediction for one candidate.

    For each group G_i in order: the communication of the previous group
    starts when both the computation so far and the previous communication
    are done (t_m^acc = max(t_p^acc, t_m^acc) + t_m), then the group's own
    computation time gemm/T*|G_i| is added to t_p^acc. After the last group
    its communication is added the same way. The first group has no previous
    group; its t_m is 0 (reading). ``comm_us_of_group(j)`` gives the
    interpolated latency of group j (0-based).
    """
    acc_p = acc_m = 0.0
    for i, g in enumerate(sizes):
        t_m = comm_us_of_group(i - 1) if i > 0 else 0.0
        t_p = gemm_us / T * g
        acc_m = max(acc_p, acc_m) + t_m
        acc_p = acc_p + t_p
    return max(acc_p, acc_m) + comm_us_of_group(len(sizes) - 1)


def predictive_search(T: int, gemm_us: float, comm_us_for_partition,
                      s_first: int = 2, s_last: int = 4,
                      cands: Optional[List[Tuple[int, ...]]] = None):
    """Algorithm 1: keep the candidate with the strictly smallest predicted
    latency (the earliest candidate wins ties). ``comm_us_for_partition(sizes)``
    returns a function j -> latency of group j for that partition."""
    best, best_t = None, math.inf
    for g in (candidates(T, s_first, s_last) if cands is None else cands):
        t = predicted_latency(g, T, gemm_us, comm_us_for_partition(g))
        if t < best_t:
            best, best_t = g, t
    return best, best_t


# --------------------------------------------------------------------------
# The plan: map, groups, counters, segments (Sections 3.2 and 3.3)
# --------------------------------------------------------------------------

@dataclasses.dataclass
class Plan:
    M: int
    N: int
    BM: int
    BN: int
    tiles_m: int
    tiles_n: int
    W: int
    T: int
    pattern: str
    num_dest: int
    order: List[int]              # dispatch position -> tile
    tile_to_slot: np.ndarray      # tile -> slot
    first: List[int]              # group j owns slots [first[j], first[j+1])
    targets: List[int]            # tiles per group = final counter value
    slot_group: np.ndarray        # slot -> group
    sizes: Tuple[int, ...]
    unit: str
    sigma: Optional[np.ndarray] = None
    bucket: Optional[np.ndarray] = None
    # subtoken (All-to-All) pool bookkeeping
    rows_of: Optional[dict] = None        # (tm, b) -> ascending row list
    pool_base: Optional[np.ndarray] = None  # [tiles + 1, B]: subtokens of pool b before slot s
    pool_off: Optional[np.ndarray] = None   # [B + 1]: first subtoken of pool b

    @property
    def tiles(self) -> int:
        return self.tiles_m * self.tiles_n

    @property
    def P(self) -> int:
        return len(self.targets)


def make_plan(M: int, N: int, BM: int, BN: int, *, num_cus: int, wg_per_cu: int = 1,
              reserved_cus: int = 0, order: str = "rowmajor", group_m: int = 4,
              num_xcds: int = 8, pattern: str = TILE, num_dest: int = 0,
              sigma=None, bucket=None, sizes: Sequence[int] = (), unit: str = "waves",
              exec_order: Optional[Sequence[int]] = None) -> Plan:
    """Plan of a GEMM of [M, N] outputs in BM x BN tiles. ``sizes`` is the
    wave-group partition (in waves, or in tiles when unit == "tiles").
    ``exec_order`` (position -> tile) overrides the dispatch-order formula."""
    assert M % BM == 0 and N % BN == 0
    tiles_m, tiles_n = M // BM, N // BN
    tiles = tiles_m * tiles_n
    W = wave_width(num_cus, wg_per_cu, reserved_cus)
    T = num_waves(tiles, W)
    ordr = (list(exec_order) if exec_order is not None
            else dispatch_order(tiles_m, tiles_n, order, group_m, num_xcds))
    assert sorted(ordr) == list(range(tiles))
    # slot = dispatch position: earlier waves first, a wave's tiles together
    # (Section 3.3 Approach (1); order inside a wave is fixed to the
    # dispatch order, one of the orders the paper allows).
    t2s = np.empty(tiles, dtype=np.int64)
    for p, t in enumerate(ordr):
        t2s[t] = p
    total = T if unit == "waves" else tiles
    assert all(s >= 1 for s in sizes) and sum(sizes) == total, (sizes, total)
    first = group_first_slots(sizes, unit, W, tiles)
    targets = [first[j + 1] - first[j] for j in range(len(sizes))]
    slot_group = np.empty(tiles, dtype=np.int64)
    for j in range(len(sizes)):
        slot_group[first[j]:first[j + 1]] = j
    plan = Plan(M=M, N=N, BM=BM, BN=BN, tiles_m=tiles_m, tiles_n=tiles_n, W=W, T=T,
                pattern=pattern, num_dest=num_dest, order=ordr, tile_to_slot=t2s,
                first=first, targets=targets, slot_group=slot_group,
                sizes=tuple(sizes), unit=unit)
    if pattern == SUBTILE:
        assert BM % num_dest == 0
        plan.sigma = np.asarray(sigma if sigma is not None else np.arange(num_dest), dtype=np.int64)
    if pattern == SUBTOKEN:
        B = num_dest
        bucket = np.asarray(bucket, dtype=np.int64)
        plan.bucket = bucket
        rows_of = {}
        for tm in range(tiles_m):
            for b in range(B):
                rows_of[(tm, b)] = [i for i in range(tm * BM, (tm + 1) * BM) if bucket[i] == b]
        plan.rows_of = rows_of
        base = np.zeros((tiles + 1, B), dtype=np.int64)
        for s in range(tiles):
            tm = ordr[s] // tiles_n
            for b in range(B):
                base[s + 1, b] = base[s, b] + len(rows_of[(tm, b)])
        plan.pool_base = base
        off = np.zeros(B + 1, dtype=np.int64)
        for b in range(B):
            off[b + 1] = off[b] + base[tiles, b]
        plan.pool_off = off
    return plan


def slot_range_bytes(plan: Plan, f0: int, f1: int, elem_bytes: int = 2, all_dest: bool = False) -> int:
    """Data a group owning slots [f0, f1) hands to the communication
    (Algorithm 1, get_data_size). For the All-to-All pattern the largest
    per-destination piece stands in for the slowest destination (Section 4.2:
    the maximum across GPUs is taken for the imbalanced All-to-All); with
    ``all_dest`` every piece counts (one device moving all of them, which is
    what a one-GPU stand-in of the exchange does)."""
    if plan.pattern == SUBTOKEN and not all_dest:
        return int(max(plan.pool_base[f1, b] - plan.pool_base[f0, b]
                       for b in range(plan.num_dest))) * plan.BN * elem_bytes
    return (f1 - f0) * plan.BM * plan.BN * elem_bytes


def search_partition(plan: Plan, gemm_us: float, curve_bytes, curve_us,
                     s_first: int = 2, s_last: int = 4, elem_bytes: int = 2, all_dest: bool = False,
                     last_curve=None):
    """Algorithm 1 on a plan's geometry (its waves, tiles and pools; its own
    partition is ignored). Returns (partition in waves, predicted us).
    ``last_curve`` = (bytes, us): the latency curve of the last group's
    communication, which runs once the GEMM is over; None: the one curve for
    every group. (The paper has one curve; a second one for the last group
    is this implementation's reading for a one-GPU stand-in of the
    communication, which shares the device with the GEMM until then.)"""
    T = plan.T

    def comm_for(sizes):
        first = group_first_slots(sizes, "waves", plan.W, plan.tiles)
        lat = []
        for j in range(len(sizes)):
            xs, ys = (curve_bytes, curve_us) if last_curve is None or j < len(sizes) - 1 else last_curve
            lat.append(interp_latency(xs, ys, slot_range_bytes(plan, first[j], first[j + 1], elem_bytes, all_dest)))
        return lambda j: lat[j]

    return predictive_search(T, gemm_us, comm_for, s_first, s_last)


# --------------------------------------------------------------------------
# Partitions reused across sizes (Section 4.2, online stage)
# --------------------------------------------------------------------------

def nearest_size(cached_ms: Sequence[int], M: int) -> int:
    """Section 4.2: for dynamic shapes the search runs ahead of time on
    representative GEMM sizes and an unseen size takes the partition of its
    nearest neighbour. Reading: neighbours are sizes of the same problem
    family (every parameter but M equal), the distance is |M - M_ref|, and a
    tie goes to the smaller M_ref."""
    best = None
    for m in cached_ms:
        if best is None or abs(M - m) < abs(M - best) or (abs(M - m) == abs(M - best) and m < best):
            best = m
    if best is None:
        raise KeyError("no cached size")
    return best


def rescale_partition(sizes_ref: Sequence[int], T: int) -> Tuple[int, ...]:
    """The nearest neighbour's partition applied to a problem of T waves.
    Reading (the paper reuses the partition without saying how a different
    wave count is handled): group boundaries keep their relative position. A
    boundary after wave b of the T_ref cached waves moves to after wave
    b * T / T_ref, rounded to the nearest integer with halves rounded up;
    boundaries that land on wave 0, on wave T or not after the previous kept
    boundary are dropped."""
    from fractions import Fraction
    T_ref = sum(sizes_ref)
    if T <= 0:
        return ()
    kept = []
    b = 0
    for s in list(sizes_ref)[:-1]:
        b += s
        nb = math.floor(Fraction(b * T, T_ref) + Fraction(1, 2))
        if 0 < nb < T and (not kept or nb > kept[-1]):
            kept.append(nb)
    edges = [0] + kept + [T]
    return tuple(edges[i + 1] - edges[i] for i in range(len(edges) - 1))


# --------------------------------------------------------------------------
# Explicit permutations (Section 3.3 Approach (1)-(3))
# --------------------------------------------------------------------------

def _tile_rc(plan: Plan, t: int):
    return divmod(t, plan.tiles_n)


def reorder_index(plan: Plan) -> np.ndarray:
    """perm with Cr.flat = C.flat[perm], where Cr is the buffer the GEMM
    epilogue writes (the reordered output, or the per-destination pools).

    tile:     the reordered output is a column of tiles, tile of slot s at
              rows [s*BM, (s+1)*BM) of a [tiles*BM, BN] row-major buffer.
    subtile:  each tile is cut into R slices of h = BM/R rows; in group j
              (slots first_j.., n_j tiles, starting at element E_j) slice k of
              slot s sits at E_j + k*n_j*h*BN + (s - first_j)*h*BN, so the k-th
              slices of a group are contiguous.
    subtoken: a subtoken is one tile row (BN elements). Pool b holds the rows
              whose destination is b, ordered by slot, then by row.
    rowmajor: identity.
    """
    M, N, BM, BN = plan.M, plan.N, plan.BM, plan.BN
    perm = np.empty(M * N, dtype=np.int64)
    r_idx = np.arange(BM, dtype=np.int64)[:, None]
    c_idx = np.arange(BN, dtype=np.int64)[None, :]
    if plan.pattern == ROWMAJOR:
        return np.arange(M * N, dtype=np.int64)
    for s in range(plan.tiles):
        t = plan.order[s]
        tm, tn = _tile_rc(plan, t)
        src = (tm * BM + r_idx) * N + tn * BN + c_idx          # [BM, BN]
        if plan.pattern == TILE:
            perm[s * BM * BN:(s + 1) * BM * BN] = src.reshape(-1)
        elif plan.pattern == SUBTILE:
            R = plan.num_dest
            h = BM // R
            j = int(plan.slot_group[s])
            n_j = plan.targets[j]
            E_j = plan.first[j] * BM * BN
            for k in range(R):
                o = E_j + k * n_j * h * BN + (s - plan.first[j]) * h * BN
                perm[o:o + h * BN] = src[k * h:(k + 1) * h].reshape(-1)
        elif plan.pattern == SUBTOKEN:
            for b in range(plan.num_dest):
                rows = plan.rows_of[(tm, b)]
                for rank, i in enumerate(rows):
                    o = (plan.pool_off[b] + plan.pool_base[s, b] + rank) * BN
                    perm[o:o + BN] = i * N + tn * BN + np.arange(BN)
        else:
            raise ValueError(plan.pattern)
    return perm


def dest_buffer_elems(plan: Plan) -> int:
    """Elements in the consumer's destination (all destinations together)."""
    if plan.pattern == SUBTILE:
        h = plan.BM // plan.num_dest
        return plan.num_dest * plan.tiles * h * plan.BN
    return plan.M * plan.N


def segments(plan: Plan) -> List[Tuple[int, int, int, int, int]]:
    """Contiguous pieces handed to the communication, in launch order.

    Each entry is (group j, destination d, source offset, destination
    offset, length), in elements. tile: one piece per group, the group's
    slots. subtile: one piece per (group, slice k); slice k of every tile goes
    to destination buffer sigma(k), whose layout is a column of h-row
    subtiles in slot order (destination buffers are laid end to end).
    subtoken: one piece per (group, pool b); the receive buffer mirrors the
    pools. rowmajor (plain GEMM): one piece, the whole output."""
    BM, BN = plan.BM, plan.BN
    out = []
    if plan.pattern == ROWMAJOR:
        # plain GEMM output: nothing is contiguous per group, so the whole
        # buffer is one piece, ready only when the last group is
        return [(plan.P - 1, 0, 0, 0, plan.M * plan.N)] if plan.P else []
    for j in range(plan.P):
        f0, f1 = plan.first[j], plan.first[j + 1]
        if plan.pattern == TILE:
            out.append((j, 0, f0 * BM * BN, f0 * BM * BN, (f1 - f0) * BM * BN))
        elif plan.pattern == SUBTILE:
            R = plan.num_dest
            h = BM // R
            slot_elems = plan.tiles * h * BN
            n_j = f1 - f0
            for k in range(R):
                src = f0 * BM * BN + k * n_j * h * BN
                dst = int(plan.sigma[k]) * slot_elems + f0 * h * BN
                out.append((j, k, src, dst, n_j * h * BN))
        elif plan.pattern == SUBTOKEN:
            for b in range(plan.num_dest):
                o = (plan.pool_off[b] + plan.pool_base[f0, b]) * BN
                l = (plan.pool_base[f1, b] - plan.pool_base[f0, b]) * BN
                out.append((j, b, int(o), int(o), int(l)))
    return out


def post_index(plan: Plan) -> np.ndarray:
    """gather with out.flat = dst.flat[idx]: the post-communication reorder
    (Section 3.3: the element-wise kernel after communication loads by the
    reordered index). Built directly from the destination layouts, not by
    inverting ``reorder_index``."""
    M, N, BM, BN = plan.M, plan.N, plan.BM, plan.BN
    idx = np.empty(M * N, dtype=np.int64)
    c_idx = np.arange(BN, dtype=np.int64)
    for tm in range(plan.tiles_m):
        for tn in range(plan.tiles_n):
            s = int(plan.tile_to_slot[tm * plan.tiles_n + tn])
            for r in range(BM):
                i = tm * BM + r
                o_out = i * N + tn * BN
                if plan.pattern == ROWMAJOR:
                    src = o_out
                elif plan.pattern == TILE:
                    src = (s * BM + r) * BN
                elif plan.pattern == SUBTILE:
                    h = BM // plan.num_dest
                    k, rr = divmod(r, h)
                    src = int(plan.sigma[k]) * plan.tiles * h * BN + (s * h + rr) * BN
                else:
                    b = int(plan.bucket[i])
                    rank = plan.rows_of[(tm, b)].index(i)
                    src = (plan.pool_off[b] + plan.pool_base[s, b] + rank) * BN
                idx[o_out:o_out + BN] = src + c_idx
    return idx


def apply_consumer(plan: Plan, Cr: np.ndarray, peer: Optional[np.ndarray], dtype: str) -> np.ndarray:
    """Run every segment of the communication stand-in: the sum with the
    peer's partial (AllReduce / ReduceScatter) or a copy (All-to-All)."""
    dst = np.zeros(dest_buffer_elems(plan), dtype=np.uint16)
    for (_, _, so, do, ln) in segments(plan):
        if ln == 0:
            continue
        if peer is None:
            dst[do:do + ln] = Cr[so:so + ln]
        else:
            dst[do:do + ln] = add_rne(Cr[so:so + ln], peer[so:so + ln], dtype)
    return dst


def run_path(plan: Plan, C_bits: np.ndarray, peer: Optional[np.ndarray], dtype: str,
             bias=None, gamma=None, eps: float = 1e-6, do_norm: bool = False):
    """The whole path on the CPU for a given GEMM output (row-major bits):
    pre-communication reorder, consumer, post-communication reorder, then the
    optional bias + RMSNorm. Returns (reordered, dst, out)."""
    Cr = C_bits.reshape(-1)[reorder_index(plan)]
    dst = apply_consumer(plan, Cr, peer, dtype)
    x = dst[post_index(plan)].reshape(plan.M, plan.N)
    if do_norm or bias is not None:
        x = rmsnorm(x, dtype, bias=bias, gamma=gamma, eps=eps, do_norm=do_norm)
    return Cr, dst, x
