"""Python binding of libfo, the MI355X (gfx950) signaled + reordered GEMM path.

Argument marshalling only: every step of the path runs in the HIP kernels of
``libfo.so`` (see ``include/fo.h`` for the contract of each call). Device
buffers are passed as raw device pointers (ints) or as objects with a
``data_ptr()`` method (e.g. torch tensors on a ROCm device); streams as raw
hipStream_t handles or objects with a ``cuda_stream`` attribute.

The library must be built (``python -m paper_2504_19519_amd.build``); there is
no fallback path: importing the binding without the library raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

__all__ = [
    "FoError", "Plan", "PlanCache", "plan_groups", "gemm_signal_reorder", "consume_group",
    "post_reorder", "reset_counters", "run_overlapped", "run_overlapped_noalloc", "set_poll_timeout_us",
    "get_poll_timeout_us", "device_num_cus", "set_sync_mode", "get_sync_mode",
    "set_consumer_grid", "get_consumer_grid", "Options", "options", "device_wall_clock_khz", "LIB_PATH",
    "FP16", "BF16", "TILE", "SUBTILE", "SUBTOKEN", "ROWMAJOR",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfo.so")

FP16, BF16 = 0, 1
TILE, SUBTILE, SUBTOKEN, ROWMAJOR = 0, 1, 2, 3
ORDER_ROWMAJOR, ORDER_GROUPED, ORDER_XCD = 0, 1, 2
UNIT_WAVES, UNIT_TILES = 0, 1
DISPENSER_WORDS = 8     # tile-position counters after the P group counters (FO_DISPENSER_WORDS)

_DTYPES = {"fp16": FP16, "bf16": BF16, FP16: FP16, BF16: BF16}
_PATTERNS = {"tile": TILE, "subtile": SUBTILE, "subtoken": SUBTOKEN, "rowmajor": ROWMAJOR,
             TILE: TILE, SUBTILE: SUBTILE, SUBTOKEN: SUBTOKEN, ROWMAJOR: ROWMAJOR}
_ORDERS = {"rowmajor": ORDER_ROWMAJOR, "grouped": ORDER_GROUPED, "xcd": ORDER_XCD,
           ORDER_ROWMAJOR: ORDER_ROWMAJOR, ORDER_GROUPED: ORDER_GROUPED, ORDER_XCD: ORDER_XCD}
_UNITS = {"waves": UNIT_WAVES, "tiles": UNIT_TILES, UNIT_WAVES: UNIT_WAVES, UNIT_TILES: UNIT_TILES}


class FoError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"libfo status {status}: {message}")
        self.status = status


class _Problem(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int64), ("N", ctypes.c_int64), ("K", ctypes.c_int64),
                ("dtype", ctypes.c_int32), ("tile_m", ctypes.c_int32), ("tile_n", ctypes.c_int32),
                ("order", ctypes.c_int32), ("group_m", ctypes.c_int32), ("num_xcds", ctypes.c_int32),
                ("num_cus", ctypes.c_int32), ("wg_per_cu", ctypes.c_int32),
                ("reserved_cus", ctypes.c_int32), ("pattern", ctypes.c_int32),
                ("num_dest", ctypes.c_int32),
                ("dest_perm", ctypes.POINTER(ctypes.c_int32)),
                ("row_bucket", ctypes.POINTER(ctypes.c_int32))]


class _Grouping(ctypes.Structure):
    _fields_ = [("unit", ctypes.c_int32), ("num_groups", ctypes.c_int32),
                ("sizes", ctypes.POINTER(ctypes.c_int32)), ("gemm_us", ctypes.c_double),
                ("curve_bytes", ctypes.POINTER(ctypes.c_double)),
                ("curve_us", ctypes.POINTER(ctypes.c_double)), ("curve_len", ctypes.c_int32),
                ("s_first", ctypes.c_int32), ("s_last", ctypes.c_int32),
                ("all_dest_bytes", ctypes.c_int32),
                ("last_curve_bytes", ctypes.POINTER(ctypes.c_double)),
                ("last_curve_us", ctypes.POINTER(ctypes.c_double)), ("last_curve_len", ctypes.c_int32)]


class _Options(ctypes.Structure):
    _fields_ = [("sync_producer", ctypes.c_int32), ("sync_consumer", ctypes.c_int32),
                ("consumer_blocks", ctypes.c_int32), ("consumer_threads", ctypes.c_int32),
                ("poll_timeout_us", ctypes.c_int64), ("consumer_limit", ctypes.c_int32),
                ("reserved0", ctypes.c_int32), ("tile_trace", ctypes.c_void_p),
                ("tile_trace_capacity", ctypes.c_int64)]


Options = _Options

_lib = None


def lib() -> ctypes.CDLL:
    """Load libfo.so. Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          f"`python -m paper_2504_19519_amd.build` (no fallback path exists)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32
    pi32 = ctypes.POINTER(ctypes.c_int32)
    pi64 = ctypes.POINTER(ctypes.c_int64)
    L.fo_plan_groups.argtypes = [ctypes.POINTER(_Problem), ctypes.POINTER(_Grouping), ctypes.POINTER(vp)]
    L.fo_plan_destroy.argtypes = [vp]
    L.fo_plan_cache_create.argtypes = [ctypes.POINTER(vp)]
    L.fo_plan_cache_destroy.argtypes = [vp]
    L.fo_plan_cache_add.argtypes = [vp, ctypes.POINTER(_Problem), ctypes.POINTER(_Grouping)]
    L.fo_plan_cache_lookup.argtypes = [vp, ctypes.POINTER(_Problem), ctypes.POINTER(vp), pi64]
    L.fo_plan_cache_size.argtypes, L.fo_plan_cache_size.restype = [vp], i32
    L.fo_plan_cache_entry.argtypes = [vp, i32, pi64, pi32, ctypes.POINTER(pi32)]
    for name in ("num_tiles", "wave_width", "num_waves", "num_groups", "num_counters", "num_segments"):
        f = getattr(L, f"fo_plan_{name}")
        f.argtypes, f.restype = [vp], i32
    for name in ("group_sizes", "order", "tile_to_slot", "group_first", "group_targets",
                 "pool_base", "pool_off"):
        f = getattr(L, f"fo_plan_{name}")
        f.argtypes, f.restype = [vp], pi32
    L.fo_plan_segments.argtypes, L.fo_plan_segments.restype = [vp], pi64
    L.fo_plan_dest_elems.argtypes, L.fo_plan_dest_elems.restype = [vp], i64
    L.fo_plan_predicted_us.argtypes, L.fo_plan_predicted_us.restype = [vp], ctypes.c_double
    L.fo_plan_device_bytes.argtypes, L.fo_plan_device_bytes.restype = [vp], ctypes.c_size_t
    L.fo_plan_to_device.argtypes = [vp, vp, ctypes.c_size_t, vp]
    po = ctypes.POINTER(_Options)
    L.fo_options_init.argtypes, L.fo_options_init.restype = [po], ctypes.c_int
    L.fo_gemm_signal_reorder.argtypes = [vp, vp, vp, vp, vp, vp, vp, po]
    L.fo_consume_group.argtypes = [vp, vp, vp, i64, i32, vp, u32, vp, vp, po]
    L.fo_post_reorder.argtypes = [vp, vp, vp, vp, vp, vp, ctypes.c_float, i32, vp]
    L.fo_reset_counters.argtypes = [vp, i32, vp]
    L.fo_run_overlapped.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_float, i32,
                                    vp, vp, vp, vp, vp, vp, po]
    L.fo_run_overlapped_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_float, i32,
                                            vp, vp, vp, po]
    L.fo_run_overlapped_noalloc.restype = ctypes.c_int
    L.fo_set_sync_mode.argtypes, L.fo_set_sync_mode.restype = [i32, i32], ctypes.c_int
    L.fo_get_sync_mode.argtypes = [pi32, pi32]
    L.fo_set_consumer_grid.argtypes, L.fo_set_consumer_grid.restype = [i32, i32], ctypes.c_int
    L.fo_device_wall_clock_khz.argtypes, L.fo_device_wall_clock_khz.restype = [pi32], ctypes.c_int
    L.fo_get_consumer_grid.argtypes = [pi32, pi32]
    L.fo_set_poll_timeout_us.argtypes = [i64]
    L.fo_get_poll_timeout_us.restype = i64
    L.fo_device_num_cus.argtypes = [i32, pi32]
    L.fo_status_string.argtypes, L.fo_status_string.restype = [ctypes.c_int], ctypes.c_char_p
    L.fo_last_error.restype = ctypes.c_char_p
    for f in (L.fo_plan_cache_create, L.fo_plan_cache_add, L.fo_plan_cache_lookup, L.fo_plan_cache_entry):
        f.restype = ctypes.c_int
    for f in (L.fo_plan_groups, L.fo_plan_to_device, L.fo_gemm_signal_reorder, L.fo_consume_group,
              L.fo_post_reorder, L.fo_reset_counters, L.fo_run_overlapped, L.fo_device_num_cus):
        f.restype = ctypes.c_int
    _lib = L
    return L


def _check(status: int) -> None:
    if status != 0:
        L = lib()
        msg = L.fo_last_error().decode() or L.fo_status_string(status).decode()
        raise FoError(status, msg)


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, (int, np.integer)):
        return int(x) or None
    if hasattr(x, "data_ptr"):
        return int(x.data_ptr())
    raise TypeError(f"cannot take a device pointer of {type(x)}")


def _need(x, nbytes: int, what: str) -> None:
    """A tensor argument must hold at least `nbytes` (raw pointers are taken
    as given: the C ABI cannot see buffer sizes)."""
    if x is not None and hasattr(x, "numel") and hasattr(x, "element_size"):
        have = int(x.numel()) * int(x.element_size())
        if have < nbytes:
            raise ValueError(f"{what}: {have} bytes, the call needs {nbytes}")


def _stream(s) -> Optional[int]:
    if s is None:
        return None
    if isinstance(s, (int, np.integer)):
        return int(s) or None
    if hasattr(s, "cuda_stream"):
        return int(s.cuda_stream) or None
    raise TypeError(f"cannot take a stream handle of {type(s)}")


def _event(e) -> Optional[int]:
    if e is None:
        return None
    if isinstance(e, (int, np.integer)):
        return int(e) or None
    if hasattr(e, "cuda_event"):
        h = int(e.cuda_event)
        if not h:
            raise ValueError("event not created yet: record it once before passing it")
        return h
    raise TypeError(f"cannot take an event handle of {type(e)}")


def _i32_array(values) -> Optional[ctypes.Array]:
    if values is None:
        return None
    a = np.ascontiguousarray(np.asarray(values, dtype=np.int32))
    return (ctypes.c_int32 * a.size).from_buffer_copy(a.tobytes()) if a.size else (ctypes.c_int32 * 1)()


def _f64_array(values) -> Optional[ctypes.Array]:
    if values is None:
        return None
    a = np.ascontiguousarray(np.asarray(values, dtype=np.float64))
    return (ctypes.c_double * a.size).from_buffer_copy(a.tobytes())


class Plan:
    """Owner of an fo_plan (host memory); arrays are copied out as numpy."""

    def __init__(self, handle: int, M: int, N: int, K: int, dtype: int, tile_m: int, tile_n: int,
                 pattern: int, num_dest: int):
        self._h = ctypes.c_void_p(handle)
        self.M, self.N, self.K, self.dtype = M, N, K, dtype
        self.tile_m, self.tile_n, self.pattern, self.num_dest = tile_m, tile_n, pattern, num_dest

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.fo_plan_destroy(h)
            self._h = None

    @property
    def handle(self) -> ctypes.c_void_p:
        return self._h

    def _arr(self, fn, n, dtype=np.int32):
        if n <= 0:
            return np.zeros(0, dtype=dtype)
        p = fn(self._h)
        return np.ctypeslib.as_array(p, shape=(n,)).copy()

    @property
    def tiles(self) -> int: return lib().fo_plan_num_tiles(self._h)
    @property
    def W(self) -> int: return lib().fo_plan_wave_width(self._h)
    @property
    def T(self) -> int: return lib().fo_plan_num_waves(self._h)
    @property
    def P(self) -> int: return lib().fo_plan_num_groups(self._h)
    @property
    def num_counters(self) -> int:
        """Length of the counters array of a signalling run: P group counters,
        the GEMM's tile-position counters, then the two words an overlapped run
        uses to hand work between its streams."""
        return lib().fo_plan_num_counters(self._h)
    @property
    def sizes(self) -> np.ndarray: return self._arr(lib().fo_plan_group_sizes, self.P)
    @property
    def order(self) -> np.ndarray: return self._arr(lib().fo_plan_order, self.tiles)
    @property
    def tile_to_slot(self) -> np.ndarray: return self._arr(lib().fo_plan_tile_to_slot, self.tiles)
    @property
    def group_first(self) -> np.ndarray: return self._arr(lib().fo_plan_group_first, self.P + 1)
    @property
    def targets(self) -> np.ndarray: return self._arr(lib().fo_plan_group_targets, self.P)
    @property
    def predicted_us(self) -> float: return lib().fo_plan_predicted_us(self._h)
    @property
    def dest_elems(self) -> int: return lib().fo_plan_dest_elems(self._h)
    @property
    def device_bytes(self) -> int: return lib().fo_plan_device_bytes(self._h)

    @property
    def segments(self) -> np.ndarray:
        n = lib().fo_plan_num_segments(self._h)
        return self._arr(lib().fo_plan_segments, 5 * n, np.int64).reshape(n, 5)

    @property
    def pool_base(self) -> Optional[np.ndarray]:
        if self.pattern != SUBTOKEN:
            return None
        return self._arr(lib().fo_plan_pool_base, (self.tiles + 1) * self.num_dest).reshape(
            self.tiles + 1, self.num_dest)

    @property
    def pool_off(self) -> Optional[np.ndarray]:
        if self.pattern != SUBTOKEN:
            return None
        return self._arr(lib().fo_plan_pool_off, self.num_dest + 1)

    def to_device(self, dev_buf, nbytes: Optional[int] = None, stream=None) -> None:
        nb = self.device_bytes if nbytes is None else nbytes
        _check(lib().fo_plan_to_device(self._h, _ptr(dev_buf), nb, _stream(stream)))


def _problem(M: int, N: int, K: int, *, dtype="fp16", tile_m: int = 256, tile_n: int = 128,
             order="xcd", group_m: int = 4, num_xcds: int = 8, num_cus: int = 256,
             wg_per_cu: int = 1, reserved_cus: int = 0, pattern="tile", num_dest: int = 0,
             dest_perm: Optional[Sequence[int]] = None, row_bucket=None):
    """An fo_problem and the arrays it points to (keep them alive with it)."""
    perm = _i32_array(dest_perm)
    buck = _i32_array(row_bucket)
    prob = _Problem(M=M, N=N, K=K, dtype=_DTYPES[dtype], tile_m=tile_m, tile_n=tile_n,
                    order=_ORDERS[order], group_m=group_m, num_xcds=num_xcds, num_cus=num_cus,
                    wg_per_cu=wg_per_cu, reserved_cus=reserved_cus, pattern=_PATTERNS[pattern],
                    num_dest=num_dest,
                    dest_perm=ctypes.cast(perm, ctypes.POINTER(ctypes.c_int32)) if perm is not None else None,
                    row_bucket=ctypes.cast(buck, ctypes.POINTER(ctypes.c_int32)) if buck is not None else None)
    return prob, (perm, buck)


_DEST_BYTES = {"largest": 0, "all": 1}


def _grouping(sizes: Optional[Sequence[int]] = None, unit="waves", gemm_us: float = 0.0,
              curve_bytes=None, curve_us=None, s_first: int = 2, s_last: int = 4, dest_bytes: str = "largest",
              last_curve_bytes=None, last_curve_us=None):
    """An fo_grouping and the arrays it points to."""
    sz = _i32_array(sizes)
    cb, cu = _f64_array(curve_bytes), _f64_array(curve_us)
    lb, lu = _f64_array(last_curve_bytes), _f64_array(last_curve_us)
    grp = _Grouping(unit=_UNITS[unit], num_groups=0 if sizes is None else len(sizes),
                    sizes=ctypes.cast(sz, ctypes.POINTER(ctypes.c_int32)) if sz is not None else None,
                    gemm_us=gemm_us,
                    curve_bytes=ctypes.cast(cb, ctypes.POINTER(ctypes.c_double)) if cb is not None else None,
                    curve_us=ctypes.cast(cu, ctypes.POINTER(ctypes.c_double)) if cu is not None else None,
                    curve_len=0 if curve_bytes is None else len(curve_bytes),
                    s_first=s_first, s_last=s_last, all_dest_bytes=_DEST_BYTES[dest_bytes],
                    last_curve_bytes=ctypes.cast(lb, ctypes.POINTER(ctypes.c_double)) if lb is not None else None,
                    last_curve_us=ctypes.cast(lu, ctypes.POINTER(ctypes.c_double)) if lu is not None else None,
                    last_curve_len=0 if last_curve_bytes is None else len(last_curve_bytes))
    return grp, (sz, cb, cu, lb, lu)


_PROBLEM_KEYS = ("dtype", "tile_m", "tile_n", "order", "group_m", "num_xcds", "num_cus", "wg_per_cu",
                 "reserved_cus", "pattern", "num_dest", "dest_perm", "row_bucket")


def _split(kw):
    prob_kw = {k: v for k, v in kw.items() if k in _PROBLEM_KEYS}
    grp_kw = {k: v for k, v in kw.items() if k not in _PROBLEM_KEYS}
    return prob_kw, grp_kw


def _plan_of(handle: int, M: int, N: int, K: int, prob_kw) -> Plan:
    return Plan(handle, M, N, K, _DTYPES[prob_kw.get("dtype", "fp16")], prob_kw.get("tile_m", 256),
                prob_kw.get("tile_n", 128), _PATTERNS[prob_kw.get("pattern", "tile")], prob_kw.get("num_dest", 0))


def plan_groups(M: int, N: int, K: int, **kw) -> Plan:
    """fo_plan_groups. Keywords: the fo_problem fields (dtype, tile_m, tile_n,
    order, group_m, num_xcds, num_cus, wg_per_cu, reserved_cus, pattern,
    num_dest, dest_perm, row_bucket) and the fo_grouping ones (sizes, unit,
    gemm_us, curve_bytes, curve_us, s_first, s_last, dest_bytes = "largest" or
    "all": an All-to-All group's data size in the estimate, last_curve_bytes /
    last_curve_us: the last group's latency curve); sizes=None runs the
    Algorithm 1 search (needs gemm_us and the latency curve)."""
    L = lib()
    prob_kw, grp_kw = _split(kw)
    prob, keep_p = _problem(M, N, K, **prob_kw)
    grp, keep_g = _grouping(**grp_kw)
    out = ctypes.c_void_p()
    _check(L.fo_plan_groups(ctypes.byref(prob), ctypes.byref(grp), ctypes.byref(out)))
    return _plan_of(out.value, M, N, K, prob_kw)


class PlanCache:
    """fo_plan_cache: partitions searched ahead of time for representative
    sizes of a problem family, reused by nearest M for unseen sizes (Section
    4.2, online stage)."""

    def __init__(self):
        L = lib()
        h = ctypes.c_void_p()
        _check(L.fo_plan_cache_create(ctypes.byref(h)))
        self._h = h

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.fo_plan_cache_destroy(h)
            self._h = None

    def add(self, M: int, N: int, K: int, **kw) -> None:
        """fo_plan_cache_add: same keywords as plan_groups."""
        prob_kw, grp_kw = _split(kw)
        prob, keep_p = _problem(M, N, K, **prob_kw)
        grp, keep_g = _grouping(**grp_kw)
        _check(lib().fo_plan_cache_add(self._h, ctypes.byref(prob), ctypes.byref(grp)))

    def lookup(self, M: int, N: int, K: int, **kw):
        """fo_plan_cache_lookup: (Plan, M of the entry used). Takes the
        problem keywords of plan_groups (grouping keywords are ignored: the
        partition comes from the cache)."""
        prob_kw, _ = _split(kw)
        prob, keep_p = _problem(M, N, K, **prob_kw)
        out, matched = ctypes.c_void_p(), ctypes.c_int64()
        _check(lib().fo_plan_cache_lookup(self._h, ctypes.byref(prob), ctypes.byref(out), ctypes.byref(matched)))
        return _plan_of(out.value, M, N, K, prob_kw), int(matched.value)

    def __len__(self) -> int:
        return int(lib().fo_plan_cache_size(self._h))

    def entries(self):
        """[(M, wave partition)] in insertion order."""
        L, res = lib(), []
        for e in range(len(self)):
            m, n, sz = ctypes.c_int64(), ctypes.c_int32(), ctypes.POINTER(ctypes.c_int32)()
            _check(L.fo_plan_cache_entry(self._h, e, ctypes.byref(m), ctypes.byref(n), ctypes.byref(sz)))
            res.append((int(m.value), [int(sz[j]) for j in range(n.value)]))
        return res


def options(**fields) -> _Options:
    """fo_options: the process defaults (fo_options_init) with the given
    fields changed (sync_producer, sync_consumer, consumer_blocks,
    consumer_threads, poll_timeout_us, consumer_limit, tile_trace: a device
    buffer, tile_trace_capacity)."""
    o = _Options()
    _check(lib().fo_options_init(ctypes.byref(o)))
    for k, v in fields.items():
        if k not in dict(_Options._fields_):
            raise TypeError(f"unknown option {k!r}")
        setattr(o, k, _ptr(v) if k == "tile_trace" else int(v))
    return o


def _opts(o):
    """A pointer to an fo_options (None = the process defaults); a dict of
    fields is turned into options(**dict)."""
    if o is None:
        return None
    if isinstance(o, dict):
        o = options(**o)
    return ctypes.byref(o)


def gemm_signal_reorder(plan: Plan, dev_plan, A, W, C_out, counters=None, stream=None, opts=None) -> None:
    _need(A, 2 * plan.M * plan.K, "A")
    _need(W, 2 * plan.N * plan.K, "W")
    _need(C_out, 2 * plan.M * plan.N, "C_out")
    _need(counters, 4 * (plan.P + DISPENSER_WORDS), "counters")
    _check(lib().fo_gemm_signal_reorder(plan.handle, _ptr(dev_plan), _ptr(A), _ptr(W), _ptr(C_out),
                                        _ptr(counters), _stream(stream), _opts(opts)))


def consume_group(src, peer, dst, length: int, dtype, counter=None, target: int = 0,
                  status_word=None, stream=None, opts=None) -> None:
    _need(src, 2 * int(length), "src")
    _need(peer, 2 * int(length), "peer")
    _need(dst, 2 * int(length), "dst")
    _check(lib().fo_consume_group(_ptr(src), _ptr(peer), _ptr(dst), int(length), _DTYPES[dtype],
                                  _ptr(counter), int(target), _ptr(status_word), _stream(stream),
                                  _opts(opts)))


def post_reorder(plan: Plan, dev_plan, src, out, bias=None, gamma=None, eps: float = 1e-6,
                 do_rmsnorm: bool = False, stream=None) -> None:
    _need(src, 2 * (plan.dest_elems if plan.pattern != ROWMAJOR else plan.M * plan.N), "src")
    _need(out, 2 * plan.M * plan.N, "out")
    _need(bias, 2 * plan.N, "bias")
    _need(gamma, 2 * plan.N, "gamma")
    _check(lib().fo_post_reorder(plan.handle, _ptr(dev_plan), _ptr(src), _ptr(out), _ptr(bias),
                                 _ptr(gamma), float(eps), int(bool(do_rmsnorm)), _stream(stream)))


def reset_counters(counters, n: int, stream=None) -> None:
    _check(lib().fo_reset_counters(_ptr(counters), int(n), _stream(stream)))


def run_overlapped(plan: Plan, dev_plan, A, W, C_out, peer, dst, out=None, bias=None, gamma=None,
                   eps: float = 1e-6, do_rmsnorm: bool = False, counters=None, status_word=None,
                   gemm_stream=None, comm_stream=None, gemm_begin_event=None,
                   gemm_end_event=None, opts=None) -> None:
    _need(A, 2 * plan.M * plan.K, "A")
    _need(W, 2 * plan.N * plan.K, "W")
    _need(C_out, 2 * plan.M * plan.N, "C_out")
    _need(peer, 2 * plan.M * plan.N, "peer")
    _need(dst, 2 * plan.dest_elems, "dst")
    _need(out, 2 * plan.M * plan.N, "out")
    _need(bias, 2 * plan.N, "bias")
    _need(gamma, 2 * plan.N, "gamma")
    _need(counters, 4 * plan.num_counters, "counters")
    _need(status_word, 4, "status_word")
    _check(lib().fo_run_overlapped(plan.handle, _ptr(dev_plan), _ptr(A), _ptr(W), _ptr(C_out),
                                   _ptr(peer), _ptr(dst), _ptr(out), _ptr(bias), _ptr(gamma),
                                   float(eps), int(bool(do_rmsnorm)), _ptr(counters),
                                   _ptr(status_word), _stream(gemm_stream), _stream(comm_stream),
                                   _event(gemm_begin_event), _event(gemm_end_event), _opts(opts)))


NOALLOC_MAX_COUNTERS = 1024    # FO_NOALLOC_MAX_COUNTERS


def run_overlapped_noalloc(plan: Plan, dev_plan, A, W, C_out, peer, dst, out=None, bias=None, gamma=None,
                           eps: float = 1e-6, do_rmsnorm: bool = False, status_word=None,
                           gemm_stream=None, comm_stream=None, opts=None) -> None:
    """fo_run_overlapped_noalloc: the overlapped run with the library's static
    counters array (no device allocation; calls on one device must not
    overlap)."""
    _need(A, 2 * plan.M * plan.K, "A")
    _need(W, 2 * plan.N * plan.K, "W")
    _need(C_out, 2 * plan.M * plan.N, "C_out")
    _need(peer, 2 * plan.M * plan.N, "peer")
    _need(dst, 2 * plan.dest_elems, "dst")
    _need(out, 2 * plan.M * plan.N, "out")
    _need(bias, 2 * plan.N, "bias")
    _need(gamma, 2 * plan.N, "gamma")
    _need(status_word, 4, "status_word")
    _check(lib().fo_run_overlapped_noalloc(plan.handle, _ptr(dev_plan), _ptr(A), _ptr(W), _ptr(C_out),
                                           _ptr(peer), _ptr(dst), _ptr(out), _ptr(bias), _ptr(gamma),
                                           float(eps), int(bool(do_rmsnorm)), _ptr(status_word),
                                           _stream(gemm_stream), _stream(comm_stream), _opts(opts)))


SYNC_FENCE_ALL, SYNC_FENCE_ONE, SYNC_COHERENT = 0, 1, 2


def set_sync_mode(producer: int, consumer: int) -> None:
    _check(lib().fo_set_sync_mode(int(producer), int(consumer)))


def get_sync_mode():
    p, c = ctypes.c_int32(), ctypes.c_int32()
    lib().fo_get_sync_mode(ctypes.byref(p), ctypes.byref(c))
    return int(p.value), int(c.value)


def set_consumer_grid(max_blocks: int, threads: int = 64) -> None:
    """Grid of the consumer launches that run beside the GEMM: at most
    `max_blocks` workgroups (1..256) of `threads` threads (64, 128, 256);
    process-wide."""
    _check(lib().fo_set_consumer_grid(int(max_blocks), int(threads)))


def get_consumer_grid():
    b, t = ctypes.c_int32(), ctypes.c_int32()
    lib().fo_get_consumer_grid(ctypes.byref(b), ctypes.byref(t))
    return int(b.value), int(t.value)


def device_wall_clock_khz() -> int:
    k = ctypes.c_int32()
    _check(lib().fo_device_wall_clock_khz(ctypes.byref(k)))
    return int(k.value)


def set_poll_timeout_us(us: int) -> None:
    lib().fo_set_poll_timeout_us(int(us))


def get_poll_timeout_us() -> int:
    return int(lib().fo_get_poll_timeout_us())


def device_num_cus(device: int = 0) -> int:
    v = ctypes.c_int32()
    _check(lib().fo_device_num_cus(device, ctypes.byref(v)))
    return int(v.value)
