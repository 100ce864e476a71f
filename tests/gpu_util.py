"""Helpers for the GPU parity tests: device buffers from stored bits, the
value tolerance, and a runner for one whole path through the C ABI."""
from __future__ import annotations

import math
import sys

import numpy as np

import oracle
import paper_2504_19519_amd as fo
import workloads

ATOL, RTOL = 2e-3, 1e-2      # |gpu - ref| <= ATOL + RTOL * |ref| for fp16/bf16 values
NAN_BITS = {"fp16": 0x7E00, "bf16": 0x7FC0}


def torch_mod():
    import torch
    return torch


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(bits: np.ndarray):
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).reshape(-1).view(np.int16)).to("cuda")


def from_dev(t) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint16).copy()


def empty16(n: int, poison: str | None = None):
    torch = torch_mod()
    t = torch.empty(max(int(n), 8), dtype=torch.int16, device="cuda")
    if poison:
        b = NAN_BITS[poison]
        t.fill_(b - 65536 if b >= 32768 else b)
    return t


def zeros_u32(n: int):
    torch = torch_mod()
    return torch.zeros(max(int(n), 1), dtype=torch.int32, device="cuda")


def dev_plan(plan: fo.Plan):
    torch = torch_mod()
    buf = torch.empty(plan.device_bytes // 4 + 4, dtype=torch.int32, device="cuda")
    plan.to_device(buf)
    torch.cuda.synchronize()
    return buf


def assert_close_bits(got: np.ndarray, ref: np.ndarray, dtype: str, what: str = "") -> None:
    g = oracle.decode(got.reshape(-1), dtype)
    r = oracle.decode(ref.reshape(-1), dtype)
    assert np.all(np.isfinite(g)), f"{what}: non-finite values in GPU result"
    err = np.abs(g - r)
    bound = ATOL + RTOL * np.abs(r)
    bad = err > bound
    if bad.any():
        i = int(np.argmax(err - bound))
        raise AssertionError(f"{what}: {int(bad.sum())} of {g.size} outside tolerance; worst at {i}: "
                             f"gpu={g[i]!r} ref={r[i]!r}")


def plan_for(w: workloads.Workload, inp: workloads.Inputs, *, num_cus=256, sizes=None, unit=None,
             pattern=None, group_m=4, num_xcds=8):
    pattern = pattern or w.pattern
    nd = w.num_dest if pattern in ("subtile", "subtoken") else 0
    kw = dict(dtype=w.dtype, tile_m=w.tile_m, tile_n=w.tile_n, order=w.order, num_cus=num_cus,
              group_m=group_m, num_xcds=num_xcds, pattern=pattern, num_dest=nd,
              dest_perm=inp.sigma if pattern == "subtile" else None,
              row_bucket=inp.bucket if pattern == "subtoken" else None)
    tiles = (w.M // w.tile_m) * (w.N // w.tile_n)
    T = -(-tiles // num_cus) if tiles else 0
    if sizes is None:
        if w.groups is not None and unit is None:
            sizes, unit = list(w.groups), w.group_unit
        else:
            sizes, unit = [1] * T, "waves"
    unit = unit or "waves"
    p = fo.plan_groups(w.M, w.N, w.K, sizes=sizes, unit=unit, **kw)
    o = oracle.make_plan(w.M, w.N, w.tile_m, w.tile_n, num_cus=num_cus, order=w.order,
                         group_m=group_m, num_xcds=num_xcds, pattern=pattern, num_dest=nd,
                         sigma=inp.sigma, bucket=inp.bucket,
                         sizes=sizes, unit=unit)
    return p, o
