"""A consumer workgroup must fit on a compute unit beside a GEMM workgroup.

The consumer kernels poll and stream while the persistent GEMM holds one
workgroup per compute unit; if a consumer workgroup did not fit beside it, it
would take the compute unit away from the GEMM for as long as it waits. The
budget is checked on the compiler's resource report that the build writes
(gfx950: 512 registers per SIMD lane, allocated in blocks of 8; 160 KiB of
LDS per compute unit; a consumer workgroup has one wave per SIMD).
"""
import json
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
USAGE = os.path.join(ROOT, "paper_2504_19519_amd", "_build", "resource_usage.json")


def _round8(n):
    return (n + 7) // 8 * 8


def _usage():
    if not os.path.exists(USAGE):
        pytest.fail("no resource report: build the library first (python -m paper_2504_19519_amd.build)")
    with open(USAGE) as f:
        return json.load(f)


def _regs(v):
    """Registers per lane of one wave: the VGPRs (rounded up to the 4 at which
    the accumulation registers start) followed by the AGPRs, rounded to 8."""
    return _round8((v["vgpr"] + 3) // 4 * 4 + v.get("agpr", 0))


def test_consumer_fits_beside_every_gemm_kernel():
    u = _usage()
    gemm = {k: v for k, v in u.items()
            if "gemm_signal_kernel" in k or "gemm_w4_kernel" in k or "gemm_w4n_kernel" in k}
    cons = {k: v for k, v in u.items() if "consume_kernel" in k}
    assert len(gemm) >= 6 and len(cons) >= 8
    c_regs = max(_regs(v) for v in cons.values())
    c_lds = max(v["lds"] for v in cons.values())
    for name, v in gemm.items():
        # register spills may only go to other registers (no scratch memory)
        assert v.get("scratch", 0) == 0, name
        if "gemm_w4_kernel" in name or "gemm_w4n_kernel" in name:
            per_simd = 1                   # 4 waves of 128 x 128 (128 x 64): one per SIMD
        else:
            # waves of one GEMM workgroup per SIMD (template arguments: dtype,
            # tile_m, tile_n, waves_m, waves_n, stages, k step): 4 waves -> 1, 8 -> 2
            m = re.search(r"gemm_signal_kernelILi(\d+)ELi(\d+)ELi(\d+)ELi(\d+)ELi(\d+)ELi(\d+)ELi(\d+)E", name)
            assert m, name
            per_simd = (int(m.group(4)) * int(m.group(5)) + 3) // 4
        regs = per_simd * _regs(v)
        assert regs + c_regs <= 512, (name, regs, c_regs)
        assert v["lds"] + c_lds <= 160 * 1024, (name, v["lds"], c_lds)
