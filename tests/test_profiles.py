"""The committed rocprofv3 summaries: their commands run committed files only,
their figures agree with each other, and bench.py reads the GEMM's HBM traffic
from them only for the workload and GEMM sources they were taken with."""
import glob
import os
import re

import pytest

from paper_2504_19519_amd import profsum

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
STEP = sorted(glob.glob(os.path.join(ROOT, "profiles", "gemm_step_*.md")))


def figures(path):
    kv = {}
    with open(path) as f:
        for line in f:
            m = re.match(r"^(\w+): (\S+)$", line.strip())
            if m:
                kv[m.group(1)] = m.group(2)
    return kv


def test_every_large_workload_has_a_summary():
    names = {os.path.basename(p)[len("gemm_step_"):-3] for p in STEP}
    assert {"rs_8192x8192x3584", "ar_rmsnorm_16384x4096x3584_bf16", "a2a_4096x7168x2048"} <= names
    for n in names:
        assert os.path.exists(os.path.join(ROOT, "profiles", f"serial_step_and_gemm_{n}.md"))


@pytest.mark.parametrize("path", STEP + sorted(glob.glob(os.path.join(ROOT, "profiles", "serial_step_*.md"))),
                         ids=os.path.basename)
def test_commands_run_committed_files_only(path):
    text = open(path).read()
    cmds = [l for l in text.splitlines() if l.startswith("rocprofv3 ")]
    assert cmds, "a summary lists the commands that made it"
    for c in cmds:
        prog = c.split(" -- ", 1)[1].split()
        assert prog[0] == "python3" and prog[1] == "R/bench.py", c
        assert "_work" not in c and "gpurun" not in c


@pytest.mark.parametrize("path", STEP, ids=os.path.basename)
def test_traffic_is_the_scaled_counter_sum(path):
    kv = figures(path)
    w = os.path.basename(path)[len("gemm_step_"):-3]
    assert kv["workload"] == w
    traffic = (float(kv["gemm_fetch_kib"]) * float(kv["fetch_scale"]) +
               float(kv["gemm_write_kib"]) * float(kv["write_scale"])) * 1024.0
    assert abs(traffic - float(kv["traffic_bytes_per_launch"])) <= 1e-4 * traffic + 2048
    assert float(kv["gemm_trace_avg_us"]) > 0
    if kv["gemm_sources_sha256"] == profsum.gemm_sources_sha256():
        assert profsum.read_traffic(path, w) == pytest.approx(float(kv["traffic_bytes_per_launch"]))
    else:
        assert profsum.read_traffic(path, w) is None
    assert profsum.read_traffic(path, w + "_other") is None
