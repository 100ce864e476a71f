"""Host-side derivations of bench.py, on the CPU: the step's lower bound
(Section 6.4: the last group's communication cannot be hidden, nor the whole
communication before the first group's compute), the fractions of the
theoretical speedup and performance, and the one-GPU guard."""
import os
import subprocess
import sys
import types

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def plan_with(targets):
    return types.SimpleNamespace(targets=list(targets))


def test_bound_is_the_last_groups_share_or_the_first_groups_compute():
    # GEMM 400, consumer 80, post 40: with [512, 256, 256] tiles the last
    # group's share (1/4) of the consumer follows the GEMM
    assert bench.theoretical(plan_with([512, 256, 256]), 400.0, 80.0, 40.0) == pytest.approx(400 + 20 + 40)
    # a consumer much longer than the GEMM behind a large first group: the
    # first group's compute + the whole consumer
    assert bench.theoretical(plan_with([768, 256]), 400.0, 900.0, 0.0) == pytest.approx(300 + 900)
    assert bench.theoretical(plan_with([256, 768]), 400.0, 900.0, 0.0) == pytest.approx(400 + 675)
    # one group: nothing overlaps, the bound is the serialized step
    assert bench.theoretical(plan_with([1024]), 400.0, 80.0, 40.0) == pytest.approx(520.0)


def rounds(ov, se):
    return {"overlapped_step_us": ov, "serial_step_us": se, "gemm_consume_overlapped_us": 300.0,
            "gemm_alone_us": 280.0, "consume_alone_us": 60.0, "gemm_in_overlapped_us": 290.0,
            "gemm_in_serial_us": 280.0}


def test_fractions_of_the_theoretical_bound():
    bound = 400.0
    at_bound = bench.overlap_fields(rounds(400.0, 480.0), bound)
    assert at_bound["fraction_of_theoretical_speedup"] == pytest.approx(1.0)
    assert at_bound["fraction_of_theoretical_performance"] == pytest.approx(1.0)
    assert at_bound["theoretical_speedup"] == pytest.approx(1.2)
    no_gain = bench.overlap_fields(rounds(480.0, 480.0), bound)
    assert no_gain["fraction_of_theoretical_speedup"] == pytest.approx(0.0)
    half = bench.overlap_fields(rounds(480.0 / 1.1, 480.0), bound)
    assert half["fraction_of_theoretical_speedup"] == pytest.approx(0.5, abs=1e-4)
    assert half["overlapped_gemm_consume_over_max"] == pytest.approx(300.0 / 280.0, abs=1e-4)
    # a bound no better than the serialized step has no theoretical speedup
    assert bench.overlap_fields(rounds(480.0, 480.0), 480.0)["fraction_of_theoretical_speedup"] is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stdout
