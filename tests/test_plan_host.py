"""Planner invariants checked on the host: tests/plan_check.cpp is built with
g++ against csrc/plan.cpp (no HIP), with AddressSanitizer and
UndefinedBehaviorSanitizer (the kernels trust the planner's tables and
padding), and run on the shape lists of every workload, a ragged set and
random shapes."""
import os
import subprocess

import numpy as np
import pytest

from paper_2606_27153_amd.workloads import WORKLOAD_KEYS, get_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def plan_check(tmp_path_factory):
    exe = tmp_path_factory.mktemp("plan") / "plan_check"
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "plan_check.cpp"),
                    os.path.join(ROOT, "paper_2606_27153_amd", "csrc", "plan.cpp"), "-o", str(exe)],
                   check=True)
    return str(exe)


def _run(exe, shapes, precision=0, wave_bytes=0, aspect=2.0, restart=0):
    inp = "\n".join(f"{r} {c}" for r, c in shapes)
    out = subprocess.run([exe, str(precision), str(wave_bytes), str(aspect), str(restart)], input=inp,
                         capture_output=True, text=True)
    assert out.returncode == 0 and out.stdout.startswith("OK"), out.stdout + out.stderr


@pytest.mark.parametrize("key", WORKLOAD_KEYS)
def test_workload_plans(plan_check, key):
    shapes = [(m.rows, m.cols) for m in get_workload(key).matrices]
    _run(plan_check, shapes)
    _run(plan_check, shapes, wave_bytes=1 << 30)
    _run(plan_check, shapes, aspect=0.0)
    _run(plan_check, shapes, precision=2)


def test_ragged_and_random_plans(plan_check):
    rng = np.random.default_rng(0)
    ragged = [(1, 1), (1, 300), (300, 1), (7, 13), (65, 200), (200, 65), (130, 700), (700, 130),
              (257, 513), (513, 257), (1000, 1000), (96, 4304), (1152, 1200), (2304, 9000), (4100, 4100)]
    _run(plan_check, ragged)
    _run(plan_check, ragged, precision=1)
    _run(plan_check, ragged, precision=2)
    _run(plan_check, ragged, aspect=1.0)
    _run(plan_check, ragged, aspect=0.0)
    # segments of one, two (shared square buffers), three and all steps
    for restart in (1, 2, 3, 16):
        _run(plan_check, ragged, aspect=1.0, restart=restart)
    # more than 65535 tiles along one dimension
    _run(plan_check, [(1, 1 << 22), ((1 << 22) + 5, 3), (70, 1 << 18)])
    for trial in range(5):
        shapes = [(int(rng.integers(1, 3000)), int(rng.integers(1, 3000))) for _ in range(40)]
        _run(plan_check, shapes, wave_bytes=int(rng.integers(1, 4)) << 28)
