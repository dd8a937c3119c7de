"""Host-side pieces of bench.py: the CLI contract for more than one GPU and
the algorithmic byte counts used for the roofline, on host-only plans."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2606_27153_amd.optim import MuonPlan  # noqa: E402


def test_more_than_one_gpu_is_refused():
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True)
    assert out.returncode == 2 and "one GPU" in out.stderr


@pytest.mark.parametrize("aspect", [0.0, 2.0])
def test_gemm_algorithmic_bytes(lib, aspect):
    # one wide 512 x 2048 matrix (bf16 NS, 256 tiles) and its transpose
    plan = MuonPlan([(512, 2048, "bf16", "bf16"), (2048, 512, "bf16", "bf16")], host_only=True,
                    gram_min_aspect=aspect)
    cls = "bf16_t256"
    assert plan.matrix_info(0)["kernel_class"] == plan.matrix_info(1)["kernel_class"] == 0
    m, n, k = 512.0, 2048.0, 5
    got = {kind: bench.gemm_algorithmic_bytes(plan, k, kind, cls) for kind in ("gram", "poly", "bx", "symm")}
    if aspect:
        want = {"gram": 2 * (m * n + m * m), "poly": k * 4 * m * m, "symm": (k - 1) * 9 * 2 * m * m,
                "bx": 2 * (m * m + m * n) + 4 * m * n}
    else:
        want = {"gram": k * 2 * (m * n + m * m), "poly": k * 4 * m * m, "symm": 0.0,
                "bx": k * 2 * (m * m + m * n) + (k - 1) * 2 * m * n + 4 * m * n}
    for kind in want:
        assert got[kind] == pytest.approx(2 * want[kind]), kind   # two matrices
    assert bench.gemm_algorithmic_bytes(plan, k, "bx", "f32_t64") == 0.0
    plan.close()
