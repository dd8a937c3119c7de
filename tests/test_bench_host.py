"""Host-side pieces of bench.py: the CLI contract for more than one GPU, the
algorithmic byte counts used for the roofline, the per-matrix cost and the
LPT split of the owner-share diagnostic, on host-only plans."""
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2606_27153_amd.optim import MuonPlan  # noqa: E402
from paper_2606_27153_amd.workloads import get_workload  # noqa: E402


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
    pb = [2, 2]   # bf16 parameters: the last B*X reads and writes W, 4 bytes per element
    got = {kind: bench.gemm_algorithmic_bytes(plan, k, kind, cls, pb) for kind in ("gram", "poly", "bx", "symm")}
    if aspect:
        want = {"gram": 2 * (m * n + m * m), "poly": k * 4 * m * m, "symm": (k - 1) * 9 * 2 * m * m,
                "bx": 2 * (m * m + m * n) + 4 * m * n}
    else:
        want = {"gram": k * 2 * (m * n + m * m), "poly": k * 4 * m * m, "symm": 0.0,
                "bx": k * 2 * (m * m + m * n) + (k - 1) * 2 * m * n + 4 * m * n}
    for kind in want:
        assert got[kind] == pytest.approx(2 * want[kind]), kind   # two matrices
    assert bench.gemm_algorithmic_bytes(plan, k, "bx", "f32_t64", pb) == 0.0
    plan.close()


def test_kernel_keys():
    assert bench.kernel_key("_ZN4muon12_GLOBAL__N_114ns_gemm_kernelIDF16bLi256ELi2ELi4ELi3EEEvNS0_8GemmArgsE") \
        == "symm:bf16_t256"
    assert bench.kernel_key("_ZN4muon12_GLOBAL__N_114ns_gemm_kernelIfLi64ELi2ELi2ELi2EEEvNS0_8GemmArgsE") \
        == "bx:f32_t64"
    assert bench.kernel_key("_ZN4muon12_GLOBAL__N_114ns_gemm_kernelIDF16_Li256ELi2ELi4ELi2EEEvNS0_8GemmArgsE") \
        == "bx:f16_t256"
    assert bench.kernel_key("muon::(anonymous namespace)::apply_kernel(...)") == "apply"


def test_traffic_summary_round_trip(tmp_path):
    # counter files as rocprofv3 writes them: a 1 MiB copy reads 512 KiB and
    # writes 1024 KiB by the counters, so the scales are 2 and 1
    sym = "_ZN4muon12_GLOBAL__N_114ns_gemm_kernelIDF16bLi256ELi2ELi4ELi3EEEvNS0_8GemmArgsE"
    rows = [("__amd_rocclr_copyBuffer", "FETCH_SIZE", 512.0), ("__amd_rocclr_copyBuffer", "WRITE_SIZE", 1024.0),
            (sym, "FETCH_SIZE", 100.0), (sym, "FETCH_SIZE", 300.0), (sym, "WRITE_SIZE", 50.0)]
    d = tmp_path / "pmc"
    d.mkdir()
    with open(d / "run_counter_collection.csv", "w") as f:
        f.write("Kernel_Name,Counter_Name,Counter_Value\n")
        for k, c, v in rows:
            f.write(f"{k},{c},{v}\n")
    out = tmp_path / "traffic.txt"
    bench.write_traffic_summary(str(tmp_path), "symm:bf16_t256", 1, "cmd", path=str(out))
    got = bench.read_traffic("symm:bf16_t256", path=str(out))
    assert got == pytest.approx((200.0 * 2 + 50.0 * 1) * 1024)
    assert bench.read_traffic("bx:bf16_t256", path=str(out)) is None


def test_ns_cost_matches_the_plan_accounting():
    # the LPT cost of each matrix is the algorithmic flops of the form the
    # plan gives it (Eq. 4 or Eq. 2), summed as the plan reports them
    for key in ("1b", "8b", "vla"):
        wl = get_workload(key)
        plan = MuonPlan([(m.rows, m.cols, m.param, m.grad) for m in wl.matrices], host_only=True)
        info = plan.info()
        want = plan.ns_flops(5)
        got = sum(bench.ns_cost(m.rows, m.cols, 5) for m in wl.matrices)
        assert abs(got - want) <= 1e-9 * want, key
        plan.close()


def test_lpt_partition_against_brute_force():
    import itertools
    rng = np.random.default_rng(5)
    for trial in range(40):
        n_items = int(rng.integers(1, 9))
        n_owners = int(rng.integers(1, 4))
        costs = [float(c) for c in rng.integers(1, 50, size=n_items)]
        owners, loads = bench.lpt_partition(costs, n_owners)
        assert sorted(i for o in owners for i in o) == list(range(n_items))
        for r, o in enumerate(owners):
            assert abs(loads[r] - sum(costs[i] for i in o)) < 1e-9
        best = min(max(sum(costs[i] for i in range(n_items) if a[i] == r) for r in range(n_owners))
                   for a in itertools.product(range(n_owners), repeat=n_items))
        # Graham's bound for LPT: makespan <= (4/3 - 1/(3N)) * optimum
        assert max(loads) <= (4 / 3 - 1 / (3 * n_owners)) * best + 1e-9


def test_percentile_and_share_of_the_8b_set():
    assert bench.percentile([3.0, 1.0, 2.0], 0.5) == 2.0
    assert bench.percentile([1.0, 2.0], 0.9) == pytest.approx(1.9)
    wl = get_workload("8b")
    costs = [bench.ns_cost(m.rows, m.cols) for m in wl.matrices]
    owners, loads = bench.lpt_partition(costs, 8)
    # 224 matrices in three shapes split into 8 nearly equal shares
    assert max(loads) / (sum(loads) / 8) < 1.02
    assert sum(len(o) for o in owners) == 224


def test_eq2_work_of_the_8b_and_moe_sets():
    # Eq. 2 work, symmetry-aware: 5 (3 m^2 n + m^3) per matrix; 4.72e14 for
    # the 8B set, and 2.67e14 for the MoE set once its zero-gradient experts
    # are left out (they have no NS work at all)
    wl = get_workload("8b")
    ffn = 5 * (3 * 4096 ** 2 * 14336 + 4096 ** 3)
    sq = 5 * 4 * 4096 ** 3
    kv = 5 * (3 * 1024 ** 2 * 4096 + 1024 ** 3)
    got = sum(bench.eq2_work_flops(m.rows, m.cols) for m in wl.matrices)
    assert got == pytest.approx(96 * ffn + 64 * sq + 64 * kv, rel=1e-12)
    assert got == pytest.approx(4.72e14, rel=2e-3)
    moe = get_workload("moe")
    live = sum(bench.eq2_work_flops(m.rows, m.cols) for m in moe.matrices if not m.zero_grad)
    assert sum(m.zero_grad for m in moe.matrices) == 1152
    assert live == pytest.approx(2.67e14, rel=3e-3)


def test_live_flop_share():
    # four equal matrices, one with a zero gradient: three quarters of every
    # launch group's flops are executed
    descs = [(1024, 4096, "bf16", "bf16")] * 4
    plan = MuonPlan(descs, host_only=True)
    share = bench.live_flop_share(plan, 5, [True, False, False, False])
    assert sorted(k[0] for k in share) == ["bx", "gram", "poly", "symm"]
    assert all(v == pytest.approx(0.75) for v in share.values())
    assert bench.live_flop_share(plan, 5, [False] * 4) == {k: 1.0 for k in share}
    assert bench.live_flop_share(plan, 5, [True] * 4) == {k: 0.0 for k in share}
    plan.close()
    # Gram-space (n >= 1.4m) and Eq. 2 matrices in one class: with restarts
    # every 2 steps (segments 2, 2, 1) the former's Gram and B*X run 3 times,
    # the latter's k = 5 times
    descs = [(1024, 4096, "bf16", "bf16"), (1024, 1024, "bf16", "bf16")]
    plan = MuonPlan(descs, host_only=True)
    infos = [plan.matrix_info(i) for i in range(2)]
    assert [i["gram_space"] for i in infos] == [1, 0] and infos[0]["kernel_class"] == infos[1]["kernel_class"]
    from paper_2606_27153_amd import _lib as L
    cls = L.KERNEL_CLASSES[infos[0]["kernel_class"]]
    share = bench.live_flop_share(plan, 5, [False, True])
    g_rect, g_sq = 3 * 1024 ** 2 * 4096, 5 * 1024 ** 3
    assert share[("gram", cls)] == pytest.approx(g_rect / (g_rect + g_sq))
    assert share[("symm", cls)] == pytest.approx(1.0)   # only the Gram-space matrix has symmetric products
    assert share[("bx", cls)] == pytest.approx(3 * 2 * 1024 ** 2 * 4096 / (3 * 2 * 1024 ** 2 * 4096 + 5 * 2 * 1024 ** 3))
    plan.close()


def test_kernel_sources_hash_covers_files_only():
    """The hash that keys the committed traffic summary reads the kernel
    source files and passes over sub-directories (the diagnostic probe)."""
    import re
    h = bench.kernel_sources_hash()
    assert re.fullmatch(r"[0-9a-f]{16}", h)
