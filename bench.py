"""Benchmark of the single-GPU Muon optimizer step (one JSON line on stdout).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 8b]
    python bench.py --sweep [--config 8b]          # per-shape batch sweep (table)
    python bench.py --owner-share 8 [--owner 0]    # one owner's cost-balanced share

A step is one muon_step over every matrix of the chosen synthetic set:
momentum + Nesterov, Frobenius normalisation, 5 Newton-Schulz steps, apply.
Inputs (params, grads, momentum) are resident in HBM before the timed
region.  Per-launch durations come from HIP events recorded by the library
on its stream during the timed steps; the dominant kernel's achieved rate is
its algorithmic work per launch over its mean launch duration.  The fp64
oracle is timed on the host cores on a bounded sample as a reference point.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "Muon optimizer-step ms per step (1 GPU) + MFMA util % on Newton–Schulz GEMMs"
PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 matrix peak: 256 CU x 2.4 GHz x 4096 flop/clk
PEAK_F32_TFLOPS = 157.3       # MI355X fp32 matrix peak
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
GEMM_KINDS = ("gram", "poly", "bx", "symm")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_sources_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_27153_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if not os.path.isfile(os.path.join(csrc, name)):
            continue  # diag/: the ceiling probe, not a kernel the traffic was taken on
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "traffic_summary.txt")


def read_traffic(kernel_key: str, path: str = TRAFFIC_SUMMARY):
    """HBM bytes per launch of ``kernel_key`` from the committed rocprofv3
    --pmc summary, if it was taken on the current kernel sources."""
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if line.startswith("#") or "=" not in line:
                continue
            k, v = line.split("=", 1)
            vals[k.strip()] = v.strip()
    if vals.get("sources_sha256_16") != kernel_sources_hash():
        return None
    try:
        return float(vals[f"{kernel_key} hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _kernel_patterns():
    pats = []
    for e, cls in (("DF16b", "bf16"), ("f", "f32"), ("DF16_", "f16")):
        for tile, wg in ((256, "2ELi4"), (128, "2ELi2"), (64, "2ELi2")):
            if e == "f" and tile == 256:
                continue
            for stage, kind in enumerate(("gram", "poly", "bx", "symm")):
                pats.append((rf"ns_gemm_kernelI{e}Li{tile}ELi{wg}ELi{stage}E", f"{kind}:{cls}_t{tile}"))
    return pats


KERNEL_RE = _kernel_patterns() + [
    # (regex on the mangled or plain kernel name, readable key)
    (r"momentum_kernel", "momentum"),
    (r"finalize_kernel", "finalize"),
    (r"apply_kernel", "apply"),
    (r"__amd_rocclr_copyBuffer", "copy (device copy)"),
]


def kernel_key(name: str) -> str:
    import re
    for pat, key in KERNEL_RE:
        if re.search(pat, name):
            return key
    return "other: " + name[:60]


def rocprof_summary(root: str) -> str:
    """Markdown summary of rocprofv3 CSV output found under ``root``:
    kernel statistics (--kernel-trace --stats) and per-dispatch FETCH_SIZE /
    WRITE_SIZE counters (--pmc), scaled by the device-copy calibration."""
    import csv
    import glob
    lines = []
    for path in sorted(glob.glob(os.path.join(root, "**", "*kernel_stats.csv"), recursive=True)):
        rows = list(csv.DictReader(open(path)))
        agg = {}
        for r in rows:
            k = kernel_key(r["Name"])
            a = agg.setdefault(k, [0, 0.0])
            a[0] += int(r["Calls"])
            a[1] += float(r["TotalDurationNs"])
        total = sum(v[1] for v in agg.values())
        lines += [f"### kernel statistics ({os.path.relpath(path, root)})", "",
                  "| kernel | calls | total ms | mean ms | share |", "|---|---|---|---|---|"]
        for k, (calls, ns) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
            lines.append(f"| {k} | {calls} | {ns / 1e6:.3f} | {ns / 1e6 / max(1, calls):.4f} | "
                         f"{100 * ns / total:.1f}% |")
        lines.append("")
    counters = {}
    shader = {}   # pass directory -> kernel -> counter -> [dispatches, sum, sum of durations]
    for path in sorted(glob.glob(os.path.join(root, "**", "*counter_collection.csv"), recursive=True)):
        for r in csv.DictReader(open(path)):
            k = kernel_key(r["Kernel_Name"])
            cname = r["Counter_Name"]
            if cname in ("FETCH_SIZE", "WRITE_SIZE"):
                c = counters.setdefault(cname, {}).setdefault(k, [0, 0.0])
                c[0] += 1
                c[1] += float(r["Counter_Value"])
            else:
                dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
                c = shader.setdefault(os.path.relpath(os.path.dirname(path), root), {}).setdefault(k, {}) \
                    .setdefault(cname, [0, 0.0, 0.0])
                c[0] += 1
                c[1] += float(r["Counter_Value"])
                c[2] += dur
    if shader:
        lines += ["### Shader counters per dispatch (rocprofv3 --pmc)", "",
                  "Clock = GRBM_GUI_ACTIVE / 8 XCDs / dispatch duration; MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / "
                  "(GRBM_GUI_ACTIVE / 8 x 1024 SIMDs); L2 hit = TCC_HIT / (TCC_HIT + TCC_MISS).", "",
                  "| pass | kernel | dispatches | mean ms | clock GHz | MFMA busy | L2 hit | counters (mean) |",
                  "|---|---|---|---|---|---|---|---|"]
        for pas, per in sorted(shader.items()):
            for k, cs in sorted(per.items()):
                if k.startswith("other") or k.startswith("copy"):
                    continue
                mean = {c: v[1] / v[0] for c, v in cs.items()}
                n, _, dsum = next(iter(cs.values()))
                ms = dsum / n * 1e3
                clk = busy = hit = ""
                if "GRBM_GUI_ACTIVE" in mean and ms > 0:
                    cyc = mean["GRBM_GUI_ACTIVE"] / 8
                    clk = f"{cyc / (ms * 1e-3) / 1e9:.2f}"
                    if "SQ_VALU_MFMA_BUSY_CYCLES" in mean:
                        busy = f"{100 * mean['SQ_VALU_MFMA_BUSY_CYCLES'] / (cyc * 1024):.1f}%"
                hs = [mean.get(c) for c in ("TCC_HIT_sum", "TCC_MISS_sum")]
                if all(v is not None for v in hs) and sum(hs) > 0:
                    hit = f"{100 * hs[0] / sum(hs):.1f}%"
                rest = ", ".join(f"{c} {v:.4g}" for c, v in sorted(mean.items()))
                lines.append(f"| {pas} | {k} | {n} | {ms:.3f} | {clk} | {busy} | {hit} | {rest} |")
        lines.append("")
    if counters:
        copy = "copy (device copy)"
        lines += ["### HBM traffic per dispatch (rocprofv3 --pmc, KiB per dispatch)", ""]
        cal = {}
        for cname in ("FETCH_SIZE", "WRITE_SIZE"):
            if cname in counters and copy in counters[cname]:
                n, v = counters[cname][copy]
                cal[cname] = v / n
        lines.append(f"device-copy calibration (mean KiB per copy dispatch): {cal}")
        lines += ["", "| kernel | counter | dispatches | mean KiB | mean GB |", "|---|---|---|---|---|"]
        for cname, per in sorted(counters.items()):
            for k, (n, v) in sorted(per.items()):
                lines.append(f"| {k} | {cname} | {n} | {v / n:.0f} | {v / n * 1024 / 1e9:.4f} |")
        lines.append("")
    return "\n".join(lines)


def write_traffic_summary(root: str, kernels: str, copy_mib: int, command: str, path: str = TRAFFIC_SUMMARY) -> str:
    """Writes profiles/traffic_summary.txt for the comma-separated kernel keys
    from the FETCH_SIZE and WRITE_SIZE passes under ``root``.  Each counter is
    scaled by the ratio of the known size of the calibration copy to what the
    same counter read for it."""
    import csv
    import glob
    per = {}
    for csv_path in sorted(glob.glob(os.path.join(root, "**", "*counter_collection.csv"), recursive=True)):
        for r in csv.DictReader(open(csv_path)):
            k = kernel_key(r["Kernel_Name"])
            c = per.setdefault(r["Counter_Name"], {}).setdefault(k, [0, 0.0])
            c[0] += 1
            c[1] += float(r["Counter_Value"])
    known_kib = copy_mib * 1024.0
    factor = {c: known_kib / per[c]["copy (device copy)"][1] for c in ("FETCH_SIZE", "WRITE_SIZE")}
    lines = [
        "# HBM traffic per launch (rocprofv3 --pmc, one counter per run)",
        f"# command: {command}",
        f"# FETCH_SIZE and WRITE_SIZE scaled by a {copy_mib} MiB device-to-device copy in the same run",
        f"sources_sha256_16 = {kernel_sources_hash()}",
        f"fetch_scale = {factor['FETCH_SIZE']:.4f}",
        f"write_scale = {factor['WRITE_SIZE']:.4f}",
    ]
    for kernel in kernels.split(","):
        kib = {}
        for c in ("FETCH_SIZE", "WRITE_SIZE"):
            n, v = per[c][kernel]
            kib[c] = v / n
        total = sum(kib[c] * factor[c] * 1024.0 for c in kib)
        lines += [f"{kernel} fetch_kib_per_launch = {kib['FETCH_SIZE']:.0f}",
                  f"{kernel} write_kib_per_launch = {kib['WRITE_SIZE']:.0f}",
                  f"{kernel} hbm_bytes_per_launch = {total:.0f}"]
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    return path


def cpu_baseline(wl, budget_s: float):
    """Times the fp64 oracle on one matrix per shape bucket and extrapolates
    to the whole set by bucket counts."""
    import numpy as np
    import torch

    from oracle import muon_ref as R
    from paper_2606_27153_amd.workloads import make_grad, make_param

    try:
        from threadpoolctl import threadpool_info
        threads = max([d.get("num_threads", 1) for d in threadpool_info() if d.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    buckets = {}
    for i, m in enumerate(wl.matrices):
        buckets.setdefault((min(m.rows, m.cols), max(m.rows, m.cols)), []).append(i)
    order = sorted(buckets.items(), key=lambda kv: kv[0][0] * kv[0][0] * kv[0][1])
    total_ms = 0.0
    sampled = []
    spent = 0.0
    lr, mu, wd = wl.lr, wl.momentum, wl.weight_decay
    per_flop_ms = None
    for (m, n), idx in order:
        i = idx[0]
        flops = R.ns_flops(m, n, wl.ns_steps)
        if spent < budget_s or per_flop_ms is None:
            w = make_param(torch, wl, i, "cpu").double().numpy()
            g = make_grad(torch, wl, i, 0, "cpu").double().numpy()
            t0 = time.perf_counter()
            R.muon_step_matrix(w, g, np.zeros_like(g), lr=lr, momentum=mu, weight_decay=wd,
                               ns_steps=wl.ns_steps, nesterov=wl.nesterov, param_dtype=wl.matrices[i].param)
            dt = time.perf_counter() - t0
            spent += dt
            per_flop_ms = dt * 1e3 / flops
            sampled.append(f"{wl.matrices[i].rows}x{wl.matrices[i].cols} {dt:.2f}s")
            total_ms += dt * 1e3 * len(idx)
        else:
            total_ms += per_flop_ms * flops * len(idx)
            sampled.append(f"{m}x{n} extrapolated by flops")
    return {"value": round(total_ms, 1), "unit": "ms", "cores": int(threads), "kind": "oracle",
            "sample": ("fp64 numpy oracle, one matrix per shape bucket, one step each ("
                       + "; ".join(sampled) + "), scaled by bucket counts to the whole set"),
            "cpu_model": cpu_model(), "affinity_cores": len(os.sched_getaffinity(0)),
            "blas_threads": int(threads)}


def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo), or '' if unknown."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


GRAM_MIN_M = 256      # smaller matrices stay on Eq. 2
GRAM_RESTART = 2     # NS steps per Gram-space segment (the library's default)


def gram_segments(k: int, restart: int = GRAM_RESTART) -> list:
    """Lengths of the Gram-space segments of k NS steps."""
    return [min(restart, k - s0) for s0 in range(0, k, restart)]


def ns_cost(rows: int, cols: int, k: int = 5, gram_min_aspect: float = 1.4, restart: int = GRAM_RESTART) -> float:
    """Algorithmic NS flops of one matrix in the form the plan gives it
    (16-bit classes; Eq. 4 when n >= aspect * m and m >= 256, else Eq. 2).
    Eq. 4 restarts every ``restart`` steps; a segment of L steps costs
    3 m^2 n + (4L - 3) m^3."""
    m, n = min(rows, cols), max(rows, cols)
    if gram_min_aspect > 0 and n >= gram_min_aspect * m and m >= GRAM_MIN_M:
        return sum(3.0 * m * m * n + (4 * L - 3) * float(m) ** 3 for L in gram_segments(k, restart))
    return k * (3.0 * m * m * n + float(m) ** 3)


def eq2_work_flops(rows: int, cols: int, k: int = 5) -> float:
    """The NS work of one matrix as the method states it (Eq. 2, symmetry-aware:
    per step m^2 n for X X^T, m^3 for A A and 2 m^2 n for B X), whichever form
    the plan runs; a zero-gradient matrix has none."""
    m, n = min(rows, cols), max(rows, cols)
    return k * (3.0 * m * m * n + float(m) ** 3)


def live_flop_share(plan, k: int, zero) -> dict:
    """(kind, kernel class) -> the share of that launch group's algorithmic
    flops that belongs to matrices with a nonzero gradient.  The library
    counts every matrix of a launch; the tiles of a zero-gradient matrix exit
    before their K loop, so only this share is executed.  Per matrix and step:
    Eq. 2 runs Gram (m^2 n), A*A (m^3) and B*X (2 m^2 n) k times; the Gram-space
    form runs, per segment of L steps, Gram and B*X once, P_i L times and
    3L - 3 symmetric m^3 products."""
    from paper_2606_27153_amd import _lib as L
    tot: dict = {}
    live: dict = {}
    for i in range(plan.n):
        mi = plan.matrix_info(i)
        cls = L.KERNEL_CLASSES[mi["kernel_class"]]
        m, n = float(mi["m"]), float(mi["n"])
        if mi["gram_space"]:
            segs = gram_segments(k, plan.info()["gram_restart"])
            per = {"gram": len(segs) * m * m * n, "poly": k * m ** 3,
                   "symm": sum(3 * L - 3 for L in segs) * m ** 3, "bx": len(segs) * 2 * m * m * n}
        else:
            per = {"gram": k * m * m * n, "poly": k * m ** 3, "symm": 0.0, "bx": k * 2 * m * m * n}
        for kind, f in per.items():
            tot[(kind, cls)] = tot.get((kind, cls), 0.0) + f
            if not zero[i]:
                live[(kind, cls)] = live.get((kind, cls), 0.0) + f
    return {key: (live.get(key, 0.0) / v if v > 0 else 1.0) for key, v in tot.items()}


def measure_peaks(torch, dev, copy_mib: int = 1024, reps: int = 5) -> dict:
    """Rates the same box reaches outside this library, as context for the
    vendor peaks: a device-to-device copy (HBM read + write) and the vendor
    BLAS (torch.bmm, bf16, contiguous operands) on the B*X shape of the 8B
    set's MLP matrices, a full product with no symmetry to exploit."""
    def timed(fn):
        fn()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        b.synchronize()
        return a.elapsed_time(b) / reps * 1e-3
    nb = copy_mib << 20
    src = torch.ones(nb, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    t_copy = timed(lambda: dst.copy_(src))
    del src, dst
    batch, m, n, k = 8, 4096, 14336, 4096
    x = torch.randn(batch, m, k, device=dev, dtype=torch.bfloat16)
    y = torch.randn(batch, k, n, device=dev, dtype=torch.bfloat16)
    z = torch.empty(batch, m, n, device=dev, dtype=torch.bfloat16)
    t_mm = timed(lambda: torch.bmm(x, y, out=z))
    del x, y, z
    ceil = measure_mfma_ceiling(torch, dev, timed)
    return {"hbm_device_copy_gbs": round(2.0 * nb / t_copy / 1e9, 1),
            "bf16_bmm_tflops": round(2.0 * batch * m * n * k / t_mm / 1e12, 1),
            **ceil,
            "what": f"device-to-device copy of {copy_mib} MiB (read + write bytes); torch.bmm bf16 "
                    f"{batch} x ({m}x{k} @ {k}x{n}), the vendor BLAS on the B*X shape; the bf16 matrix-core "
                    f"rate sustained with no global-memory traffic (libmuon_diag.so): MFMAs alone on random "
                    f"operands, with the 256-tile K loop's LDS reads (6 per 8 MFMAs), and on constant operands"}


DIAG_LIB = os.path.join(ROOT, "paper_2606_27153_amd", "libmuon_diag.so")


def measure_mfma_ceiling(torch, dev, timed, blocks: int = 1024, iters: int = 20000) -> dict:
    """Runs the three modes of muon_diag_mfma_ceiling (4 blocks of 8 waves per
    CU) and returns their rates in TFLOP/s."""
    import ctypes
    if not os.path.exists(DIAG_LIB):
        raise RuntimeError(f"{DIAG_LIB} is missing: run __graft_entry__.build() first")
    lib = ctypes.CDLL(DIAG_LIB)
    fn = lib.muon_diag_mfma_ceiling
    fn.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    out = torch.empty(blocks * 512, dtype=torch.float32, device=dev)
    stream = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    rates = {}
    for mode, key, nmfma in ((0, "mfma_bf16_random_tflops", 16), (1, "mfma_bf16_lds_mix_tflops", 8),
                             (2, "mfma_bf16_const_tflops", 16)):
        def launch():
            if fn(blocks, iters, mode, ctypes.c_void_p(out.data_ptr()), stream) != 0:
                raise RuntimeError(f"muon_diag_mfma_ceiling mode {mode} failed")
        t = timed(launch)
        rates[key] = round(blocks * 8 * iters * nmfma * 32768.0 / t / 1e12, 1)
    del out
    return rates


def lpt_partition(costs, n_owners: int):
    """Longest-processing-time assignment: matrices in decreasing cost, each
    to the owner with the least load so far (ties to the lowest rank).
    Returns (owners, loads); owners[r] lists matrix indices in input order."""
    owners = [[] for _ in range(n_owners)]
    loads = [0.0] * n_owners
    for i in sorted(range(len(costs)), key=lambda i: (-costs[i], i)):
        r = min(range(n_owners), key=lambda r: (loads[r], r))
        owners[r].append(i)
        loads[r] += costs[i]
    return [sorted(o) for o in owners], loads


def time_steps(plan, params, grads, moms, kw, warmup: int, steps: int):
    """Runs warmup steps, then times ``steps`` steps as one block (returns ms
    per step) and each step on its own with events on the step's stream
    (returns the per-step list)."""
    import torch
    for _ in range(warmup):
        plan.step(params, grads, moms, **kw)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    stream = kw["stream"]
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(steps):
        plan.step(params, grads, moms, **kw)
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    return (t1 - t0) * 1e3 / steps, [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]


def percentile(vals, q: float) -> float:
    v = sorted(vals)
    if not v:
        return 0.0
    pos = (len(v) - 1) * q
    lo = int(pos)
    hi = min(lo + 1, len(v) - 1)
    return v[lo] + (v[hi] - v[lo]) * (pos - lo)


def batch_sweep(wl, precision: str, gram_min_aspect: float, batches=(1, 2, 4, 8, 16), steps: int = 5) -> str:
    """Per distinct (rows, cols, dtypes) of the set: the step time of a plan
    holding b copies, for each batch size b, and the per-matrix time
    normalised to b = 1 (the measured c_{s,b} of Sec. 3.4)."""
    import dataclasses

    import torch

    from paper_2606_27153_amd.optim import MuonPlan
    from paper_2606_27153_amd.workloads import make_grads, make_state

    shapes = []
    for m in wl.matrices:
        key = (m.rows, m.cols, m.param, m.grad)
        if key not in shapes:
            shapes.append(key)
    dev = "cuda:0"
    lines = [f"# Batch sweep, {wl.key} set, {precision} NS, {wl.ns_steps} NS steps: ms per muon_step over b "
             f"copies of one shape (median of {steps} steps)", "",
             "| rows x cols | b | ms / step | ms / matrix | per-matrix vs b = 1 |", "|---|---|---|---|---|"]
    for rows, cols, pd, gd in shapes:
        base = None
        for b in batches:
            same = [m for m in wl.matrices if (m.rows, m.cols, m.param, m.grad) == (rows, cols, pd, gd)]
            spec = ([m for m in same if not m.zero_grad] or same)[0]   # a matrix that runs the NS chain
            sub = dataclasses.replace(wl, key=f"{rows}x{cols}", description="", matrices=[spec] * b)
            plan = MuonPlan([(rows, cols, pd, gd)] * b, precision=precision, gram_min_aspect=gram_min_aspect)
            params, moms = make_state(torch, sub, dev)
            grads = make_grads(torch, sub, 0, dev)
            kw = dict(lr=wl.lr, momentum=wl.momentum, weight_decay=wl.weight_decay, ns_steps=wl.ns_steps,
                      nesterov=wl.nesterov, workspace=plan.workspace(dev), stream=torch.cuda.current_stream(dev))
            _, per = time_steps(plan, params, grads, moms, kw, 2, steps)
            ms = percentile(per, 0.5)
            base = ms if base is None else base
            lines.append(f"| {rows} x {cols} | {b} | {ms:.3f} | {ms / b:.4f} | {ms / b / base:.3f} |")
            log(f"[sweep] {rows}x{cols} b={b}: {ms:.3f} ms/step")
            plan.close()
            del params, moms, grads, plan
            torch.cuda.empty_cache()
    return "\n".join(lines)


def gemm_algorithmic_bytes(plan, k: int, kind: str, kclass: str, param_bytes) -> float:
    """HBM bytes one muon_step must move for the launches of one GEMM kind and
    kernel class, each operand read once and each output written once:
      Eq. 2, per step:  Gram  read X, write A;  A*A  read A, write B;
                        B*X   read B and X, write X' (on the last step read
                              and write the parameters W instead)
      Gram space:       Gram  read X0, write G (once);  P_i  read G, write P (k times);
                        m^3 products  read two, write one (3 (k - 1) times);
                        B*X   read Q and X0, read and write W (once).
    param_bytes[i] is the element size of matrix i's parameters."""
    from paper_2606_27153_amd import _lib as L
    total = 0.0
    for i in range(plan.n):
        mi = plan.matrix_info(i)
        if L.KERNEL_CLASSES[mi["kernel_class"]] != kclass:
            continue
        m, n = float(mi["m"]), float(mi["n"])
        e = 4.0 if mi["fp32_ns"] else 2.0
        w = 2.0 * param_bytes[i] * m * n
        if mi["gram_space"]:
            per = {"gram": e * (m * n + m * m), "poly": k * 2 * e * m * m, "symm": (k - 1) * 3 * 3 * e * m * m,
                   "bx": e * (m * m + m * n) + w}
        else:
            per = {"gram": k * e * (m * n + m * m), "poly": k * 2 * e * m * m, "symm": 0.0,
                   "bx": k * e * (m * m + m * n) + (k - 1) * e * m * n + w}
        total += per[kind]
    return total


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="8b", choices=["tiny", "1b", "8b", "vla", "moe"])
    ap.add_argument("--precision", default="bf16", choices=["bf16", "fp16", "fp32"])
    ap.add_argument("--wave-bytes", type=int, default=0)
    ap.add_argument("--gram-min-aspect", type=float, default=None,
                    help="Gram-space recurrence (Eq. 4) for matrices with n >= this * m; 0 = Eq. 2 only")
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle time to sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-peaks", action="store_true", help="skip the copy and vendor-BLAS reference rates")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run one device-to-device copy of this size first (HBM counter calibration)")
    ap.add_argument("--rocprof-summary", metavar="DIR", help="summarise rocprofv3 CSV output and exit")
    ap.add_argument("--write-traffic", metavar="KERNELS",
                    help="with --rocprof-summary: write profiles/traffic_summary.txt for these comma-separated "
                         "kernel keys")
    ap.add_argument("--traffic-command", default="", help="command recorded in the traffic summary")
    ap.add_argument("--sweep", action="store_true",
                    help="print the per-shape batch sweep (b = 1, 2, 4, 8, 16) as a table instead of the JSON line")
    ap.add_argument("--owner-share", type=int, default=1, metavar="N",
                    help="time one of N owners' shares of the set (LPT on algorithmic cost): the per-GPU work "
                         "of an N-GPU run, as a diagnostic")
    ap.add_argument("--owner", type=int, default=0, help="which owner's share with --owner-share")
    ap.add_argument("--autotune", action="store_true",
                    help="measure each shape's GEMM tile first (cached on disk, see --tune-cache) and plan with it")
    ap.add_argument("--tune-cache", default=None, help="tile cache file for --autotune")
    ap.add_argument("--graph", action="store_true",
                    help="also time replays of one step captured in a HIP graph (graph_ms_per_step)")
    args = ap.parse_args(argv)

    if args.gram_min_aspect is None:
        from paper_2606_27153_amd.optim import default_gram_min_aspect
        args.gram_min_aspect = default_gram_min_aspect(args.precision)
    if args.rocprof_summary:
        print(rocprof_summary(args.rocprof_summary))
        if args.write_traffic:
            print(write_traffic_summary(args.rocprof_summary, args.write_traffic, args.copy_calibration_mib or 1024,
                                        args.traffic_command))
        return 0

    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the Muon step here runs on one GPU's matrices with no "
              f"collectives; --gpus {args.gpus} is not supported", file=sys.stderr)
        return 2

    import torch

    from paper_2606_27153_amd.optim import MuonPlan
    from paper_2606_27153_amd.workloads import get_workload, make_grads, make_state

    if not torch.cuda.is_available():
        log("bench.py needs a GPU")
        return 1
    dev = "cuda:0"
    wl = get_workload(args.config)
    if args.sweep:
        print(batch_sweep(wl, args.precision, args.gram_min_aspect), flush=True)
        return 0
    share = None
    if args.owner_share > 1:
        import dataclasses
        if not 0 <= args.owner < args.owner_share:
            log("--owner must be in [0, --owner-share)")
            return 2
        costs = [ns_cost(m.rows, m.cols, wl.ns_steps, args.gram_min_aspect) for m in wl.matrices]
        owners, loads = lpt_partition(costs, args.owner_share)
        mine = owners[args.owner]
        share = {"owners": args.owner_share, "owner": args.owner, "matrices": len(mine),
                 "cost_share": round(loads[args.owner] / sum(costs), 4),
                 "imbalance": round(max(loads) / (sum(loads) / len(loads)), 4)}
        wl = dataclasses.replace(wl, key=f"{wl.key}/owner{args.owner}of{args.owner_share}",
                                 description=f"{wl.description}; owner {args.owner} of {args.owner_share} (LPT)",
                                 matrices=[wl.matrices[i] for i in mine])
    log(f"[bench] workload {wl.key}: {wl.description}; {wl.elements() / 1e9:.2f} G elements")
    descs = [(m.rows, m.cols, m.param, m.grad) for m in wl.matrices]
    tuned = None
    if args.autotune:
        from paper_2606_27153_amd.autotune import tune
        t0 = time.perf_counter()
        hints = tune(descs, precision=args.precision, gram_min_aspect=args.gram_min_aspect, ns_steps=wl.ns_steps,
                     cache_path=args.tune_cache)
        descs = [d + (h,) for d, h in zip(descs, hints)]
        tuned = {"seconds": round(time.perf_counter() - t0, 1),
                 "tiles": sorted({f"{min(d[0], d[1])}x{max(d[0], d[1])}:{d[4]}" for d in descs})}
        log(f"[bench] autotune: {tuned}")
    plan = MuonPlan(descs, precision=args.precision, wave_bytes=args.wave_bytes,
                    gram_min_aspect=args.gram_min_aspect)
    info = plan.info()
    log(f"[bench] plan: {info['n_waves']} waves, {info['n_buckets']} buckets, "
        f"{info['launches_per_step']} launches/step at max steps, workspace {info['workspace_bytes'] / 2**30:.2f} GiB")
    if args.copy_calibration_mib > 0:
        nb = args.copy_calibration_mib << 20
        src = torch.ones(nb, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {nb} bytes done")
        del src, dst
    params, moms = make_state(torch, wl, dev)
    grads = make_grads(torch, wl, 0, dev)
    ws = plan.workspace(dev)
    stream = torch.cuda.current_stream(dev)
    kw = dict(lr=wl.lr, momentum=wl.momentum, weight_decay=wl.weight_decay, ns_steps=wl.ns_steps,
              nesterov=wl.nesterov, workspace=ws, stream=stream)
    torch.cuda.synchronize()
    for i in range(args.warmup):
        plan.step(params, grads, moms, **kw)
        torch.cuda.synchronize()
        log(f"[bench] warmup step {i + 1}/{args.warmup} done")

    plan.set_timing(True)
    plan.timing_read(reset=True)
    ms_per_step, per_step = time_steps(plan, params, grads, moms, kw, 0, args.steps)
    plan.set_timing(False)
    stats = plan.timing_read(reset=True)
    log(f"[bench] {args.steps} timed steps: {ms_per_step:.3f} ms/step")
    zero = [m.zero_grad for m in wl.matrices]
    if any(zero):
        flop_share = live_flop_share(plan, wl.ns_steps, zero)
        for s in stats:
            if s["kind"] in GEMM_KINDS:
                s["algo_flops"] *= flop_share.get((s["kind"], s["kernel_class"]), 1.0)

    # fp16 MFMA has the bf16 dense peak
    peak_mm = PEAK_F32_TFLOPS if args.precision == "fp32" else PEAK_BF16_TFLOPS
    per_kernel = []
    for s in sorted(stats, key=lambda s: -s["total_ms"]):
        mean_ms = s["total_ms"] / max(1, s["launches"])
        row = {"kind": s["kind"], "class": s["kernel_class"], "launches_per_step": s["launches"] / args.steps,
               "ms_per_step": round(s["total_ms"] / args.steps, 4), "mean_launch_ms": round(mean_ms, 5)}
        if s["kind"] in GEMM_KINDS and s["total_ms"] > 0:
            row["tflops"] = round(s["algo_flops"] / (s["total_ms"] * 1e-3) / 1e12, 2)
        if s["kind"] in ("momentum", "apply") and s["total_ms"] > 0:
            row["gbs"] = round(s["algo_bytes"] / (s["total_ms"] * 1e-3) / 1e9, 1)
        per_kernel.append(row)
        log(f"[bench]   {json.dumps(row)}")

    gemm = [s for s in stats if s["kind"] in GEMM_KINDS]
    gemm_ms = sum(s["total_ms"] for s in gemm) / args.steps
    gemm_flops = sum(s["algo_flops"] for s in gemm) / args.steps
    ew = [s for s in stats if s["kind"] in ("momentum", "apply")]
    ew_bytes = sum(s["algo_bytes"] for s in ew) / args.steps
    ns_tflops = gemm_flops / (gemm_ms * 1e-3) / 1e12 if gemm_ms > 0 else 0.0
    mfma_util = 100.0 * ns_tflops / peak_mm
    eq2_flops = sum(eq2_work_flops(m.rows, m.cols, wl.ns_steps) for m in wl.matrices if not m.zero_grad)
    eq2_tflops = eq2_flops / (gemm_ms * 1e-3) / 1e12 if gemm_ms > 0 else 0.0

    dom = max(stats, key=lambda s: s["total_ms"])
    dom_key = f"{dom['kind']}:{dom['kernel_class']}"
    dom_mean_s = dom["total_ms"] * 1e-3 / dom["launches"]
    if dom["kind"] in GEMM_KINDS:
        achieved = dom["algo_flops"] / dom["launches"] / dom_mean_s / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak_mm, "unit": "TFLOP/s",
                "frac": round(achieved / peak_mm, 4)}
    else:
        achieved = dom["algo_bytes"] / dom["launches"] / dom_mean_s / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roof["kernel"] = dom_key
    roof["mean_launch_ms"] = round(dom["total_ms"] / dom["launches"], 4)
    traffic = read_traffic(dom_key)
    roof["traffic"] = None if traffic is None else round(traffic)
    if dom["kind"] in GEMM_KINDS:
        launches_per_step = dom["launches"] / args.steps
        alg = gemm_algorithmic_bytes(plan, wl.ns_steps, dom["kind"], dom["kernel_class"],
                                     [2 if m.param == "bf16" else 4 for m in wl.matrices])
        roof["algorithmic_bytes"] = round(alg / launches_per_step)
        roof["flop_per_byte"] = round(dom["algo_flops"] / dom["launches"] / roof["algorithmic_bytes"], 1)
        if traffic is not None:
            roof["traffic_vs_algorithmic"] = round(traffic / roof["algorithmic_bytes"], 2)

    graph_ms = None
    if args.graph:
        # the eager steps above uploaded the pointer table for these buffers,
        # so a step now only enqueues kernels and can be captured
        kw_g = {k: v for k, v in kw.items() if k != "stream"}
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            plan.step(params, grads, moms, **kw_g)
        graph.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            graph.replay()
        torch.cuda.synchronize()
        graph_ms = (time.perf_counter() - t0) * 1e3 / args.steps
        log(f"[bench] {args.steps} graph replays: {graph_ms:.3f} ms/step")
        del graph
    floor_ms = (gemm_flops / (peak_mm * 1e12) + ew_bytes / (PEAK_HBM_GBS * 1e9)) * 1e3
    peaks = None
    if not args.no_peaks and args.copy_calibration_mib == 0:
        peaks = measure_peaks(torch, dev)
        log(f"[bench] measured on this box: {peaks}")
        if roof["bound"] == "mfma" and args.precision != "fp32":
            # the dominant kernel against the vendor BLAS on the same box
            # (box-to-box clock differences move both alike)
            roof["vs_vendor_bf16_bmm"] = round(roof["achieved"] / peaks["bf16_bmm_tflops"], 3)
            roof["vs_measured_mfma_ceiling"] = round(roof["achieved"] / peaks["mfma_bf16_lds_mix_tflops"], 3)
    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the fp64 oracle on a sample of the same set ...")
        cpu = cpu_baseline(wl, args.cpu_budget)
        log(f"[bench] oracle: {cpu}")

    out = {
        "metric": METRIC,
        "value": round(ms_per_step, 3),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"bf16": "bf16", "fp16": "f16", "fp32": "f32"}[args.precision],
        "data": "synthetic",
        "config": {"workload": wl.key, "description": wl.description, "matrices": wl.n,
                   "elements": wl.elements(), "ns_steps": wl.ns_steps,
                   "params": sorted({m.param for m in wl.matrices}), "momentum": "f32",
                   "ns_operands": args.precision, "gram_space_matrices": info["n_gram"],
                   "gram_min_aspect": args.gram_min_aspect, "autotune": tuned, "parallelism": "single GPU"},
        "mfma_util_pct_ns_gemms": round(mfma_util, 2),
        "ns_gemm_tflops": round(ns_tflops, 2),
        "ns_gemm_ms_per_step": round(gemm_ms, 3),
        "ns_eq2_work_tflops": round(eq2_tflops, 2),
        "ns_eq2_work_pct_of_peak": round(100.0 * eq2_tflops / peak_mm, 2),
        "graph_ms_per_step": None if graph_ms is None else round(graph_ms, 3),
        "step_ms_median": round(percentile(per_step, 0.5), 3),
        "step_ms_p10": round(percentile(per_step, 0.1), 3),
        "step_ms_p90": round(percentile(per_step, 0.9), 3),
        "step_roofline_floor_ms": round(floor_ms, 3),
        "step_roofline_frac": round(floor_ms / ms_per_step, 4),
        "roofline": roof,
        "measured_peaks": peaks,
        "cpu_baseline": cpu,
        "owner_share": share,
        "kernels": per_kernel,
    }
    print(json.dumps(out), flush=True)
    plan.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
