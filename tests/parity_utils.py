"""Shared helpers of the GPU parity tests: run the HIP step through the C ABI
and the fp64 oracle side by side on the same seeded inputs.

The oracle runs free: it starts from the same seeded parameters and zero
momentum, takes the same seeded gradients each step, and carries its own
stored state from step to step.  Nothing the HIP path produced is ever fed
to the oracle.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from oracle import muon_ref as R
from paper_2606_27153_amd.optim import MuonPlan
from paper_2606_27153_amd.workloads import Workload, make_grads, make_state

# Bounds of the contract: relative Frobenius error of the orthogonalised
# update per matrix, bf16 NS path and fp32 validation path.  The fp16 path
# has no stated bound; its unit roundoff is 8x smaller than bf16's (2^-11 vs
# 2^-8), and an fp32-accumulate emulation with fp16 stores measured at most
# 3.3e-3 (m = 32, Gram space) and 1.7e-3 for m >= 64, so it is held to 5e-3.
TOL_O = {"bf16": 2e-2, "fp32": 1e-5, "fp16": 5e-3}
# Momentum is one fp32 fused multiply-add per element on both sides.
TOL_M = 1e-6


def to64(t) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def rel(a: np.ndarray, b: np.ndarray) -> float:
    nb = float(np.linalg.norm(b))
    na = float(np.linalg.norm(a - b))
    if nb == 0.0:
        return 0.0 if na == 0.0 else math.inf
    return na / nb


def bf16_ulp(x: np.ndarray) -> np.ndarray:
    """Spacing of the bfloat16 grid at |x| (2^-133 below the normal range)."""
    ax = np.abs(x)
    e = np.floor(np.log2(np.where(ax > 0, ax, 1.0)))
    e = np.maximum(e, -126)
    return np.where(ax > 0, np.ldexp(1.0, (e - 7).astype(np.int64)), np.ldexp(1.0, -133))


@dataclass
class MatrixReport:
    index: int
    step: int
    o_rel: float
    m_rel: float
    w_err: float
    w_bound: float
    zero: bool


@dataclass
class ParityResult:
    reports: List[MatrixReport] = field(default_factory=list)

    def worst(self, attr: str) -> float:
        vals = [getattr(r, attr) for r in self.reports if not r.zero]
        return max(vals) if vals else 0.0


def run_parity(wl: Workload, *, precision: str = "bf16", steps: Optional[int] = None,
               check: Optional[Sequence[int]] = None, ns_steps: Optional[int] = None,
               nesterov: Optional[bool] = None, wave_bytes: int = 0, device: str = "cuda:0",
               plan: Optional[MuonPlan] = None, abc: Optional[Sequence[float]] = None,
               gram_min_aspect: float = 2.0) -> ParityResult:
    """Runs ``steps`` HIP Muon steps over the whole workload and checks the
    matrices in ``check`` against the free-running oracle after every step."""
    steps = wl.steps if steps is None else steps
    ns = wl.ns_steps if ns_steps is None else ns_steps
    nest = wl.nesterov if nesterov is None else nesterov
    check = list(range(wl.n)) if check is None else list(check)
    lr, mu, wd = (float(np.float32(v)) for v in (wl.lr, wl.momentum, wl.weight_decay))
    descs = [(m.rows, m.cols, m.param, m.grad) for m in wl.matrices]
    own_plan = plan is None
    if own_plan:
        plan = MuonPlan(descs, precision=precision, wave_bytes=wave_bytes, abc=abc,
                        gram_min_aspect=gram_min_aspect)
    # the oracle takes the fp32 values the ABI passes (one triple or a schedule)
    if abc is None:
        abc = R.QUINTIC_ABC
    elif len(abc) == 3 and all(np.ndim(v) == 0 for v in abc):
        abc = tuple(float(np.float32(v)) for v in abc)
    else:
        abc = [tuple(float(np.float32(v)) for v in t) for t in abc]
    params, moms = make_state(torch, wl, device)
    torch.cuda.synchronize()
    # oracle state: its own stored values, starting from the same seeded ones
    ow = {i: to64(params[i]) for i in check}
    om = {i: np.zeros((wl.matrices[i].rows, wl.matrices[i].cols)) for i in check}
    res = ParityResult()
    tol = TOL_O[precision]
    for step in range(steps):
        grads = make_grads(torch, wl, step, device)
        outs = [None] * wl.n
        for i in check:
            outs[i] = torch.empty(wl.matrices[i].rows, wl.matrices[i].cols, device=device, dtype=torch.float32)
        plan.step(params, grads, moms, lr=lr, momentum=mu, weight_decay=wd, ns_steps=ns,
                  nesterov=nest, update_out=outs)
        torch.cuda.synchronize()
        for i in check:
            spec = wl.matrices[i]
            g = to64(grads[i])
            ref = R.muon_step_matrix(ow[i], g, om[i], lr=lr, momentum=mu, weight_decay=wd, ns_steps=ns,
                                     nesterov=nest, param_dtype=spec.param, abc=abc)
            o_gpu = to64(outs[i])
            m_gpu = to64(moms[i])
            w_gpu = to64(params[i])
            zero = not np.any(ref["o"])
            o_rel = rel(o_gpu, ref["o"]) if not zero else float(np.max(np.abs(o_gpu)))
            m_rel = rel(m_gpu, ref["m"]) if np.any(ref["m"]) else float(np.max(np.abs(m_gpu)))
            # W: the two sides drift apart by the O error of each step plus at
            # most one rounding step of the stored dtype per element and step.
            w_err = float(np.linalg.norm(w_gpu - ref["w"]))
            s = R.shape_scale(spec.rows, spec.cols)
            if spec.param == "bf16":
                rnd = float(np.linalg.norm(bf16_ulp(ref["w"])))
            else:
                rnd = float(np.linalg.norm(np.abs(ref["w"]) * 2.0 ** -23))
            w_bound = (step + 1) * (lr * s * tol * float(np.linalg.norm(ref["o"])) + rnd)
            res.reports.append(MatrixReport(i, step, o_rel, m_rel, w_err, w_bound, zero))
            ow[i] = ref["w"]
            om[i] = ref["m"]
        del grads, outs
    if own_plan:
        plan.close()
    return res


def assert_parity(res: ParityResult, precision: str, label: str = "") -> None:
    tol = TOL_O[precision]
    for r in res.reports:
        where = f"{label} matrix {r.index} step {r.step}"
        if r.zero:
            assert r.o_rel == 0.0, f"{where}: zero-gradient matrix has nonzero O"
            continue
        assert r.o_rel <= tol, f"{where}: O rel err {r.o_rel:.3e} > {tol}"
        assert r.m_rel <= TOL_M, f"{where}: M rel err {r.m_rel:.3e} > {TOL_M}"
        assert r.w_err <= r.w_bound, f"{where}: W err {r.w_err:.3e} > bound {r.w_bound:.3e}"
