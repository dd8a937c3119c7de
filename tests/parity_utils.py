"""Shared helpers of the GPU parity tests: run the HIP step through the C ABI
and the fp64 oracle side by side on the same seeded inputs.

The oracle runs free: it starts from the same seeded parameters and zero
momentum, takes the same seeded gradients each step, and carries its own
stored state from step to step.  Nothing the HIP path produced is fed to the
free-running oracle.  One check (P4) asks a second question of the oracle's
apply step (Eq. 1): given the parameters the GPU held before the step and the
update O the GPU computed, does the stored result equal the oracle's
round-to-nearest-even of W*(1 - lr*wd) - lr*s*O?  That isolates the apply
from the error of the Newton-Schulz chain, so it can be held to (almost) the
bit.

Checks per matrix and step:
  O      relative Frobenius error against the oracle (the contract bar), and
         the worst 64 x 64 tile: the tile's error over the error the tile
         would carry at the matrix's own RMS of O.  A wrong block, a skipped
         epilogue region (the debug output is NaN-filled before every step)
         or a mask error shows up there, where the matrix norm would hide it.
  M      relative Frobenius error (one fp32 FMA per element on both sides).
  W      P4 as above; plus the free-running drift bound.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

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
# Worst 64 x 64 tile, relative to the matrix's RMS of O (1.5x the matrix bar:
# a tile of 4096 elements averages the rounding noise almost as well as the
# whole matrix; a wrong 32 x 32 block scores about 0.5).
TOL_TILE = {"bf16": 3e-2, "fp32": 1.5e-5, "fp16": 7.5e-3}
TILE = 64
TILE_MIN = 1024
# Momentum is one fp32 fused multiply-add per element on both sides.
TOL_M = 1e-6
# P4: the stored W against the oracle's rounding of the GPU's own update.
# The GPU forms W*decay - lrs*O in fp32, the oracle in fp64, then both round
# once to the stored dtype.  Measured in ulps (fp32) of the larger term, B =
# max(|W*decay|, |lr*s*O|), a relative rounding of 2^-24 on a term is at most
# one such ulp, so the fp32 intermediate is off the fp64 value by at most:
# one for decay = 1 - lr*wd, a half for W*decay, one each for the square root
# and the product in lrs = lr*sqrt(max(1, rows/cols)), and one for the final
# fused multiply-add (the result can reach 2B): 4.5.  The budget delta is 5
# ulps of B.  fp32 W: |W_gpu - exact| <= delta.  bf16 W: the result must be
# the rounding of some value within delta of the exact one, which makes it
# the oracle's own rounding except where the exact value lies within delta
# of a bf16 rounding boundary -- at most 1e-3 of the elements (mostly where
# the two terms cancel and the result is tiny).
P4_BF16_MAX_FRAC = 1e-3


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


def worst_tile(o_gpu: np.ndarray, o_ref: np.ndarray, tile: int = TILE) -> Tuple[float, Tuple[int, int]]:
    """Worst tile x tile block of o_gpu - o_ref: its Frobenius error over
    rms(o_ref) * sqrt(max(elements of the block, TILE_MIN)), and the block's
    (row, col) index.  Edge blocks of a ragged matrix can hold a handful of
    elements, whose rounding noise does not average out; counting them as
    TILE_MIN elements keeps their score on the scale of a full block's (an
    entirely wrong block of 8 elements still scores about 0.09).  Non-finite
    values in o_gpu give +inf at their block."""
    rows, cols = o_ref.shape
    rms = float(np.linalg.norm(o_ref)) / math.sqrt(rows * cols)
    tr, tc = -(-rows // tile), -(-cols // tile)
    d2 = np.zeros((tr * tile, tc * tile))
    cnt = np.zeros((tr * tile, tc * tile))
    diff = o_gpu - o_ref
    d2[:rows, :cols] = np.where(np.isfinite(diff), diff * diff, np.inf)
    cnt[:rows, :cols] = 1.0
    s = d2.reshape(tr, tile, tc, tile).sum(axis=(1, 3))
    n = cnt.reshape(tr, tile, tc, tile).sum(axis=(1, 3))
    if rms == 0.0:
        err = np.where(s == 0.0, 0.0, np.inf)
    else:
        err = np.sqrt(s) / (rms * np.sqrt(np.maximum(n, TILE_MIN)))
    k = int(np.argmax(err))
    return float(err.flat[k]), (k // tc, k % tc)


def _ordered_bits(x: np.ndarray, dtype: str) -> np.ndarray:
    """Stored values as integers that count representable values in order
    (a difference of two is a distance in ulps); +0 and -0 coincide."""
    u = x.astype(np.float32).view(np.uint32).astype(np.int64)
    if dtype == "bf16":
        u = u >> 16
        sign, mag = u >> 15, u & 0x7FFF
    else:
        sign, mag = u >> 31, u & 0x7FFFFFFF
    return np.where(sign == 1, -mag, mag)


def ulp_distance(a: np.ndarray, b: np.ndarray, dtype: str) -> np.ndarray:
    """Distance in units of the stored dtype's grid between stored values a and b."""
    return np.abs(_ordered_bits(a, dtype) - _ordered_bits(b, dtype))


@dataclass
class MatrixReport:
    index: int
    step: int
    o_rel: float
    m_rel: float
    w_err: float
    w_bound: float
    zero: bool
    tile_err: float = 0.0
    tile_at: Tuple[int, int] = (0, 0)
    p4_max_ulp: float = 0.0
    p4_frac: float = 0.0
    p4_outside: int = 0
    param: str = "bf16"
    finite: bool = True


@dataclass
class ParityResult:
    reports: List[MatrixReport] = field(default_factory=list)
    outputs: dict = field(default_factory=dict)   # index -> O_gpu of the last step (keep_outputs)

    def worst(self, attr: str) -> float:
        vals = [getattr(r, attr) for r in self.reports if not r.zero]
        return max(vals) if vals else 0.0

    def worst_report(self, attr: str) -> Optional[MatrixReport]:
        live = [r for r in self.reports if not r.zero]
        return max(live, key=lambda r: getattr(r, attr)) if live else None

    def summary(self) -> str:
        o = self.worst_report("o_rel")
        t = self.worst_report("tile_err")
        s = f"worst O {self.worst('o_rel'):.3e}"
        if o is not None:
            s += f" (matrix {o.index} step {o.step})"
        if t is not None:
            s += f", worst tile {t.tile_err:.3e} (matrix {t.index} step {t.step} tile {t.tile_at})"
        s += f", M {self.worst('m_rel'):.3e}"
        for dt in ("bf16", "f32"):
            rs = [r for r in self.reports if r.param == dt]
            if rs:
                p4 = max(r.p4_max_ulp for r in rs)
                p4f = max(r.p4_frac for r in rs)
                s += f", P4 ({dt} W) differs on {p4f:.2e} of elements, by at most {p4:.3g} ulp"
        return s


def compare_matrix(index: int, step: int, spec, o_gpu: np.ndarray, w_gpu: np.ndarray, m_gpu: np.ndarray,
                   w_prev_gpu: np.ndarray, ref: dict, *, lr: float, wd: float, tol: float) -> MatrixReport:
    """All per-matrix checks of one step (see the module docstring)."""
    finite = bool(np.all(np.isfinite(o_gpu)))
    zero = not np.any(ref["o"])
    if zero:
        o_rel = 0.0 if (finite and not np.any(o_gpu)) else math.inf
        tile_err, tile_at = o_rel, (0, 0)
    else:
        o_rel = rel(o_gpu, ref["o"]) if finite else math.inf
        tile_err, tile_at = worst_tile(o_gpu, ref["o"])
    m_rel = rel(m_gpu, ref["m"]) if np.any(ref["m"]) else float(np.max(np.abs(m_gpu)))
    # free-running drift: the O error of each step plus at most one rounding
    # step of the stored dtype per element and step
    w_err = float(np.linalg.norm(w_gpu - ref["w"]))
    s = R.shape_scale(spec.rows, spec.cols)
    if spec.param == "bf16":
        rnd = float(np.linalg.norm(bf16_ulp(ref["w"])))
    else:
        rnd = float(np.linalg.norm(np.abs(ref["w"]) * 2.0 ** -23))
    w_bound = (step + 1) * (lr * s * tol * float(np.linalg.norm(ref["o"])) + rnd)
    # P4: the oracle's apply of the GPU's own O to the GPU's own previous W
    o_used = np.where(np.isfinite(o_gpu), o_gpu, 0.0)
    exact = R.apply_update(w_prev_gpu, o_used, lr, wd)
    big = np.maximum(np.abs(w_prev_gpu * (1.0 - lr * wd)), np.abs(lr * s * o_used))
    delta = 5.0 * np.ldexp(1.0, np.maximum(np.floor(np.log2(np.where(big > 0, big, 1.0))), -126).astype(np.int64) - 23)
    if spec.param == "bf16":
        near = R.store_round(exact, "bf16")
        inside = (w_gpu >= R.store_round(exact - delta, "bf16")) & (w_gpu <= R.store_round(exact + delta, "bf16"))
        p4_max = float(ulp_distance(w_gpu, near, "bf16").max()) if w_gpu.size else 0.0
        p4_frac = float(np.count_nonzero(w_gpu != near)) / max(1, w_gpu.size)
    else:
        dist = np.abs(w_gpu - exact) / delta
        inside = dist <= 1.0
        p4_max = 5.0 * float(dist.max()) if dist.size else 0.0   # in ulps of the larger term
        p4_frac = float(np.count_nonzero(w_gpu != R.store_round(exact, "f32"))) / max(1, w_gpu.size)
    p4_outside = int(np.count_nonzero(~inside))
    return MatrixReport(index, step, o_rel, m_rel, w_err, w_bound, zero, tile_err, tile_at, p4_max, p4_frac,
                        p4_outside, spec.param, finite)


def run_parity(wl: Workload, *, precision: str = "bf16", steps: Optional[int] = None,
               check: Optional[Sequence[int]] = None, ns_steps: Optional[int] = None,
               nesterov: Optional[bool] = None, wave_bytes: int = 0, device: str = "cuda:0",
               plan: Optional[MuonPlan] = None, abc: Optional[Sequence[float]] = None,
               gram_min_aspect: float = 2.0, grads_fn=None, progress=None,
               keep_outputs: bool = False, check_at=None) -> ParityResult:
    """Runs ``steps`` HIP Muon steps over the whole workload and checks the
    matrices in ``check`` against the free-running oracle after every step.

    ``check_at(step)`` instead names the matrices to check at each step, and
    the oracle is then teacher-forced: it starts each checked step from the
    parameters and momentum the GPU holds before it, so a matrix can be
    checked at any one step without the oracle following it through the
    earlier ones (M is bitwise equal on both sides, and W enters only
    through the decay term).  ``grads_fn(step)`` may replace the workload's
    seeded gradients (a list of device tensors, one per matrix);
    ``progress(msg)`` is called after each step."""
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
    ow = {} if check_at is not None else {i: to64(params[i]) for i in check}
    om = {} if check_at is not None else {i: np.zeros((wl.matrices[i].rows, wl.matrices[i].cols)) for i in check}
    res = ParityResult()
    tol = TOL_O[precision]
    for step in range(steps):
        grads = grads_fn(step) if grads_fn is not None else make_grads(torch, wl, step, device)
        outs = [None] * wl.n
        w_prev = {}
        if check_at is not None:
            check = list(check_at(step))
            for i in check:   # teacher forcing: the oracle starts from the GPU's state
                ow[i] = to64(params[i])
                om[i] = to64(moms[i])
        for i in check:
            # NaN-filled, so that any element the step fails to write shows
            outs[i] = torch.full((wl.matrices[i].rows, wl.matrices[i].cols), float("nan"), device=device,
                                 dtype=torch.float32)
            w_prev[i] = to64(params[i])
        plan.step(params, grads, moms, lr=lr, momentum=mu, weight_decay=wd, ns_steps=ns,
                  nesterov=nest, update_out=outs)
        torch.cuda.synchronize()
        for i in check:
            spec = wl.matrices[i]
            g = to64(grads[i])
            ref = R.muon_step_matrix(ow[i], g, om[i], lr=lr, momentum=mu, weight_decay=wd, ns_steps=ns,
                                     nesterov=nest, param_dtype=spec.param, abc=abc)
            o_gpu = to64(outs[i])
            res.reports.append(compare_matrix(i, step, spec, o_gpu, to64(params[i]), to64(moms[i]),
                                              w_prev[i], ref, lr=lr, wd=wd, tol=tol))
            if keep_outputs:
                res.outputs[i] = (o_gpu, ref["o"])
            ow[i] = ref["w"]
            om[i] = ref["m"]
        del grads, outs
        if progress is not None:
            progress(f"step {step + 1}/{steps} checked ({len(check)} matrices)")
    if own_plan:
        plan.close()
    return res


def assert_parity(res: ParityResult, precision: str, label: str = "", *, tol: Optional[float] = None,
                  tile_tol: Optional[float] = None) -> None:
    tol = TOL_O[precision] if tol is None else tol
    tile_tol = TOL_TILE[precision] if tile_tol is None else tile_tol
    for r in res.reports:
        where = f"{label} matrix {r.index} step {r.step}"
        assert r.finite, f"{where}: O has non-finite elements (unwritten or NaN)"
        if r.zero:
            assert r.o_rel == 0.0, f"{where}: zero-gradient matrix has nonzero O"
        else:
            assert r.o_rel <= tol, f"{where}: O rel err {r.o_rel:.3e} > {tol}"
            assert r.tile_err <= tile_tol, f"{where}: tile {r.tile_at} err {r.tile_err:.3e} > {tile_tol}"
            assert r.m_rel <= TOL_M, f"{where}: M rel err {r.m_rel:.3e} > {TOL_M}"
            assert r.w_err <= r.w_bound, f"{where}: W err {r.w_err:.3e} > bound {r.w_bound:.3e}"
        assert r.p4_outside == 0, \
            f"{where}: W is not RNE(W_prev*decay - lr*s*O_gpu) on {r.p4_outside} elements (up to {r.p4_max_ulp:.3g} ulp)"
        if r.param == "bf16":
            assert r.p4_frac <= P4_BF16_MAX_FRAC, \
                f"{where}: W differs from RNE(W_prev*decay - lr*s*O_gpu) on {r.p4_frac:.2e} of elements"
