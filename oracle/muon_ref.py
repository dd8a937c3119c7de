"""fp64 reference for one Muon optimizer step over a set of weight matrices.

TEST INFRASTRUCTURE ONLY.  This module is the oracle the HIP path is checked
against.  Nothing on the product path may import or call it: only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` use it.
It shares no kernels, headers, helpers, tables or pre/post-processing with the
HIP library, and it never reads anything the HIP path produced.

What is computed, per matrix (DMuon, Sec. 2.1, Eq. 1 and Eq. 2):

  1. momentum:   M <- mu*M + G ; Nesterov input u = G + mu*M  (else u = M)
  2. orient:     X = u^T if rows > cols (so X is m x n with m <= n)
  3. normalise:  X0 = X / (||X||_F + eps)
  4. Eq. 2, k times:  A = X X^T ; B = b*A + c*A A ; X <- a*X + B X
     (this is X <- aX + bXX^TX + c(XX^T)^2 X regrouped; the paper leaves
     (a,b,c) open, the quintic set used is (3.4445, -4.7750, 2.0315)).  A
     schedule of one (a_i, b_i, c_i) per step may replace the fixed triple
     (Sec. 4, "Configurations": the paper's default is a per-step set):
     step i then uses its own triple.
  5. O = X^T if transposed else X
  6. Eq. 1 with decoupled weight decay and the shape scale:
        W <- W*(1 - lr*wd) - lr*sqrt(max(1, rows/cols))*O

Readings taken where the paper is silent (momentum form, eps, shape scale,
decay form, orientation) are listed in the design notes of the repository.

Pins (tests/test_oracle_pins.py): SVD closed form U p^{ok}(s/||s||) V^T
(and U (p_{k-1} o ... o p_0)(s/||s||) V^T for a per-step schedule, with
hand-computed 1 x 1 values that fix the order),
transpose / sign / scale / orthogonal equivariance, rank-1 closed form,
2x2 and 3x3 brute force against numpy.linalg.svd, the Gram-space identity of
Eq. 4, the momentum closed form under constant gradients, the apply special
cases, and the bf16 rounding against torch's conversion.

Every floating-point operation is fp64.  Narrowing to the stored dtype is a
single round-to-nearest-even from the fp64 value.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "QUINTIC_ABC",
    "step_coefficients",
    "DEFAULT_EPS",
    "bf16_round",
    "f32_round",
    "store_round",
    "momentum_update",
    "newton_schulz",
    "newton_schulz_gram",
    "orthogonalize",
    "shape_scale",
    "apply_update",
    "muon_step_matrix",
    "muon_step",
    "ns_flops",
]

# Quintic coefficients of the Newton-Schulz step (Eq. 2).  The paper names
# (a, b, c) without fixing values; this is the standard quintic set.
QUINTIC_ABC = (3.4445, -4.7750, 2.0315)

# Guard added to the Frobenius norm before dividing (not given in the paper).
DEFAULT_EPS = 1e-7


# --------------------------------------------------------------------------
# Narrowing stores
# --------------------------------------------------------------------------

def f32_round(x):
    """Round fp64 values to the nearest fp32 value (ties to even), as fp64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def bf16_round(x):
    """Round fp64 values to the nearest bfloat16 value (ties to even), as fp64.

    bfloat16 keeps fp32's 8 exponent bits and 8 significant bits (7 stored).
    Normal numbers: the spacing in [2^e, 2^(e+1)) is 2^(e-7).  Below the
    smallest normal 2^-126 the spacing is fixed at 2^-133 (subnormals).
    Values whose rounded magnitude reaches 2^128 become +-inf.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.array(x, dtype=np.float64, copy=True)
    finite = np.isfinite(x) & (x != 0.0)
    xf = x[finite]
    _, e = np.frexp(xf)             # xf = f * 2**e with 0.5 <= |f| < 1
    e = e - 1                       # now |xf| in [2**e, 2**(e+1))
    e = np.maximum(e, -126)         # subnormal range shares the 2^-133 step
    step = np.ldexp(1.0, e - 7)
    r = np.rint(xf / step) * step   # np.rint rounds half to even
    r[np.abs(r) >= 2.0 ** 128] = np.inf * np.sign(r[np.abs(r) >= 2.0 ** 128])
    out[finite] = r
    return out


def store_round(x, dtype: str):
    """Narrow fp64 values to the stored dtype ('f32' or 'bf16')."""
    if dtype == "f32":
        return f32_round(x)
    if dtype == "bf16":
        return bf16_round(x)
    raise ValueError(f"unknown dtype {dtype!r}")


# --------------------------------------------------------------------------
# The step
# --------------------------------------------------------------------------

def momentum_update(m, g, mu: float, nesterov: bool = True):
    """Momentum-smoothed gradient fed to Newton-Schulz (M_t of Sec. 2.1).

    Heavy-ball accumulation M <- mu*M + G; with Nesterov the NS input is the
    look-ahead u = G + mu*M (using the updated M), otherwise u = M.
    Returns (M_new, u), both fp64 and unrounded.
    """
    m = np.asarray(m, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    m_new = mu * m + g
    u = g + mu * m_new if nesterov else m_new.copy()
    return m_new, u


def step_coefficients(abc, steps: int):
    """The (a, b, c) of each of ``steps`` NS steps.

    ``abc`` is either one triple, used for every step, or a schedule of at
    least ``steps`` triples, step i taking the i-th (Sec. 4,
    "Configurations").
    """
    seq = list(abc)
    if len(seq) == 3 and all(np.ndim(v) == 0 for v in seq):
        return [tuple(float(v) for v in seq)] * int(steps)
    if len(seq) < int(steps):
        raise ValueError("coefficient schedule shorter than the step count")
    out = []
    for t in seq[:int(steps)]:
        a, b, c = (float(v) for v in t)
        out.append((a, b, c))
    return out


def newton_schulz(x, steps: int, abc=QUINTIC_ABC):
    """k steps of the quintic Newton-Schulz iteration (Eq. 2) on an m x n X.

    Each step forms the Gram matrix A = X X^T, the polynomial part
    B = b*A + c*A*A, and X <- a*X + B*X, which equals
    a*X + b*X X^T X + c*(X X^T)^2 X.  X is used as given (no orientation,
    no normalisation).  ``abc`` is a triple or a per-step schedule.
    """
    x = np.array(x, dtype=np.float64, copy=True)
    for a, b, c in step_coefficients(abc, steps):
        gram = x @ x.T
        poly = b * gram + c * (gram @ gram)
        x = a * x + poly @ x
    return x


def newton_schulz_gram(x, steps: int, abc=QUINTIC_ABC, restart=None):
    """The same iteration carried in Gram space (Eq. 4).

    With G_0 = X_0 X_0^T and P_i = a I + b G_i + c G_i^2, the Gram matrix
    obeys G_{i+1} = P_i G_i P_i and X_k = P_{k-1} ... P_0 X_0.  In exact
    arithmetic this equals ``newton_schulz``.  With a per-step schedule, P_i
    takes step i's (a_i, b_i, c_i).  ``restart`` (a step count, or None for
    never) ends a segment after that many steps: X_j = P_{j-1} ... X_0 is
    formed and the recurrence starts again from G = X_j X_j^T -- in exact
    arithmetic the same G_j, so the result is unchanged.
    """
    x = np.asarray(x, dtype=np.float64)
    m = x.shape[0]
    eye = np.eye(m)
    coefs = step_coefficients(abc, steps)
    seg = len(coefs) if restart is None else int(restart)
    for s0 in range(0, len(coefs), max(1, seg)):
        gram = x @ x.T
        q = eye.copy()
        for a, b, c in coefs[s0:s0 + seg]:
            p = a * eye + b * gram + c * (gram @ gram)
            gram = p @ gram @ p
            q = p @ q
        x = q @ x
    return x


def orthogonalize(u, steps: int, abc=QUINTIC_ABC, eps: float = DEFAULT_EPS):
    """NS_k of Eq. 1: orient, Frobenius-normalise, iterate, un-orient.

    A tall input (rows > cols) is transposed so the Gram matrix is the
    smaller min(rows, cols)^2 one; the result is transposed back.  An
    all-zero input returns exact zeros.
    """
    u = np.asarray(u, dtype=np.float64)
    if u.ndim != 2:
        raise ValueError("orthogonalize expects a matrix")
    rows, cols = u.shape
    transposed = rows > cols
    x = u.T if transposed else u
    ss = float(np.sum(x * x))
    if ss == 0.0:
        return np.zeros_like(u)
    x = x / (math.sqrt(ss) + eps)
    x = newton_schulz(x, steps, abc)
    return x.T if transposed else x


def shape_scale(rows: int, cols: int) -> float:
    """Update scale sqrt(max(1, rows/cols)) on the stored (rows, cols) shape."""
    return math.sqrt(max(1.0, rows / cols))


def apply_update(w, o, lr: float, weight_decay: float):
    """Eq. 1 with decoupled, lr-multiplied weight decay and the shape scale."""
    w = np.asarray(w, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    rows, cols = w.shape
    return w * (1.0 - lr * weight_decay) - lr * shape_scale(rows, cols) * o


def muon_step_matrix(w, g, m, *, lr, momentum, weight_decay, ns_steps,
                     nesterov=True, abc=QUINTIC_ABC, eps=DEFAULT_EPS,
                     param_dtype="f32", momentum_dtype="f32"):
    """One Muon step for one matrix.

    ``w``, ``g``, ``m`` are the stored values (already exact in fp64).
    Returns a dict with the stored results ``w`` and ``m`` (narrowed to their
    dtypes), the unrounded fp64 ``w_exact`` and ``m_exact``, and ``o`` (the
    orthogonalised update before lr and shape scale).
    """
    m_new, u = momentum_update(m, g, momentum, nesterov)
    o = orthogonalize(u, ns_steps, abc, eps)
    w_new = apply_update(w, o, lr, weight_decay)
    return {
        "w": store_round(w_new, param_dtype),
        "m": store_round(m_new, momentum_dtype),
        "w_exact": w_new,
        "m_exact": m_new,
        "o": o,
    }


def muon_step(params, grads, moms, *, lr, momentum, weight_decay, ns_steps,
              nesterov=True, abc=QUINTIC_ABC, eps=DEFAULT_EPS,
              param_dtypes=None, momentum_dtype="f32"):
    """One Muon step over a list of matrices; matrices are independent."""
    n = len(params)
    if param_dtypes is None:
        param_dtypes = ["f32"] * n
    out = []
    for i in range(n):
        out.append(muon_step_matrix(
            params[i], grads[i], moms[i], lr=lr, momentum=momentum,
            weight_decay=weight_decay, ns_steps=ns_steps, nesterov=nesterov,
            abc=abc, eps=eps, param_dtype=param_dtypes[i],
            momentum_dtype=momentum_dtype))
    return out


def ns_flops(rows: int, cols: int, steps: int = 5) -> int:
    """Symmetry-aware algorithmic flops of k NS steps on one matrix.

    Per step: half of the 2 m^2 n Gram product, half of the 2 m^3 A*A
    product, and the full 2 m^2 n B*X product: 3 m^2 n + m^3.
    """
    m, n = min(rows, cols), max(rows, cols)
    return int(steps) * (3 * m * m * n + m ** 3)
