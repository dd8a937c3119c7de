"""Pins for the fp64 oracle: checks against what the mathematics fixes.

None of these re-types the oracle's iteration.  They compare it with the SVD
closed form of Eq. 2 (each step maps a singular value x to
p(x) = a x + b x^3 + c x^5), with brute force through numpy.linalg.svd, with
the Gram-space recurrence of Eq. 4, with symmetry invariants, with the
closed form of the momentum recurrence under a constant gradient, and with
torch's own bfloat16 conversion.  The last test plants mistakes in copies of
the oracle and shows the pins catch each one.
"""
import math
import os

import numpy as np
import pytest

from oracle import muon_ref as R

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "scalar_map.txt")
ABC = R.QUINTIC_ABC


def _golden():
    vals = {"compose": {}, "fixed_point": []}
    with open(GOLDEN) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            parts = line.split()
            if parts[0] == "compose":
                vals["compose"][int(parts[1])] = float(parts[2])
            elif parts[0] == "fixed_point":
                vals["fixed_point"].append(float(parts[1]))
            else:
                vals[parts[0]] = float(parts[1])
    return vals


def _p(x):
    a, b, c = ABC
    return a * x + b * x ** 3 + c * x ** 5


def _pk(x, k):
    for _ in range(k):
        x = _p(x)
    return x


def _orthonormal(rng, n, k):
    q, r = np.linalg.qr(rng.standard_normal((n, k)))
    return q * np.sign(np.diag(r))


def _svd_input(rng, rows, cols, svals):
    r = len(svals)
    u = _orthonormal(rng, rows, r)
    v = _orthonormal(rng, cols, r)
    return u, np.asarray(svals, dtype=np.float64), v


def _rel(a, b):
    return np.linalg.norm(a - b) / np.linalg.norm(b)


# ---------------------------------------------------------------- golden

def test_golden_scalar_map_by_hand():
    g = _golden()
    # p(1) = a + b + c = 3.4445 - 4.7750 + 2.0315 = 0.701 (hand arithmetic)
    assert abs(g["compose"][1] - 0.701) < 1e-15
    assert abs(_pk(1.0, 5) - g["compose"][5]) < 1e-13
    for fp in g["fixed_point"]:
        assert abs(_p(fp) - fp) < 1e-13
    assert abs(g["derivative_at_1"] - (-0.723)) < 1e-15


# ---------------------------------------------------------------- closed forms

@pytest.mark.parametrize("rows,cols", [(6, 11), (11, 6), (9, 9), (1, 7), (7, 1), (16, 40)])
@pytest.mark.parametrize("k", [0, 1, 2, 5])
def test_svd_closed_form(rows, cols, k):
    rng = np.random.default_rng(rows * 100 + cols + k)
    r = min(rows, cols)
    s = rng.uniform(0.05, 3.0, size=r)
    u, s, v = _svd_input(rng, rows, cols, s)
    g = (u * s) @ v.T
    got = R.orthogonalize(g, k, ABC, eps=0.0)
    want = (u * _pk(s / np.linalg.norm(s), k)) @ v.T
    assert _rel(got, want) < 1e-12


def test_svd_closed_form_with_eps():
    rng = np.random.default_rng(3)
    u, s, v = _svd_input(rng, 12, 30, rng.uniform(0.1, 1.0, size=12))
    g = (u * s) @ v.T
    got = R.orthogonalize(g, 5, ABC)           # default eps
    want = (u * _pk(s / np.linalg.norm(s), 5)) @ v.T
    assert _rel(got, want) < 1e-6


def test_rank_one_closed_form():
    g = _golden()
    rng = np.random.default_rng(7)
    for rows, cols in [(5, 8), (8, 5), (1, 1), (13, 13)]:
        a = rng.standard_normal(rows)
        b = rng.standard_normal(cols)
        got = R.orthogonalize(np.outer(a, b), 5, ABC, eps=0.0)
        want = g["compose"][5] * np.outer(a, b) / (np.linalg.norm(a) * np.linalg.norm(b))
        assert np.max(np.abs(got - want)) < 1e-13


def test_one_by_one():
    g = _golden()
    for x in [3.7, -0.002, 1e-30]:
        got = R.orthogonalize(np.array([[x]]), 5, ABC, eps=0.0)
        assert abs(got[0, 0] - math.copysign(g["compose"][5], x)) < 1e-14


@pytest.mark.parametrize("n", [2, 3])
def test_brute_force_small(n):
    rng = np.random.default_rng(11 + n)
    for trial in range(50):
        rows = n
        cols = n + int(rng.integers(0, 2))
        if trial % 2:
            rows, cols = cols, rows
        g = rng.standard_normal((rows, cols))
        u, s, vt = np.linalg.svd(g, full_matrices=False)
        want = (u * _pk(s / np.linalg.norm(s), 5)) @ vt
        got = R.orthogonalize(g, 5, ABC, eps=0.0)
        assert np.max(np.abs(got - want)) < 1e-12


def test_rank_deficient_keeps_zero_singular_values():
    rng = np.random.default_rng(5)
    u, s, v = _svd_input(rng, 10, 25, [2.0, 1.0, 0.5, 0.0, 0.0])
    got = R.orthogonalize((u * s) @ v.T, 5, ABC, eps=0.0)
    sv = np.linalg.svd(got, compute_uv=False)
    assert np.all(sv[3:] < 1e-12)
    np.testing.assert_allclose(sv[:3], np.sort(_pk(s[:3] / np.linalg.norm(s), 5))[::-1], atol=1e-12)


def test_zero_steps_is_normalised_input():
    rng = np.random.default_rng(2)
    g = rng.standard_normal((7, 19))
    got = R.orthogonalize(g, 0, ABC, eps=0.0)
    assert np.max(np.abs(got - g / np.sqrt(np.sum(g * g)))) < 1e-15


def test_zero_matrix_gives_zero():
    assert np.all(R.orthogonalize(np.zeros((4, 9)), 5) == 0.0)
    assert np.all(R.orthogonalize(np.zeros((9, 4)), 5) == 0.0)


# ---------------------------------------------------------------- invariants

def test_transpose_equivariance():
    rng = np.random.default_rng(1)
    for rows, cols in [(8, 21), (21, 8), (3, 64)]:
        g = rng.standard_normal((rows, cols))
        a = R.orthogonalize(g.T, 5)
        b = R.orthogonalize(g, 5).T
        assert np.array_equal(a, b)        # orientation makes it exact
    g = rng.standard_normal((12, 12))
    assert np.max(np.abs(R.orthogonalize(g.T, 5) - R.orthogonalize(g, 5).T)) < 1e-12


def test_odd_and_scale_invariance():
    rng = np.random.default_rng(4)
    g = rng.standard_normal((9, 30))
    base = R.orthogonalize(g, 5, eps=0.0)
    assert np.array_equal(R.orthogonalize(-g, 5, eps=0.0), -base)
    for alpha in [1e-4, 0.3, 250.0]:
        assert np.max(np.abs(R.orthogonalize(alpha * g, 5, eps=0.0) - base)) < 1e-12


def test_orthogonal_equivariance():
    rng = np.random.default_rng(6)
    g = rng.standard_normal((10, 17))
    q1 = _orthonormal(rng, 10, 10)
    q2 = _orthonormal(rng, 17, 17)
    lhs = R.orthogonalize(q1 @ g @ q2, 5, eps=0.0)
    rhs = q1 @ R.orthogonalize(g, 5, eps=0.0) @ q2
    assert np.max(np.abs(lhs - rhs)) < 1e-12


# ---------------------------------------------------------------- per-step schedules
# Sec. 4 ("Configurations"): a schedule gives each NS step its own (a, b, c).
# Step i then maps a singular value x to p_i(x), so k steps apply the
# composition p_{k-1} o ... o p_0, in that order.

CLASSIC = (15 / 8, -10 / 8, 3 / 8)   # the textbook quintic, p(1) = 1
CUBIC = (1.5, -0.5, 0.0)             # Newton-Schulz cubic, p(1) = 1
SCHEDULE = [ABC, ABC, CLASSIC, CUBIC, CLASSIC]


def _p_of(t, x):
    a, b, c = t
    return a * x + b * x ** 3 + c * x ** 5


def _compose(schedule, x):
    for t in schedule:
        x = _p_of(t, x)
    return x


def test_schedule_worked_values_by_hand():
    # 1 x 1 inputs normalise to +-1.  cubic then quintic: p_c(1) = 1.5 - 0.5
    # = 1, then p(1) = 0.701.  quintic then cubic: p(1) = 0.701, then
    # 1.5 * 0.701 - 0.5 * 0.701^3 = 1.0515 - 0.5 * 0.344472101 = 0.8792639495.
    got = R.orthogonalize(np.array([[2.5]]), 2, [CUBIC, ABC], eps=0.0)[0, 0]
    assert abs(got - 0.701) < 1e-14
    got = R.orthogonalize(np.array([[-0.3]]), 2, [ABC, CUBIC], eps=0.0)[0, 0]
    assert abs(got + 0.8792639495) < 1e-12


@pytest.mark.parametrize("rows,cols", [(6, 11), (11, 6), (9, 9), (16, 40)])
def test_schedule_svd_closed_form(rows, cols):
    rng = np.random.default_rng(rows * 31 + cols)
    u, s, v = _svd_input(rng, rows, cols, rng.uniform(0.05, 3.0, size=min(rows, cols)))
    g = (u * s) @ v.T
    for k in (1, 3, 5):
        got = R.orthogonalize(g, k, SCHEDULE, eps=0.0)
        want = (u * _compose(SCHEDULE[:k], s / np.linalg.norm(s))) @ v.T
        assert _rel(got, want) < 1e-12
    # the order matters: the reversed schedule is a different map
    rev = R.orthogonalize(g, 5, SCHEDULE[::-1], eps=0.0)
    assert _rel(rev, R.orthogonalize(g, 5, SCHEDULE, eps=0.0)) > 1e-3


def test_schedule_of_one_triple_is_the_fixed_iteration():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((7, 19))
    assert np.array_equal(R.orthogonalize(x, 5, [ABC] * 5), R.orthogonalize(x, 5, ABC))
    # a longer schedule uses only its first k triples
    assert np.array_equal(R.orthogonalize(x, 3, SCHEDULE), R.orthogonalize(x, 3, SCHEDULE[:3]))
    with pytest.raises(ValueError):
        R.orthogonalize(x, 6, SCHEDULE)


def test_gram_space_identity_with_schedule():
    rng = np.random.default_rng(9)
    for rows, cols in [(6, 40), (12, 30)]:
        x = rng.standard_normal((rows, cols))
        x /= np.linalg.norm(x)
        assert _rel(R.newton_schulz_gram(x, 5, SCHEDULE), R.newton_schulz(x, 5, SCHEDULE)) < 1e-11


def test_pins_catch_schedule_taken_in_reverse(monkeypatch):
    orig = R.step_coefficients

    def reversed_schedule(abc, steps):
        return orig(abc, steps)[::-1]
    monkeypatch.setattr(R, "step_coefficients", reversed_schedule)
    rng = np.random.default_rng(6 * 31 + 11)
    u, s, v = _svd_input(rng, 6, 11, rng.uniform(0.05, 3.0, size=6))
    g = (u * s) @ v.T
    got = R.orthogonalize(g, 5, SCHEDULE, eps=0.0)
    want = (u * _compose(SCHEDULE, s / np.linalg.norm(s))) @ v.T
    assert not _rel(got, want) < 1e-6


def test_gram_space_identity():
    rng = np.random.default_rng(8)
    for rows, cols in [(6, 40), (16, 16), (20, 33)]:
        x = rng.standard_normal((rows, cols))
        x /= np.linalg.norm(x)
        a = R.newton_schulz(x, 5)
        for restart in (None, 1, 2, 3):
            b = R.newton_schulz_gram(x, 5, restart=restart)
            assert _rel(b, a) < 1e-11, restart


def test_gram_space_restart_matches_the_svd_map():
    # restarted segments on a known spectrum: still U p^{o5}(s) V^T
    rng = np.random.default_rng(10)
    u, _ = np.linalg.qr(rng.standard_normal((12, 12)))
    v, _ = np.linalg.qr(rng.standard_normal((30, 12)))
    s = np.logspace(0, -2, 12)
    s /= np.linalg.norm(s)
    x = (u * s) @ v.T
    want = (u * _pk(s, 5)) @ v.T
    for restart in (1, 2, 4):
        assert _rel(R.newton_schulz_gram(x, 5, restart=restart), want) < 1e-11


# ---------------------------------------------------------------- momentum / apply

def test_momentum_closed_form_constant_gradient():
    rng = np.random.default_rng(9)
    g = rng.standard_normal((5, 6))
    mu = 0.95
    m = np.zeros_like(g)
    for t in range(1, 8):
        m, u = R.momentum_update(m, g, mu, nesterov=True)
        geo = (1 - mu ** t) / (1 - mu)
        np.testing.assert_allclose(m, geo * g, rtol=1e-13)
        np.testing.assert_allclose(u, g + mu * geo * g, rtol=1e-13)
        m_plain, u_plain = R.momentum_update(m, g, mu, nesterov=False)
        np.testing.assert_array_equal(u_plain, m_plain)


def test_first_step_nesterov_from_zero_is_scaled_gradient():
    g = np.arange(12.0).reshape(3, 4) - 5
    m, u = R.momentum_update(np.zeros_like(g), g, 0.95, nesterov=True)
    np.testing.assert_array_equal(m, g)
    np.testing.assert_allclose(u, 1.95 * g, rtol=1e-15)


def test_apply_special_cases():
    rng = np.random.default_rng(10)
    w = rng.standard_normal((6, 4))
    o = rng.standard_normal((6, 4))
    np.testing.assert_array_equal(R.apply_update(w, o, 0.0, 0.1), w)
    np.testing.assert_allclose(R.apply_update(w, np.zeros_like(w), 0.02, 0.01), w * (1 - 2e-4), rtol=1e-15)


@pytest.mark.parametrize("rows,cols", [(64, 16), (16, 64), (24, 24), (1024, 256)])
def test_apply_shape_scale_spectral(rows, cols):
    # with lambda = 0 and O having all singular values 1, ||dW||_2 = lr*sqrt(max(1, rows/cols))
    rng = np.random.default_rng(rows + cols)
    r = min(rows, cols)
    o = _orthonormal(rng, rows, r) @ _orthonormal(rng, cols, r).T
    lr = 0.02
    dw = R.apply_update(np.zeros((rows, cols)), o, lr, 0.0)
    assert abs(np.linalg.norm(dw, 2) - lr * math.sqrt(max(1.0, rows / cols))) < 1e-14


def test_full_step_closed_form():
    rng = np.random.default_rng(12)
    rows, cols = 24, 10
    u, s, v = _svd_input(rng, rows, cols, rng.uniform(0.2, 2.0, size=10))
    g = (u * s) @ v.T
    w = rng.standard_normal((rows, cols)) * 0.02
    lr, mu, wd = 0.02, 0.95, 0.01
    out = R.muon_step_matrix(w, g, np.zeros_like(g), lr=lr, momentum=mu, weight_decay=wd,
                             ns_steps=5, eps=0.0)
    o = (u * _pk(s / np.linalg.norm(s), 5)) @ v.T
    want = w * (1 - lr * wd) - lr * math.sqrt(rows / cols) * o
    assert np.max(np.abs(out["w_exact"] - want)) < 1e-13
    np.testing.assert_array_equal(out["m_exact"], g)


# ---------------------------------------------------------------- narrowing

def test_bf16_round_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(13)
    bits = rng.integers(0, 2 ** 32, size=200000, dtype=np.uint64).astype(np.uint32)
    x32 = bits.view(np.float32)
    x32 = x32[np.isfinite(x32)]
    extra = np.array([0.0, -0.0, 1.0, 1.00390625, 1.005859375, 3.0e38, -3.3e38, 1e-40, -1e-45,
                      1.1754944e-38, 9.1835e-41], dtype=np.float32)
    x32 = np.concatenate([x32, extra])
    want = torch.from_numpy(x32.copy()).to(torch.bfloat16).to(torch.float64).numpy()
    got = R.bf16_round(x32.astype(np.float64))
    assert np.array_equal(np.isinf(got), np.isinf(want))
    fin = np.isfinite(want)
    assert np.array_equal(got[fin], want[fin])


def test_bf16_round_ties_to_even():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties go to the even 1.0
    assert R.bf16_round(np.array([1.0 + 2.0 ** -8]))[0] == 1.0
    assert R.bf16_round(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6


def _f32_from_bits(bits):
    return np.asarray(bits, dtype=np.uint32).view(np.float32).astype(np.float64)


def test_f32_round_halfway_cases_from_the_grid():
    # Neighbouring fp32 values lo < hi are built from their bit patterns
    # (normal and subnormal, both signs); the fp64 midpoint of each pair is
    # exact.  Round-to-nearest-even sends the midpoint to the one whose last
    # significand bit is 0, and anything off the midpoint by a quarter step to
    # the nearer one.  A truncating or ties-away narrowing fails here.
    rng = np.random.default_rng(17)
    mags = np.concatenate([rng.integers(1 << 23, 0x7F7FFFFF, size=4000),   # normal
                           rng.integers(1, 1 << 23, size=1000),            # subnormal
                           [1, (1 << 23) - 1, 1 << 23, 0x3F800000, 0x7F7FFFFE]]).astype(np.uint64)
    for sign in (0, 1 << 31):
        lo_bits = mags | np.uint64(sign)
        lo = _f32_from_bits(lo_bits)
        hi = _f32_from_bits(lo_bits + np.uint64(1))   # next magnitude, same sign
        mid = (lo + hi) / 2.0
        even = np.where((mags & np.uint64(1)) == 0, lo, hi)
        assert np.array_equal(R.f32_round(mid), even)
        quarter = (hi - lo) / 4.0
        assert np.array_equal(R.f32_round(mid - quarter), lo)
        assert np.array_equal(R.f32_round(mid + quarter), hi)
        assert np.array_equal(R.f32_round(lo), lo) and np.array_equal(R.f32_round(hi), hi)


def test_f32_round_range_ends():
    top = _f32_from_bits(0x7F7FFFFF)           # largest finite fp32
    half_ulp = 2.0 ** (127 - 24)
    with np.errstate(over="ignore"):
        assert R.f32_round(np.array([top + 0.5 * half_ulp]))[0] == top
        # the midpoint between the largest finite and 2^128 rounds to even: inf
        assert np.isposinf(R.f32_round(np.array([top + half_ulp]))[0])
        assert np.isneginf(R.f32_round(np.array([-(top + half_ulp)]))[0])
    tiny = 2.0 ** -149                         # smallest subnormal
    assert R.f32_round(np.array([0.5 * tiny]))[0] == 0.0          # tie to the even 0
    assert R.f32_round(np.array([0.75 * tiny]))[0] == tiny
    assert R.f32_round(np.array([1.5 * tiny]))[0] == 2 * tiny     # tie to the even 2
    assert R.f32_round(np.array([-0.0]))[0] == 0.0


def _f32_truncate(x):
    # planted mistake: chops the significand (rounds toward zero)
    x = np.asarray(x, dtype=np.float64)
    r = np.asarray(x, dtype=np.float32).astype(np.float64)
    down = np.abs(r) > np.abs(x)
    r[down] = np.nextafter(r[down].astype(np.float32), np.float32(0)).astype(np.float64)
    return r


def _f32_ties_away(x):
    # planted mistake: halfway cases go away from zero
    x = np.asarray(x, dtype=np.float64)
    r = np.asarray(x, dtype=np.float32).astype(np.float64)
    other = np.nextafter(r.astype(np.float32), np.where(x > r, np.float32(np.inf), np.float32(-np.inf)))
    other = other.astype(np.float64)
    tie = (np.abs(other - x) == np.abs(r - x)) & (np.abs(other) > np.abs(r))
    r[tie] = other[tie]
    return r


@pytest.mark.parametrize("mutant", [_f32_truncate, _f32_ties_away], ids=["truncate", "ties-away"])
def test_pins_catch_planted_f32_rounding_mistakes(monkeypatch, mutant):
    monkeypatch.setattr(R, "f32_round", mutant)
    with pytest.raises(AssertionError):
        test_f32_round_halfway_cases_from_the_grid()


def test_zero_gradient_bf16_param_is_bitwise_unchanged():
    torch = pytest.importorskip("torch")
    g = torch.Generator().manual_seed(0)
    w = (torch.randn(64, 48, generator=g) * 0.02).to(torch.bfloat16).double().numpy()
    out = R.muon_step_matrix(w, np.zeros_like(w), np.zeros_like(w), lr=0.02, momentum=0.95,
                             weight_decay=0.01, ns_steps=5, param_dtype="bf16")
    assert np.array_equal(out["w"], w)
    assert np.all(out["o"] == 0.0) and np.all(out["m"] == 0.0)


def test_ns_flops_counts():
    assert R.ns_flops(4096, 14336) == R.ns_flops(14336, 4096) == 5 * (3 * 4096 ** 2 * 14336 + 4096 ** 3)


# ---------------------------------------------------------------- planted mistakes

def _mutant_ns(kind):
    def ns(x, steps, abc=ABC):
        a, b, c = abc
        x = np.array(x, dtype=np.float64, copy=True)
        for _ in range(steps):
            gram = x @ x.T
            if kind == "drop_c":
                poly = b * gram
            elif kind == "sign_b":
                poly = -b * gram + c * (gram @ gram)
            elif kind == "cube_not_square":
                poly = b * gram + c * (gram @ gram @ gram)
            else:
                poly = b * gram + c * (gram @ gram)
            if kind == "right_multiply":
                x = a * x + x @ poly.T if x.shape[0] == x.shape[1] else a * x + poly @ x
            else:
                x = a * x + poly @ x
        return x
    return ns


@pytest.mark.parametrize("kind", ["drop_c", "sign_b", "cube_not_square", "right_multiply"])
def test_pins_catch_planted_iteration_mistakes(monkeypatch, kind):
    monkeypatch.setattr(R, "newton_schulz", _mutant_ns(kind))
    caught = False
    for (rows, cols) in [(6, 11), (9, 9)]:
        rng = np.random.default_rng(rows * 100 + cols + 5)
        u, s, v = _svd_input(rng, rows, cols, rng.uniform(0.05, 3.0, size=min(rows, cols)))
        g = (u * s) @ v.T
        with np.errstate(all="ignore"):
            got = R.orthogonalize(g, 5, ABC, eps=0.0)
        want = (u * _pk(s / np.linalg.norm(s), 5)) @ v.T
        # X @ poly(X X^T) on a square X equals U p(S) V^T only when X is normal;
        # a random square G is not, so the closed form catches that one too.
        if not _rel(got, want) < 1e-6:
            caught = True
    assert caught, kind


def test_pins_catch_planted_momentum_mistake(monkeypatch):
    def wrong(m, g, mu, nesterov=True):       # Nesterov from the stale M
        m = np.asarray(m, dtype=np.float64)
        m_new = mu * m + g
        return m_new, g + mu * m
    monkeypatch.setattr(R, "momentum_update", wrong)
    g = np.ones((2, 3))
    m = np.zeros_like(g)
    for t in range(1, 4):
        m, u = R.momentum_update(m, g, 0.9)
    geo = (1 - 0.9 ** 3) / 0.1
    assert not np.allclose(u, g + 0.9 * geo * g)


def test_pins_catch_missing_untranspose(monkeypatch):
    orig = R.orthogonalize

    def wrong(u, steps, abc=ABC, eps=R.DEFAULT_EPS):
        u = np.asarray(u, dtype=np.float64)
        x = u.T if u.shape[0] > u.shape[1] else u
        return orig(x, steps, abc, eps)        # forgets to transpose back
    rng = np.random.default_rng(0)
    g = rng.standard_normal((12, 5))
    assert wrong(g, 5).shape != g.shape
