"""Pins of the PVS oracle (quantisation, residual bound, guard, intervals)
against closed forms, brute force and exact rationals (Sec. 2.3.1, App. A.1)."""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import pvs
from paper_2608_07152_amd import datagen

F32 = np.float32


def _nearest_int_brute(x: np.float32) -> int:
    """Integer nearest to x, halves away from zero, by exact comparison."""
    fx = Fraction(float(x))
    lo = math.floor(fx)
    hi = lo + 1
    dlo, dhi = fx - lo, hi - fx
    if dlo < dhi:
        return lo
    if dhi < dlo:
        return hi
    return hi if abs(hi) > abs(lo) else lo


def test_zero_vector_closed_form():
    e = pvs.quantize(np.zeros((1, 16), dtype=np.float32))
    assert e.s[0] == F32(1)
    assert not e.z.any()
    assert e.norm[0] == 0 and e.enorm[0] == 0 and e.hnorm[0] == 0


@pytest.mark.parametrize("a", [127 / 128, -127 / 128, 254.0, -0.5 * 127])
def test_scaled_basis_vector_is_exact(a):
    # a / 127 is a power of two, so s * 127 == a exactly and the residual is 0
    v = np.zeros((1, 8), dtype=np.float32)
    v[0, 3] = a
    e = pvs.quantize(v)
    assert Fraction(float(e.s[0])) * 127 == abs(Fraction(a))
    assert e.z[0, 3] == (127 if a > 0 else -127)
    assert np.count_nonzero(e.z) == 1
    assert e.enorm[0] == 0


def test_scaled_basis_vector_generic():
    v = np.zeros((1, 8), dtype=np.float32)
    v[0, 5] = F32(0.3)
    e = pvs.quantize(v)
    assert e.z[0, 5] == 127 and np.count_nonzero(e.z) == 1
    # residual is the rounding error of s = fl(0.3/127), far below one ulp of 0.3
    assert 0 < e.enorm[0] < 1e-7


def test_half_way_ties_round_away_from_zero():
    s = 2.0 ** -7
    vals = [127 * s, 0.5 * s, -0.5 * s, 2.5 * s, -2.5 * s, 3.5 * s, -126.5 * s]
    e = pvs.quantize(np.array([vals], dtype=np.float32))
    assert e.s[0] == F32(s)
    assert list(e.z[0]) == [127, 1, -1, 3, -3, 4, -127]


def test_just_below_half_rounds_to_zero():
    s = 2.0 ** -7
    below_half = np.nextafter(F32(0.5), F32(0))          # 0.49999997
    v = np.array([[127 * s, float(below_half) * s, -float(below_half) * s]], dtype=np.float32)
    e = pvs.quantize(v)
    assert list(e.z[0]) == [127, 0, 0]


def test_codes_match_brute_force_nearest_integer():
    rng = np.random.default_rng(7)
    v = (rng.standard_normal((40, 64)) * rng.uniform(1e-3, 10, size=(40, 1))).astype(np.float32)
    e = pvs.quantize(v)
    for i in range(v.shape[0]):
        mu = max(abs(Fraction(float(x))) for x in v[i])
        # s is the float32 nearest to mu / 127
        s = e.s[i]
        t = mu / 127
        for nb in (np.nextafter(s, F32(np.inf)), np.nextafter(s, F32(0))):
            assert abs(Fraction(float(s)) - t) <= abs(Fraction(float(nb)) - t)
        for j in range(v.shape[1]):
            x = np.float32(v[i, j] / s)
            want = max(-127, min(127, _nearest_int_brute(x)))
            assert e.z[i, j] == want


def test_underflowing_scale_uses_smallest_subnormal():
    tiny = np.nextafter(F32(0), F32(1))
    v = np.array([[tiny, 0.0, -tiny]], dtype=np.float32)
    e = pvs.quantize(v)
    assert e.s[0] == tiny
    assert list(e.z[0]) == [1, 0, -1]


def test_non_finite_rejected():
    with pytest.raises(ValueError):
        pvs.quantize(np.array([[1.0, np.nan]], dtype=np.float32))


def test_norms_rounded_up():
    rng = np.random.default_rng(3)
    v = rng.standard_normal((50, 96)).astype(np.float32)
    e = pvs.quantize(v)
    for i in range(50):
        exact_sq = sum(Fraction(float(x)) ** 2 for x in v[i])
        assert Fraction(float(e.norm[i])) ** 2 >= exact_sq
        # and not more than a couple of float32 ulps above
        assert float(e.norm[i]) <= math.sqrt(float(exact_sq)) * (1 + 3 * 2.0 ** -23)
        resid = [Fraction(float(v[i, j])) - Fraction(float(e.s[i])) * int(e.z[i, j]) for j in range(96)]
        assert Fraction(float(e.enorm[i])) ** 2 >= sum(r * r for r in resid)


@pytest.mark.parametrize("m", [1, 128, 384, 768, 4096])
def test_gamma_brackets(m):
    a = (8 * m + 64) * 2.0 ** -23
    gm = float(pvs.gamma(m))
    # a/(1-a) = a + a^2 + a^3 + ... lies in [a + a^2, a + 2 a^2] for a < 1/2
    assert gm >= a + a * a
    assert gm <= (a + 2 * a * a) * (1 + 2.0 ** -23)


def test_gamma_rejects_too_large_dimension():
    with pytest.raises(ValueError):
        pvs.gamma((2 ** 23) // 8)


def _tight_pair(side: str):
    """(q, v) with one residual exactly parallel to the other vector, so the
    Cauchy-Schwarz residual bound is attained (see the construction in the
    test body)."""
    rng = np.random.default_rng(11)
    m = 32
    za = rng.integers(-100, 101, size=m)
    zb = rng.integers(-100, 101, size=m)
    za[0] = 127          # sets ||.||_inf so the scale is exactly 2^-7
    zb[1] = 127
    zb[0] = 0            # residual direction (from za) is 0 where zb peaks
    za[1] = 0
    a = (za / 128.0).astype(np.float32)       # exactly representable, zero residual
    # b = bhat + t * a with t = 2^-10 : |t * a_j| < s/2, quantisation unchanged
    b = ((zb + za * 2.0 ** -10) / 128.0).astype(np.float32)
    assert np.all(b.astype(np.float64) == (zb + za * 2.0 ** -10) / 128.0)
    if side == "item":     # q exact, v carries a residual parallel to q_hat
        return a, b
    return b, a            # v exact, q carries a residual parallel to v


@pytest.mark.parametrize("side", ["item", "query"])
def test_residual_bound_is_tight(side):
    q, v = _tight_pair(side)
    qe, ve = pvs.quantize(q), pvs.quantize(v)
    iv = pvs.intervals(qe, ve, q.shape[0])
    s_exact = sum(Fraction(float(x)) * Fraction(float(y)) for x, y in zip(q, v))
    c_exact = Fraction(float(qe.s[0])) * Fraction(float(ve.s[0])) * int(
        np.dot(qe.z[0].astype(np.int64), ve.z[0].astype(np.int64)))
    gap = abs(s_exact - c_exact)
    assert gap > 0
    E = Fraction(float(iv.E[0, 0]))
    assert E >= gap                                    # the bound holds ...
    assert E <= gap * (1 + Fraction(1, 10 ** 5))      # ... and is attained


def test_center_score_exact_for_dyadic_inputs():
    # scales are powers of two: c = s_q s_v <z_q, z_v> is exact in float32
    q = np.array([[127 / 128, 0.25, -0.5]], dtype=np.float32)
    v = np.array([[0.5, 127 / 64, 1.0]], dtype=np.float32)
    qe, ve = pvs.quantize(q), pvs.quantize(v)
    iv = pvs.intervals(qe, ve, 3)
    assert iv.c[0, 0] == F32(q[0] @ v[0])
    assert iv.E[0, 0] == 0
    assert iv.lo[0, 0] < iv.c[0, 0] < iv.hi[0, 0]


def _f32_dot_orders(q, v):
    """float32 inner products accumulated in three different orders."""
    out = []
    acc = F32(0)
    for x, y in zip(q, v):
        acc = F32(acc + F32(x * y))
    out.append(acc)
    acc = F32(0)
    for x, y in zip(q[::-1], v[::-1]):
        acc = F32(acc + F32(x * y))
    out.append(acc)
    p = (q * v).astype(np.float32)
    while len(p) > 1:
        if len(p) % 2:
            p = np.append(p, F32(0))
        p = (p[0::2] + p[1::2]).astype(np.float32)
    out.append(p[0])
    return out


def test_intervals_contain_exact_and_f32_scores():
    w = datagen.workload("tiny", n=400)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=6)
    qe, ve = pvs.quantize(q), pvs.quantize(x)
    iv = pvs.intervals(qe, ve, w.d)
    s64 = q.astype(np.float64) @ x.astype(np.float64).T
    assert np.all(iv.lo <= s64) and np.all(s64 <= iv.hi)
    # pure Cauchy-Schwarz part alone: |s - c| <= E (no guard)
    assert np.all(np.abs(s64 - iv.c.astype(np.float64)) <= iv.E.astype(np.float64) * (1 + 1e-6))
    for b in range(3):
        for i in range(0, 400, 37):
            for s32 in _f32_dot_orders(q[b], x[i]):
                assert iv.lo[b, i] <= s32 <= iv.hi[b, i]


def test_intervals_contain_scores_on_hard_inputs():
    # heavy-tailed coordinates, mixed magnitudes and exact zeros
    rng = np.random.default_rng(5)
    m = 256
    x = rng.standard_cauchy((300, m)).astype(np.float32)
    x[::7, ::3] = 0
    x[5] = 0
    q = rng.standard_cauchy((4, m)).astype(np.float32)
    qe, ve = pvs.quantize(q), pvs.quantize(x)
    iv = pvs.intervals(qe, ve, m)
    s64 = q.astype(np.float64) @ x.astype(np.float64).T
    assert np.all(iv.lo <= s64) and np.all(s64 <= iv.hi)
    # outward rounding: the interval strictly contains the centre score
    assert np.all(iv.lo < iv.c) and np.all(iv.c < iv.hi)


def test_interval_widens_with_guard():
    w = datagen.workload("tiny", n=50)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=2)
    qe, ve = pvs.quantize(q), pvs.quantize(x)
    iv = pvs.intervals(qe, ve, w.d)
    width = iv.hi.astype(np.float64) - iv.lo.astype(np.float64)
    assert np.all(width >= 2 * (iv.E.astype(np.float64) + iv.G.astype(np.float64)))
    assert np.all(iv.G > 0)


# ---------------------------------------------------------------------------
# Global-scale scalar quantisation (the alternative generator of Sec. 4.4)

def test_global_scale_reduces_to_per_vector_when_row_maxima_agree():
    # every row has the same largest magnitude, so the shared scale is each
    # row's own scale and the two encoders must agree exactly
    rng = np.random.default_rng(11)
    x = rng.uniform(-0.9, 0.9, (50, 64)).astype(np.float32)
    x[np.arange(50), rng.integers(0, 64, 50)] = np.where(rng.random(50) < 0.5, F32(-1.25), F32(1.25))
    g, p = pvs.quantize_global(x), pvs.quantize(x)
    for f in ("s", "z", "norm", "enorm", "hnorm"):
        assert np.array_equal(getattr(g, f), getattr(p, f)), f


def test_global_scale_is_the_largest_row_scale():
    # f32 division by 127 is monotone, so fl32(max|v| / 127) equals the
    # largest per-row scale of the nonzero rows
    w = datagen.workload("tiny", n=300)
    x, _ = datagen.corpus(w)
    assert pvs.quantize_global(x).s[0] == pvs.quantize(x).s.max()


def test_global_scale_dyadic_closed_form():
    # max |entry| = 127 * 2^-6 and every entry a multiple of 2^-6: the scale
    # is 2^-6, the codes are the multipliers and the residual is zero
    rng = np.random.default_rng(3)
    k = rng.integers(-127, 128, (20, 32))
    k[4, 7] = 127
    x = (k * 2.0 ** -6).astype(np.float32)
    e = pvs.quantize_global(x)
    assert np.all(e.s == F32(2.0 ** -6))
    assert np.array_equal(e.z.astype(np.int64), k)
    assert np.all(e.enorm == 0)


def test_global_codes_are_nearest_integers_and_residual_bounded():
    rng = np.random.default_rng(8)
    x = rng.standard_normal((40, 48)).astype(np.float32)
    e = pvs.quantize_global(x)
    s = e.s[0]
    for i in range(0, 40, 3):
        for j in range(0, 48, 5):
            assert int(e.z[i, j]) == _nearest_int_brute(F32(x[i, j] / s))
    resid = np.abs(x.astype(np.float64) - np.float64(s) * e.z.astype(np.float64))
    # |v - s z| <= s/2 up to the rounding of the f32 quotient
    assert np.all(resid <= np.float64(s) * (0.5 + 2.0 ** -20))


def test_global_zero_matrix_and_clipping_with_a_fixed_scale():
    e = pvs.quantize_global(np.zeros((3, 8), dtype=np.float32))
    assert np.all(e.s == F32(1)) and not np.any(e.z)
    # rows inserted after the scale was fixed: codes clip at +-127 and the
    # residual norm accounts for what was clipped
    x = np.array([[1.0, -3.0, 0.5]], dtype=np.float32)
    e = pvs.quantize_global(x, scale=F32(1.0 / 127))
    assert list(e.z[0]) == [127, -127, 64]
    r = x.astype(np.float64)[0] - np.float64(F32(1.0 / 127)) * e.z[0].astype(np.float64)
    assert e.enorm[0] >= np.sqrt(np.sum(r * r))


@pytest.mark.parametrize("clip", [False, True])
def test_global_intervals_contain_exact_scores(clip):
    w = datagen.workload("tiny", n=400)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=5)
    ve = pvs.quantize_global(x, scale=(pvs.quantize_global(x).s[0] * F32(0.5)) if clip else None)
    iv = pvs.intervals(pvs.quantize(q), ve, w.d)
    s64 = q.astype(np.float64) @ x.astype(np.float64).T
    assert np.all(iv.lo <= s64) and np.all(s64 <= iv.hi)
    assert np.all(np.abs(s64 - iv.c.astype(np.float64)) <= iv.E.astype(np.float64) * (1 + 1e-6))
