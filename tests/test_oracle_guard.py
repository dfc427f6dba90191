"""Exact-rational pins of the PVS interval (Sec. 2.3.1, App. A.1).

For every (query, row) pair the oracle's float32 values c, E, G and the
endpoints [lo, hi] are compared with the paper's definitions evaluated
exactly, from the raw float32 vectors rather than from anything the oracle
stored:

    c* = s_q s_v <z_q, z_v>                           (Sec. 2.3.1)
    E* = ||e_q|| ||v|| + ||q_hat|| ||e_v||            (Sec. 2.3.1, Cauchy-Schwarz)
    G* = (|c*| + E* + ||q|| ||v||) a_m / (1 - a_m)    (App. A.1, the least gamma_m allowed)

with every norm computed exactly (to 2^-120) from q, v, s and z.  The oracle
rounds each operation to float32 and stores norms rounded up, so its values
may differ from these by a few float32 roundings; the tolerances below are
derived from the number of roundings, and each planted mistake (a dropped
||q|| ||v|| term, a_m in place of gamma_m, ||q_hat|| in place of ||q||, no
outward step, the wrong endpoint) moves a value far outside them.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import pvs
from paper_2608_07152_amd import datagen

F32 = np.float32
U = Fraction(1, 2 ** 24)          # unit roundoff of float32 round-to-nearest
SQRT_BITS = 120


def _fr(x) -> Fraction:
    return Fraction(float(x))


def _sqrt_lo(x: Fraction) -> Fraction:
    """A lower bound of sqrt(x) within 2^-SQRT_BITS (x >= 0)."""
    if x == 0:
        return Fraction(0)
    scaled = x * 2 ** (2 * SQRT_BITS)
    return Fraction(math.isqrt(scaled.numerator // scaled.denominator), 2 ** SQRT_BITS)


def _rn32(x: Fraction) -> Fraction:
    """x rounded to the nearest float32 (ties to even), by exact arithmetic."""
    if x == 0:
        return Fraction(0)
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = math.floor(math.log2(a.numerator) - math.log2(a.denominator))
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)                         # subnormal range shares the last binade's ulp
    ulp = Fraction(2) ** (e - 23)
    k = a / ulp
    n = math.floor(k)
    rem = k - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return sign * n * ulp


def _ulp32(x: Fraction) -> Fraction:
    a = abs(x)
    if a == 0:
        return Fraction(2) ** -149
    e = math.floor(math.log2(float(a)))
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    return Fraction(2) ** (max(e, -126) - 23)


def _next32(x: Fraction, up: bool) -> Fraction:
    f = np.float32(float(x))
    assert _fr(f) == x, "not a float32 value"
    return _fr(np.nextafter(f, F32(np.inf if up else -np.inf)))


def exact_terms(q32, v32, qe, ve, b, i, m):
    """c*, E*, G* of pair (b, i) from the raw vectors (see the module docstring)."""
    qb = [_fr(t) for t in q32[b]]
    vi = [_fr(t) for t in v32[i]]
    sq, sv = _fr(qe.s[b]), _fr(ve.s[i])
    zq = [int(t) for t in qe.z[b]]
    zv = [int(t) for t in ve.z[i]]
    c = sq * sv * sum(x * y for x, y in zip(zq, zv))
    nq = _sqrt_lo(sum(t * t for t in qb))
    nv = _sqrt_lo(sum(t * t for t in vi))
    neq = _sqrt_lo(sum((t - sq * z) ** 2 for t, z in zip(qb, zq)))
    nev = _sqrt_lo(sum((t - sv * z) ** 2 for t, z in zip(vi, zv)))
    nqh = _sqrt_lo(sum((sq * z) ** 2 for z in zq))
    E = neq * nv + nqh * nev
    a = (8 * m + 64) * Fraction(1, 2 ** 23)
    G = (abs(c) + E + nq * nv) * (a / (1 - a))
    return c, E, G


def check_guard(q32, v32, qe, ve, m, iv, pairs):
    """Assert the oracle's interval of every listed pair against the exact terms."""
    gamma_ok = _fr(pvs.gamma(m))
    a = (8 * m + 64) * Fraction(1, 2 ** 23)
    assert gamma_ok >= a / (1 - a)
    assert gamma_ok <= (a / (1 - a)) * (1 + 2 * U)
    for b, i in pairs:
        c, E, G = exact_terms(q32, v32, qe, ve, b, i, m)
        c_o, E_o, G_o = _fr(iv.c[b, i]), _fr(iv.E[b, i]), _fr(iv.G[b, i])
        lo_o, hi_o = _fr(iv.lo[b, i]), _fr(iv.hi[b, i])
        # c: two roundings (s_q s_v, then the product with the exact dot)
        assert abs(c_o - c) <= 2 * U * abs(c) + Fraction(2) ** -149, ("c", b, i)
        # E: norms rounded up (<= 2^-23 each), two products and a sum
        assert E * (1 - 3 * U) <= E_o <= E * (1 + 16 * U) + Fraction(2) ** -149, ("E", b, i)
        # G: the stored ||q||, ||v|| rounded up, five float32 roundings, gamma
        # rounded up from a_m / (1 - a_m)
        assert G * (1 - 8 * U) <= G_o <= G * (1 + 24 * U), ("G", b, i, float(G_o / G - 1))
        # endpoints: one ulp outward of the float32 sum and difference
        w_o = _rn32(E_o + G_o)
        assert lo_o == _next32(_rn32(c_o - w_o), up=False), ("lo step", b, i)
        assert hi_o == _next32(_rn32(c_o + w_o), up=True), ("hi step", b, i)
        # and close to the exact endpoints c* -/+ (E* + G*)
        w = E + G
        slack_lo = 40 * U * (abs(c) + w) + 2 * _ulp32(c - w)
        slack_hi = 40 * U * (abs(c) + w) + 2 * _ulp32(c + w)
        assert abs(lo_o - (c - w)) <= slack_lo, ("lo", b, i)
        assert abs(hi_o - (c + w)) <= slack_hi, ("hi", b, i)
        assert lo_o < c - E and c + E < hi_o, ("guard not outside E", b, i)


def _coarse_queries(m, rng):
    """Queries whose coordinates sit just below half a quantisation step
    from the grid: large ||e_q||, so ||q_hat|| and ||q|| differ clearly."""
    out = np.zeros((3, m), dtype=np.float32)
    for r in range(3):
        k = rng.integers(-120, 121, size=m).astype(np.float64)
        x = (k + np.sign(rng.standard_normal(m)) * 0.49) / 127.0
        x[r] = 1.0                                  # ||q||_inf = 1, s_q = fl(1/127)
        out[r] = x.astype(np.float32)
    return out


def _cases():
    rng = np.random.default_rng(2027)
    cases = []
    # clustered unit vectors of the Tiny workload (d = 128)
    w = datagen.workload("tiny", n=40)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=3)
    cases.append(("tiny", q, x, w.d))
    # passage dimension, random unit vectors, negative and positive scores
    m = 768
    x = rng.standard_normal((12, m))
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    qv = rng.standard_normal((2, m))
    qv /= np.linalg.norm(qv, axis=1, keepdims=True)
    cases.append(("d768", qv.astype(np.float32), x.astype(np.float32), m))
    # coarse queries against heavy-tailed rows with zeros and a zero row
    m = 96
    x = rng.standard_cauchy((10, m)).astype(np.float32)
    x[::3, ::4] = 0
    x[4] = 0
    cases.append(("coarse", _coarse_queries(m, rng), x, m))
    return cases


@pytest.mark.parametrize("name,q32,v32,m", _cases(), ids=lambda c: c if isinstance(c, str) else "")
def test_interval_terms_match_exact_definition(name, q32, v32, m):
    qe, ve = pvs.quantize(q32), pvs.quantize(v32)
    iv = pvs.intervals(qe, ve, m)
    pairs = [(b, i) for b in range(q32.shape[0]) for i in range(v32.shape[0])]
    check_guard(q32, v32, qe, ve, m, iv, pairs)


def test_query_hat_norm_rounded_up():
    rng = np.random.default_rng(4)
    q = _coarse_queries(64, rng)
    qe = pvs.quantize(q)
    for b in range(q.shape[0]):
        exact_sq = sum((_fr(qe.s[b]) * int(z)) ** 2 for z in qe.z[b])
        assert _fr(qe.hnorm[b]) ** 2 >= exact_sq
        assert float(qe.hnorm[b]) <= math.sqrt(float(exact_sq)) * (1 + 3 * 2.0 ** -23)


def _mutant(qe, ve, m, kind):
    """The oracle's interval arithmetic with one planted mistake."""
    g = pvs.gamma(m)
    if kind == "a_m":
        g = F32(float((8 * m + 64) * Fraction(1, 2 ** 23)))
    dot = qe.z.astype(np.int64) @ ve.z.astype(np.int64).T
    sqv = (qe.s[:, None] * ve.s[None, :]).astype(np.float32)
    c = (sqv * dot.astype(np.float32)).astype(np.float32)
    E = ((qe.enorm[:, None] * ve.norm[None, :]).astype(np.float32)
         + (qe.hnorm[:, None] * ve.enorm[None, :]).astype(np.float32)).astype(np.float32)
    nq = qe.hnorm if kind == "qhat_for_q" else qe.norm
    nqv = (nq[:, None] * ve.norm[None, :]).astype(np.float32)
    if kind == "no_norm_term":
        nqv = np.zeros_like(nqv)
    G = (((np.abs(c) + E).astype(np.float32) + nqv).astype(np.float32) * g).astype(np.float32)
    w = (E + G).astype(np.float32)
    if kind == "endpoint_E_only":
        w = E
    lo = (c - w).astype(np.float32)
    hi = (c + w).astype(np.float32)
    if kind != "no_outward_step":
        lo = np.nextafter(lo, F32(-np.inf)).astype(np.float32)
        hi = np.nextafter(hi, F32(np.inf)).astype(np.float32)
    return pvs.Intervals(c, E, G, lo, hi)


@pytest.mark.parametrize("kind", ["no_norm_term", "a_m", "qhat_for_q", "no_outward_step",
                                  "endpoint_E_only"])
def test_planted_mistakes_are_caught(kind):
    # the check above must reject each plausible mistake in the guard
    rng = np.random.default_rng(1729)
    m = 96
    q = _coarse_queries(m, rng)
    x = rng.standard_normal((6, m)).astype(np.float32)
    qe, ve = pvs.quantize(q), pvs.quantize(x)
    pairs = [(b, i) for b in range(q.shape[0]) for i in range(x.shape[0])]
    check_guard(q, x, qe, ve, m, _mutant(qe, ve, m, "none"), pairs)   # the unmutated copy passes
    with pytest.raises(AssertionError):
        check_guard(q, x, qe, ve, m, _mutant(qe, ve, m, kind), pairs)
