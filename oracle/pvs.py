"""PVS quantisation and deterministic score intervals (oracle).

Follows Sec. 2.3.1 (per-vector scale, Int8 encoding, quantised centre score,
Cauchy-Schwarz residual bound) and App. A.1 (finite-precision guard).

Readings where the paper is silent (each also listed in the design notes):

* round() of v_j / s_v is round-half-away-from-zero (the paper's implementation
  is Rust, whose ``f32::round`` does that), applied to the correctly rounded
  float32 quotient.
* s_v is the float32 nearest to ||v||_inf / 127; if that underflows to zero
  for a nonzero v, the smallest positive float32 is used.
* ||v||_2, ||e_v||_2, ||q||_2, ||q_hat||_2, ||e_q||_2 are computed in float64,
  inflated by (1 + 2^-40) to absorb float64 rounding, and stored as the
  smallest float32 not below that ("rounded up").
* The interval is evaluated in float32 round-to-nearest, one rounding per
  operation, in this order:
      sqv = s_q * s_v;  c = sqv * float(dot)
      E   = ||e_q|| * ||v|| + ||q_hat|| * ||e_v||
      G   = ((|c| + E) + ||q|| * ||v||) * gamma_m
      w   = E + G;  lo = down(c - w);  hi = up(c + w)
  where down/up step one float32 ulp outward (nextafter).
* gamma_m is the smallest float32 not below a_m / (1 - a_m),
  a_m = (8m + 64) * 2^-23 (numerator and denominator are exact in float32).

Parity: pinned by closed forms (zero vector, scaled basis vectors, exact
half-way ties, dyadic inputs), brute-force nearest-integer and nearest-scale
search, the bracket of gamma, tightness of the residual bound, containment
of exact and float32 scores, and an exact-rational recomputation of c, E, G
and both endpoints from the raw vectors (each within its stated number of
float32 roundings, the endpoints exactly one ulp outward), which rejects
planted mistakes in the guard (a dropped ||q|| ||v|| term, a_m in place of
gamma_m, ||q_hat|| in place of ||q||, no outward step, a wrong endpoint).
This module is test infrastructure: only the tests, the smoke check and the
CPU baseline of the benchmark use it.
"""
from __future__ import annotations

import dataclasses
from fractions import Fraction

import numpy as np

F32 = np.float32
EPS32 = Fraction(1, 2 ** 23)       # f32::EPSILON
NORM_INFLATE = 1.0 + 2.0 ** -40
TINY32 = np.nextafter(F32(0), F32(1))


def up32(x64: np.ndarray) -> np.ndarray:
    """Smallest float32 >= x64 * (1 + 2^-40), elementwise (x64 >= 0)."""
    x = np.asarray(x64, dtype=np.float64) * NORM_INFLATE
    f = x.astype(np.float32)
    low = f.astype(np.float64) < x
    f = np.where(low, np.nextafter(f, F32(np.inf)), f)
    return f.astype(np.float32)


def round_half_away(x32: np.ndarray) -> np.ndarray:
    """Nearest integer to each float32 value, halves away from zero (float64,
    where |x| + 0.5 is exact for |x| < 2^29)."""
    x = np.asarray(x32, dtype=np.float32).astype(np.float64)
    return np.sign(x) * np.floor(np.abs(x) + 0.5)


@dataclasses.dataclass
class Encoded:
    """Per-vector PVS record: scale s, codes z, and rounded-up norms."""
    s: np.ndarray        # float32 [n]
    z: np.ndarray        # int8 [n, m]
    norm: np.ndarray     # float32 [n]  ||v||_2 rounded up
    enorm: np.ndarray    # float32 [n]  ||v - s z||_2 rounded up
    hnorm: np.ndarray    # float32 [n]  ||s z||_2 rounded up (used for queries)


def quantize(v32: np.ndarray) -> Encoded:
    """Encode rows of a float32 matrix [n, m] (a 1-D vector is one row)."""
    v = np.atleast_2d(np.asarray(v32, dtype=np.float32))
    if not np.all(np.isfinite(v)):
        raise ValueError("non-finite input")
    mu = np.max(np.abs(v), axis=1)                      # ||v||_inf, exact
    s = (mu / F32(127)).astype(np.float32)              # correctly rounded f32 divide
    s = np.where((mu > 0) & (s == 0), TINY32, s).astype(np.float32)
    s = np.where(mu == 0, F32(1), s).astype(np.float32)
    x = (v / s[:, None]).astype(np.float32)             # correctly rounded f32 divide
    z = np.clip(round_half_away(x), -127, 127).astype(np.int8)
    v64 = v.astype(np.float64)
    vh64 = s.astype(np.float64)[:, None] * z.astype(np.float64)   # exact products
    e64 = v64 - vh64
    norm = up32(np.sqrt(np.sum(v64 * v64, axis=1)))
    enorm = up32(np.sqrt(np.sum(e64 * e64, axis=1)))
    hnorm = up32(np.sqrt(np.sum(vh64 * vh64, axis=1)))
    return Encoded(s, z, norm, enorm, hnorm)


def quantize_global(v32: np.ndarray, scale=None) -> Encoded:
    """Scalar quantisation with one scale shared by every row: the interval
    generator Sec. 3.5 and Sec. 4.4 (Table 4-1) compare PVS with.

    Reading: the shared scale is the per-vector rule applied to the whole
    matrix, s = fl32(max_ij |v_ij| / 127) (1 if every entry is zero, the
    smallest positive float32 if the quotient underflows); codes, norms and
    intervals are then those of Sec. 2.3.1 with s_v = s for every row.  A
    given ``scale`` (rows inserted after the scale was fixed) is used as is,
    and codes that would exceed 127 in magnitude are clipped.
    """
    v = np.atleast_2d(np.asarray(v32, dtype=np.float32))
    if not np.all(np.isfinite(v)):
        raise ValueError("non-finite input")
    if scale is None:
        mu = F32(np.max(np.abs(v))) if v.size else F32(0)
        sc = F32(mu / F32(127))
        if mu > 0 and sc == 0:
            sc = TINY32
        if mu == 0:
            sc = F32(1)
    else:
        sc = F32(scale)
    n = v.shape[0]
    s = np.full(n, sc, dtype=np.float32)
    x = (v / sc).astype(np.float32)                      # correctly rounded f32 divide
    z = np.clip(round_half_away(x), -127, 127).astype(np.int8)
    v64 = v.astype(np.float64)
    vh64 = np.float64(sc) * z.astype(np.float64)         # exact products
    e64 = v64 - vh64
    norm = up32(np.sqrt(np.sum(v64 * v64, axis=1)))
    enorm = up32(np.sqrt(np.sum(e64 * e64, axis=1)))
    hnorm = up32(np.sqrt(np.sum(vh64 * vh64, axis=1)))
    return Encoded(s, z, norm, enorm, hnorm)


def gamma(m: int) -> np.float32:
    """Smallest float32 >= a_m / (1 - a_m) with a_m = (8m + 64) eps (App. A.1)."""
    a = (8 * m + 64) * EPS32
    if a >= 1:
        raise ValueError("a_m >= 1: dimension too large for the guard")
    target = a / (1 - a)
    f = np.float32(float(target))
    while Fraction(float(f)) < target:
        f = np.nextafter(f, F32(np.inf))
    while Fraction(float(np.nextafter(f, F32(-np.inf)))) >= target:
        f = np.nextafter(f, F32(-np.inf))
    return np.float32(f)


@dataclasses.dataclass
class Intervals:
    c: np.ndarray    # float32 [B, n] quantised centre score
    E: np.ndarray    # float32 [B, n] residual bound
    G: np.ndarray    # float32 [B, n] finite-precision guard
    lo: np.ndarray   # float32 [B, n]
    hi: np.ndarray   # float32 [B, n]


def intervals(q: Encoded, v: Encoded, m: int) -> Intervals:
    """Score intervals for every (query, row) pair, float32 [B, n]."""
    g = gamma(m)
    dot = q.z.astype(np.int64) @ v.z.astype(np.int64).T             # exact integers
    if np.any(np.abs(dot) >= 2 ** 31):
        raise OverflowError("integer accumulator overflow")
    sqv = (q.s[:, None] * v.s[None, :]).astype(np.float32)
    c = (sqv * dot.astype(np.float32)).astype(np.float32)
    E = ((q.enorm[:, None] * v.norm[None, :]).astype(np.float32)
         + (q.hnorm[:, None] * v.enorm[None, :]).astype(np.float32)).astype(np.float32)
    nqv = (q.norm[:, None] * v.norm[None, :]).astype(np.float32)
    G = (((np.abs(c) + E).astype(np.float32) + nqv).astype(np.float32) * g).astype(np.float32)
    w = (E + G).astype(np.float32)
    lo = np.nextafter((c - w).astype(np.float32), F32(-np.inf)).astype(np.float32)
    hi = np.nextafter((c + w).astype(np.float32), F32(np.inf)).astype(np.float32)
    return Intervals(c, E, G, lo, hi)
