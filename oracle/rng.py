"""Perturbation Z regenerated from a counter (oracle side).

Paper: Section 3 ("ZO-Act") samples Z ~ N(0, I) in the r x n coefficient space of
every adapted layer, and Algorithm 2 draws a fresh Z_l^(j) per step and query.
The paper fixes only "Gaussian"; the generator below is this build's reading,
chosen so that Z is a pure function of (seed, step, query, arena index) and is
never stored:

* Uniform bits: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random
  Numbers: As Easy as 1, 2, 3", SC'11).  key = (lo32(seed), hi32(seed));
  counter = (lo32(e >> 2), hi32(e >> 2), step, query); arena index e takes
  output lane e & 3.
* Gaussian: Box-Muller (Box & Muller 1958) with the angle measured in quarter
  turns.  Words (w0, w1) give lanes 0 and 1 as (R cos, R sin); words (w2, w3)
  give lanes 2 and 3.
    u1 = ((w0 >> 8) + 1) * 2^-24 in (0, 1];  ln u1 = (E - 24) ln 2 + ln m with
    (w0 >> 8) + 1 = m 2^E, m in [sqrt(1/2), sqrt(2)), ln m = 2s(1 + s^2/3 + s^4/5 +
    s^6/7 + s^8/9), s = (m - 1)/(m + 1);  R = sqrt(-2 ln u1).
    quadrant q = w1 >> 30, fraction f = ((w1 >> 8) & 0x3FFFFF) 2^-22;
    sin(pi f/2), cos(pi f/2) from their Maclaurin series to degree 13 / 14
    (Horner in f^2); the quadrant rotates (c, s) -> (-s, c) -> (-c, -s) -> (s, -c).
  Every operation is a single fp32 operation (no fused multiply-add), division
  and square root are IEEE correctly rounded, in the exact order written below.
  |z| <= sqrt(2 * 24 ln 2) ~ 5.77 (the truncation at u1 >= 2^-24).

Pins (tests/test_oracle_rng.py): a second, scalar pure-Python implementation;
moments E z = 0, E z^2 = 1, E z^4 = 3 and E||z||^6 = k(k+2)(k+4) (the sixth
moment used in Appendix A's proof); a Kolmogorov-Smirnov test against N(0,1);
chi-square uniformity of the Philox words; determinism.
"""
from __future__ import annotations

import math

import numpy as np

# Philox4x32 round multipliers and Weyl key increments (Salmon et al., SC'11).
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
_MASK32 = 0xFFFFFFFF

_F = np.float32
# fp32 constants, each computed from its definition in float64 and rounded once.
LN2 = _F(math.log(2.0))
SQRT2 = _F(math.sqrt(2.0))
INV_ODD = {n: _F(1.0 / n) for n in (3, 5, 7, 9)}
# sin(pi x / 2) = sum_k (-1)^k (pi/2)^(2k+1) x^(2k+1) / (2k+1)!, k = 0..6
SIN_C = [_F((-1) ** k * (math.pi / 2) ** (2 * k + 1) / math.factorial(2 * k + 1)) for k in range(7)]
# cos(pi x / 2) = sum_k (-1)^k (pi/2)^(2k) x^(2k) / (2k)!, k = 0..7
COS_C = [_F((-1) ** k * (math.pi / 2) ** (2 * k) / math.factorial(2 * k)) for k in range(8)]


def philox4x32_10(c0, c1, c2, c3, k0: int, k1: int):
    """Ten Philox4x32 rounds on uint32 arrays; returns the four output words."""
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint32) for c in (c0, c1, c2, c3))
    m0, m1 = np.uint64(PHILOX_M0), np.uint64(PHILOX_M1)
    for rnd in range(10):
        if rnd:
            k0 = (k0 + PHILOX_W0) & _MASK32
            k1 = (k1 + PHILOX_W1) & _MASK32
        p0 = c0.astype(np.uint64) * m0
        p1 = c2.astype(np.uint64) * m1
        hi0 = (p0 >> np.uint64(32)).astype(np.uint32)
        lo0 = p0.astype(np.uint32)
        hi1 = (p1 >> np.uint64(32)).astype(np.uint32)
        lo1 = p1.astype(np.uint32)
        c0, c1, c2, c3 = hi1 ^ c1 ^ np.uint32(k0), lo1, hi0 ^ c3 ^ np.uint32(k1), lo0
    return c0, c1, c2, c3


def _ln_u1(w: np.ndarray) -> np.ndarray:
    """ln(((w >> 8) + 1) 2^-24) in fp32 by exponent split + atanh series."""
    n = (w >> np.uint32(8)) + np.uint32(1)                 # 1 .. 2^24, exact in fp32
    bits = n.astype(np.float32).view(np.uint32)
    e = (bits >> np.uint32(23)).astype(np.int32) - 127
    m = ((bits & np.uint32(0x007FFFFF)) | np.uint32(0x3F800000)).view(np.float32)
    big = m >= SQRT2
    m = np.where(big, m * _F(0.5), m).astype(np.float32)
    e = e + big.astype(np.int32)
    s = (m - _F(1.0)) / (m + _F(1.0))
    s2 = s * s
    p = INV_ODD[9]
    p = p * s2 + INV_ODD[7]
    p = p * s2 + INV_ODD[5]
    p = p * s2 + INV_ODD[3]
    p = p * s2 + _F(1.0)
    lnm = (s + s) * p
    return (e - 24).astype(np.float32) * LN2 + lnm


def _quarter_turn_sincos(w: np.ndarray):
    """(cos, sin) of 2 pi u for the angle encoded in w: quadrant w >> 30 plus 22 fraction bits."""
    q = (w >> np.uint32(30)).astype(np.int32)
    f = ((w >> np.uint32(8)) & np.uint32(0x3FFFFF)).astype(np.float32) * _F(2.0 ** -22)
    f2 = f * f
    sp = SIN_C[6]
    for k in (5, 4, 3, 2, 1, 0):
        sp = sp * f2 + SIN_C[k]
    sn = f * sp
    cp = COS_C[7]
    for k in (6, 5, 4, 3, 2, 1, 0):
        cp = cp * f2 + COS_C[k]
    cs = cp
    cos_out = np.select([q == 0, q == 1, q == 2], [cs, -sn, -cs], sn).astype(np.float32)
    sin_out = np.select([q == 0, q == 1, q == 2], [sn, cs, -sn], -cs).astype(np.float32)
    return cos_out, sin_out


def box_muller(wa: np.ndarray, wb: np.ndarray):
    """Two N(0,1) fp32 values (R cos, R sin) from two uint32 words."""
    r = np.sqrt(_F(-2.0) * _ln_u1(wa))
    c, s = _quarter_turn_sincos(wb)
    return (r * c).astype(np.float32), (r * s).astype(np.float32)


def gauss(seed: int, step: int, query: int, e) -> np.ndarray:
    """Z values (float32) at arena indices e (int64 array-like)."""
    e = np.asarray(e, dtype=np.int64)
    blk = (e >> 2).astype(np.uint64)
    lane = (e & 3).astype(np.int64)
    k0, k1 = int(seed) & _MASK32, (int(seed) >> 32) & _MASK32
    c0 = (blk & np.uint64(_MASK32)).astype(np.uint32)
    c1 = (blk >> np.uint64(32)).astype(np.uint32)
    c2 = np.full(e.shape, np.uint32(step & _MASK32), dtype=np.uint32)
    c3 = np.full(e.shape, np.uint32(query & _MASK32), dtype=np.uint32)
    w0, w1, w2, w3 = philox4x32_10(c0, c1, c2, c3, k0, k1)
    z0, z1 = box_muller(w0, w1)
    z2, z3 = box_muller(w2, w3)
    return np.select([lane == 0, lane == 1, lane == 2], [z0, z1, z2], z3).astype(np.float32)


def gauss_range(seed: int, step: int, query: int, e0: int, n: int) -> np.ndarray:
    """Z over the contiguous arena range [e0, e0 + n)."""
    return gauss(seed, step, query, np.arange(e0, e0 + n, dtype=np.int64))
