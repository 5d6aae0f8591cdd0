"""Pins for the oracle's perturbation generator (oracle/rng.py).

The paper fixes only that Z is standard Gaussian (Section 3; Algorithm 2 draws a
fresh Z per step and query).  The oracle is pinned by (1) a second implementation
written independently here with scalar Python integers and fp64-then-fp32
rounding (exact for +, -, *, /, sqrt since 53 >= 2*24 + 2), (2) the Gaussian
moments, including E||z||^6 = k(k+2)(k+4), the sixth moment Appendix A's proof
uses, (3) a Kolmogorov-Smirnov test, and (4) uniformity of the raw Philox words.
"""
import math
import struct

import numpy as np
import pytest
from scipy import stats

from oracle import rng


def f32(x: float) -> float:
    return struct.unpack("<f", struct.pack("<f", x))[0]


def philox_scalar(ctr, key):
    """Philox4x32-10 on Python ints (independent of the vectorised oracle)."""
    c = list(ctr)
    k = list(key)
    for i in range(10):
        if i > 0:
            k = [(k[0] + 0x9E3779B9) % 2**32, (k[1] + 0xBB67AE85) % 2**32]
        a = 0xD2511F53 * c[0]
        b = 0xCD9E8D57 * c[2]
        c = [(b >> 32) ^ c[1] ^ k[0], b % 2**32, (a >> 32) ^ c[3] ^ k[1], a % 2**32]
    return c


def ln_u1_scalar(w: int) -> float:
    n = (w >> 8) + 1
    e = n.bit_length() - 1                      # floor(log2 n)
    m = n / 2.0**e                              # exact, in [1, 2)
    if m >= f32(math.sqrt(2.0)):
        m *= 0.5
        e += 1
    s = f32(f32(m - 1.0) / f32(m + 1.0))
    s2 = f32(s * s)
    p = f32(1.0 / 9.0)
    for c in (1.0 / 7.0, 1.0 / 5.0, 1.0 / 3.0):
        p = f32(f32(p * s2) + f32(c))
    p = f32(f32(p * s2) + 1.0)
    lnm = f32(f32(s + s) * p)
    return f32(f32(float(e - 24) * f32(math.log(2.0))) + lnm)


def sincos_scalar(w: int):
    q = w >> 30
    f = float((w >> 8) & 0x3FFFFF) * 2.0**-22
    f2 = f32(f * f)
    h = math.pi / 2
    sp = f32((-1) ** 6 * h**13 / math.factorial(13))
    for k in range(5, -1, -1):
        sp = f32(f32(sp * f2) + f32((-1) ** k * h ** (2 * k + 1) / math.factorial(2 * k + 1)))
    sn = f32(f * sp)
    cp = f32((-1) ** 7 * h**14 / math.factorial(14))
    for k in range(6, -1, -1):
        cp = f32(f32(cp * f2) + f32((-1) ** k * h ** (2 * k) / math.factorial(2 * k)))
    cs = cp
    return [(cs, sn), (-sn, cs), (-cs, -sn), (sn, -cs)][q]


def gauss_scalar(seed: int, step: int, query: int, e: int) -> float:
    blk = e >> 2
    w = philox_scalar([blk % 2**32, blk >> 32, step, query], [seed % 2**32, seed >> 32])
    pair = (w[0], w[1]) if (e & 3) < 2 else (w[2], w[3])
    r = f32(math.sqrt(f32(-2.0 * ln_u1_scalar(pair[0]))))
    c, s = sincos_scalar(pair[1])
    return f32(r * (c if (e & 1) == 0 else s))


CASES = [
    (0, 1, 0), (12345, 7, 0), (2**40 + 17, 3, 5), (2**64 - 1, 2**32 - 1, 2**32 - 1), (99, 0, 1),
]


@pytest.mark.parametrize("seed,step,query", CASES)
def test_matches_scalar_implementation(seed, step, query):
    r = np.random.default_rng(seed % 1000)
    idx = np.concatenate([
        np.arange(0, 64),
        r.integers(0, 2**31, 200),
        np.array([2**32 - 4, 2**32 - 1, 2**32, 2**32 + 3, 2**34 + 2, 44_040_191, 104_857_599]),
        r.integers(2**32, 2**40, 50),
    ]).astype(np.int64)
    got = rng.gauss(seed, step, query, idx)
    want = np.array([gauss_scalar(seed, step, query, int(e)) for e in idx], dtype=np.float32)
    np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32))


def test_philox_words_match_scalar():
    r = np.random.default_rng(1)
    for _ in range(50):
        ctr = [int(x) for x in r.integers(0, 2**32, 4, dtype=np.uint64)]
        key = [int(x) for x in r.integers(0, 2**32, 2, dtype=np.uint64)]
        got = rng.philox4x32_10(*[np.array([c], np.uint32) for c in ctr], key[0], key[1])
        assert [int(g[0]) for g in got] == philox_scalar(ctr, key)


def test_series_accuracy_against_libm():
    """The series ln/sin/cos stay within a few fp32 ulps of the true functions."""
    w = np.random.default_rng(3).integers(0, 2**32, 200_000, dtype=np.uint64).astype(np.uint32)
    lnu = rng._ln_u1(w).astype(np.float64)
    exact = np.log((((w >> 8) + 1).astype(np.float64)) * 2.0**-24)
    assert np.all(np.abs(lnu - exact) <= 1e-6 * np.maximum(1.0, np.abs(exact)))
    c, s = rng._quarter_turn_sincos(w)
    ang = ((w >> 30).astype(np.float64) + ((w >> 8) & 0x3FFFFF).astype(np.float64) * 2.0**-22) * (np.pi / 2)
    assert np.max(np.abs(c - np.cos(ang))) < 5e-7
    assert np.max(np.abs(s - np.sin(ang))) < 5e-7


@pytest.fixture(scope="module")
def big_sample():
    return rng.gauss_range(2024, 1, 0, 0, 4_000_000).astype(np.float64)


def test_moments(big_sample):
    z = big_sample
    n = z.size
    assert abs(z.mean()) < 5 / math.sqrt(n)
    assert abs((z**2).mean() - 1) < 5 * math.sqrt(2 / n)
    assert abs((z**4).mean() - 3) < 5 * math.sqrt(96 / n)
    assert abs((z**3).mean()) < 5 * math.sqrt(15 / n)
    assert np.abs(z).max() <= math.sqrt(2 * 24 * math.log(2)) + 1e-5


@pytest.mark.parametrize("k", [4, 8])
def test_sixth_moment_of_norm(big_sample, k):
    """E||z||^6 = k(k+2)(k+4) for z ~ N(0, I_k) (Appendix A, bound on E||z||^3)."""
    blocks = big_sample.reshape(-1, k)
    nrm6 = (blocks**2).sum(axis=1) ** 3
    mk = k * (k + 2) * (k + 4)
    m12 = math.prod(k + 2 * i for i in range(6))
    se = math.sqrt((m12 - mk**2) / blocks.shape[0])
    assert abs(nrm6.mean() - mk) < 5 * se


def test_estimator_second_moment(big_sample):
    """E<g,z>^2||z||^2 = (k+2)||g||^2 and E<g,z>z = g (Section 4, variance of a_t)."""
    k = 8
    zb = big_sample.reshape(-1, k)
    g = np.array([0.5, -1.0, 2.0, 0.0, 0.25, 1.5, -0.75, 1.0])
    a = (zb @ g)[:, None] * zb
    n = zb.shape[0]
    assert np.all(np.abs(a.mean(axis=0) - g) < 6 * a.std(axis=0) / math.sqrt(n))
    sq = (a**2).sum(axis=1)
    assert abs(sq.mean() - (k + 2) * (g @ g)) < 6 * sq.std() / math.sqrt(n)


def test_ks_normal(big_sample):
    res = stats.kstest(big_sample[:1_000_000], "norm")
    assert res.pvalue > 1e-4


def test_philox_word_uniformity():
    n = 1 << 18
    blk = np.arange(n, dtype=np.uint32)
    words = rng.philox4x32_10(blk, np.zeros(n, np.uint32), np.full(n, 5, np.uint32),
                              np.zeros(n, np.uint32), 77, 0)
    for w in words:
        counts = np.bincount((w >> 24).astype(np.int64), minlength=256)
        chi2 = ((counts - n / 256) ** 2 / (n / 256)).sum()
        assert stats.chi2.sf(chi2, 255) > 1e-5
        bits = np.unpackbits(w.view(np.uint8)).reshape(-1, 32).mean(axis=0)
        assert np.all(np.abs(bits - 0.5) < 6 * 0.5 / math.sqrt(n))


def test_streams_are_distinct_and_deterministic():
    a = rng.gauss_range(5, 1, 0, 0, 100_000)
    b = rng.gauss_range(5, 2, 0, 0, 100_000)
    c = rng.gauss_range(5, 1, 1, 0, 100_000)
    d = rng.gauss_range(6, 1, 0, 0, 100_000)
    np.testing.assert_array_equal(a, rng.gauss_range(5, 1, 0, 0, 100_000))
    for other in (b, c, d):
        assert abs(np.corrcoef(a, other)[0, 1]) < 0.02
    # lanes of one counter block are not correlated either
    lanes = a.reshape(-1, 4)
    cc = np.corrcoef(lanes.T)
    assert np.max(np.abs(cc - np.eye(4))) < 0.03
    # any sub-range equals the same indices of the full range
    np.testing.assert_array_equal(rng.gauss_range(5, 1, 0, 1234, 999), a[1234:1234 + 999])
