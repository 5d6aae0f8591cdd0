"""Pins for oracle/basis.py (Algorithm 1)."""
import numpy as np
import pytest

import synth
from oracle import basis


def _gapped(t=200, d=48, seed=0):
    """X with a clear spectral gap after the 8th singular value."""
    r = np.random.default_rng(seed)
    q, _ = np.linalg.qr(r.standard_normal((d, d)))
    sv = np.concatenate([np.linspace(20, 10, 8), np.linspace(3, 0.5, d - 8)])
    a, _ = np.linalg.qr(r.standard_normal((t, d)))
    return (a * sv) @ q.T


@pytest.mark.parametrize("r", [1, 4, 8])
def test_matches_brute_force_svd(r):
    x = _gapped()
    u, lam = basis.basis_init(x, r)
    _, s, vt = np.linalg.svd(x, full_matrices=False)
    assert basis.overlap(u, vt[:r].T) > 1 - 1e-10
    np.testing.assert_allclose(lam, s[:r] ** 2, rtol=1e-10)
    assert np.all(np.diff(lam) <= 0)


def test_orthonormal_and_canonical_sign():
    u, _ = basis.basis_init(_gapped(), 8)
    assert np.max(np.abs(u.T @ u - np.eye(8))) < 1e-5
    idx = np.argmax(np.abs(u), axis=0)
    assert np.all(u[idx, np.arange(8)] > 0)


def test_eckart_young_residual():
    x = _gapped(seed=2)
    r = 8
    u, _ = basis.basis_init(x, r)
    s = np.linalg.svd(x, compute_uv=False)
    res = x - (x @ u) @ u.T
    assert np.sum(res**2) == pytest.approx(np.sum(s[r:] ** 2), rel=1e-9)


def test_restricted_least_squares_gap():
    """Section 4: min ||X V_r B - R||^2 - min ||X dW - R||^2 = sum_{i>r} ||u_i^T R||^2."""
    x = _gapped(t=120, d=40, seed=3)
    rr = np.random.default_rng(4).standard_normal((120, 6))
    r = 8
    v, _ = basis.basis_init(x, r)
    full = np.linalg.lstsq(x, rr, rcond=None)
    f_star = np.sum((x @ full[0] - rr) ** 2)
    bsol = np.linalg.lstsq(x @ v, rr, rcond=None)[0]
    phi_v = np.sum((x @ v @ bsol - rr) ** 2)
    uu, s, _ = np.linalg.svd(x, full_matrices=False)
    rank = int(np.sum(s > 1e-10 * s[0]))
    gap = np.sum((uu[:, r:rank].T @ rr) ** 2)
    assert phi_v - f_star == pytest.approx(gap, rel=1e-8)


def test_recovers_planted_subspace():
    x, q = synth.planted_lowrank(2048, 256, n_dirs=16, frac=0.9, decay=0.8, seed=5)
    u, _ = basis.basis_init(x, 4)
    # top-4 basis lies in the planted span
    resid = u - q @ (q.T @ u)
    assert np.linalg.norm(resid) < 0.1


def test_too_few_tokens_is_an_error():
    with pytest.raises(ValueError):
        basis.basis_init(np.ones((3, 8)), 4)
