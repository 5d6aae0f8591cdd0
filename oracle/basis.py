"""One-shot activation basis, Algorithm 1 (oracle side).

Algorithm 1 runs one forward pass on a calibration batch, collects the input
activations X_l (tokens x d_in) of every adapted linear layer and keeps the top-r
right singular vectors V_{l,r} of X_l, frozen from then on (Section 3).  The right
singular vectors of X are the eigenvectors of the uncentred Gram X^T X with
eigenvalues sigma_i^2, so the oracle forms X^T X in float64 and calls a dense
symmetric eigensolver (LAPACK through NumPy / SciPy) as one step.

Conventions (this build's reading; the paper leaves them open): uncentred Gram;
eigenvalues unnormalised, in descending order; each basis column's sign is chosen
so that its largest-magnitude entry is positive (lowest index on ties); layers that
read the same input (q/k/v, gate/up) share one basis; fewer tokens than r is an
error.  The top-r subspace is only defined when lambda_r > lambda_{r+1}, so test
inputs have a gap there.

Pins (tests/test_oracle_basis.py): brute-force SVD of X on small inputs (the
subspace overlap ||U_a^T U_b||_F^2 / r of Section 5.3 equals 1), U^T U = I (the
theory's assumption, Appendix A), Eckart-Young ||X - X U U^T||_F^2 =
sum_{i>r} sigma_i^2, the restricted least-squares gap of Section 4
(sum_{i>r} ||u_i^T R||^2) against a direct lstsq, and recovery of a planted
subspace.
"""
from __future__ import annotations

import numpy as np


def gram(x: np.ndarray) -> np.ndarray:
    """Uncentred Gram X^T X in float64 (x: tokens x d)."""
    xf = np.asarray(x, dtype=np.float64)
    return xf.T @ xf


def canonical_sign(u: np.ndarray) -> np.ndarray:
    """Flip columns so the largest-|.| entry (first on ties) is positive."""
    u = np.array(u, dtype=np.float64, copy=True)
    idx = np.argmax(np.abs(u), axis=0)
    s = np.sign(u[idx, np.arange(u.shape[1])])
    s[s == 0] = 1.0
    return u * s[None, :]


def top_eigvecs(g: np.ndarray, r: int):
    """Top-r eigenpairs of a symmetric matrix, descending, canonical sign."""
    d = g.shape[0]
    if d > 4096:
        import scipy.linalg
        w, v = scipy.linalg.eigh(g, subset_by_index=[d - r, d - 1])
    else:
        w, v = np.linalg.eigh(g)
    order = np.argsort(w)[::-1][:r]
    return w[order], canonical_sign(v[:, order])


def basis_init(x: np.ndarray, r: int):
    """Algorithm 1 for one input site: returns (U [d][r] float64, eigenvalues [r])."""
    x = np.asarray(x)
    if r < 1 or x.shape[0] < r:
        raise ValueError("basis init needs 1 <= r <= number of calibration tokens")
    lam, u = top_eigvecs(gram(x), r)
    return u, lam


def overlap(ua: np.ndarray, ub: np.ndarray) -> float:
    """Subspace overlap ||U_a^T U_b||_F^2 / r (Section 5.3's stability measure)."""
    m = np.asarray(ua, dtype=np.float64).T @ np.asarray(ub, dtype=np.float64)
    return float((m * m).sum() / ua.shape[1])
