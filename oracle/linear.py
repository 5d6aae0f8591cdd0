"""Adapted linear layer with the +/- coefficient perturbation (oracle side).

Paper, Section 3 ("ZO-Act"): each adapted layer's weight is W_eff = W + V_r B with
W and V_r frozen and B trainable (zero at initialisation); a perturbation Z in the
r x n coefficient space gives W + V_r (B + mu Z), evaluated without forming W_eff
as Y+ = X W + (X V_r)(B + mu Z).  The two-sided step evaluates this with +mu Z and
with -mu Z on stacked halves of the batch.

Orientation used by the library (PyTorch style): x [T][d_in], W [d_out][d_in],
U^T [r][d_in] (U = V_r), C = B^T [d_out][r], Z [d_out][r], so that
    y_h = x_h W^T + b + (x_h U) C_h^T,   C_h = C + s_h eps Z,  s = (+1, -1).
Coefficient C[n][i] of a layer whose block starts at arena offset `off` has arena
index off + n * r + i; Z at that index comes from oracle.rng.

Modes:
  "fp32": all products and sums in float64; inputs are fp32 values.
  "bf16": x, W, U, P = xU, C_h and y are bf16 values; products are summed in
          float64, and each stored tensor is rounded once (oracle.numerics).
          C_h = bf16(C + s (eps Z)) with the sum formed in fp32.

Pins (tests/test_oracle_core.py): C = 0, eps = 0 reproduces x W^T + b bitwise;
the factored form equals x (W + C U^T)^T (materialised W_eff); y+ - y- = 2 eps
(xU) Z^T in fp64; INT4 dequantisation error bound.
"""
from __future__ import annotations

import numpy as np

from . import rng
from .numerics import rne_bf16


def coef_index(off: int, n_rows: int, r: int, row0: int = 0) -> np.ndarray:
    """Arena indices [n_rows][r] of coefficient rows row0 .. row0+n_rows of a block at `off`."""
    rows = np.arange(row0, row0 + n_rows, dtype=np.int64)[:, None]
    return off + rows * r + np.arange(r, dtype=np.int64)[None, :]


def z_block(seed: int, step: int, query: int, off: int, n_rows: int, r: int, row0: int = 0) -> np.ndarray:
    """Z [n_rows][r] (float32) for a coefficient block."""
    return rng.gauss(seed, step, query, coef_index(off, n_rows, r, row0))


def perturbed_coeffs(c: np.ndarray, z: np.ndarray, eps: float, sign: int, mode: str) -> np.ndarray:
    """C + sign eps Z for sign in {-1, 0, +1}: fp32 ops (eps*z first) then bf16 rounding in
    bf16 mode; float64 in fp32 mode.  Sign 0 is the unperturbed C (Algorithm 2's reference
    loss in the one-sided form)."""
    if mode == "bf16":
        c32 = c.astype(np.float32)
        if sign == 0:
            return rne_bf16(c32).astype(np.float64)
        ez = np.float32(eps) * z.astype(np.float32)
        ch = (c32 + ez) if sign > 0 else (c32 - ez)
        return rne_bf16(ch.astype(np.float32)).astype(np.float64)
    if sign == 0:
        return c.astype(np.float64)
    return c.astype(np.float64) + sign * float(np.float32(eps)) * z.astype(np.float64)


def project(x: np.ndarray, ut: np.ndarray, mode: str) -> np.ndarray:
    """P = x U for x [T][d_in], U^T [r][d_in]; bf16-rounded in bf16 mode."""
    p = x.astype(np.float64) @ ut.astype(np.float64).T
    return rne_bf16(p.astype(np.float32)).astype(np.float64) if mode == "bf16" else p


def adapted_linear(x, w, bias, ut, c, z, eps, sign, mode, p=None, round_out=True):
    """One half of the adapted linear: x W^T + b + (x U)(C + sign eps Z)^T.

    Returns float64 values (bf16-rounded when mode == "bf16" and round_out).
    r = 0 layers (ut is None) reduce to x W^T + b.
    """
    y = x.astype(np.float64) @ w.astype(np.float64).T
    if ut is not None and ut.shape[0] > 0:
        if p is None:
            p = project(x, ut, mode)
        ch = perturbed_coeffs(c, z, eps, sign, mode)
        y = y + p @ ch.T
    if bias is not None:
        y = y + bias.astype(np.float64)[None, :]
    if mode == "bf16" and round_out:
        y = rne_bf16(y.astype(np.float32)).astype(np.float64)
    return y


def adapted_linear_pm(x_pm, w, bias, ut, c, eps, seed, step, query, off, mode, p_pm=None):
    """Both halves: y_pm[0] with C + eps Z, y_pm[1] with C - eps Z (x_pm [2][T][d_in])."""
    r = 0 if ut is None else ut.shape[0]
    z = z_block(seed, step, query, off, w.shape[0], r) if r else None
    out = []
    for h, sign in ((0, +1), (1, -1)):
        p = None if p_pm is None else p_pm[h]
        out.append(adapted_linear(x_pm[h], w, bias, ut, c, z, eps, sign, mode, p=p))
    return np.stack(out)


def dequant_int4(packed: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """INT4 group-128 weights to bf16 values: w = bf16(float(q) * float(s)).

    packed [N][K/2] uint8, even k in the low nibble, two's complement in [-7, 7];
    scales [N][K/128] bf16 values.  The product can need 11 significand bits, so the
    bf16 rounding is part of the dequantised value.
    """
    packed = np.asarray(packed, dtype=np.uint8)
    lo = (packed & 0xF).astype(np.int16)
    hi = (packed >> 4).astype(np.int16)
    lo = np.where(lo >= 8, lo - 16, lo)
    hi = np.where(hi >= 8, hi - 16, hi)
    n = packed.shape[0]
    q = np.empty((n, packed.shape[1] * 2), dtype=np.float32)
    q[:, 0::2] = lo
    q[:, 1::2] = hi
    s = np.repeat(np.asarray(scales, dtype=np.float32), 128, axis=1)
    return rne_bf16((q * s).astype(np.float32))
