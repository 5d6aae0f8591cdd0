"""Projected-gradient scalar and ZO-Adam on the coefficient arena (oracle side).

Algorithm 2 forms the estimate g_B = a Z from loss differences and updates every
B_l with a first-order optimiser; Section 5 and Appendix B use Adam with weight
decay 0 and a "constant with warmup" schedule.  The two-sided form used on the
hot path is a = (L+ - L-) / (2 eps) with the same regenerated Z.

The paper does not give Adam's constants; the reading here is PyTorch's Adam:
beta1 = 0.9, beta2 = 0.999, eps_A = 1e-8, bias correction on.  Host-side scalars
are computed in float64 and rounded once to fp32:
    step_size = lr_t / (1 - beta1^t), inv_sqrt_bc2 = 1 / sqrt(1 - beta2^t),
    one_minus_beta1 = 1 - beta1, one_minus_beta2 = 1 - beta2.
Per coefficient, in fp32, one rounding per operation, in this order:
    gh = g * z                         (+ wd * c when weight decay is non-zero)
    m  = beta1 * m + one_minus_beta1 * gh
    v  = beta2 * v + one_minus_beta2 * (gh * gh)
    d  = sqrt(v) * inv_sqrt_bc2 + eps_A
    c  = c - step_size * (m / d)
with C stored bf16 (rounded to nearest even after the update) when requested.  A
non-finite g leaves C, m, v unchanged and raises bit 0 of the status word.

Pins (tests/test_oracle_core.py): with m = v = 0 the first step moves each
coefficient by lr * gh / (|gh| + eps_A) (about lr * sign(gh)) within a few fp32
ulps; g = 0 leaves C unchanged; bias-corrected moments of a constant gradient
stay equal to it.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from .numerics import rne_bf16

_F = np.float32


@dataclass
class AdamScalars:
    lr: float
    beta1: float
    beta2: float
    eps: float
    weight_decay: float
    t: int
    step_size: np.float32
    inv_sqrt_bc2: np.float32
    one_minus_beta1: np.float32
    one_minus_beta2: np.float32


def adam_scalars(lr: float, t: int, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
                 weight_decay: float = 0.0) -> AdamScalars:
    """Host-side Adam scalars for step t >= 1 (float64 then one fp32 rounding)."""
    if t < 1:
        raise ValueError("Adam step t starts at 1")
    return AdamScalars(lr, beta1, beta2, eps, weight_decay, t,
                       _F(lr / (1.0 - beta1 ** t)), _F(1.0 / math.sqrt(1.0 - beta2 ** t)),
                       _F(1.0 - beta1), _F(1.0 - beta2))


def projected_grad(loss_plus, loss_minus, eps: float) -> np.float32:
    """a = (L+ - L-) / (2 eps) in fp32 (2 eps formed as eps + eps, exact)."""
    e = _F(eps)
    return _F(_F(loss_plus) - _F(loss_minus)) / (e + e)


def zo_adam(c: np.ndarray, m: np.ndarray, v: np.ndarray, g, z: np.ndarray, hp: AdamScalars,
            c_bf16: bool = False):
    """One ZO-Adam update.  Returns (c, m, v, status); inputs are not modified."""
    g = _F(g)
    if not np.isfinite(g):
        return c.copy(), m.copy(), v.copy(), 1
    return adam_on_estimate(c, m, v, g * np.asarray(z, dtype=np.float32), hp, c_bf16)


def adam_on_estimate(c: np.ndarray, m: np.ndarray, v: np.ndarray, gh: np.ndarray, hp: AdamScalars,
                     c_bf16: bool = False):
    """Adam on a given per-coefficient estimate gh (fp32), in the order stated above."""
    c32 = np.asarray(c, dtype=np.float32)
    gh = np.asarray(gh, dtype=np.float32)
    if hp.weight_decay != 0.0:
        gh = gh + _F(hp.weight_decay) * c32
    m1 = _F(hp.beta1) * np.asarray(m, dtype=np.float32) + hp.one_minus_beta1 * gh
    v1 = _F(hp.beta2) * np.asarray(v, dtype=np.float32) + hp.one_minus_beta2 * (gh * gh)
    d = np.sqrt(v1) * hp.inv_sqrt_bc2 + _F(hp.eps)
    c1 = c32 - hp.step_size * (m1 / d)
    if c_bf16:
        c1 = rne_bf16(c1)
    return c1.astype(np.float32), m1.astype(np.float32), v1.astype(np.float32), 0


def zo_sgd(c: np.ndarray, g, z: np.ndarray, lr: float, c_bf16: bool = False):
    """ZO-SGD variant (the paper's 'Full SGD' row): c = c - lr * (g * z), fp32."""
    g = _F(g)
    if not np.isfinite(g):
        return np.asarray(c).copy(), 1
    c1 = np.asarray(c, dtype=np.float32) - _F(lr) * (g * np.asarray(z, dtype=np.float32))
    return (rne_bf16(c1) if c_bf16 else c1).astype(np.float32), 0


# ------------------------------------------------------------------ one-sided, q queries
# Section 3's averaged forward-difference estimate and the inner loop of Algorithm 2:
# with the unperturbed loss L and L_j = L(B + mu Z^(j)) for j = 1..q,
#     a_j = (L_j - L) / mu,    g_B = (1/q) sum_j a_j Z^(j),
# accumulated in the algorithm's order (j ascending, then one division by q).  Reading of
# the precision: fp32, one rounding per operation; Z^(j) is Z(seed, t, query j).

def query_coeffs(losses, eps: float) -> np.ndarray:
    """a_j = (L_j - L_0) / eps for j = 1..q in fp32 (losses = [L, L_1, .., L_q])."""
    ls = np.asarray(losses, dtype=np.float32)
    return (ls[1:] - ls[0]) / _F(eps)


def query_estimate(a: np.ndarray, zs: np.ndarray) -> np.ndarray:
    """g = (sum_j a_j Z^(j)) / q for zs [q][k] (fp32, j ascending)."""
    acc = np.zeros(zs.shape[1], np.float32)
    for j in range(zs.shape[0]):
        acc = acc + _F(a[j]) * zs[j].astype(np.float32)
    return acc / _F(zs.shape[0])


def zo_adam_q(c, m, v, losses, zs, eps: float, hp: AdamScalars, c_bf16: bool = False):
    """One-sided q-query ZO-Adam update.  Returns (c, m, v, status)."""
    a = query_coeffs(losses, eps)
    if not np.all(np.isfinite(a)):
        return np.asarray(c).copy(), np.asarray(m).copy(), np.asarray(v).copy(), 1
    return adam_on_estimate(c, m, v, query_estimate(a, zs), hp, c_bf16)


def zo_sgd_q(c, losses, zs, eps: float, lr: float, c_bf16: bool = False):
    """One-sided q-query ZO-SGD update: c = c - lr * g.  Returns (c, status)."""
    a = query_coeffs(losses, eps)
    if not np.all(np.isfinite(a)):
        return np.asarray(c).copy(), 1
    c1 = np.asarray(c, dtype=np.float32) - _F(lr) * query_estimate(a, zs)
    return (rne_bf16(c1) if c_bf16 else c1).astype(np.float32), 0
