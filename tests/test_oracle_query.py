"""Pins for the one-sided q-query form of Algorithm 2 in the oracle (oracle/adam.py
query_coeffs, query_estimate, zo_adam_q, zo_sgd_q; oracle/linear.py sign 0;
oracle/model.py zo_step_q).

Section 3 averages q forward differences against the unperturbed loss:
g = (1/q) sum_j (L(B + mu Z^(j)) - L(B)) / mu * Z^(j).  The pins evaluate real loss
functions at perturbed coefficients and compare with what the mathematics fixes: the
closed form of the estimate for a linear loss, its agreement with the two-sided
difference there, its unbiasedness for a quadratic loss over many queries, and the
unperturbed evaluation (sign 0) against eps = 0.
"""
import math

import numpy as np

import synth
from oracle import adam, linear, loss, rng
from oracle import model as om
from oracle.basis import basis_init


def _layer(t=32, k=32, n=16, r=4, seed=5):
    x = synth.bf16_round(synth.normal((t, k), 1.0, seed, 1))
    w = synth.bf16_round(synth.normal((n, k), 0.02, seed, 2))
    b = synth.bf16_round(synth.normal((n,), 0.1, seed, 3))
    u, _ = basis_init(x, r)
    return x, w, b, u.T.astype(np.float32), synth.normal((n, r), 0.01, seed, 4)


def _zs(seed, t, q, k):
    return np.stack([rng.gauss_range(seed, t, j, 0, k) for j in range(1, q + 1)])


def test_linear_loss_closed_form_and_normalisation():
    """For f(C) = <G, C> at C = 0, a_j = <G, Z_j> and the estimate is (1/q) Z^T Z G."""
    k, q, eps = 40, 3, 1e-2
    G = synth.normal((k,), 1.0, 2, 2).astype(np.float64)
    zs = _zs(9, 4, q, k)

    def f(c):
        return float(G @ c)

    losses = [f(np.zeros(k))] + [f(np.float32(eps) * zs[j].astype(np.float64)) for j in range(q)]
    got = adam.query_estimate(adam.query_coeffs(losses, eps), zs).astype(np.float64)
    z64 = zs.astype(np.float64)
    want = z64.T @ (z64 @ G) / q
    np.testing.assert_allclose(got, want, rtol=2e-5, atol=2e-5 * np.abs(want).max())
    # dividing by q + 1 or by 2 eps, or differencing consecutive losses, would miss this
    assert np.abs(got - want).max() < 0.05 * np.abs(want).max() / q


def test_one_query_equals_two_sided_on_linear_loss():
    """With a linear loss the one-sided and the two-sided differences give the same
    estimate (the second-order term they differ by vanishes)."""
    k, eps = 24, 1e-2
    G = synth.normal((k,), 1.0, 3, 3).astype(np.float64)
    c = synth.normal((k,), 0.1, 3, 4).astype(np.float32)
    z = rng.gauss_range(4, 2, 1, 0, k)
    e32 = np.float32(eps)
    f = lambda cc: np.float32(G @ cc.astype(np.float64))
    one = adam.query_estimate(adam.query_coeffs([f(c), f(c + e32 * z)], eps), z[None])
    two = adam.projected_grad(f(c + e32 * z), f(c - e32 * z), eps) * z
    np.testing.assert_allclose(one, two, rtol=1e-3, atol=1e-3 * np.abs(two).max())


def test_quadratic_loss_unbiased_over_many_queries():
    """phi(C) = MSE of one adapted layer is quadratic in C; E[a Z] = grad phi for Gaussian
    Z (the second-order term has zero third moment), so the q-query average converges to
    the gradient at the 1/sqrt(q) rate."""
    x, w, b, ut, c = _layer()
    tgt = synth.normal((x.shape[0], w.shape[0]), 0.5, 9, 8).astype(np.float64)
    p = x.astype(np.float64) @ ut.astype(np.float64).T
    base = x.astype(np.float64) @ w.astype(np.float64).T + b
    phi = lambda cc: loss.mse(base + p @ cc.T, tgt)
    res = base + p @ c.astype(np.float64).T - tgt
    grad = (2.0 / res.size * res.T @ p).reshape(-1)
    n, r = c.shape
    q, eps = 3000, 1e-2
    zs = np.stack([linear.z_block(13, 7, j, 0, n, r).reshape(-1) for j in range(1, q + 1)])
    e32 = float(np.float32(eps))
    c64 = c.astype(np.float64)
    losses = [phi(c64)] + [phi(c64 + e32 * zs[j].reshape(n, r)) for j in range(q)]
    g = adam.query_estimate(adam.query_coeffs(losses, eps), zs).astype(np.float64)
    per = (np.asarray(losses[1:]) - losses[0])[:, None] / e32 * zs.astype(np.float64)
    se = per.std(axis=0) / math.sqrt(q)
    assert np.all(np.abs(g - grad) < 6 * se)
    # a sign error or a factor 2 on eps is far outside that band
    assert np.abs(-g - grad).max() > 6 * se.max() and np.abs(0.5 * g - grad).max() > 6 * se.max()


def test_update_given_estimate_and_guard():
    k = 10
    c = synth.normal((k,), 0.1, 1, 1).astype(np.float32)
    m = np.zeros(k, np.float32)
    z = rng.gauss_range(2, 1, 1, 0, k)
    losses = [np.float32(1.25), np.float32(1.5)]
    hp = adam.adam_scalars(1e-3, 1)
    a = adam.query_coeffs(losses, 1e-3)
    # q = 1: the estimate is a_1 Z exactly, so the q-query update is the two-sided one's
    # with g = a_1 (same operation order from there on)
    c1, m1, v1, st = adam.zo_adam_q(c, m, m, losses, z[None], 1e-3, hp)
    c2, m2, v2, _ = adam.zo_adam(c, m, m, a[0], z, hp)
    assert st == 0
    np.testing.assert_array_equal(c1, c2)
    np.testing.assert_array_equal(v1, v2)
    # SGD moves against the estimate by lr
    s1, _ = adam.zo_sgd_q(c, losses, z[None], 1e-3, 0.5)
    np.testing.assert_allclose(s1, c - 0.5 * a[0] * z, rtol=1e-6, atol=1e-7)
    # a non-finite loss leaves everything unchanged and raises the status bit
    c3, m3, v3, st = adam.zo_adam_q(c, m, m, [np.float32(1.0), np.float32(np.inf)], z[None], 1e-3, hp)
    assert st == 1 and np.array_equal(c3, c)
    _, st = adam.zo_sgd_q(c, [np.float32(np.nan), np.float32(1.0)], z[None], 1e-3, 0.5)
    assert st == 1


def test_sign_zero_is_the_unperturbed_layer():
    x, w, b, ut, c = _layer()
    z = linear.z_block(1, 1, 3, 0, w.shape[0], ut.shape[0])
    for mode in ("fp32", "bf16"):
        y0 = linear.adapted_linear(x, w, b, ut, c, z, 1e-2, 0, mode)
        ye = linear.adapted_linear(x, w, b, ut, c, z, 0.0, +1, mode)
        np.testing.assert_array_equal(y0, ye)


def test_model_step_q_losses_and_reference():
    """zo_step_q on the tiny model: L is the unperturbed loss, L_j the +eps Z^(j) losses,
    and with eps -> small the estimate's directional component tracks the two-sided one."""
    m = om.Model(synth.TINY, 0, "fp32")
    m.basis_init(synth.uniform_tokens(4, 32, synth.TINY.vocab, 0, 1))
    tok = synth.uniform_tokens(2, 32, synth.TINY.vocab, 0, 2)
    k = m.k
    c = synth.normal((k,), 0.02, 5, 5).astype(np.float32)
    zero = np.zeros(k, np.float32)
    c1, m1, v1, losses = om.zo_step_q(m, tok, c, zero, zero, 1, 1e-3, 1e-3, 21, 2)
    assert len(losses) == 3
    assert losses[0] == m.loss(tok, c, +1, 0.0, (21, 1, 1))
    assert losses[2] == m.loss(tok, c, +1, 1e-3, (21, 1, 2))
    # first Adam step moves every coefficient by about lr against its estimate
    a = adam.query_coeffs(losses, 1e-3)
    g = adam.query_estimate(a, _zs(21, 1, 2, k))
    moved = c1 - c
    big = np.abs(g) > 1e-3 * np.abs(g).max()
    assert np.all(np.sign(moved[big]) == -np.sign(g[big]))
    np.testing.assert_allclose(np.abs(moved[big]), 1e-3, rtol=1e-2)
