"""Pins for oracle/numerics.py, oracle/linear.py, oracle/loss.py and oracle/adam.py.

Every check compares the oracle with something the paper or the mathematics fixes,
not with a retyped copy of the oracle's own formula.
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import adam, linear, loss, rng
from oracle.basis import basis_init
from oracle.numerics import rne_bf16


# ---------------------------------------------------------------- bf16 rounding
def test_rne_bf16_matches_torch_cast():
    r = np.random.default_rng(0)
    bits = r.integers(0, 2**32, 2_000_000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x) & (np.abs(x) < 1e38)]
    want = torch.from_numpy(x.copy()).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(rne_bf16(x).view(np.uint32), want.view(np.uint32))


def test_rne_bf16_ties_to_even():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to the even mantissa (1.0)
    assert rne_bf16(np.float32(1 + 2**-8)) == np.float32(1.0)
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 and 1 + 2^-6: ties to 1 + 2^-6
    assert rne_bf16(np.float32(1 + 3 * 2**-8)) == np.float32(1 + 2**-6)


# ---------------------------------------------------------------- adapted linear
def _layer(t=40, k=64, n=48, r=8, seed=3):
    x = synth.bf16_round(synth.normal((t, k), 1.0, seed, 1))
    w = synth.bf16_round(synth.normal((n, k), 0.02, seed, 2))
    b = synth.bf16_round(synth.normal((n,), 0.1, seed, 3))
    u, _ = basis_init(x, r)
    ut = u.T.astype(np.float32)
    c = synth.normal((n, r), 0.01, seed, 4)
    return x, w, b, ut, c


def test_zero_coefficients_reproduce_base_layer_bitwise():
    """B = 0 at initialisation gives W_eff = W (Section 3; Algorithm 2 init)."""
    x, w, b, ut, c = _layer()
    zero = np.zeros_like(c)
    y = linear.adapted_linear_pm(np.stack([x, x]), w, b, synth.bf16_round(ut), zero, 0.0, 1, 1, 0, 0, "bf16")
    base = rne_bf16((x.astype(np.float64) @ w.astype(np.float64).T + b).astype(np.float32))
    np.testing.assert_array_equal(y[0], base)
    np.testing.assert_array_equal(y[1], base)


def test_factored_equals_materialised_effective_weight():
    """X W + (X V_r)(B + mu Z) = X (W + V_r (B + mu Z)) (Section 3, both forms)."""
    x, w, b, ut, c = _layer()
    eps, seed, step, off = 1e-3, 11, 4, 100
    y = linear.adapted_linear_pm(np.stack([x, x]), w, b, ut, c, eps, seed, step, 0, off, "fp32")
    z = rng.gauss(seed, step, 0, off + np.arange(w.shape[0])[:, None] * ut.shape[0] + np.arange(ut.shape[0]))
    u = ut.astype(np.float64).T
    for h, sgn in ((0, 1.0), (1, -1.0)):
        ch = c.astype(np.float64) + sgn * float(np.float32(eps)) * z.astype(np.float64)
        w_eff = w.astype(np.float64) + ch @ u.T          # [n][k] = (W_paper + V_r B)^T
        want = x.astype(np.float64) @ w_eff.T + b
        np.testing.assert_allclose(y[h], want, rtol=1e-12, atol=1e-12)


def test_pm_difference_is_rank_r_output_perturbation():
    """y+ - y- = 2 eps (X U) Z^T, and with U = V_r this equals 2 eps U_r D_r Z (Section 3, Motivation)."""
    x, w, b, ut, c = _layer()
    eps, seed, step = 1e-2, 2, 9
    y = linear.adapted_linear_pm(np.stack([x, x]), w, b, ut, c, eps, seed, step, 0, 0, "fp32")
    z = linear.z_block(seed, step, 0, 0, w.shape[0], ut.shape[0]).astype(np.float64)
    xu = x.astype(np.float64) @ ut.astype(np.float64).T
    np.testing.assert_allclose(y[0] - y[1], 2 * float(np.float32(eps)) * xu @ z.T, rtol=1e-9, atol=1e-12)
    # X V_r = U_r D_r from the thin SVD of X
    uu, dd, vt = np.linalg.svd(x.astype(np.float64), full_matrices=False)
    r = ut.shape[0]
    sgn = np.sign(np.sum(vt[:r] * ut.astype(np.float64), axis=1))
    np.testing.assert_allclose(xu, (uu[:, :r] * dd[:r]) * sgn, rtol=1e-4, atol=1e-4)


def test_coefficient_index_layout():
    idx = linear.coef_index(1000, 3, 4)
    assert idx.tolist() == [[1000, 1001, 1002, 1003], [1004, 1005, 1006, 1007], [1008, 1009, 1010, 1011]]


def test_int4_dequant_bound_and_packing():
    w = synth.bf16_round(synth.normal((16, 256), 0.02, 5, 1))
    w[3, 128:256] = 0.0                                  # an all-zero group
    packed, s = synth.quantize_int4_g128(w)
    what = linear.dequant_int4(packed, s)
    srep = np.repeat(s, 128, axis=1)
    ulp = np.abs(what) * 2.0**-8
    assert np.all(np.abs(w - what) <= srep / 2 + ulp / 2 + 1e-12)
    assert np.all(what[3, 128:] == 0)
    # low nibble holds the even column: unpack column 0 and 1 of row 0 by hand
    q0 = int(packed[0, 0] & 0xF)
    q1 = int(packed[0, 0] >> 4)
    q0 = q0 - 16 if q0 >= 8 else q0
    q1 = q1 - 16 if q1 >= 8 else q1
    assert what[0, 0] == rne_bf16(np.float32(q0 * s[0, 0])) and what[0, 1] == rne_bf16(np.float32(q1 * s[0, 0]))
    assert -7 <= q0 <= 7 and -7 <= q1 <= 7
    # the group absmax maps to +/-7
    g = np.abs(w[0, :128])
    j = int(np.argmax(g))
    assert abs(what[0, j]) == rne_bf16(np.float32(7 * s[0, 0]))


# ---------------------------------------------------------------- losses
def test_uniform_logits_give_log_vocab():
    v = 512
    tok = synth.uniform_tokens(3, 17, v, 0, 1)
    assert loss.next_token_ce(np.zeros((3, 17, v)), tok) == pytest.approx(math.log(v), rel=1e-14)


def test_ce_against_torch():
    r = np.random.default_rng(0)
    lg = r.standard_normal((2, 9, 33)) * 3
    tok = r.integers(0, 33, (2, 9))
    want = torch.nn.functional.cross_entropy(torch.from_numpy(lg[:, :-1].reshape(-1, 33)),
                                             torch.from_numpy(tok[:, 1:].reshape(-1))).item()
    assert loss.next_token_ce(lg, tok) == pytest.approx(want, rel=1e-12)


def test_loss_symmetry_under_z_sign():
    """L+(Z) = L-(-Z): the + half with Z is the - half with -Z."""
    x, w, b, ut, c = _layer()
    tgt = synth.normal((x.shape[0], w.shape[0]), 1.0, 9, 9)
    z = linear.z_block(1, 1, 0, 0, w.shape[0], ut.shape[0])
    yp = linear.adapted_linear(x, w, b, ut, c, z, 1e-3, +1, "fp32")
    ym = linear.adapted_linear(x, w, b, ut, c, -z, 1e-3, -1, "fp32")
    assert loss.mse(yp, tgt) == loss.mse(ym, tgt)
    assert loss.mse(tgt, tgt) == 0.0


# ---------------------------------------------------------------- estimator
def test_central_difference_exact_on_quadratic_and_mc_moments():
    """For the MSE of one adapted layer phi(C) is quadratic in C, so the two-sided
    difference equals <grad phi, Z> up to rounding; averaged over many Z the estimate
    g Z is unbiased for grad phi (Section 4)."""
    x, w, b, ut, c = _layer(t=32, k=32, n=16, r=4)
    tgt = synth.normal((x.shape[0], w.shape[0]), 0.5, 9, 8).astype(np.float64)
    p = x.astype(np.float64) @ ut.astype(np.float64).T
    base = x.astype(np.float64) @ w.astype(np.float64).T + b

    def phi(cc):
        return loss.mse(base + p @ cc.T, tgt)

    res = base + p @ c.astype(np.float64).T - tgt
    grad = 2.0 / res.size * res.T @ p                     # d phi / d C, [n][r]
    eps = 1e-3
    est = []
    for step in range(1, 4001):
        z = linear.z_block(77, step, 0, 0, w.shape[0], ut.shape[0]).astype(np.float64)
        e32 = float(np.float32(eps))
        fd = (phi(c + e32 * z) - phi(c - e32 * z)) / (2 * e32)
        if step <= 5:
            assert fd == pytest.approx(float((grad * z).sum()), rel=1e-7, abs=1e-12)
        est.append(fd * z)
    est = np.array(est)
    k = grad.size
    mean = est.mean(axis=0)
    se = est.std(axis=0) / math.sqrt(len(est))
    assert np.all(np.abs(mean - grad) < 6 * se)
    sq = (est**2).sum(axis=(1, 2))
    assert abs(sq.mean() - (k + 2) * (grad**2).sum()) < 6 * sq.std() / math.sqrt(len(est))


def test_central_difference_error_decays_quadratically():
    """Smooth non-quadratic phi: the central-difference error of the directional
    derivative falls ~100x per decade of eps (remainder bound, Appendix A)."""
    x, w, b, ut, c = _layer(t=16, k=32, n=8, r=4)
    tok = np.random.default_rng(1).integers(0, 8, (1, 16))
    p = x.astype(np.float64) @ ut.astype(np.float64).T
    base = x.astype(np.float64) @ w.astype(np.float64).T

    def phi(cc):
        return loss.next_token_ce((base + p @ cc.T)[None] * 5.0, tok)

    z = linear.z_block(3, 1, 0, 0, 8, 4).astype(np.float64)
    c64 = c.astype(np.float64)
    lg = torch.tensor((base)[None] * 5.0, dtype=torch.float64)
    cc = torch.tensor(c64, requires_grad=True)
    out = lg + 5.0 * (torch.tensor(p) @ cc.T)[None]
    l = torch.nn.functional.cross_entropy(out[0, :-1], torch.tensor(tok[0, 1:]))
    l.backward()
    exact = float((cc.grad.numpy() * z).sum())
    errs = [abs((phi(c64 + e * z) - phi(c64 - e * z)) / (2 * e) - exact) for e in (1e-1, 1e-2)]
    assert errs[1] < errs[0] / 30


# ---------------------------------------------------------------- Adam
def test_projected_grad_scalar():
    assert adam.projected_grad(2.5, 2.0, 0.25) == np.float32(1.0)
    assert adam.projected_grad(1.0, 1.0, 1e-3) == np.float32(0.0)


def test_adam_first_step_closed_form():
    """With m = v = 0 PyTorch-style Adam moves each coefficient by lr*gh/(|gh| + eps_A)."""
    r = np.random.default_rng(0)
    c = r.standard_normal(1000).astype(np.float32)
    z = r.standard_normal(1000).astype(np.float32)
    hp = adam.adam_scalars(1e-3, 1)
    g = np.float32(0.7)
    c1, m1, v1, st = adam.zo_adam(c, np.zeros_like(c), np.zeros_like(c), g, z, hp)
    gh = (g * z).astype(np.float64)
    want = c - 1e-3 * gh / (np.abs(gh) + 1e-8)
    assert st == 0
    np.testing.assert_allclose(c1, want, rtol=0, atol=4 * np.spacing(np.abs(c)).max())
    # agrees with torch.optim.Adam on the same gradient
    t = torch.tensor(c.copy(), dtype=torch.float32, requires_grad=True)
    opt = torch.optim.Adam([t], lr=1e-3, betas=(0.9, 0.999), eps=1e-8)
    t.grad = torch.tensor((g * z).astype(np.float32))
    opt.step()
    np.testing.assert_allclose(c1, t.detach().numpy(), rtol=0, atol=4 * np.spacing(np.abs(c)).max())


def test_adam_tracks_torch_over_steps_and_zero_grad():
    r = np.random.default_rng(1)
    c = r.standard_normal(500).astype(np.float32)
    m = np.zeros_like(c)
    v = np.zeros_like(c)
    t = torch.tensor(c.copy(), requires_grad=True)
    opt = torch.optim.Adam([t], lr=5e-3)
    for step in range(1, 11):
        z = rng.gauss_range(1, step, 0, 0, 500)
        g = np.float32(0.3 * (-1) ** step)
        c, m, v, _ = adam.zo_adam(c, m, v, g, z, adam.adam_scalars(5e-3, step))
        t.grad = torch.tensor(g * z)
        opt.step()
    np.testing.assert_allclose(c, t.detach().numpy(), rtol=0, atol=1e-5)
    c2, _, _, _ = adam.zo_adam(c, np.zeros_like(c), np.zeros_like(c), 0.0, z, adam.adam_scalars(1e-3, 1))
    np.testing.assert_array_equal(c2, c)


def test_adam_nonfinite_guard_and_bf16_storage():
    c = np.ones(8, np.float32)
    out = adam.zo_adam(c, c * 0, c * 0, np.float32(np.nan), c, adam.adam_scalars(1e-3, 1))
    assert out[3] == 1 and np.array_equal(out[0], c)
    cb = rne_bf16(np.linspace(-1, 1, 64).astype(np.float32))
    c1, _, _, _ = adam.zo_adam(cb, cb * 0, cb * 0, 1.0, np.ones(64, np.float32), adam.adam_scalars(0.1, 1),
                               c_bf16=True)
    np.testing.assert_array_equal(c1, rne_bf16(c1))
    np.testing.assert_allclose(c1, cb - 0.1, atol=2**-7)
