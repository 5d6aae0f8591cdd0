"""GPU parity of the one-sided q-query form of Algorithm 2 (Section 3's averaged
forward difference against the unperturbed loss): the general perturbation pair in
the coefficient pass and in the fused GEMM, the q-query Adam / SGD update, and a whole
model step, against the oracle.

Bars: the coefficient pass and the updates bit-exact (teacher-forced losses); GEMM
outputs within the bf16 bar of gpu_helpers; model losses within 2e-2 relative.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import adam as oadam
from oracle import linear as olin
from oracle import model as om
from oracle import rng as orng
from paper_2607_01125_amd import model as gm
from paper_2607_01125_amd import zoact as Z

from gpu_helpers import announce, assert_bf16_close, assert_rel_close, dev, host, t_bf16, t_f32, t_i32

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("c_bf16", [False, True])
@pytest.mark.parametrize("queries,signs", [((0, 1), (0, 1)), ((2, 3), (1, 1)), ((5, 5), (-1, 0)), ((0, 0), (1, -1))])
def test_perturb_pair_bitwise(c_bf16, queries, signs):
    announce("perturb pair", c_bf16, queries, signs)
    e0, n = 5, 3001
    k = e0 + n + 2
    c = synth.normal((k,), 0.01, 4, 4)
    if c_bf16:
        c = synth.bf16_round(c)
    ct = t_bf16(c) if c_bf16 else t_f32(c)
    arena = Z.Arena(ct, torch.zeros(k, device=dev()), torch.zeros(k, device=dev()))
    out = torch.empty(2 * n, dtype=torch.bfloat16, device=dev())
    Z.perturb_coeffs(arena, e0, n, Z.pert_pair(31, 7, queries, signs, 1e-3), out)
    got = host(out).reshape(2, n)
    for h in range(2):
        z = orng.gauss_range(31, 7, queries[h], e0, n)
        want = olin.perturbed_coeffs(c[e0:e0 + n], z, 1e-3, signs[h], "bf16")
        np.testing.assert_array_equal(got[h], want)


def _pair_layer(T, K, N, r, seed):
    x = synth.bf16_round(synth.normal((2, T, K), 1.0, seed, 1))
    w = synth.bf16_round(synth.normal((N, K), 0.05, seed, 2))
    ut = synth.bf16_round(synth.normal((r, K), 1.0 / np.sqrt(K), seed, 3))
    c = synth.normal((N * r,), 0.05, seed, 4)
    return x, w, ut, c


@pytest.mark.parametrize("T,K,N,r,precomputed", [
    (200, 512, 336, 32, False), (200, 512, 336, 32, True), (130, 256, 512, 128, True), (64, 384, 256, 8, False),
    (100, 256, 256, 3, False), (100, 256, 256, 72, False),      # the kernels that form C_h for other ranks
])
def test_linear_pair_against_oracle(T, K, N, r, precomputed):
    """Half 0 unperturbed (sign 0), half 1 with +eps Z^(3); in-kernel and precomputed."""
    announce("linear pair", T, K, N, r, precomputed)
    x, w, ut, c = _pair_layer(T, K, N, r, T + N)
    eps, seed, step = 1e-2, 17, 2
    pp = Z.pert_pair(seed, step, (0, 3), (0, 1), eps)
    xt = t_bf16(x.reshape(2 * T, K))
    p = torch.empty(2 * T, r, dtype=torch.bfloat16, device=dev())
    Z.project(xt, t_bf16(ut), p)
    layer = Z.Linear(t_bf16(w), K, N, r, t_bf16(ut), 0)
    arena = Z.Arena(t_f32(c), torch.zeros(N * r, device=dev()), torch.zeros(N * r, device=dev()))
    if precomputed:
        ch = torch.empty(2 * N * r, dtype=torch.bfloat16, device=dev())
        Z.perturb_coeffs(arena, 0, N * r, pp, ch)
        layer.ch, layer.ch_stride = ch, N * r
    y = torch.empty(2 * T, N, dtype=torch.bfloat16, device=dev())
    Z.linear_fwd_pm(layer, arena, xt, T, p, y, pp)
    got = host(y).reshape(2, T, N)
    cm = c.reshape(N, r)
    z0 = olin.z_block(seed, step, 0, 0, N, r)
    z3 = olin.z_block(seed, step, 3, 0, N, r)
    ref0 = olin.adapted_linear(x[0], w, None, ut, cm, z0, eps, 0, "bf16")
    ref1 = olin.adapted_linear(x[1], w, None, ut, cm, z3, eps, +1, "bf16")
    assert_bf16_close(got, np.stack([ref0, ref1]), what="linear pair")
    # the unperturbed half does not depend on Z or eps
    pp0 = Z.pert_pair(seed + 1, step, (0, 3), (0, 1), 0.5)
    if precomputed:
        Z.perturb_coeffs(arena, 0, N * r, pp0, layer.ch)
    y2 = torch.empty_like(y)
    Z.linear_fwd_pm(layer, arena, xt, T, p, y2, pp0)
    np.testing.assert_array_equal(host(y2).reshape(2, T, N)[0], got[0])


@pytest.mark.parametrize("c_bf16", [False, True])
@pytest.mark.parametrize("q,k", [(1, 4096), (3, 100_003), (8, 70_001)])
def test_step_q_adam_bitwise(c_bf16, q, k):
    announce("step_q adam", c_bf16, q, k)
    rs = np.random.default_rng(q)
    c = (rs.standard_normal(k) * 0.01).astype(np.float32)
    if c_bf16:
        c = synth.bf16_round(c).astype(np.float32)
    m = (rs.standard_normal(k) * 1e-3).astype(np.float32)
    v = (rs.random(k) * 1e-5).astype(np.float32)
    losses = (2.0 + rs.standard_normal(q + 1) * 1e-3).astype(np.float32)
    seed, step, eps, lr = 23, 4, 1e-3, 5e-5
    ct = t_bf16(c) if c_bf16 else t_f32(c)
    arena = Z.Arena(ct, t_f32(m), t_f32(v))
    status = torch.zeros(1, dtype=torch.int32, device=dev())
    Z.step_q(arena, t_f32(losses), q, seed, step, eps, Z.adam_desc(lr, step), status)
    zs = np.stack([orng.gauss_range(seed, step, j, 0, k) for j in range(1, q + 1)])
    c1, m1, v1, st = oadam.zo_adam_q(c, m, v, losses, zs, eps, oadam.adam_scalars(lr, step), c_bf16=c_bf16)
    assert st == 0 and int(status.item()) == 0
    np.testing.assert_array_equal(host(arena.m).astype(np.float32).view(np.uint32), m1.view(np.uint32))
    np.testing.assert_array_equal(host(arena.v).astype(np.float32).view(np.uint32), v1.view(np.uint32))
    np.testing.assert_array_equal(host(arena.c).astype(np.float32).view(np.uint32), c1.view(np.uint32))


@pytest.mark.parametrize("c_bf16", [False, True])
def test_step_q_sgd_bitwise_and_guard(c_bf16):
    announce("step_q sgd", c_bf16)
    k, q = 50_001, 5
    rs = np.random.default_rng(1)
    c = (rs.standard_normal(k) * 0.01).astype(np.float32)
    if c_bf16:
        c = synth.bf16_round(c).astype(np.float32)
    losses = (1.0 + rs.standard_normal(q + 1) * 1e-3).astype(np.float32)
    ct = t_bf16(c) if c_bf16 else t_f32(c)
    arena = Z.Arena(ct, torch.zeros(k, device=dev()), torch.zeros(k, device=dev()))
    Z.step_q_sgd(arena, t_f32(losses), q, 3, 9, 1e-3, 1e-4)
    zs = np.stack([orng.gauss_range(3, 9, j, 0, k) for j in range(1, q + 1)])
    want, _ = oadam.zo_sgd_q(c, losses, zs, 1e-3, 1e-4, c_bf16=c_bf16)
    np.testing.assert_array_equal(host(arena.c).astype(np.float32).view(np.uint32), want.view(np.uint32))
    # a non-finite query loss: no update anywhere, status bit 0
    before = host(arena.c).copy()
    bad = losses.copy()
    bad[3] = np.inf
    status = torch.zeros(1, dtype=torch.int32, device=dev())
    Z.step_q_sgd(arena, t_f32(bad), q, 3, 10, 1e-3, 1e-4, status)
    assert int(status.item()) & 1
    np.testing.assert_array_equal(host(arena.c), before)


LLAMA_S = synth.shrink(synth.LLAMA3_8B, n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, d_ff=512, vocab=512,
                       rank=16)


@pytest.mark.parametrize("q,mode", [(3, "bf16"), (2, "fp32")])
def test_model_step_q(q, mode):
    """ceil((q+1)/2) stacked forwards give L and L_1..L_q within the loss bar; the update
    given the GPU's own losses is the oracle's, bit for bit."""
    announce("model step_q", q, mode)
    shape = LLAMA_S if mode == "bf16" else synth.TINY
    W = synth.model_weights(shape, 4, mode)
    o = om.Model(shape, 4, mode, weights=W)
    o.basis_init(synth.uniform_tokens(4, 32, shape.vocab, 4, 1))
    g = gm.Decoder(shape, W, mode)
    g.set_basis({key: o.U[key].T for key in g.site_dims()})
    k = o.k
    c = synth.normal((k,), 0.02, 4, 2).astype(np.float32)
    if g.c_bf16:
        c = synth.bf16_round(c).astype(np.float32)
    g.arena.c.copy_(torch.from_numpy(c).to(g.arena.c.dtype))
    tok = synth.uniform_tokens(2, 48, shape.vocab, 4, 3)
    eps, lr, seed = 1e-2, 1e-4, 8
    losses = host(g.step_q(t_i32(tok), seed, eps, lr, q))
    want = [o.loss(tok, c, 0, eps, (seed, 1, 0))] + [o.loss(tok, c, +1, eps, (seed, 1, j)) for j in range(1, q + 1)]
    assert_rel_close(losses[:q + 1], want, 2e-2 if mode == "bf16" else 1e-4, "q-query losses")
    if len(losses) > q + 1:
        assert losses[q + 1] == losses[0]          # the spare half re-evaluates L
    zs = np.stack([orng.gauss_range(seed, 1, j, 0, k) for j in range(1, q + 1)])
    z0 = np.zeros(k, np.float32)
    c1, m1, v1, st = oadam.zo_adam_q(c, z0, z0, losses[:q + 1].astype(np.float32), zs, eps,
                                     oadam.adam_scalars(lr, 1), c_bf16=g.c_bf16)
    np.testing.assert_array_equal(host(g.arena.c).astype(np.float32), c1)
    np.testing.assert_array_equal(host(g.arena.m), m1)
