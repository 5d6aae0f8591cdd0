"""GPU parity at the full widths of the paper's models (Section 5, Appendix B): one
decoder layer of the Llama-3-8B shape (d = 4096, 32 query / 8 key-value heads of 128,
SwiGLU FFN 14336, vocabulary 128256, r = 32 on all seven projections) in bf16 and with
INT4 weights, and of the OPT-13B shape (d = 5120, 40 heads, ReLU FFN 20480, vocabulary
50272, r = 64 on q, v, out, fc1, fc2), against the oracle on the same seeded weights.

The full depth is not needed for parity: every layer runs the same kernels on the same
shapes, so one layer at full width covers every launch configuration a step of the
full model makes (the LM head and the fused cross entropy included).  The basis is a
seeded random orthonormal U per site (Algorithm 1 itself is tested elsewhere; here it
would need eigensolves of 14336- and 20480-wide Grams on the host).

Bars: logits of both halves element-wise within 2e-2 (relative, plus 2e-2 of the rms),
losses within 2e-2 relative, the update given the GPU's own losses bit for bit.  With
16 sequences of 256 tokens per half the Llama attention runs its whole-sequence-resident
kernel with the rotary inside (a grid that fills the chip); the oracle then runs two of
the sequences, which attention keeps independent of the others, and their logits are
compared row by row.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import adam as oadam
from oracle import model as om
from oracle import rng as orng
from oracle.numerics import rne_bf16
from paper_2607_01125_amd import model as gm
from paper_2607_01125_amd import zoact as Z

from gpu_helpers import announce, assert_bf16_close, assert_rel_close, dev, host, t_bf16, t_f32, t_i32

pytestmark = pytest.mark.gpu

LLAMA_1L = synth.shrink(synth.LLAMA3_8B, n_layers=1)
OPT_1L = synth.shrink(synth.OPT_13B, n_layers=1, max_pos=512)
LINEARS = ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "w1", "w2")


def _random_basis(shape, dims, mode, seed):
    """Seeded orthonormal U [d_in][r] per adapted site (QR of a Gaussian), bf16 values in bf16 mode."""
    U = {}
    for key, d_in in sorted(dims.items()):
        stream = synth.gen(seed, 880, key[0], gm.SITES.index(key[1]))
        q, _ = np.linalg.qr(stream.standard_normal((d_in, shape.rank)))
        U[key] = rne_bf16(q.astype(np.float32)).astype(np.float64) if mode != "fp32" else q
    return U


def _int4_weights(W, shape):
    """(GPU weights with (packed, scales) linears, oracle weights holding the dequantised values)."""
    from oracle import linear as olin
    Wg = {k: v for k, v in W.items() if not isinstance(k, int)}
    Wo = dict(Wg)
    for l in range(shape.n_layers):
        Lg, Lo = dict(W[l]), dict(W[l])
        for name in LINEARS:
            if name in W[l]:
                packed, scales = synth.quantize_int4_g128(W[l][name])
                Lg[name] = (packed, synth.bf16_round(scales))
                Lo[name] = olin.dequant_int4(packed, scales).astype(np.float32)
        Wg[l], Wo[l] = Lg, Lo
    return Wg, Wo


def _build(shape, mode, seed):
    W = synth.model_weights(shape, seed, "bf16")
    Wg, Wo = _int4_weights(W, shape) if mode == "int4" else (W, W)
    om_m = om.Model(shape, seed, "bf16", weights=Wo)
    g = gm.Decoder(shape, Wg, mode)
    dims = g.site_dims()
    U = _random_basis(shape, dims, mode, seed)
    om_m.U = dict(U)
    g.set_basis({k: U[k].T for k in dims})
    return om_m, g


def _logits_close(got, want, rel, what):
    """The bar: norm-relative error <= rel over the compared logits.  Element-wise, no logit
    beyond rel |want| + 3 rel rms(want): each logit is a 4096- or 5120-term dot product of
    bf16 activations that differ from the oracle's by rounding decisions, so its error is a
    sum of many small independent terms (a normal tail), and millions of logits reach
    several standard deviations of it."""
    rms = np.sqrt(np.mean(want ** 2))
    err = np.linalg.norm(got - want) / np.linalg.norm(want)
    print(f"[parity] {what}: norm-relative {err:.3e}, max |d|/rms {np.max(np.abs(got - want)) / rms:.3e}",
          flush=True)
    assert err <= rel, f"{what}: norm-relative error {err:.3e} > {rel}"
    bound = rel * np.abs(want) + 3 * rel * rms
    bad = np.abs(got - want) > bound
    assert not bad.any(), f"{what}: {bad.sum()} elements outside {rel} (first {np.argwhere(bad)[0]})"


@pytest.fixture(scope="module")
def llama_bf16():
    announce("full-width llama bf16: weights")
    return _build(LLAMA_1L, "bf16", 21)


def _forward_and_step(om_m, g, B, S, seed, name):
    """Logits of both halves with random C against the oracle; then one step from C = 0:
    losses against the oracle and the update bit for bit given the GPU's losses."""
    shape = g.s
    c = synth.normal((om_m.k,), 0.05, seed, 9)
    if g.c_bf16:
        c = synth.bf16_round(c)
    g.arena.c.copy_(torch.from_numpy(c).to(g.arena.c.dtype))
    tok = synth.uniform_tokens(B, S, shape.vocab, seed, 4)
    eps, z_ctx = 1e-2, (5, 3, 0)
    announce(name, "forward", B, S)
    logits = g.forward(t_i32(tok), Z.Pert(*z_ctx, eps))
    rows = np.random.default_rng(seed).choice(B * S, 48, replace=False)
    got = host(logits.reshape(2, B * S, -1)[:, torch.from_numpy(rows).to(dev())])
    for h, sign in ((0, +1), (1, -1)):
        want = om_m.forward(tok, c, sign, eps, z_ctx).reshape(B * S, -1)[rows]
        _logits_close(got[h], want, 2e-2, f"{name} half {h}")
    assert np.any(got[0] != got[1])
    del logits
    # one step from C = 0 (m = v = 0)
    g.arena.c.zero_()
    g.arena.m.zero_()
    g.arena.v.zero_()
    g.t = 0
    k = om_m.k
    c0 = np.zeros(k, np.float32)
    eps, lr, zseed = 1e-3, 5e-5, 11
    announce(name, "step")
    lpm = host(g.step(t_i32(tok), zseed, eps, lr))
    lp = om_m.loss(tok, c0, +1, eps, (zseed, 1, 0))
    lm = om_m.loss(tok, c0, -1, eps, (zseed, 1, 0))
    assert_rel_close(lpm, [lp, lm], 2e-2, f"{name} losses")
    gg = oadam.projected_grad(np.float32(lpm[0]), np.float32(lpm[1]), eps)
    z = orng.gauss_range(zseed, 1, 0, 0, k)
    c1, m1, v1, st = oadam.zo_adam(c0, c0, c0, gg, z, oadam.adam_scalars(lr, 1), c_bf16=g.c_bf16)
    np.testing.assert_array_equal(host(g.arena.c).astype(np.float32), c1)
    np.testing.assert_array_equal(host(g.arena.m).astype(np.float32), m1)
    np.testing.assert_array_equal(host(g.arena.v).astype(np.float32), v1)


def test_llama_full_width_bf16(llama_bf16):
    """One Llama-3-8B-shape layer in bf16, 2 x 256 tokens per half."""
    om_m, g = llama_bf16
    _forward_and_step(om_m, g, 2, 256, 21, "llama full width bf16")


def test_llama_full_width_resident_attention(llama_bf16):
    """16 x 256 tokens per half (the benchmark's batch): the resident attention kernel with
    the rotary applied inside, the shared first projection, the fused LM head and loss at
    8192 stacked rows.  The oracle runs sequences 0 and 11 of each half."""
    om_m, g = llama_bf16
    B, S, seed = 16, 256, 22
    c = synth.normal((om_m.k,), 0.05, seed, 9)
    g.arena.c.copy_(torch.from_numpy(c))
    tok = synth.uniform_tokens(B, S, g.s.vocab, seed, 4)
    eps, z_ctx = 1e-2, (6, 2, 0)
    announce("llama full width resident attention: forward", B, S)
    logits = g.forward(t_i32(tok), Z.Pert(*z_ctx, eps))
    pick = [0, 11]
    got = host(logits[:, pick])
    # the fused head + cross entropy against the stored-logits loss of the same forward
    stored = torch.zeros(2, dtype=torch.float32, device=dev())
    Z.xent_pm(logits.reshape(2 * B * S, -1), t_i32(tok), stored, g.loss_ws)
    del logits
    fused = torch.full((2,), float("nan"), dtype=torch.float32, device=dev())
    g._loss_pair(t_i32(tok), Z.Pert(*z_ctx, eps), fused)
    np.testing.assert_allclose(host(fused), host(stored), rtol=2e-6)
    for h, sign in ((0, +1), (1, -1)):
        want = om_m.forward(tok[pick], c, sign, eps, z_ctx)
        _logits_close(got[h], want, 2e-2, f"resident attention half {h}")


def test_llama_full_width_shared_first_layer_bitwise(llama_bf16):
    """The first projection in its shared-input form gives the same logits, bit for bit,
    as the stacked form (both halves fed the same embedding rows twice)."""
    _, g = llama_bf16
    tok = t_i32(synth.uniform_tokens(4, 256, g.s.vocab, 23, 4))
    pert = Z.Pert(8, 4, 0, 1e-2)
    announce("llama full width shared first layer")
    g.shared_first = True
    a = g.forward(tok, pert).clone()
    g.shared_first = False
    b = g.forward(tok, pert)
    g.shared_first = True
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_llama_full_width_int4():
    """One Llama-3-8B-shape layer with INT4 weights (group 128, bf16 scales) and bf16 C; the
    INT4 GEMM that converts the packed weights in LDS (int4_dequant=False) gives the same
    logits bit for bit as the decoder's default dequantise-then-bf16 path."""
    announce("full-width llama int4: weights")
    om_m, g = _build(LLAMA_1L, "int4", 24)
    c = synth.bf16_round(synth.normal((om_m.k,), 0.05, 24, 10))
    g.arena.c.copy_(torch.from_numpy(c).to(g.arena.c.dtype))
    tok = t_i32(synth.uniform_tokens(2, 256, LLAMA_1L.vocab, 24, 5))
    pert = Z.Pert(5, 3, 0, 1e-2)
    announce("full-width llama int4: dequantised vs converted in the GEMM")
    a = g.forward(tok, pert).clone()
    g.int4_dequant = False
    b = g.forward(tok, pert)
    g.int4_dequant = True
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    del a, b
    _forward_and_step(om_m, g, 2, 256, 24, "llama full width int4")


def test_opt_full_width_bf16():
    """One OPT-13B-shape layer in bf16 (r = 64 on q, v, out, fc1, fc2), with nonzero norm
    weights and biases, 2 x 256 tokens per half."""
    announce("full-width opt bf16: weights")
    shape = OPT_1L
    W = synth.model_weights(shape, 25, "bf16")
    g0 = synth.gen(25, 4243)
    L = W[0]
    for n in ("n1", "n2"):
        L[n] = synth.bf16_round((1.0 + 0.2 * g0.standard_normal(shape.d_model)).astype(np.float32))
    for n in ("n1b", "n2b", "bq", "bk", "bv", "bo", "b2"):
        L[n] = synth.bf16_round((0.05 * g0.standard_normal(L[n].shape[0])).astype(np.float32))
    L["b1"] = synth.bf16_round((0.05 * g0.standard_normal(shape.d_ff)).astype(np.float32))
    om_m = om.Model(shape, 25, "bf16", weights=W)
    g = gm.Decoder(shape, W, "bf16")
    dims = g.site_dims()
    U = _random_basis(shape, dims, "bf16", 25)
    om_m.U = dict(U)
    g.set_basis({k: U[k].T for k in dims})
    _forward_and_step(om_m, g, 2, 256, 25, "opt full width bf16")


def test_headline_shared_x_mse_equals_stacked_full_size():
    """The single-layer workload's own launch (K = N = 4096, 8192 tokens per half, r = 32,
    the regression loss in the epilogue): the shared-input form gives the stacked form's
    losses bit for bit, and the stacked form's rows match the oracle on a sample."""
    from oracle import linear as olin
    T, K, N, r = 8192, 4096, 4096, 32
    announce("headline shared x vs stacked, full size")
    x, q = synth.planted_lowrank(T, K, seed=0)
    x = synth.bf16_round(x)
    w = synth.bf16_round(synth.normal((N, K), 0.02, 0, 2))
    ut = synth.bf16_round(q[:, :r].T.copy())
    c = synth.normal((N * r,), 0.01, 0, 3)
    layer = Z.Linear(t_bf16(w), K, N, r, t_bf16(ut), 0)
    arena = Z.Arena(t_f32(c), torch.zeros(N * r, device=dev()), torch.zeros(N * r, device=dev()))
    pert = Z.Pert(1, 3, 0, 1e-3)
    ch = torch.empty(2 * N * r, dtype=torch.bfloat16, device=dev())
    Z.perturb_coeffs(arena, 0, N * r, pert, ch)
    layer.ch, layer.ch_stride = ch, N * r
    x1 = t_bf16(x)
    x2 = torch.cat([x1, x1]).contiguous()
    p1 = torch.empty(T, r, dtype=torch.bfloat16, device=dev())
    Z.project(x1, t_bf16(ut), p1)
    p2 = torch.cat([p1, p1]).contiguous()
    tgt = t_bf16(synth.bf16_round(synth.normal((T, N), 1.0, 0, 5)))
    ws = torch.empty(Z.linear_mse_workspace_bytes(T, N), dtype=torch.uint8, device=dev())
    ls = torch.full((2,), float("nan"), dtype=torch.float32, device=dev())
    lt = torch.full((2,), float("nan"), dtype=torch.float32, device=dev())
    Z.linear_mse(layer, arena, x1, T, p1, pert, tgt, ls, ws, flags=Z.SHARED_X)
    Z.linear_mse(layer, arena, x2, T, p2, pert, tgt, lt, ws)
    np.testing.assert_array_equal(host(ls), host(lt))
    assert host(ls)[0] != host(ls)[1]
    # stored outputs of both forms, bit for bit, and sampled rows against the oracle
    ys = torch.empty(2 * T, N, dtype=torch.bfloat16, device=dev())
    yt = torch.empty(2 * T, N, dtype=torch.bfloat16, device=dev())
    Z.linear_fwd_pm(layer, arena, x1, T, p1, ys, pert, flags=Z.SHARED_X)
    Z.linear_fwd_pm(layer, arena, x2, T, p2, yt, pert)
    assert torch.equal(ys.view(torch.int16), yt.view(torch.int16))
    rows = np.concatenate([np.random.default_rng(3).choice(T, 30, replace=False), [0, T - 1]])
    xs = x[rows]
    ref = olin.adapted_linear_pm(np.stack([xs, xs]), w, None, ut, c.reshape(N, r), 1e-3, 1, 3, 0, 0, "bf16")
    assert_bf16_close(host(ys).reshape(2, T, N)[:, rows], ref, what="headline rows vs oracle")
    # both losses against the oracle's, over every row (float64 products, 2 x 275 GFLOP)
    from oracle import loss as oloss
    full = olin.adapted_linear_pm(np.stack([x, x]), w, None, ut, c.reshape(N, r), 1e-3, 1, 3, 0, 0, "bf16")
    tg = host(tgt)
    assert_rel_close(host(ls), [oloss.mse(full[0], tg), oloss.mse(full[1], tg)], 2e-2, "headline losses")
