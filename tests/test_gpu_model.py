"""End-to-end GPU parity of the decoder models: the whole perturbed forward of both
halves, the losses, Algorithm 1 over a model and the two-sided ZO-Adam step, against
the oracle model on the same seeded weights and tokens.

Bars: fp32 mode losses within 1e-4 relative; bf16 / INT4 mode logits within 2e-2
relative (norm-wise, plus an element-wise bound) and losses within 2e-2 relative; the
Adam update given the GPU's own losses bit-exact.  The oracle's basis is installed in
the GPU model for the forward and trajectory checks, so they test the forward and the
step; the GPU's own Algorithm 1 over a model is checked separately against the oracle
eigensolver on the same captured activations.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import adam as oadam
from oracle import basis as obasis
from oracle import model as om
from oracle import rng as orng
from paper_2607_01125_amd import model as gm
from paper_2607_01125_amd import zoact as Z

from gpu_helpers import announce, assert_rel_close, dev, host, t_i32

pytestmark = pytest.mark.gpu

LLAMA_S = synth.shrink(synth.LLAMA3_8B, n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, d_ff=512, vocab=512,
                       rank=16)
OPT_S = synth.shrink(synth.OPT_13B, n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, d_ff=1024, vocab=512,
                     rank=16, max_pos=64)
LINEARS = ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "w1", "w2")


def _perturb_params(W, shape, seed):
    """Non-trivial norm weights and biases, so a transposed or dropped parameter shows."""
    for l in range(shape.n_layers):
        for name, a in list(W[l].items()):
            if name.startswith("n") or name.startswith("b"):
                base = 1.0 if name in ("n1", "n2") else 0.0
                W[l][name] = synth.bf16_round(base + synth.normal(a.shape, 0.1, seed, 50 + l, sum(map(ord, name))))
    return W


def _int4(W, shape):
    """(GPU weights with (packed, scales) linears, oracle weights with the dequantised values)."""
    Wg = {k: v for k, v in W.items() if not isinstance(k, int)}
    Wo = dict(Wg)
    for l in range(shape.n_layers):
        Lg, Lo = dict(W[l]), dict(W[l])
        for name in LINEARS:
            if name in W[l]:
                packed, scales = synth.quantize_int4_g128(W[l][name])
                Lg[name] = (packed, synth.bf16_round(scales))
                Lo[name] = _dequant(packed, scales)
        Wg[l], Wo[l] = Lg, Lo
    return Wg, Wo


def _dequant(packed, scales):
    from oracle import linear as olin
    return olin.dequant_int4(packed, scales).astype(np.float32)


def _models(shape, mode, seed=0, perturb=False):
    """mode "int4-inreg": INT4 weights on the in-register INT4 GEMM instead of the
    dequantise-then-bf16 path the decoder takes by default."""
    inreg = mode == "int4-inreg"
    mode = "int4" if inreg else mode
    W = synth.model_weights(shape, seed, "fp32" if mode == "fp32" else "bf16")
    if perturb:
        W = _perturb_params(W, shape, seed)
    Wg, Wo = _int4(W, shape) if mode == "int4" else (W, W)
    om_m = om.Model(shape, seed, "fp32" if mode == "fp32" else "bf16", weights=Wo)
    om_m.basis_init(synth.uniform_tokens(4, 32, shape.vocab, seed, 1))
    g = gm.Decoder(shape, Wg, mode, int4_dequant=not inreg)
    g.set_basis({k: om_m.U[k].T for k in g.site_dims()})
    return om_m, g


def _logits_close(got, want, rel, what):
    """The bar: norm-relative error <= rel.  Element-wise, no logit beyond rel |want| +
    3 rel rms(want): a logit is a dot product of bf16 activations that differ from the
    oracle's by rounding decisions, so its error is a sum of many small terms with a
    normal tail, which thousands of logits sample out to several standard deviations."""
    rms = np.sqrt(np.mean(want ** 2))
    err = np.linalg.norm(got - want) / np.linalg.norm(want)
    print(f"[parity] {what}: norm-relative {err:.3e}, max |d|/rms {np.max(np.abs(got - want)) / rms:.3e}",
          flush=True)
    assert err <= rel, f"{what}: norm-relative error {err:.3e} > {rel}"
    bound = rel * np.abs(want) + 3 * rel * rms
    bad = np.abs(got - want) > bound
    assert not bad.any(), f"{what}: {bad.sum()} elements outside {rel} (first {np.argwhere(bad)[0]})"


# ------------------------------------------------------------------ tiny fp32 model, 20 steps
def test_tiny_fp32_twenty_steps():
    """2 layers, d=128, 4 heads, FFN 512, V=512, r=8 on q and v, 4x64 tokens, eps 1e-3, lr 1e-4."""
    announce("tiny fp32 20 steps")
    shape, seed = synth.TINY, 0
    om_m, g = _models(shape, "fp32", seed)
    tok = synth.uniform_tokens(4, 64, shape.vocab, seed, 2)
    tok_d = t_i32(tok)
    k = om_m.k
    c, m, v = np.zeros(k, np.float32), np.zeros(k, np.float32), np.zeros(k, np.float32)
    eps, lr, zseed = 1e-3, 1e-4, 0
    for t in range(1, 21):
        c, m, v, (lp, lm, gg) = om.zo_step(om_m, tok, c, m, v, t, eps, lr, zseed)
        lpm = host(g.step(tok_d, zseed, eps, lr))
        assert_rel_close(lpm, [lp, lm], 1e-4, f"losses at step {t}")
    assert int(host(g.status)[0]) == 0
    cg = host(g.arena.c)
    # the trajectories agree in direction and size (g differs at fp32 rounding level)
    assert np.linalg.norm(cg - c) <= 0.05 * np.linalg.norm(c)


# ------------------------------------------------------------------ bf16 / INT4 forward of both halves
@pytest.mark.parametrize("name,shape,mode,B,S", [
    ("llama-bf16", LLAMA_S, "bf16", 2, 64),
    ("llama-bf16-ragged", LLAMA_S, "bf16", 3, 50),
    ("opt-bf16", OPT_S, "bf16", 2, 40),
    ("llama-int4", LLAMA_S, "int4", 2, 64),
    ("llama-int4-inreg", LLAMA_S, "int4-inreg", 2, 64),
    ("opt-int4-inreg", OPT_S, "int4-inreg", 2, 40),       # q|k|v with k plain, INT4 converted in the GEMM
    ("llama-bf16-r1", synth.shrink(LLAMA_S, rank=1), "bf16", 2, 64),
    ("llama-bf16-r128", synth.shrink(LLAMA_S, rank=128), "bf16", 2, 48),
    ("llama-int4-r1", synth.shrink(LLAMA_S, rank=1), "int4", 2, 40),
])
def test_forward_pm_matches_oracle(name, shape, mode, B, S):
    announce("forward pm", name)
    om_m, g = _models(shape, mode, seed=3, perturb=True)
    c = synth.normal((om_m.k,), 0.05, 3, 9)
    if g.c_bf16:
        c = synth.bf16_round(c)
    g.arena.c.copy_(torch.from_numpy(c).to(g.arena.c.dtype))
    tok = synth.uniform_tokens(B, S, shape.vocab, 3, 4)
    eps, z_ctx = 1e-2, (5, 3, 0)
    logits = host(g.forward(t_i32(tok), Z.Pert(*z_ctx, eps)))
    for h, sign in ((0, +1), (1, -1)):
        want = om_m.forward(tok, c, sign, eps, z_ctx)
        _logits_close(logits[h], want, 2e-2, f"{name} half {h}")
    # the two halves differ by the perturbation (the correction is live)
    assert np.any(logits[0] != logits[1])


def test_eps_zero_halves_bitwise_equal():
    announce("eps 0 halves")
    om_m, g = _models(LLAMA_S, "bf16", seed=1)
    g.arena.c.copy_(torch.from_numpy(synth.normal((om_m.k,), 0.05, 1, 9)))
    tok = t_i32(synth.uniform_tokens(2, 64, LLAMA_S.vocab, 1, 4))
    logits = host(g.forward(tok, Z.Pert(7, 1, 0, 0.0)))
    np.testing.assert_array_equal(logits[0], logits[1])
    lpm = host(g.losses(tok, 7, 1, 0.0))
    assert lpm[0] == lpm[1]


# ------------------------------------------------------------------ one full bf16 step
@pytest.mark.parametrize("shape,mode", [(LLAMA_S, "bf16"), (OPT_S, "bf16"), (LLAMA_S, "int4")],
                         ids=["llama-bf16", "opt-bf16", "llama-int4"])
def test_one_step(shape, mode):
    announce("one step", shape.name, mode)
    om_m, g = _models(shape, mode, seed=2)
    tok = synth.uniform_tokens(2, 64, shape.vocab, 2, 5)
    k = om_m.k
    c0 = np.zeros(k, np.float32)
    eps, lr, zseed = 1e-3, 5e-5, 11
    lpm = host(g.step(t_i32(tok), zseed, eps, lr))
    lp = om_m.loss(tok, c0, +1, eps, (zseed, 1, 0))
    lm = om_m.loss(tok, c0, -1, eps, (zseed, 1, 0))
    assert_rel_close(lpm, [lp, lm], 2e-2, "losses")
    # the update given the GPU's own losses is the oracle's, bit for bit
    gg = oadam.projected_grad(np.float32(lpm[0]), np.float32(lpm[1]), eps)
    z = orng.gauss_range(zseed, 1, 0, 0, k)
    c1, m1, v1, st = oadam.zo_adam(c0, c0, c0, gg, z, oadam.adam_scalars(lr, 1), c_bf16=g.c_bf16)
    np.testing.assert_array_equal(host(g.arena.c).astype(np.float32), c1)
    np.testing.assert_array_equal(host(g.arena.m).astype(np.float32), m1)
    np.testing.assert_array_equal(host(g.arena.v).astype(np.float32), v1)


# ------------------------------------------------------------------ Algorithm 1 over a model
@pytest.mark.parametrize("shape,mode", [(synth.TINY, "fp32"), (LLAMA_S, "bf16"), (OPT_S, "bf16")],
                         ids=["tiny-fp32", "llama-bf16", "opt-bf16"])
def test_basis_init_over_model(shape, mode):
    """The calibration forward hands each site's inputs to zoact_basis_init; the basis
    matches the oracle eigensolver on the same captured activations."""
    announce("basis over model", shape.name, mode)
    W = synth.model_weights(shape, 4, "fp32" if mode == "fp32" else "bf16")
    g = gm.Decoder(shape, W, mode)
    calib = synth.uniform_tokens(4, 64, shape.vocab, 4, 1)
    captured = {}
    dims = g.site_dims()
    ws = torch.empty(max(Z.basis_init_workspace_bytes(d, shape.rank) for d in dims.values()), dtype=torch.uint8,
                     device=dev())

    def hook(l, site, x):
        if (l, site) in dims:
            captured[(l, site)] = host(x)
            ut = torch.empty(shape.rank, dims[(l, site)], dtype=g.act, device=dev())
            master = torch.empty(shape.rank, dims[(l, site)], dtype=torch.float32, device=dev())
            Z.basis_init(x, shape.rank, ut, ws, ut_master=master)
            captured[(l, site, "u")] = host(master).T

    tok = t_i32(calib.reshape(2, 2, 64))
    g.forward(tok, Z.Pert(0, 0, 0, 0.0), calibrate=hook, distinct_halves=True)
    assert set(k for k in captured if len(k) == 2) == set(dims)
    for key in dims:
        x = captured[key]
        assert x.shape == (4 * 64, dims[key])
        u_ref, _ = obasis.basis_init(x, shape.rank)
        u = captured[key + ("u",)]
        assert obasis.overlap(u, u_ref) >= 1 - 1e-6, key
        assert np.max(np.abs(u - u_ref)) <= 1e-3, key
    # the calibration activations are the oracle's (all calibration sequences, in order)
    om_m = om.Model(shape, 4, "fp32" if mode == "fp32" else "bf16", weights=W)
    cap = {}
    om_m.forward(calib, capture=cap)
    for key in dims:
        want = cap[key]
        got = captured[key]
        err = np.linalg.norm(got - want) / np.linalg.norm(want)
        assert err <= (1e-5 if mode == "fp32" else 2e-2), (key, err)
    # and the driver's own basis_init installs one basis per adapted site
    ut = g.basis_init(t_i32(calib))
    assert set(ut) == set(dims)
    for key, u in ut.items():
        um = host(u).T
        assert np.max(np.abs(um.T @ um - np.eye(shape.rank))) <= (1e-5 if mode == "fp32" else 2e-2)


# ------------------------------------------------------------------ fused LM head + cross entropy
@pytest.mark.parametrize("shape,mode", [(LLAMA_S, "bf16"), (OPT_S, "bf16")], ids=["llama", "opt"])
def test_basis_init_concurrent_sites_bitwise(shape, mode):
    """Decoder.basis_init solving several sites at once (copies of their inputs, one stream
    and workspace per host thread) gives each site the same basis, eigenvalues and report
    bits as solving them one at a time inside the forward."""
    announce("basis init concurrent", shape.name)
    W = synth.model_weights(shape, 6, "bf16")
    g = gm.Decoder(shape, W, mode)
    calib = t_i32(synth.uniform_tokens(4, 64, shape.vocab, 6, 1))
    opts = Z.EigOpts(oversample=shape.rank, max_iter=24, seed=0x5eed, tol=1e-4, adaptive=1, check_every=4)
    runs = []
    for k in (1, 4):
        g.basis_init(calib, opts, keep_eigvals=True, report=True, concurrency=k)
        runs.append(({key: host(v.view(torch.int16)) for key, v in g.ut.items()},
                     {key: host(v) for key, v in g.eigvals.items()}, dict(g.basis_report)))
    (u1, e1, r1), (u4, e4, r4) = runs
    assert set(u1) == set(u4) == set(g.site_dims())
    for key in u1:
        np.testing.assert_array_equal(u1[key], u4[key])
        np.testing.assert_array_equal(e1[key].view(np.uint32), e4[key].view(np.uint32))
        assert r1[key] == r4[key], key


@pytest.mark.parametrize("shape,B,S", [(LLAMA_S, 2, 64), (OPT_S, 3, 40)], ids=["llama", "opt"])
def test_fused_head_xent_matches_stored_logits(shape, B, S):
    """The LM head with the cross entropy in its epilogue (logits never stored) gives the
    losses of the stored-logits path up to summation order."""
    announce("fused head xent", shape.name, B, S)
    om_m, g = _models(shape, "bf16", seed=6, perturb=True)
    g.arena.c.copy_(torch.from_numpy(synth.normal((om_m.k,), 0.05, 6, 9)).to(g.arena.c.dtype))
    tok = t_i32(synth.uniform_tokens(B, S, shape.vocab, 6, 4))
    pert = Z.Pert(3, 2, 0, 1e-2)
    logits = g.forward(tok, pert)
    stored = torch.zeros(2, dtype=torch.float32, device=dev())
    Z.xent_pm(logits.reshape(2 * B * S, -1), tok, stored, g.loss_ws)
    fused = torch.full((2,), float("nan"), dtype=torch.float32, device=dev())
    g._loss_pair(tok, pert, fused)
    np.testing.assert_allclose(host(fused), host(stored), rtol=2e-6)
    assert host(fused)[0] != host(fused)[1]


# ------------------------------------------------------------------ the step's own fusions
def test_steps_with_the_update_pass_forming_the_next_perturbation():
    """Decoder.step in bf16: the update pass writes the next step's C +/- eps Z and the next
    forward reads it instead of forming it again.  Three steps give the same losses and
    arena, bit for bit, as three steps that form it afresh each time; a torch-side write to C
    between steps is seen (the perturbation is formed again)."""
    announce("step chain with the fused update pass")
    om_m, g1 = _models(LLAMA_S, "bf16", seed=8)
    _, g2 = _models(LLAMA_S, "bf16", seed=8)
    tok = t_i32(synth.uniform_tokens(2, 64, LLAMA_S.vocab, 8, 5))
    for t in range(3):
        l1 = host(g1.step(tok, 5, 1e-3, 5e-5))
        g2._ch_next = None                  # forget what the update pass wrote
        l2 = host(g2.step(tok, 5, 1e-3, 5e-5))
        np.testing.assert_array_equal(l1, l2)
    for a, b in ((g1.arena.c, g2.arena.c), (g1.arena.m, g2.arena.m), (g1.arena.v, g2.arena.v)):
        assert torch.equal(a, b)
    assert g1._ch_next is not None
    # an outside write to C invalidates the cached perturbation
    g1.arena.c.add_(1e-3)
    g2.arena.c.add_(1e-3)
    l1 = host(g1.step(tok, 5, 1e-3, 5e-5))
    g2._ch_next = None
    l2 = host(g2.step(tok, 5, 1e-3, 5e-5))
    np.testing.assert_array_equal(l1, l2)


@pytest.mark.parametrize("mode", ["bf16", "int4"])
def test_shared_first_projection_bitwise(mode):
    """Layer 0's q|k|v in its shared-input form (both halves read the same embedding rows):
    logits bit for bit those of the stacked form."""
    announce("shared first projection", mode)
    om_m, g = _models(LLAMA_S, mode, seed=9)
    g.arena.c.copy_(torch.from_numpy(synth.normal((om_m.k,), 0.05, 9, 9)).to(g.arena.c.dtype))
    tok = t_i32(synth.uniform_tokens(2, 64, LLAMA_S.vocab, 9, 4))
    pert = Z.Pert(4, 2, 0, 1e-2)
    calls = []
    g.linear_hook = lambda stage, lin, T, flags: calls.append(flags) if stage == "pre" else None
    a = host(g.forward(tok, pert))
    g.linear_hook = None
    assert calls[0] & Z.SHARED_X and not any(f & Z.SHARED_X for f in calls[1:])
    g.shared_first = False
    b = host(g.forward(tok, pert))
    np.testing.assert_array_equal(a, b)
