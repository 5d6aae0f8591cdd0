"""Pins for oracle/model.py (decoder forward, arena layout, Algorithm 1 over a model,
the two-sided step)."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import linear as olin
from oracle import model as om
from oracle import rng as orng


def tiny(**kw):
    return synth.shrink(synth.TINY, **kw)


# ------------------------------------------------------------------ arena size = k of Section 4
def _k_from_paper(shape):
    """k = sum over adapted linears of r * n_l (n_l = output width), Section 4."""
    d, dkv, ff = shape.d_model, shape.n_kv_heads * shape.head_dim, shape.d_ff
    width = {"q": d, "k": dkv, "v": dkv, "o": d, "gate": ff, "up": ff, "down": d, "fc1": ff, "fc2": d}
    if shape.family == "opt":
        width["k"] = width["v"] = d
    return shape.n_layers * shape.rank * sum(width[p] for p in shape.adapted)


@pytest.mark.parametrize("shape", [synth.TINY, synth.LLAMA3_8B, synth.OPT_13B], ids=lambda s: s.name)
def test_arena_size_is_k(shape):
    assert om.arena_size(shape) == _k_from_paper(shape)


def test_arena_sizes_of_the_workloads():
    assert om.arena_size(synth.TINY) == 4096
    assert om.arena_size(synth.LLAMA3_8B) == 44_040_192
    assert om.arena_size(synth.OPT_13B) == 104_857_600


def test_gate_up_rows_partition():
    g, u = om.gate_up_rows(64)
    allr = np.sort(np.concatenate([g, u]))
    np.testing.assert_array_equal(allr, np.arange(128))
    assert g[17] == 33 and u[17] == 49


# ------------------------------------------------------------------ independent torch fp64 model
def torch_forward(shape, W, U, c, tokens, sign, eps, z_ctx):
    """Same model written with torch ops: complex rotary, SDPA, materialised W_eff."""
    dt = torch.float64
    B, S = tokens.shape
    d, H, Hkv, hd = shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim
    blocks = {(b.layer, b.name): b for b in om.arena_layout(shape)}
    c = c if torch.is_tensor(c) else torch.tensor(c, dtype=dt)
    tt = lambda a: torch.tensor(np.asarray(a, np.float64), dtype=dt)

    def weff(l, name, w, rows, site):
        w = tt(w)
        if (l, name) not in blocks:
            return w
        b = blocks[(l, name)]
        idx = b.offset + np.asarray(rows)[:, None] * b.r + np.arange(b.r)[None, :]
        z = torch.tensor(orng.gauss(*z_ctx, idx).astype(np.float64), dtype=dt)
        cb = c[torch.tensor(idx)] + sign * float(np.float32(eps)) * z
        return w + cb @ tt(U[(l, site)]).T

    def rms(x, wt):
        return x * torch.rsqrt((x * x).mean(-1, keepdim=True) + shape.norm_eps) * tt(wt)

    h = tt(W["emb"])[torch.tensor(tokens.reshape(-1).astype(np.int64))]
    j = torch.arange(hd // 2, dtype=dt)
    ang = torch.arange(S, dtype=dt)[:, None] * (shape.rope_theta ** (-2.0 * j / hd))[None, :]
    # the model's rotary table holds fp32-rounded cos/sin values
    rot = torch.complex(torch.cos(ang).float().double(), torch.sin(ang).float().double())

    def rope(x):  # x [B][S][h][hd]
        xc = torch.complex(x[..., : hd // 2], x[..., hd // 2:]) * rot[None, :, None, :]
        return torch.cat([xc.real, xc.imag], dim=-1)

    for l in range(shape.n_layers):
        L = W[l]
        a = rms(h, L["n1"])
        ar = np.arange
        qn = "qkv" if (l, "qkv") in blocks else "qv"
        q = a @ weff(l, qn, L["wq"], ar(d), "attn").T
        k = a @ (weff(l, qn, L["wk"], d + ar(Hkv * hd), "attn") if qn == "qkv" else tt(L["wk"])).T
        v_rows = d + (Hkv * hd if qn == "qkv" else 0) + ar(Hkv * hd)
        v = a @ weff(l, qn, L["wv"], v_rows, "attn").T
        q = rope(q.reshape(B, S, H, hd)).transpose(1, 2)
        k = rope(k.reshape(B, S, Hkv, hd)).transpose(1, 2).repeat_interleave(H // Hkv, dim=1)
        v = v.reshape(B, S, Hkv, hd).transpose(1, 2).repeat_interleave(H // Hkv, dim=1)
        o = F.scaled_dot_product_attention(q, k, v, is_causal=True, scale=float(np.float32(1 / math.sqrt(hd))))
        o = o.transpose(1, 2).reshape(B * S, d)
        h = h + o @ weff(l, "o", L["wo"], ar(d), "o").T
        m = rms(h, L["n2"])
        gr, ur = om.gate_up_rows(shape.d_ff)
        g = m @ weff(l, "gu", L["wg"], gr, "mlp").T
        u = m @ weff(l, "gu", L["wu"], ur, "mlp").T
        h = h + (F.silu(g) * u) @ weff(l, "down", L["wd"], ar(d), "down").T
    logits = rms(h, W["nf"]) @ tt(W["head"]).T
    return logits.reshape(B, S, -1)


def _setup(shape, seed=0):
    m = om.Model(shape, seed, "fp32")
    cal = synth.uniform_tokens(2, 16, shape.vocab, seed, 1)
    m.basis_init(cal)
    tok = synth.uniform_tokens(2, 16, shape.vocab, seed, 2)
    c = synth.normal((m.k,), 0.05, seed, 3).astype(np.float64)
    return m, tok, c


@pytest.mark.parametrize("shape", [tiny(n_layers=1, d_model=64, n_heads=4, n_kv_heads=4, d_ff=128, vocab=97),
                                   tiny(n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, d_ff=96, vocab=80,
                                        adapted=("q", "k", "v", "o", "gate", "up", "down"), rank=4)],
                         ids=["mha-qv", "gqa-all"])
def test_numpy_model_matches_torch_model(shape):
    m, tok, c = _setup(shape)
    for sign in (+1, -1):
        got = m.forward(tok, c, sign, 1e-2, (5, 3, 0))
        want = torch_forward(shape, m.W, m.U, c, tok, sign, 1e-2, (5, 3, 0)).numpy()
        np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-10)


def test_zero_coefficients_are_the_base_model():
    shape = tiny(n_layers=1, d_model=64, n_heads=4, n_kv_heads=4, d_ff=128, vocab=97)
    m, tok, _ = _setup(shape)
    c0 = np.zeros(m.k)
    base = m.forward(tok)
    np.testing.assert_array_equal(m.forward(tok, c0, +1, 0.0, (1, 1, 0)), base)
    np.testing.assert_array_equal(m.forward(tok, c0, -1, 0.0, (1, 1, 0)), base)


def test_zero_head_gives_log_vocab():
    shape = tiny(n_layers=1, d_model=64, n_heads=4, n_kv_heads=4, d_ff=128, vocab=97)
    m, tok, c = _setup(shape)
    m.W["head"] = np.zeros_like(m.W["head"])
    assert m.loss(tok, c, +1, 1e-3, (1, 1, 0)) == pytest.approx(math.log(97), rel=1e-14)


def test_central_difference_matches_directional_derivative():
    """(L+ - L-)/(2 eps) -> <grad_C L, Z> with error O(eps^2) (remainder bound, Appendix A)."""
    shape = tiny(n_layers=1, d_model=64, n_heads=4, n_kv_heads=4, d_ff=128, vocab=97)
    m, tok, c = _setup(shape)
    z_ctx = (9, 1, 0)
    ct = torch.tensor(c, requires_grad=True)
    lg = torch_forward(shape, m.W, m.U, ct, tok, 0, 0.0, z_ctx)
    lt = F.cross_entropy(lg[:, :-1].reshape(-1, lg.shape[-1]), torch.tensor(tok[:, 1:].reshape(-1).astype(np.int64)))
    lt.backward()
    z = orng.gauss_range(*z_ctx, 0, m.k).astype(np.float64)
    exact = float((ct.grad.numpy() * z).sum())
    errs = []
    for eps in (1e-1, 1e-2, 1e-3):
        e32 = float(np.float32(eps))
        fd = (m.loss(tok, c, +1, eps, z_ctx) - m.loss(tok, c, -1, eps, z_ctx)) / (2 * e32)
        errs.append(abs(fd - exact))
    assert errs[1] < errs[0] / 30 and errs[2] < errs[1] / 30


def test_basis_init_over_model():
    shape = tiny(n_layers=2, d_model=64, n_heads=4, n_kv_heads=4, d_ff=128, vocab=97)
    m = om.Model(shape, 0, "fp32")
    U = m.basis_init(synth.uniform_tokens(4, 32, 97, 0, 1))
    for key, u in U.items():
        assert u.shape == (64 if key[1] != "down" else 128, shape.rank)
        assert np.max(np.abs(u.T @ u - np.eye(shape.rank))) < 1e-8


def test_bf16_and_opt_variants_run():
    for shape in (synth.shrink(synth.LLAMA3_8B, n_layers=1, d_model=128, n_heads=4, n_kv_heads=2, d_ff=256,
                               vocab=300, rank=8),
                  synth.shrink(synth.OPT_13B, n_layers=1, d_model=128, n_heads=4, n_kv_heads=4, d_ff=256,
                               vocab=300, rank=8, max_pos=64)):
        m = om.Model(shape, 1, "bf16")
        m.basis_init(synth.uniform_tokens(2, 32, 300, 1, 1))
        tok = synth.uniform_tokens(2, 16, 300, 1, 2)
        c = np.zeros(m.k, np.float32)
        lp = m.loss(tok, c, +1, 1e-3, (1, 1, 0))
        assert abs(lp - math.log(300)) < 0.2
        c1, _, _, (a, b, g) = om.zo_step(m, tok, c, np.zeros_like(c), np.zeros_like(c), 1, 1e-3, 1e-4, 7)
        assert np.isfinite(g) and np.any(c1 != 0)
