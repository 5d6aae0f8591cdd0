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


# ------------------------------------------------------------------ OPT family: independent torch fp64 model
def torch_forward_opt(shape, W, U, c, tokens, sign, eps, z_ctx):
    """The OPT decoder written with torch ops (float64): F.layer_norm, learned positions
    looked up at index s + 2, multi-head attention through SDPA, a ReLU MLP, biases on
    every projection, a final LayerNorm and the LM head tied to the token embedding.
    Adapted projections (q, v, out, fc1, fc2) use the materialised W + C_h U^T; k is
    plain (Section 3's W_eff; the adapted list of Appendix B's OPT runs)."""
    dt = torch.float64
    B, S = tokens.shape
    d, H, hd = shape.d_model, shape.n_heads, shape.head_dim
    blocks = {(b.layer, b.name): b for b in om.arena_layout(shape)}
    c = c if torch.is_tensor(c) else torch.tensor(c, dtype=dt)
    tt = lambda a: torch.tensor(np.asarray(a, np.float64), dtype=dt)

    def weff(l, name, w, rows, site):
        w = tt(w)
        b = blocks[(l, name)]
        idx = b.offset + np.asarray(rows)[:, None] * b.r + np.arange(b.r)[None, :]
        z = torch.tensor(orng.gauss(*z_ctx, idx).astype(np.float64), dtype=dt)
        cb = c[torch.tensor(idx)] + sign * float(np.float32(eps)) * z
        return w + cb @ tt(U[(l, site)]).T

    def ln(x, wt, bs):
        return F.layer_norm(x, (d,), tt(wt), tt(bs), eps=shape.norm_eps)

    ids = torch.tensor(tokens.astype(np.int64))
    pos = torch.arange(S)[None, :].expand(B, S) + 2
    h = (F.embedding(ids, tt(W["emb"])) + F.embedding(pos, tt(W["pos"]))).reshape(B * S, d)
    ar = np.arange
    for l in range(shape.n_layers):
        L = W[l]
        a = ln(h, L["n1"], L["n1b"])
        q = F.linear(a, weff(l, "qv", L["wq"], ar(d), "attn"), tt(L["bq"]))
        k = F.linear(a, tt(L["wk"]), tt(L["bk"]))
        v = F.linear(a, weff(l, "qv", L["wv"], d + ar(d), "attn"), tt(L["bv"]))
        q, k, v = (t.reshape(B, S, H, hd).transpose(1, 2) for t in (q, k, v))
        o = F.scaled_dot_product_attention(q, k, v, is_causal=True, scale=float(np.float32(1 / math.sqrt(hd))))
        o = o.transpose(1, 2).reshape(B * S, d)
        h = h + F.linear(o, weff(l, "out", L["wo"], ar(d), "o"), tt(L["bo"]))
        m = ln(h, L["n2"], L["n2b"])
        f = F.relu(F.linear(m, weff(l, "fc1", L["w1"], ar(shape.d_ff), "mlp"), tt(L["b1"])))
        h = h + F.linear(f, weff(l, "fc2", L["w2"], ar(d), "down"), tt(L["b2"]))
    logits = F.linear(ln(h, W["nf"], W["nfb"]), tt(W["emb"]))
    return logits.reshape(B, S, -1)


def _opt_shape(**kw):
    base = dict(n_layers=2, d_model=64, n_heads=4, d_ff=96, vocab=90, rank=4, max_pos=40)
    base.update(kw)
    base["n_kv_heads"] = base["n_heads"]          # OPT attention is multi-head
    return synth.shrink(synth.OPT_13B, **base)


def _randomise_norms_and_biases(W, shape, seed=0):
    """Nonzero norm weights, norm biases and projection biases: with the init values
    (ones and zeros) a dropped bias or a unit norm weight in the wrong place would not
    show."""
    g = synth.gen(seed, 4242)
    d, dkv, ff = shape.d_model, shape.n_kv_heads * shape.head_dim, shape.d_ff
    for l in range(shape.n_layers):
        L = W[l]
        for n in ("n1", "n2"):
            L[n] = (1.0 + 0.3 * g.standard_normal(d)).astype(np.float32)
        for n in ("n1b", "n2b"):
            L[n] = (0.2 * g.standard_normal(d)).astype(np.float32)
        for n, w in (("bq", d), ("bk", dkv), ("bv", dkv), ("bo", d), ("b1", ff), ("b2", d)):
            L[n] = (0.1 * g.standard_normal(w)).astype(np.float32)
    W["nf"] = (1.0 + 0.3 * g.standard_normal(d)).astype(np.float32)
    W["nfb"] = (0.2 * g.standard_normal(d)).astype(np.float32)
    # position rows large enough that a shifted lookup changes the logits visibly
    W["pos"] = (W["pos"] * 20.0).astype(np.float32)


def _setup_opt(shape, seed=0):
    m = om.Model(shape, seed, "fp32")
    _randomise_norms_and_biases(m.W, shape, seed)
    m.basis_init(synth.uniform_tokens(2, 16, shape.vocab, seed, 1))
    tok = synth.uniform_tokens(2, 16, shape.vocab, seed, 2)
    c = synth.normal((m.k,), 0.05, seed, 3).astype(np.float64)
    return m, tok, c


@pytest.mark.parametrize("shape", [_opt_shape(), _opt_shape(n_layers=1, d_model=96, n_heads=3, d_ff=128, rank=8)],
                         ids=["2l-d64", "1l-d96"])
def test_numpy_opt_model_matches_torch_model(shape):
    m, tok, c = _setup_opt(shape)
    for sign in (+1, -1):
        got = m.forward(tok, c, sign, 1e-2, (5, 3, 0))
        want = torch_forward_opt(shape, m.W, m.U, c, tok, sign, 1e-2, (5, 3, 0)).numpy()
        np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-10)


def test_opt_position_offset_and_variance_are_seen():
    """The OPT comparison above fails for the plausible slips: positions without the
    offset of 2, and LayerNorm with the unbiased variance."""
    shape = _opt_shape(n_layers=1)
    m, tok, c = _setup_opt(shape)
    want = torch_forward_opt(shape, m.W, m.U, c, tok, +1, 1e-2, (5, 3, 0)).numpy()
    W2 = dict(m.W)
    W2["pos"] = np.concatenate([m.W["pos"][2:], m.W["pos"][:2]])      # offset 0 instead of 2
    shifted = torch_forward_opt(shape, W2, m.U, c, tok, +1, 1e-2, (5, 3, 0)).numpy()
    assert np.max(np.abs(shifted - want)) > 1e-3
    orig = om.layernorm
    try:
        def unbiased(x, w, b, eps, mode):
            x = np.asarray(x, np.float64)
            mu = x.mean(axis=-1, keepdims=True)
            var = ((x - mu) ** 2).sum(axis=-1, keepdims=True) / (x.shape[-1] - 1)
            return (x - mu) / np.sqrt(var + eps) * w + b

        om.layernorm = unbiased
        slipped = m.forward(tok, c, +1, 1e-2, (5, 3, 0))
    finally:
        om.layernorm = orig
    assert np.max(np.abs(slipped - want)) > 1e-4


@pytest.mark.parametrize("family", ["llama", "opt"])
def test_zero_coefficients_are_the_base_model_both_families(family):
    if family == "opt":
        shape = _opt_shape()
        m, tok, _ = _setup_opt(shape)
    else:
        shape = tiny(n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, d_ff=96, vocab=80,
                     adapted=("q", "k", "v", "o", "gate", "up", "down"), rank=4)
        m, tok, _ = _setup(shape)
    base = m.forward(tok)
    for sign in (+1, -1):
        np.testing.assert_array_equal(m.forward(tok, np.zeros(m.k), sign, 0.0, (1, 1, 0)), base)
    # and the base model is the torch model with C = 0 and eps = 0
    fwd = torch_forward_opt if family == "opt" else torch_forward
    want = fwd(shape, m.W, m.U, np.zeros(m.k), tok, +1, 0.0, (1, 1, 0)).numpy()
    np.testing.assert_allclose(base, want, rtol=1e-10, atol=1e-10)


def test_opt_central_difference_matches_directional_derivative():
    """(L+ - L-)/(2 eps) of the OPT oracle -> <grad_C L, Z> from torch autograd.  The ReLU's
    kinks make the loss piecewise smooth: for eps above ~1e-4 the pair straddles kinks
    (error O(eps) with no clean trend); below that the O(eps^2) remainder holds."""
    shape = _opt_shape(n_layers=1)
    m, tok, c = _setup_opt(shape)
    z_ctx = (9, 1, 0)
    ct = torch.tensor(c, requires_grad=True)
    lg = torch_forward_opt(shape, m.W, m.U, ct, tok, 0, 0.0, z_ctx)
    lt = F.cross_entropy(lg[:, :-1].reshape(-1, lg.shape[-1]), torch.tensor(tok[:, 1:].reshape(-1).astype(np.int64)))
    lt.backward()
    z = orng.gauss_range(*z_ctx, 0, m.k).astype(np.float64)
    exact = float((ct.grad.numpy() * z).sum())
    e32 = float(np.float32(1e-5))
    fd = (m.loss(tok, c, +1, 1e-5, z_ctx) - m.loss(tok, c, -1, 1e-5, z_ctx)) / (2 * e32)
    assert abs(exact) > 1e-3
    assert abs(fd - exact) < 1e-8 * max(1.0, abs(exact))


# ------------------------------------------------------------------ bf16 rounding points, written again in torch
def torch_forward_bf16(shape, W, U, c, tokens, sign, eps, z_ctx):
    """Both families in bf16 mode, written with torch ops: every stored tensor goes
    through torch's bfloat16 cast (round to nearest even) at the rounding points of the
    precision reading -- embeddings and weights bf16; each linear output rounded once
    after the base product, bias, residual and the rank-r correction (P = bf16(x U),
    C_h = bf16(C + s fp32(eps Z)) formed in fp32); norms, rotary, SwiGLU and ReLU
    rounded once; attention probabilities rounded before P.V with the normaliser
    summed unrounded; logits fp32.  Products are float64."""
    dt = torch.float64
    B, S = tokens.shape
    d, H, Hkv, hd = shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim
    dkv = Hkv * hd
    opt = shape.family == "opt"
    blocks = {(b.layer, b.name): b for b in om.arena_layout(shape)}
    tt = lambda a: torch.tensor(np.asarray(a, np.float64), dtype=dt)
    rb = lambda x: x.to(torch.float32).to(torch.bfloat16).to(dt)
    c32 = torch.tensor(np.asarray(c, np.float32))

    def lin(x, w, bias, l, name, rows, site, residual=None, act=None):
        y = x @ tt(w).T
        if (l, name) in blocks:
            b = blocks[(l, name)]
            idx = b.offset + np.asarray(rows)[:, None] * b.r + np.arange(b.r)[None, :]
            p = rb(x @ tt(U[(l, site)]))
            ez = torch.tensor(np.float32(eps)) * torch.tensor(orng.gauss(*z_ctx, idx))
            ch = c32[torch.tensor(idx)] + ez if sign > 0 else c32[torch.tensor(idx)] - ez
            y = y + p @ ch.to(torch.bfloat16).to(dt).T
        if bias is not None:
            y = y + tt(bias)
        if residual is not None:
            y = residual + y
        return y if act == "raw" else rb(y)

    def norm(x, wt, bs=None):
        if opt:
            return rb(F.layer_norm(x, (d,), tt(wt), tt(bs), eps=shape.norm_eps))
        return rb(x * torch.rsqrt((x * x).mean(-1, keepdim=True) + shape.norm_eps) * tt(wt))

    ids = torch.tensor(tokens.reshape(-1).astype(np.int64))
    if opt:
        pos = (torch.arange(S) + 2).repeat(B)
        h = rb(tt(W["emb"])[ids] + tt(W["pos"])[pos])
    else:
        h = tt(W["emb"])[ids]
    j = torch.arange(hd // 2, dtype=dt)
    ang = torch.arange(S, dtype=dt)[:, None] * (shape.rope_theta ** (-2.0 * j / hd))[None, :]
    cs, sn = torch.cos(ang).float().double(), torch.sin(ang).float().double()

    def rope(x):
        lo, hi = x[..., : hd // 2], x[..., hd // 2:]
        c_, s_ = cs[None, :, None, :], sn[None, :, None, :]
        return rb(torch.cat([lo * c_ - hi * s_, hi * c_ + lo * s_], dim=-1))

    def attend(q, k, v):
        rep = q.shape[2] // k.shape[2]
        k = k.repeat_interleave(rep, dim=2)
        v = v.repeat_interleave(rep, dim=2)
        s = torch.einsum("bqhd,bkhd->bhqk", q, k) * float(np.float32(1 / math.sqrt(hd)))
        s = s.masked_fill(torch.ones(S, S, dtype=torch.bool).triu(1), float("-inf"))
        e = torch.exp(s - s.amax(-1, keepdim=True))
        o = torch.einsum("bhqk,bkhd->bqhd", rb(e), v) / e.sum(-1).transpose(1, 2)[..., None]
        return rb(o).reshape(B * S, d)

    ar = np.arange
    for l in range(shape.n_layers):
        L = W[l]
        a = norm(h, L["n1"], L.get("n1b"))
        if opt:
            q = lin(a, L["wq"], L["bq"], l, "qv", ar(d), "attn")
            k = lin(a, L["wk"], L["bk"], l, None, None, None)
            v = lin(a, L["wv"], L["bv"], l, "qv", d + ar(d), "attn")
        else:
            q = lin(a, L["wq"], None, l, "qkv", ar(d), "attn")
            k = lin(a, L["wk"], None, l, "qkv", d + ar(dkv), "attn")
            v = lin(a, L["wv"], None, l, "qkv", d + dkv + ar(dkv), "attn")
        q, k, v = q.reshape(B, S, H, hd), k.reshape(B, S, Hkv, hd), v.reshape(B, S, Hkv, hd)
        if not opt:
            q, k = rope(q), rope(k)
        o = attend(q, k, v)
        h = lin(o, L["wo"], L.get("bo"), l, "out" if opt else "o", ar(d), "o", residual=h)
        m = norm(h, L["n2"], L.get("n2b"))
        if opt:
            f = rb(F.relu(lin(m, L["w1"], L["b1"], l, "fc1", ar(shape.d_ff), "mlp", act="raw")))
            h = lin(f, L["w2"], L["b2"], l, "fc2", ar(d), "down", residual=h)
        else:
            gr, ur = om.gate_up_rows(shape.d_ff)
            g = lin(m, L["wg"], None, l, "gu", gr, "mlp", act="raw")
            u = lin(m, L["wu"], None, l, "gu", ur, "mlp", act="raw")
            f = rb(F.silu(g) * u)
            h = lin(f, L["wd"], None, l, "down", ar(d), "down", residual=h)
    hf = norm(h, W["nf"], W.get("nfb"))
    logits = (hf @ tt(W["emb"] if opt else W["head"]).T).to(torch.float32).to(dt)
    return logits.reshape(B, S, -1)


@pytest.mark.parametrize("family", ["llama", "opt"])
def test_bf16_rounding_points_match_torch(family):
    """The bf16-mode oracle against the torch bf16 rewrite: the same values except where a
    float64 sum taken in another order lands a value on the other side of a bf16
    rounding boundary, which is rare and moves a logit by bf16 noise only."""
    if family == "opt":
        shape = _opt_shape(n_layers=2, d_model=128, n_heads=4, d_ff=256, vocab=300, rank=8)
    else:
        shape = synth.shrink(synth.LLAMA3_8B, n_layers=2, d_model=128, n_heads=4, n_kv_heads=2, d_ff=256,
                             vocab=300, rank=8)
    m = om.Model(shape, 1, "bf16")
    if family == "opt":
        _randomise_norms_and_biases(m.W, shape, 1)
    m.basis_init(synth.uniform_tokens(2, 32, 300, 1, 1))
    tok = synth.uniform_tokens(2, 16, 300, 1, 2)
    c = synth.normal((m.k,), 0.05, 1, 3)
    for sign in (+1, -1):
        got = m.forward(tok, c, sign, 1e-2, (4, 2, 0))
        want = torch_forward_bf16(shape, m.W, m.U, c, tok, sign, 1e-2, (4, 2, 0)).numpy()
        exact = np.mean(got == want)
        assert exact > 0.99, exact
        np.testing.assert_allclose(got, want, rtol=0, atol=2.0 ** -6 * np.sqrt(np.mean(want ** 2)))
