"""Decoder models, Algorithm 1 over a model, and the two-sided ZO step (oracle side).

The paper adapts every linear layer except embeddings and task heads (Appendix B) of
Llama-3-8B, OPT-13B and an INT4 Llama-3-8B (Section 5).  With random-initialised
models of those shapes the build's reading of the model is:

* Llama family: token embedding; per layer RMSNorm -> q, k, v -> rotary embedding
  (rotate-half, base theta) -> causal attention with grouped K/V heads -> o projection
  + residual -> RMSNorm -> SwiGLU MLP (silu(gate) * up -> down) + residual; final
  RMSNorm; untied LM head.
* OPT family: token embedding + learned positions (offset 2); per layer LayerNorm ->
  q, k, v (biases) -> causal attention -> out projection + residual -> LayerNorm ->
  fc1 -> ReLU -> fc2 + residual; final LayerNorm; LM head tied to the embedding.

Adapted projections and the coefficient arena.  Projections that read the same input
share one basis (q/k/v read the attention input, gate/up the MLP input).  The arena is
laid out per layer, in this order, each block holding (rows x r) coefficients row-major
(row = output feature of the fused projection):
  Llama, q,k,v all adapted: [q | k | v] rows (d + 2 d_kv), o (d), gate/up (2 d_ff,
  interleaved in blocks of 16: 16 gate rows then the 16 up rows of the same features),
  down (d).  Llama with q, v adapted: [q | v] rows (2 d), o, gate/up, down as adapted.
  OPT (q, v, out, fc1, fc2): [q | v] (2 d), out (d), fc1 (d_ff), fc2 (d).
Z for coefficient (row, i) of a block at arena offset `off` is Z(off + row * r + i).

Rounding points (bf16 mode): embeddings, weights, activations between kernels and the
residual stream are bf16; GEMMs sum in float64 here and round once; norms, rotary
embedding, softmax, SwiGLU and ReLU compute in fp32/fp64 and round their output once;
attention rounds the probabilities to bf16 before multiplying by V (the normaliser is
summed unrounded); logits are fp32; the loss is summed in float64.  fp32 mode computes
in float64 throughout.

Parity: pinned by tests/test_oracle_model.py -- independent torch float64
implementations of both families (Llama: complex rotary, SDPA, materialised W_eff; OPT:
F.layer_norm, learned positions at s + 2, SDPA, ReLU MLP with biases, tied head) agree to
1e-10 with nonzero norm weights, norm biases and projection biases; a torch rewrite of
the bf16 rounding points (torch's bfloat16 cast at each stored tensor) gives the same
logits bit for bit for both families; a zero-output LM head gives ln V; with C = 0 both
halves equal the base model; the two-sided difference matches the autograd directional
derivative as eps -> 0.  Loss values of the random-initialised 8B/13B
shapes themselves are parity unpinned by the paper, which prints none.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from . import adam as oadam
from . import basis as obasis
from . import linear as olin
from . import loss as oloss
from .numerics import rne_bf16


def _round(x, mode):
    return rne_bf16(np.asarray(x, dtype=np.float32)).astype(np.float64) if mode == "bf16" else np.asarray(x, np.float64)


@dataclass
class Block:
    """One coefficient block of the arena: a fused projection's rows."""
    layer: int
    name: str          # "qkv", "qv", "o", "gu", "down", "out", "fc1", "fc2"
    rows: int
    r: int
    offset: int


def arena_layout(shape) -> list:
    """Blocks in arena order for a synth.ModelShape."""
    d, dkv, ff, r = shape.d_model, shape.n_kv_heads * shape.head_dim, shape.d_ff, shape.rank
    ad = set(shape.adapted)
    blocks, off = [], 0
    for l in range(shape.n_layers):
        if shape.family == "llama":
            names = []
            if {"q", "k", "v"} <= ad:
                names.append(("qkv", d + 2 * dkv))
            elif {"q", "v"} <= ad:
                names.append(("qv", 2 * d))
            if "o" in ad:
                names.append(("o", d))
            if {"gate", "up"} <= ad:
                names.append(("gu", 2 * ff))
            if "down" in ad:
                names.append(("down", d))
        else:
            names = [("qv", 2 * d), ("out", d), ("fc1", ff), ("fc2", d)]
        for name, rows in names:
            blocks.append(Block(l, name, rows, r, off))
            off += rows * r
    return blocks


def arena_size(shape) -> int:
    return sum(b.rows * b.r for b in arena_layout(shape))


def gate_up_rows(ff: int):
    """Fused row index of gate feature f and of up feature f (blocks of 16)."""
    f = np.arange(ff)
    g = (f // 16) * 32 + (f % 16)
    return g, g + 16


# ------------------------------------------------------------------ weights
def model_weights(shape, seed: int, mode: str):
    """Per-tensor seeded random-init weights (the seeded generator shared with the GPU side)."""
    import synth

    return synth.model_weights(shape, seed, mode)


# ------------------------------------------------------------------ support ops
def rmsnorm(x, w, eps, mode):
    x = np.asarray(x, np.float64)
    inv = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return _round(x * inv * w, mode)


def layernorm(x, w, b, eps, mode):
    x = np.asarray(x, np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return _round((x - mu) / np.sqrt(var + eps) * w + b, mode)


def rope_tables(seq: int, head_dim: int, theta: float):
    """cos/sin [seq][head_dim/2]: angles in float64, rounded once to fp32."""
    j = np.arange(head_dim // 2, dtype=np.float64)
    inv = theta ** (-2.0 * j / head_dim)
    ang = np.arange(seq, dtype=np.float64)[:, None] * inv[None, :]
    return np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)


def rope(x, cos, sin, mode):
    """Rotate-half rotary embedding on x [B][S][H][hd] with fp32 tables [S][hd/2]."""
    x = np.asarray(x, np.float64)
    h = x.shape[-1] // 2
    c = cos.astype(np.float64)[None, :, None, :]
    s = sin.astype(np.float64)[None, :, None, :]
    lo, hi = x[..., :h], x[..., h:]
    return _round(np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1), mode)


def attention(q, k, v, mode):
    """Causal attention, q [B][S][H][hd], k/v [B][S][Hkv][hd] (grouped heads)."""
    q, k, v = (np.asarray(a, np.float64) for a in (q, k, v))
    B, S, H, hd = q.shape
    rep = H // k.shape[2]
    k = np.repeat(k, rep, axis=2)
    v = np.repeat(v, rep, axis=2)
    scale = float(np.float32(1.0 / math.sqrt(hd)))
    sc = np.einsum("bqhd,bkhd->bhqk", q, k) * scale
    mask = np.triu(np.ones((S, S), bool), 1)
    sc = np.where(mask[None, None], -np.inf, sc)
    mx = sc.max(axis=-1, keepdims=True)
    p = np.exp(sc - mx)
    l = p.sum(axis=-1, keepdims=True)
    pr = _round(p, mode) if mode == "bf16" else p
    o = np.einsum("bhqk,bkhd->bqhd", pr, v) / np.transpose(l, (0, 2, 1, 3))
    return _round(o, mode)


# ------------------------------------------------------------------ model forward
class Model:
    """Oracle model: weights, bases, arena; forward of one perturbation half."""

    def __init__(self, shape, seed: int, mode: str, weights=None):
        self.s, self.mode, self.seed = shape, mode, seed
        self.W = weights if weights is not None else model_weights(shape, seed, mode)
        self.blocks = {(b.layer, b.name): b for b in arena_layout(shape)}
        self.k = arena_size(shape)
        self.U = {}          # (layer, site) -> U [d_in][r] (float64, as used: bf16-rounded in bf16 mode)

    # linear with optional adaptation of some fused rows
    def _lin(self, x, w, bias, site, block, rows, sign, c, z_ctx, eps):
        """x W^T + b (+ adapted part for `rows` of `block`), unrounded float64."""
        y = x @ w.astype(np.float64).T
        if bias is not None:
            y = y + bias.astype(np.float64)
        if block is not None and c is not None:
            b = self.blocks[block]
            u = self.U[site]
            p = olin.project(x, u.T, self.mode)                      # [T][r], rounded in bf16 mode
            idx = b.offset + rows[:, None] * b.r + np.arange(b.r)[None, :]
            cb = c[idx]
            seed, step, query = z_ctx
            z = olin.rng.gauss(seed, step, query, idx)
            ch = olin.perturbed_coeffs(cb, z, eps, sign, self.mode)
            y = y + p @ ch.T
        return y

    def forward(self, tokens, c=None, sign=0, eps=0.0, z_ctx=(0, 0, 0), capture=None):
        """Logits (float64 [B][S][V]) of one half; capture[(layer, site)] gets site inputs."""
        s, W, mode = self.s, self.W, self.mode
        B, S = tokens.shape
        d, H, Hkv, hd = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim
        dkv = Hkv * hd
        ad = set(s.adapted)
        T = B * S
        if s.family == "llama":
            h = W["emb"][tokens.reshape(-1)].astype(np.float64)
        else:
            pos = np.tile(np.arange(S) + 2, B)
            h = _round(W["emb"][tokens.reshape(-1)].astype(np.float64) + W["pos"][pos].astype(np.float64), mode)
        cos, sin = rope_tables(S, hd, s.rope_theta) if s.family == "llama" else (None, None)
        cc = c if c is not None and sign != 0 else c
        for l in range(s.n_layers):
            L = W[l]
            a = rmsnorm(h, L["n1"], s.norm_eps, mode) if s.family == "llama" else \
                layernorm(h, L["n1"], L["n1b"], s.norm_eps, mode)
            if capture is not None:
                capture[(l, "attn")] = a
            ar = lambda n: np.arange(n)
            if s.family == "llama" and {"q", "k", "v"} <= ad:
                q = self._lin(a, L["wq"], None, (l, "attn"), (l, "qkv"), ar(d), sign, cc, z_ctx, eps)
                k = self._lin(a, L["wk"], None, (l, "attn"), (l, "qkv"), d + ar(dkv), sign, cc, z_ctx, eps)
                v = self._lin(a, L["wv"], None, (l, "attn"), (l, "qkv"), d + dkv + ar(dkv), sign, cc, z_ctx, eps)
            else:
                bq, bk, bv = (L.get("bq"), L.get("bk"), L.get("bv"))
                q = self._lin(a, L["wq"], bq, (l, "attn"), (l, "qv"), ar(d), sign, cc, z_ctx, eps)
                k = self._lin(a, L["wk"], bk, None, None, None, sign, None, z_ctx, eps)
                v = self._lin(a, L["wv"], bv, (l, "attn"), (l, "qv"), d + ar(d if s.family == "opt" else dkv),
                              sign, cc, z_ctx, eps)
            q, k, v = (_round(t, mode) for t in (q, k, v))
            q = q.reshape(B, S, H, hd)
            k = k.reshape(B, S, Hkv, hd)
            v = v.reshape(B, S, Hkv, hd)
            if s.family == "llama":
                q = rope(q, cos, sin, mode)
                k = rope(k, cos, sin, mode)
            o_in = attention(q, k, v, mode).reshape(T, d)
            if capture is not None:
                capture[(l, "o")] = o_in
            oname = "o" if s.family == "llama" else "out"
            ob = (l, oname) if (l, oname) in self.blocks else None
            h = _round(h + self._lin(o_in, L["wo"], L.get("bo"), (l, "o"), ob, ar(d), sign, cc, z_ctx, eps), mode)
            m = rmsnorm(h, L["n2"], s.norm_eps, mode) if s.family == "llama" else \
                layernorm(h, L["n2"], L["n2b"], s.norm_eps, mode)
            if capture is not None:
                capture[(l, "mlp")] = m
            if s.family == "llama":
                gr, ur = gate_up_rows(s.d_ff)
                gb = (l, "gu") if (l, "gu") in self.blocks else None
                g = self._lin(m, L["wg"], None, (l, "mlp"), gb, gr, sign, cc, z_ctx, eps)
                u = self._lin(m, L["wu"], None, (l, "mlp"), gb, ur, sign, cc, z_ctx, eps)
                act = _round(g / (1.0 + np.exp(-g)) * u, mode)
                dname, dw, db = "down", L["wd"], None
            else:
                f1 = self._lin(m, L["w1"], L["b1"], (l, "mlp"), (l, "fc1"), ar(s.d_ff), sign, cc, z_ctx, eps)
                act = _round(np.maximum(f1, 0.0), mode)
                dname, dw, db = "fc2", L["w2"], L["b2"]
            if capture is not None:
                capture[(l, "down")] = act
            dbk = (l, dname) if (l, dname) in self.blocks else None
            h = _round(h + self._lin(act, dw, db, (l, "down"), dbk, ar(d), sign, cc, z_ctx, eps), mode)
        hf = rmsnorm(h, W["nf"], s.norm_eps, mode) if s.family == "llama" else \
            layernorm(h, W["nf"], W["nfb"], s.norm_eps, mode)
        head = W["head"] if s.family == "llama" else W["emb"]
        logits = hf @ head.astype(np.float64).T
        if mode == "bf16":
            logits = logits.astype(np.float32).astype(np.float64)
        return logits.reshape(B, S, -1)

    # ---------------------------------------------------------------- Algorithm 1
    def basis_init(self, calib_tokens):
        """One calibration forward (C = 0), then the top-r basis of every site's inputs."""
        cap = {}
        self.forward(calib_tokens, capture=cap)
        for key, xs in cap.items():
            u, _ = obasis.basis_init(xs, self.s.rank)
            self.U[key] = rne_bf16(u.astype(np.float32)).astype(np.float64) if self.mode == "bf16" else u
        return self.U

    def loss(self, tokens, c, sign, eps, z_ctx):
        return oloss.next_token_ce(self.forward(tokens, c, sign, eps, z_ctx), tokens)


def zo_step(model: Model, tokens, c, m, v, t: int, eps: float, lr: float, seed: int, c_bf16=False):
    """One two-sided ZO-Adam step (Algorithm 2 body with the +/- pair)."""
    z_ctx = (seed, t, 0)
    lp = model.loss(tokens, c, +1, eps, z_ctx)
    lm = model.loss(tokens, c, -1, eps, z_ctx)
    g = oadam.projected_grad(lp, lm, eps)
    z = olin.rng.gauss_range(seed, t, 0, 0, c.size)
    c1, m1, v1, st = oadam.zo_adam(c, m, v, g, z, oadam.adam_scalars(lr, t), c_bf16=c_bf16)
    return c1, m1, v1, (lp, lm, float(g))


def zo_step_q(model: Model, tokens, c, m, v, t: int, eps: float, lr: float, seed: int, q: int, c_bf16=False,
              optimizer: str = "adam"):
    """One step of Algorithm 2 in its one-sided q-query form: the unperturbed loss L, the
    losses L_j under B + mu Z^(j) (Z^(j) = Z(seed, t, query j)), the averaged estimate and
    the optimiser update."""
    losses = [model.loss(tokens, c, 0, eps, (seed, t, 0))]
    for j in range(1, q + 1):
        losses.append(model.loss(tokens, c, +1, eps, (seed, t, j)))
    zs = np.stack([olin.rng.gauss_range(seed, t, j, 0, c.size) for j in range(1, q + 1)])
    if optimizer == "adam":
        c1, m1, v1, st = oadam.zo_adam_q(c, m, v, losses, zs, eps, oadam.adam_scalars(lr, t), c_bf16=c_bf16)
    else:
        c1, st = oadam.zo_sgd_q(c, losses, zs, eps, lr, c_bf16=c_bf16)
        m1, v1 = m, v
    return c1, m1, v1, losses
