"""Decoder models on the GPU for the forward-only ZO step.

Algorithm 1 (one-shot basis from a calibration forward) and the two-sided step of
Algorithm 2 over a whole decoder, written as a sequence of libzoact calls: this module
only lays out buffers and marshals arguments; every operation of the forward, the loss
and the update runs in the library's kernels.

Models (the random-initialised shapes of the paper's Section 5 experiments):
* Llama family: token embedding; per layer RMSNorm, q/k/v, rotary embedding
  (rotate-half), causal attention with grouped K/V heads, o projection + residual,
  RMSNorm, SwiGLU MLP + residual; final RMSNorm; untied LM head.
* OPT family: token + learned position embedding (offset 2); per layer LayerNorm,
  q/k/v with biases, causal attention, out projection + residual, LayerNorm, fc1, ReLU,
  fc2 + residual; final LayerNorm; LM head tied to the embedding.

Adapted projections (Section 3, y = x W^T + (x U) C^T) read one of four input sites
per layer -- "attn" (q, k, v), "o", "mlp" (gate/up or fc1) and "down" (down or fc2) --
and projections reading the same site share its basis U.  Projections that read one
site are fused into one linear call: q|k|v (when k is not adapted, as in OPT, k is the
call's plain feature range -- no correction, no coefficient rows -- or, where the fast
schedule does not cover that, a separate plain linear beside q|v) and gate|up, whose
rows interleave blocks of 16 gate and 16 up features so the SwiGLU epilogue pairs them
inside a tile.

Coefficient arena: per layer, in order, [q|k|v] (or [q|v]), o, gate|up, down (Llama)
or [q|v], out, fc1, fc2 (OPT); each block holds rows x r coefficients row-major, where
a row is an output feature of the fused projection.  The arena size is the paper's
k = sum of r n_l over adapted linears (Section 4).

Precision modes: "fp32" (fp32 weights and activations), "bf16" (bf16 weights and
activations, fp32 logits) and "int4" (group-128 INT4 linears with bf16 scales, bf16
everything else, bf16 coefficients by default).
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import queue

import math
from dataclasses import dataclass

import numpy as np
import torch

from . import zoact as Z

SITES = ("attn", "o", "mlp", "down")
# widths covered by zoact_rmsnorm_project / zoact_layernorm_project, and the largest row
# count at which the decoder uses them
NORM_PROJECT_WIDTHS = (128, 256, 512, 1024, 2048, 4096, 5120)
NORM_PROJECT_MAX_ROWS = 4096


@dataclass
class Block:
    """One coefficient block: the fused projection `name` of `layer`, rows x r at `offset`."""
    layer: int
    name: str
    rows: int
    r: int
    offset: int
    site: str


def arena_layout(shape) -> list:
    d, dkv, ff, r = shape.d_model, shape.n_kv_heads * shape.head_dim, shape.d_ff, shape.rank
    ad = set(shape.adapted)
    out, off = [], 0
    for l in range(shape.n_layers):
        if shape.family == "llama":
            names = []
            if {"q", "k", "v"} <= ad:
                names.append(("qkv", d + 2 * dkv, "attn"))
            elif {"q", "v"} <= ad:
                names.append(("qv", 2 * d, "attn"))
            elif ad & {"q", "k", "v"}:
                raise ValueError("Llama models adapt q, k, v together or q, v")
            if "o" in ad:
                names.append(("o", d, "o"))
            if {"gate", "up"} <= ad:
                names.append(("gu", 2 * ff, "mlp"))
            elif ad & {"gate", "up"}:
                raise ValueError("gate and up are adapted together")
            if "down" in ad:
                names.append(("down", d, "down"))
        else:
            if set(shape.adapted) != {"q", "v", "o", "fc1", "fc2"}:
                raise ValueError("OPT models adapt q, v, out, fc1, fc2")
            names = [("qv", 2 * d, "attn"), ("out", d, "o"), ("fc1", ff, "mlp"), ("fc2", d, "down")]
        for name, rows, site in names:
            out.append(Block(l, name, rows, r, off, site))
            off += rows * r
    return out


def _pair_key(pert) -> tuple:
    """(seed, step, queries, signs, eps) of a Pert or PertPair."""
    pp = Z.as_pair(pert)
    return (pp.seed, pp.step, tuple(pp.query), tuple(pp.sign), float(pp.eps))


def interleave_gate_up(wg: torch.Tensor, wu: torch.Tensor) -> torch.Tensor:
    """Rows 32j..32j+15 = gate rows 16j..16j+15, rows 32j+16..32j+31 = the matching up rows."""
    ff = wg.shape[0]
    if ff % 16:
        raise ValueError("d_ff must be a multiple of 16")
    return torch.stack([wg.reshape(ff // 16, 16, *wg.shape[1:]), wu.reshape(ff // 16, 16, *wu.shape[1:])],
                       dim=1).reshape(2 * ff, *wg.shape[1:]).contiguous()


class Decoder:
    """A decoder on one GPU: frozen weights, per-site bases U, coefficient arena, Adam state.

    W holds the model's tensors under the names wq wk wv wo, wg wu wd (Llama) or w1 w2 and
    biases (OPT), norms n1 n2 (n1b n2b), emb, head or pos, nf (nfb); numpy arrays or torch
    tensors.  In mode "int4" each linear weight is given instead as a pair (packed uint8
    [N][K/2], scales [N][K/128]) in the library's INT4 format.
    """

    def __init__(self, shape, W: dict, mode: str, *, c_bf16: bool | None = None, device="cuda",
                 int4_dequant: bool = True):
        if mode not in ("fp32", "bf16", "int4"):
            raise ValueError(f"unknown mode {mode!r}")
        self.s, self.mode, self.dev = shape, mode, torch.device(device)
        self.act = torch.float32 if mode == "fp32" else torch.bfloat16
        self.c_bf16 = (mode == "int4") if c_bf16 is None else c_bf16
        s = shape
        self.d, self.H, self.Hkv, self.hd = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim
        self.dkv = self.Hkv * self.hd
        self.blocks = arena_layout(shape)
        self.bmap = {(b.layer, b.name): b for b in self.blocks}
        self.k = sum(b.rows * b.r for b in self.blocks)
        self._adapted_sites = {(b.layer, b.site) for b in self.blocks}
        self.r = s.rank
        self._pack(W, int4_dequant)
        # the fused GEMM's workspace for splitting a partly idle last round of tiles (bf16 modes)
        if self.act == torch.bfloat16:
            nb = Z.linear_workspace_bytes()
            if nb:
                lin_ws = torch.empty(nb, dtype=torch.uint8, device=self.dev)
                for P in self.layers:
                    for v in P.values():
                        if isinstance(v, tuple):
                            v[0].ws = lin_ws
        self.ut = {}                      # (layer, site) -> U^T [r][d_in] (activation dtype)
        self.arena = Z.Arena(torch.zeros(self.k, dtype=torch.bfloat16 if self.c_bf16 else torch.float32,
                                         device=self.dev),
                             torch.zeros(self.k, dtype=torch.float32, device=self.dev),
                             torch.zeros(self.k, dtype=torch.float32, device=self.dev))
        self.t = 0
        self.loss_pm = torch.zeros(2, dtype=torch.float32, device=self.dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=self.dev)
        self.loss_ws = torch.empty(Z.loss_workspace_bytes(), dtype=torch.uint8, device=self.dev)
        self._proj_ws = None     # the depth-split projection's partial sums (grown on demand)
        self._bufs = {}
        self._rope = {}
        self._ch = self._ch_all = None   # per-step C +/- eps Z of the whole arena (bf16 modes)
        # the perturbation the last update pass wrote into _ch_all for the next step:
        # (pair key, arena.c._version after the pass); any torch-side write to C bumps the
        # version and the forward forms the perturbation again
        self._ch_next = None
        # optional callable(stage, lin, T, flags) around every linear launch ("pre"/"post"),
        # for per-launch timing
        self.linear_hook = None
        # layer 0 reads the same embedding in both halves: its first projection forms x W^T
        # and x U once (ZOACT_SHARED_X) when the layer qualifies
        self.shared_first = True
        # norms that feed an adapted site (attention and MLP inputs) also form the site's
        # projection P = x U in the same pass where the library covers the width and it is
        # the faster form: up to NORM_PROJECT_MAX_ROWS rows (measured on MI355X at d = 4096,
        # r = 32: 4096 rows 25.3 us fused against 29.4 us for the norm and the projection
        # apart; 8192 rows 42.0 against 39.6 us -- the fused pass re-reads its 16-token
        # rows from L2 or memory between the statistics and the projection, and the
        # separate norm already runs near the memory rate)
        self.fuse_norm_project = mode != "fp32" and self.r <= 128 and self.d in NORM_PROJECT_WIDTHS
        # INT4 layers: True dequantises each layer once per forward into one bf16 buffer (the
        # largest layer's size, allocated on first use) and runs the bf16 schedule; False
        # keeps the INT4 GEMM that converts the packed weights in LDS.  The first is faster
        # at every batch size measured on MI355X (Llama-3-8B shape, 256 to 4096 tokens per
        # half: 24.8 vs 25.6 ms to 97.8 vs 109.3 ms per step): the INT4 GEMM converts each
        # weight once per 256-token tile, the pass once per forward, and the GEMM then reads
        # the bf16 copy mostly from the last-level cache.
        self.int4_dequant = bool(int4_dequant)
        self._wdq = None

    # ---------------------------------------------------------------- weights
    def _t(self, a, dtype=None):
        dtype = dtype or self.act
        t = a if torch.is_tensor(a) else torch.from_numpy(np.ascontiguousarray(a))
        return t.to(device=self.dev, dtype=dtype).contiguous()

    def _lin_w(self, *parts, interleave=False):
        """Device weight of a fused linear from row blocks (and the INT4 scales)."""
        if self.mode == "int4":
            packed = [self._t(p[0], torch.uint8) for p in parts]
            scales = [self._t(p[1], torch.bfloat16) for p in parts]
            if interleave:
                return interleave_gate_up(*packed), interleave_gate_up(*scales)
            return torch.cat(packed).contiguous(), torch.cat(scales).contiguous()
        ws = [self._t(p) for p in parts]
        if interleave:
            return interleave_gate_up(*ws), None
        return torch.cat(ws).contiguous(), None

    def _int4_dq(self, T: int) -> bool:
        """Whether a forward over T tokens per half runs its INT4 layers dequantised."""
        return self.mode == "int4" and self.int4_dequant

    def _pack(self, W, int4_dequant=True):
        s, d, dkv, ff = self.s, self.d, self.dkv, self.s.d_ff
        ad = set(s.adapted)
        # q and v adapted, k not (OPT): one q|k|v launch with k as its plain feature range
        # where the 64-deep schedules cover it (precomputed C +/- eps Z, range bounds on
        # 256-feature tiles; INT4 weights in whole scale groups); else q|v and k as two
        # launches
        plain_k = ({"q", "v"} <= ad and "k" not in ad and self.act == torch.bfloat16
                   and (self.mode == "bf16" or int4_dequant is True or (d % 128 == 0 and d >= 256))
                   and d % 256 == 0 and dkv % 256 == 0)
        self.layers = []
        for l in range(s.n_layers):
            L = W[l]
            P = {"n1": self._t(L["n1"]), "n2": self._t(L["n2"])}
            if s.family == "opt":
                P["n1b"], P["n2b"] = self._t(L["n1b"]), self._t(L["n2b"])
            fused_qkv = s.family == "llama" and ({"q", "k", "v"} <= ad or not (ad & {"q", "k", "v"}))
            if fused_qkv:
                w, sc = self._lin_w(L["wq"], L["wk"], L["wv"])
                P["qkv"] = self._linear(l, "qkv", w, sc, d, d + 2 * dkv)
            elif plain_k:
                w, sc = self._lin_w(L["wq"], L["wk"], L["wv"])
                bias = (torch.cat([self._t(L["bq"]), self._t(L["bk"]), self._t(L["bv"])])
                        if s.family == "opt" else None)
                lin, blk = self._linear(l, "qv", w, sc, d, d + 2 * dkv, bias)
                lin.plain = (d, d + dkv)
                P["qkv"] = (lin, blk)
            else:
                w, sc = self._lin_w(L["wq"], L["wv"])
                bias = torch.cat([self._t(L["bq"]), self._t(L["bv"])]) if s.family == "opt" else None
                P["qv"] = self._linear(l, "qv", w, sc, d, 2 * d, bias)
                w, sc = self._lin_w(L["wk"])
                P["k"] = self._linear(l, None, w, sc, d, dkv, self._t(L["bk"]) if s.family == "opt" else None)
            if s.family == "llama":
                w, sc = self._lin_w(L["wo"])
                P["o"] = self._linear(l, "o", w, sc, d, d)
                w, sc = self._lin_w(L["wg"], L["wu"], interleave=True)
                P["gu"] = self._linear(l, "gu", w, sc, d, 2 * ff)
                w, sc = self._lin_w(L["wd"])
                P["down"] = self._linear(l, "down", w, sc, ff, d)
            else:
                w, sc = self._lin_w(L["wo"])
                P["o"] = self._linear(l, "out", w, sc, d, d, self._t(L["bo"]))
                w, sc = self._lin_w(L["w1"])
                P["gu"] = self._linear(l, "fc1", w, sc, d, ff, self._t(L["b1"]))
                w, sc = self._lin_w(L["w2"])
                P["down"] = self._linear(l, "fc2", w, sc, ff, d, self._t(L["b2"]))
            self.layers.append(P)
        self.emb = self._t(W["emb"])
        self.nf = self._t(W["nf"])
        if s.family == "llama":
            self.head = Z.Linear(self._t(W["head"]), d, s.vocab)
            self.pos = None
        else:
            self.nfb = self._t(W["nfb"])
            self.head = Z.Linear(self.emb, d, s.vocab)        # tied
            self.pos = self._t(W["pos"])

    def _linear(self, l, name, w, scales, d_in, d_out, bias=None):
        b = self.bmap.get((l, name)) if name is not None else None
        return Z.Linear(w, d_in, d_out, r=0, coef_offset=b.offset if b else 0, bias=bias, w_scales=scales), b

    # ---------------------------------------------------------------- buffers
    def _buffers(self, n_seq: int, seq: int):
        """Activation buffers for 2 halves of n_seq sequences of length seq (cached per shape)."""
        key = (n_seq, seq)
        if key in self._bufs:
            return self._bufs[key]
        s, T = self.s, n_seq * seq
        e = lambda *shp, dt=None: torch.empty(*shp, dtype=dt or self.act, device=self.dev)
        fused = "qkv" in self.layers[0]
        B = {
            "h0": e(2 * T, self.d), "h1": e(2 * T, self.d), "a": e(2 * T, self.d),
            "qkv": e(2 * T, self.d + 2 * self.dkv) if fused else e(2 * T, 2 * self.d),
            "k": None if fused else e(2 * T, self.dkv),
            "att": e(2 * T, self.d), "ff": e(2 * T, s.d_ff),
            "p": e(2 * T, max(self.r, 1)),
            "logits": None,          # fp32 [2 T][vocab], allocated when a forward returns logits
        }
        self._bufs[key] = B
        return B

    def _rope_tables(self, seq: int):
        if seq not in self._rope:
            half = self.hd // 2
            j = torch.arange(half, dtype=torch.float64)
            inv = self.s.rope_theta ** (-2.0 * j / self.hd)
            ang = torch.arange(seq, dtype=torch.float64)[:, None] * inv[None, :]
            self._rope[seq] = (torch.cos(ang).float().to(self.dev).contiguous(),
                               torch.sin(ang).float().to(self.dev).contiguous())
        return self._rope[seq]

    # ---------------------------------------------------------------- forward of both halves
    def _norm_site(self, l, site, x, w, b, y, adapt, calibrate):
        """The norm of x into y, then the site's projection of y into P (U^T of the site, or
        None where it is not adapted); one fused pass where the library covers it."""
        if (adapt and self.fuse_norm_project and x.shape[0] <= NORM_PROJECT_MAX_ROWS
                and (l, site) in self._adapted_sites):
            ut = self.ut.get((l, site))
            if ut is None:
                raise RuntimeError(f"no basis for site {(l, site)}: run basis_init or set_basis first")
            p = self._cur["p"][:x.shape[0]]
            if self.s.family == "llama":
                Z.rmsnorm_project(x, w, y, self.s.norm_eps, ut, p)
            else:
                Z.layernorm_project(x, w, b, y, self.s.norm_eps, ut, p)
            return ut
        self._norm(x, w, b, y)
        return self._site(l, site, y, adapt, calibrate)

    def _norm(self, x, w, b, y):
        if self.s.family == "llama":
            Z.rmsnorm(x, w, y, self.s.norm_eps)
        else:
            Z.layernorm(x, w, b, y, self.s.norm_eps)

    def _apply(self, lin_blk, x, T, y, pert, site_ut, residual=None, flags=0, adapt=True):
        lin, blk = lin_blk
        B = self._cur
        if lin.w.dtype == torch.uint8 and self._int4_dq(T):
            n = lin.d_out * lin.d_in
            if self._wdq is None or self._wdq.numel() < n:
                n = max(n, max(l.d_out * l.d_in for P in self.layers for l, _ in
                               (v for v in P.values() if isinstance(v, tuple)) if l.w.dtype == torch.uint8))
                self._wdq = torch.empty(n, dtype=torch.bfloat16, device=self.dev)
            wdq = self._wdq[:lin.d_out * lin.d_in].view(lin.d_out, lin.d_in)
            Z.dequant_int4(lin.w, lin.w_scales, wdq)
            lin = dataclasses.replace(lin, w=wdq, w_scales=None)
        hook = self.linear_hook
        if adapt and blk is not None and site_ut is not None:
            lin.r, lin.ut = self.r, site_ut
            if self._ch is not None:
                lin.ch, lin.ch_stride = self._ch[blk.offset:], self.k
            else:
                lin.ch, lin.ch_stride = None, 0
            if hook:
                hook("pre", lin, T, flags)
            Z.linear_fwd_pm(lin, self.arena, x, T, B["p"], y, pert, residual, flags)
        else:
            lin.r, lin.ut, lin.ch, lin.ch_stride = 0, None, None, 0
            if hook:
                hook("pre", lin, T, flags)
            Z.linear_fwd_pm(lin, None, x, T, None, y, pert, residual, flags)
        if hook:
            hook("post", lin, T, flags)

    def _shared_ok(self, lin_blk, site_ut, T) -> bool:
        """Whether the shared-input form covers this projection over T tokens per half: bf16
        weights (or INT4 run on its dequantised copy), the perturbed coefficients
        precomputed, 8 <= r <= 32 with r % 8 == 0, depth a multiple of 64, no SwiGLU."""
        lin, blk = lin_blk
        return (self.shared_first and self.act == torch.bfloat16 and blk is not None and site_ut is not None
                and self._ch is not None and (lin.w.dtype == torch.bfloat16 or self._int4_dq(T))
                and 8 <= self.r <= 32 and self.r % 8 == 0 and lin.d_in % 64 == 0 and lin.d_in >= 128
                and lin.plain[0] == lin.plain[1])

    def forward(self, tokens: torch.Tensor, pert: Z.Pert | Z.PertPair, *, calibrate=None, distinct_halves=False,
                head: bool = True):
        """Both halves of the forward; logits fp32 [2][n_seq][seq][V] in the buffer set.

        tokens int32 [n_seq][seq] (or [2][n_seq][seq] with distinct_halves).  With a Pert,
        half 0 uses C + eps Z and half 1 C - eps Z; with a PertPair, half h uses
        C + sign[h] eps Z(query[h]).  With `calibrate` (a callable taking (layer, site, x))
        the linears are not adapted and each site's input [2 T][d_in] is handed over
        before it is consumed (Algorithm 1's calibration forward).
        """
        s = self.s
        n_seq, seq = tokens.shape[-2], tokens.shape[-1]
        T = n_seq * seq
        B = self._cur = self._buffers(n_seq, seq)
        adapt = calibrate is None
        # C +/- eps Z for the whole arena in one streaming pass; every adapted GEMM reads its
        # slice instead of regenerating Z per workgroup
        self._ch = None
        if adapt and self.act == torch.bfloat16 and self.k > 0:
            if self._ch_all is None:
                self._ch_all = torch.empty(2 * self.k, dtype=torch.bfloat16, device=self.dev)
            # the previous update pass may have written this step's perturbation already
            if self._ch_next != (_pair_key(pert), self.arena.c._version):
                Z.perturb_coeffs(self.arena, 0, self.k, pert, self._ch_all)
            self._ch = self._ch_all
        self._ch_next = None
        Z.embed(tokens, self.emb, B["h0"], seq, self.pos, pos_offset=2, distinct_halves=distinct_halves)
        h, h_alt = B["h0"], B["h1"]
        cos_sin = self._rope_tables(seq) if s.family == "llama" else None
        d, dkv, H, Hkv, hd = self.d, self.dkv, self.H, self.Hkv, self.hd
        scale = float(np.float32(1.0 / math.sqrt(hd)))
        for l, P in enumerate(self.layers):
            # attention block.  Layer 0 of a forward whose halves read the same tokens: both
            # halves' inputs are the same embedding rows, so the norm and the projection run
            # on one half and the fused q|k|v forms x W^T once (the same bits as stacked)
            qkv = B["qkv"]
            shared = (l == 0 and adapt and not distinct_halves and "qkv" in P
                      and self._shared_ok(P["qkv"], self.ut.get((0, "attn")), T))
            if shared:
                a1 = B["a"][:T]
                ut = self._norm_site(l, "attn", h[:T], P["n1"], P.get("n1b"), a1, adapt, calibrate)
                self._apply(P["qkv"], a1, T, qkv, pert, ut, flags=Z.SHARED_X, adapt=adapt)
                q, k, v = qkv[:, :d], qkv[:, d:d + dkv], qkv[:, d + dkv:]
            elif "qkv" in P:
                ut = self._norm_site(l, "attn", h, P["n1"], P.get("n1b"), B["a"], adapt, calibrate)
                self._apply(P["qkv"], B["a"], T, qkv, pert, ut, adapt=adapt)
                q, k, v = qkv[:, :d], qkv[:, d:d + dkv], qkv[:, d + dkv:]
            else:
                ut = self._norm_site(l, "attn", h, P["n1"], P.get("n1b"), B["a"], adapt, calibrate)
                self._apply(P["qv"], B["a"], T, qkv, pert, ut, adapt=adapt)
                self._apply(P["k"], B["a"], T, B["k"], pert, None, adapt=False)
                q, k, v = qkv[:, :d], B["k"], qkv[:, d:]
            if cos_sin is not None:
                # rotary on q and k, inside the attention where it holds the sequence in LDS
                Z.attention_rope(q, k, v, B["att"], 2 * n_seq, seq, H, Hkv, hd, scale, *cos_sin)
            else:
                Z.attention(q, k, v, B["att"], 2 * n_seq, seq, H, Hkv, hd, scale)
            ut = self._site(l, "o", B["att"], adapt, calibrate)
            self._apply(P["o"], B["att"], T, h_alt, pert, ut, residual=h, adapt=adapt)
            h, h_alt = h_alt, h
            # MLP block
            ut = self._norm_site(l, "mlp", h, P["n2"], P.get("n2b"), B["a"], adapt, calibrate)
            flags = Z.EPI_SWIGLU if s.family == "llama" else Z.EPI_RELU
            self._apply(P["gu"], B["a"], T, B["ff"], pert, ut, flags=flags, adapt=adapt)
            ut = self._site(l, "down", B["ff"], adapt, calibrate)
            self._apply(P["down"], B["ff"], T, h_alt, pert, ut, residual=h, adapt=adapt)
            h, h_alt = h_alt, h
        self._norm(h, self.nf, getattr(self, "nfb", None), B["a"])
        if not head:                 # the caller runs the LM head (fused with the loss)
            return B["a"]
        if B["logits"] is None:
            B["logits"] = torch.empty(2 * T, s.vocab, dtype=torch.float32, device=self.dev)
        Z.linear_fwd_pm(self.head, None, B["a"], T, None, B["logits"], pert)
        return B["logits"].view(2, n_seq, seq, s.vocab)

    def _site(self, l, site, x, adapt, calibrate):
        """U^T of an adapted site after projecting its input into P (None if not adapted)."""
        if not adapt:
            calibrate(l, site, x)
            return None
        ut = self.ut.get((l, site)) if (l, site) in self._adapted_sites else None
        if ut is None:
            if (l, site) in self._adapted_sites:
                raise RuntimeError(f"no basis for site {(l, site)}: run basis_init or set_basis first")
            return None
        n_tok = x.shape[0]
        need = Z.project_workspace_bytes(n_tok, x.shape[1], self.r) if self.act == torch.bfloat16 else 0
        if need and (self._proj_ws is None or self._proj_ws.numel() < need):
            self._proj_ws = torch.empty(need, dtype=torch.uint8, device=self.dev)
        Z.project(x, ut, self._cur["p"][:n_tok], self._proj_ws if need else None)
        return ut

    def site_dims(self):
        """(layer, site) -> d_in for every adapted site."""
        d_in = {"attn": self.d, "o": self.d, "mlp": self.d, "down": self.s.d_ff}
        return {(b.layer, b.site): d_in[b.site] for b in self.blocks}

    # ---------------------------------------------------------------- Algorithm 1
    def basis_init(self, calib_tokens: torch.Tensor, opts: Z.EigOpts | None = None, keep_eigvals=False,
                   report=False, concurrency: int = 4):
        """Unperturbed calibration forward, then the top-r basis of each adapted site's inputs.

        calib_tokens int32 [n_seq][seq] with n_seq even: the two halves of the stacked
        forward carry the first and second n_seq/2 sequences, so every site sees all
        n_seq * seq calibration tokens once.  With `report` each site's convergence report
        (residual, gap theta_r / theta_{r+1}, iterations, converged) lands in
        self.basis_report after the call; a site whose residual stays above opts.tol keeps
        its best-effort basis and is reported with converged = False.

        `concurrency` sites are solved at once: each site's input is copied as the forward
        produces it and handed to one of that many host threads, each with its own stream
        and workspace (the solver's small b x b steps run on one workgroup and its adaptive
        checks wait on the host, so one site leaves most of the GPU idle).  Every site's
        result is the same as when solved alone.  1 solves each site inside the forward.
        """
        n_seq, seq = calib_tokens.shape
        if n_seq % 2:
            raise ValueError("the calibration batch needs an even number of sequences")
        dims = self.site_dims()
        nws = max(Z.basis_init_workspace_bytes(dd, self.r, opts) for dd in set(dims.values()))
        k = max(1, int(concurrency))
        wss = [torch.empty(nws, dtype=torch.uint8, device=self.dev) for _ in range(k)]
        self.eigvals = {}
        reps = {}

        def outputs(key):   # the site's basis, eigenvalues and report (allocated on the current stream)
            ut = torch.empty(self.r, dims[key], dtype=self.act, device=self.dev)
            ev = torch.empty(self.r, dtype=torch.float32, device=self.dev) if keep_eigvals else None
            rep = Z.eig_report_tensor(self.dev) if report else None
            self.ut[key] = ut
            if keep_eigvals:
                self.eigvals[key] = ev
            if report:
                reps[key] = rep
            return ut, ev, rep

        tok = calib_tokens.reshape(2, n_seq // 2, seq).contiguous()
        if k == 1:
            def hook(l, site, x):
                if (l, site) in dims:
                    ut, ev, rep = outputs((l, site))
                    Z.basis_init(x, self.r, ut, wss[0], opts, eigvals=ev, report=rep)

            self.forward(tok, Z.Pert(0, 0, 0, 0.0), calibrate=hook, distinct_halves=True)
        else:
            streams = [torch.cuda.Stream(device=self.dev) for _ in range(k)]
            idle = queue.SimpleQueue()
            for i in range(k):
                idle.put(i)

            def work(x, out, ready):
                i = idle.get()
                try:
                    s = streams[i]
                    s.wait_event(ready)
                    ut, ev, rep = out
                    Z.basis_init(x, self.r, ut, wss[i], opts, eigvals=ev, report=rep, stream=s)
                    for t in (x, *out):
                        if t is not None:
                            t.record_stream(s)
                finally:
                    idle.put(i)

            futures = []
            with concurrent.futures.ThreadPoolExecutor(max_workers=k) as pool:
                def hook(l, site, x):
                    if (l, site) not in dims:
                        return
                    xc = x.clone()
                    out = outputs((l, site))
                    ready = torch.cuda.Event()
                    ready.record()
                    futures.append(pool.submit(work, xc, out, ready))

                self.forward(tok, Z.Pert(0, 0, 0, 0.0), calibrate=hook, distinct_halves=True)
                for f in futures:
                    f.result()
            for st in streams:
                st.synchronize()
        if report:
            self.basis_report = {k2: Z.read_eig_report(v) for k2, v in reps.items()}
        return self.ut

    def set_basis(self, ut: dict):
        """Install bases U^T [r][d_in] per (layer, site) (e.g. computed elsewhere)."""
        for key, d_in in self.site_dims().items():
            u = ut[key]
            self.ut[key] = self._t(u).reshape(self.r, d_in).contiguous()

    # ---------------------------------------------------------------- Algorithm 2 step
    def _loss_pair(self, tokens: torch.Tensor, pert, out: torch.Tensor):
        """Forward both halves and write their next-token cross entropies into out[0:2]; in
        bf16 modes the LM head and the loss run fused (logits not stored)."""
        if self.act == torch.bfloat16:
            a = self.forward(tokens, pert, head=False)
            T = tokens.numel()
            need = Z.linear_xent_workspace_bytes(T, self.s.vocab)
            if getattr(self, "_xent_ws", None) is None or self._xent_ws.numel() < need:
                self._xent_ws = torch.empty(need, dtype=torch.uint8, device=self.dev)
            Z.linear_xent(self.head, None, a, tokens, None, pert, out, self._xent_ws)
        else:
            self.forward(tokens, pert)
            Z.xent_pm(self._cur["logits"], tokens, out, self.loss_ws)
        return out

    def losses(self, tokens: torch.Tensor, seed: int, t: int, eps: float):
        """Forward both halves at step t and write (L+, L-) into self.loss_pm."""
        return self._loss_pair(tokens, Z.Pert(seed, t, 0, eps), self.loss_pm)

    def step(self, tokens: torch.Tensor, seed: int, eps: float, lr: float, optimizer: str = "adam"):
        """One two-sided ZO step: L+ and L-, g = (L+ - L-) / (2 eps), update C with Z regenerated.
        In bf16 modes the Adam pass also writes the next step's C +/- eps Z (one pass over the
        arena instead of two), which the next step's forward then reads."""
        self.t += 1
        pert = Z.Pert(seed, self.t, 0, eps)
        self.losses(tokens, seed, self.t, eps)
        if optimizer == "adam" and self._ch_all is not None:
            nxt = Z.Pert(seed, self.t + 1, 0, eps)
            Z.step_perturb(self.arena, self.loss_pm, pert, Z.adam_desc(lr, self.t), nxt, self._ch_all, self.status)
            self._ch_next = (_pair_key(nxt), self.arena.c._version)
        elif optimizer == "adam":
            Z.step(self.arena, self.loss_pm, pert, Z.adam_desc(lr, self.t), self.status)
        elif optimizer == "sgd":
            Z.step_sgd(self.arena, self.loss_pm, pert, lr, self.status)
        else:
            raise ValueError(optimizer)
        return self.loss_pm

    def step_q(self, tokens: torch.Tensor, seed: int, eps: float, lr: float, q: int, optimizer: str = "adam"):
        """One step of Algorithm 2 in its one-sided q-query form: the unperturbed loss L and
        L_j under C + eps Z^(j), j = 1..q (Z^(j) = Z(seed, t, query j)), evaluated two per
        stacked forward (ceil((q + 1) / 2) forwards; a spare half re-evaluates L), then the
        averaged estimate drives Adam or SGD.  Returns the device losses [L, L_1 .. L_q, spare]."""
        if not 1 <= q <= 256:
            raise ValueError("q must be in [1, 256]")
        self.t += 1
        n_fwd = (q + 2) // 2
        losses = torch.zeros(2 * n_fwd, dtype=torch.float32, device=self.dev)

        def spec(e):            # evaluation e: 0 = unperturbed, 1..q = query e, beyond = spare (unperturbed)
            return (e, 1) if 1 <= e <= q else (0, 0)

        for i in range(n_fwd):
            (q0, s0), (q1, s1) = spec(2 * i), spec(2 * i + 1)
            self._loss_pair(tokens, Z.pert_pair(seed, self.t, (q0, q1), (s0, s1), eps), losses[2 * i:2 * i + 2])
        if optimizer == "adam":
            Z.step_q(self.arena, losses, q, seed, self.t, eps, Z.adam_desc(lr, self.t), self.status)
        elif optimizer == "sgd":
            Z.step_q_sgd(self.arena, losses, q, seed, self.t, eps, lr, self.status)
        else:
            raise ValueError(optimizer)
        return losses
