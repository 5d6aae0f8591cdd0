"""Seeded synthetic inputs shared by the oracle and the HIP path.

This module holds none of the method's arithmetic: it draws weights, tokens,
activations and coefficients from seeded generators, rounds inputs to the
storage precision of the workload, and packs frozen weights into the INT4
group-128 storage format.  Both sides receive the same arrays as data.

Workload shapes follow the paper's models (Llama-3-8B, OPT-13B and an INT4
Llama-3-8B, Section 5 and Appendix B) with random initialisation, because no
pretrained weights or task datasets are used: uniform random token ids stand in
for the fine-tuning batches, and a planted low-rank activation matrix stands in
for the concentrated activation spectra the method relies on (Section 3,
Motivation; Section 4, least-squares discussion).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "gen", "normal", "bf16_round", "bf16_bits", "bits_to_f32", "uniform_tokens",
    "planted_lowrank", "quantize_int4_g128", "ModelShape", "TINY", "LLAMA3_8B",
    "OPT_13B", "shrink",
]


def gen(seed: int, *ids: int) -> np.random.Generator:
    """Independent PCG64 stream for (seed, *ids)."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), *map(int, ids)])))


def normal(shape, std: float, seed: int, *ids: int) -> np.ndarray:
    """float32 N(0, std^2) draws from the stream (seed, *ids)."""
    return (gen(seed, *ids).standard_normal(size=shape, dtype=np.float32) * np.float32(std)).astype(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """uint16 bf16 bit patterns of float32 x, round-to-nearest-even (storage conversion)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bits_to_f32(h: np.ndarray) -> np.ndarray:
    """float32 values of uint16 bf16 bit patterns (exact)."""
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 array holding bf16-representable values (RNE of x)."""
    return bits_to_f32(bf16_bits(x))


def uniform_tokens(batch: int, seq: int, vocab: int, seed: int, stream: int) -> np.ndarray:
    """int32 [batch][seq] uniform token ids in [0, vocab)."""
    return gen(seed, 7001, stream).integers(0, vocab, size=(batch, seq), dtype=np.int64).astype(np.int32)


def planted_lowrank(n_tok: int, d: int, n_dirs: int = 64, frac: float = 0.9, decay: float = 0.95,
                    seed: int = 0):
    """Activations with a planted low-rank structure.

    x = A diag(sigma) Q^T + s N, with Q (d x n_dirs) orthonormal, A and N standard normal,
    sigma_i^2 = sigma_0^2 decay^i and sum(sigma_i^2) = frac * d, noise variance (1 - frac)
    per coordinate, so each coordinate has unit variance on average and `frac` of the
    variance lies in the n_dirs planted directions.  Returns (x float32 [n_tok][d], Q).
    """
    g = gen(seed, 7101)
    q, _ = np.linalg.qr(g.standard_normal((d, n_dirs)))
    w = decay ** np.arange(n_dirs)
    sig2 = w * (frac * d / w.sum())
    a = g.standard_normal((n_tok, n_dirs))
    noise = g.standard_normal((n_tok, d))
    x = (a * np.sqrt(sig2)) @ q.T + math.sqrt(1.0 - frac) * noise
    return x.astype(np.float32), q.astype(np.float32)


def quantize_int4_g128(w: np.ndarray):
    """Pack a bf16-valued weight [N][K] into symmetric INT4 with bf16 group-128 scales.

    Storage format of the frozen INT4 backbone (the paper quantises its INT4 model with
    MagR, whose format it does not state): per (row, group of 128 along K)
    s = bf16(absmax / 7) computed in fp32, q = clamp(round_half_even(w / s), -7, 7), and
    an all-zero group stores s = 0, q = 0.  Returns (packed uint8 [N][K/2] with the even-k
    value in the low nibble, two's complement; scales as float32 bf16 values [N][K/128]).
    """
    w = np.asarray(w, dtype=np.float32)
    n, k = w.shape
    if k % 128:
        raise ValueError("K must be a multiple of 128")
    g = w.reshape(n, k // 128, 128)
    amax = np.abs(g).max(axis=2)
    s = bf16_round((amax / np.float32(7.0)).astype(np.float32))
    safe = np.where(s == 0, np.float32(1.0), s).astype(np.float32)
    q = np.rint((g / safe[:, :, None]).astype(np.float32))
    q = np.clip(q, -7, 7)
    q = np.where(s[:, :, None] == 0, 0, q).astype(np.int8).reshape(n, k)
    nib = (q.astype(np.int16) & 0xF).astype(np.uint8)
    packed = (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)
    return packed, s.astype(np.float32)


@dataclass(frozen=True)
class ModelShape:
    """Decoder-only transformer shape (random init)."""
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    d_ff: int
    vocab: int
    family: str = "llama"          # "llama" (RMSNorm, RoPE, SwiGLU) or "opt" (LayerNorm, learned pos, ReLU)
    rope_theta: float = 5.0e5
    norm_eps: float = 1e-5
    max_pos: int = 2048
    adapted: tuple = ("q", "k", "v", "o", "gate", "up", "down")
    rank: int = 32
    init_std: float = 0.02
    extra: dict = field(default_factory=dict)

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads


TINY = ModelShape("tiny-llama", 2, 128, 4, 4, 512, 512, rope_theta=1.0e4, adapted=("q", "v"), rank=8)
LLAMA3_8B = ModelShape("llama-3-8b-shape", 32, 4096, 32, 8, 14336, 128256)
OPT_13B = ModelShape("opt-13b-shape", 40, 5120, 40, 40, 20480, 50272, family="opt",
                     adapted=("q", "v", "o", "fc1", "fc2"), rank=64)


def shrink(shape: ModelShape, **kw) -> ModelShape:
    """Same family with some dimensions replaced (small parity cases)."""
    d = dict(shape.__dict__)
    d.update(kw)
    return ModelShape(**d)


# ------------------------------------------------------------------ model weights
def model_weights(shape: ModelShape, seed: int, mode: str) -> dict:
    """Per-tensor seeded random-init weights of a decoder, float32 arrays.

    Streams: embedding (seed, 1000, 0), LM head (seed, 1000, 1), learned positions
    (seed, 1000, 2), layer l tensor k (seed, l, k) with k = 1..7 for q, k, v, o and the
    MLP matrices (Llama gate, up, down; OPT fc1, fc2).  N(0, init_std^2) draws (rounded to
    bf16 values when mode is "bf16"), norm weights 1, biases 0.  Names: emb, head, pos,
    nf/nfb (final norm), and per layer wq wk wv wo, wg wu wd (Llama) or w1 w2 with biases
    bq bk bv bo b1 b2 (OPT), n1/n2 (and n1b/n2b for LayerNorm).
    """
    rnd = bf16_round if mode == "bf16" else (lambda a: a.astype(np.float32))
    d, dkv, ff, V, std = shape.d_model, shape.n_kv_heads * shape.head_dim, shape.d_ff, shape.vocab, shape.init_std
    W = {"emb": rnd(normal((V, d), std, seed, 1000, 0))}
    for l in range(shape.n_layers):
        def t(k, shp):
            return rnd(normal(shp, std, seed, l, k))
        L = {"wq": t(1, (d, d)), "wk": t(2, (dkv, d)), "wv": t(3, (dkv, d)), "wo": t(4, (d, d))}
        if shape.family == "llama":
            L.update({"wg": t(5, (ff, d)), "wu": t(6, (ff, d)), "wd": t(7, (d, ff)),
                      "n1": np.ones(d, np.float32), "n2": np.ones(d, np.float32)})
        else:
            L.update({"w1": t(5, (ff, d)), "w2": t(6, (d, ff)),
                      "n1": np.ones(d, np.float32), "n1b": np.zeros(d, np.float32),
                      "n2": np.ones(d, np.float32), "n2b": np.zeros(d, np.float32)})
            for b, n in (("bq", d), ("bk", dkv), ("bv", dkv), ("bo", d), ("b1", ff), ("b2", d)):
                L[b] = np.zeros(n, np.float32)
        W[l] = L
    W["nf"] = np.ones(d, np.float32)
    if shape.family == "llama":
        W["head"] = rnd(normal((V, d), std, seed, 1000, 1))
    else:
        W["nfb"] = np.zeros(d, np.float32)
        W["pos"] = rnd(normal((shape.max_pos + 2, d), std, seed, 1000, 2))
    return W


def device_normal(shape, std: float, seed: int, *ids: int, device="cuda", dtype=None):
    """N(0, std^2) draws generated on the device from a torch generator seeded by (seed, *ids).

    For full-size models, whose weights are too large to draw on the host quickly; the
    values differ from normal() for the same ids.
    """
    import torch

    key = int(np.random.SeedSequence([seed, *ids]).generate_state(1, np.uint64)[0] >> 1)
    g = torch.Generator(device=device)
    g.manual_seed(key)
    a = torch.randn(shape, generator=g, device=device, dtype=torch.float32).mul_(std)
    return a.to(dtype) if dtype is not None else a


def device_model_weights(shape: ModelShape, seed: int, dtype, device="cuda") -> dict:
    """model_weights() with the same names and streams, drawn on the device (torch tensors)."""
    import torch

    d, dkv, ff, V, std = shape.d_model, shape.n_kv_heads * shape.head_dim, shape.d_ff, shape.vocab, shape.init_std
    ones = lambda n: torch.ones(n, dtype=dtype, device=device)
    zeros = lambda n: torch.zeros(n, dtype=dtype, device=device)
    W = {"emb": device_normal((V, d), std, seed, 1000, 0, device=device, dtype=dtype)}
    for l in range(shape.n_layers):
        def t(k, shp):
            return device_normal(shp, std, seed, l, k, device=device, dtype=dtype)
        L = {"wq": t(1, (d, d)), "wk": t(2, (dkv, d)), "wv": t(3, (dkv, d)), "wo": t(4, (d, d))}
        if shape.family == "llama":
            L.update({"wg": t(5, (ff, d)), "wu": t(6, (ff, d)), "wd": t(7, (d, ff)), "n1": ones(d), "n2": ones(d)})
        else:
            L.update({"w1": t(5, (ff, d)), "w2": t(6, (d, ff)), "n1": ones(d), "n1b": zeros(d), "n2": ones(d),
                      "n2b": zeros(d)})
            for b, n in (("bq", d), ("bk", dkv), ("bv", dkv), ("bo", d), ("b1", ff), ("b2", d)):
                L[b] = zeros(n)
        W[l] = L
    W["nf"] = ones(d)
    if shape.family == "llama":
        W["head"] = device_normal((V, d), std, seed, 1000, 1, device=device, dtype=dtype)
    else:
        W["nfb"] = zeros(d)
        W["pos"] = device_normal((shape.max_pos + 2, d), std, seed, 1000, 2, device=device, dtype=dtype)
    return W


def device_quantize_int4_g128(w):
    """quantize_int4_g128() on a device tensor (bf16 values): (packed uint8 [N][K/2], scales bf16 [N][K/128])."""
    import torch

    n, k = w.shape
    if k % 128:
        raise ValueError("K must be a multiple of 128")
    g = w.float().reshape(n, k // 128, 128)
    s = (g.abs().amax(dim=2) / 7.0).to(torch.bfloat16)
    sf = s.float()
    safe = torch.where(sf == 0, torch.ones_like(sf), sf)
    q = torch.round(g / safe[:, :, None]).clamp_(-7, 7)
    q = torch.where(sf[:, :, None] == 0, torch.zeros_like(q), q).to(torch.int16).reshape(n, k)
    nib = (q & 0xF).to(torch.uint8)
    packed = nib[:, 0::2] | (nib[:, 1::2] << 4)
    return packed.contiguous(), s.contiguous()
