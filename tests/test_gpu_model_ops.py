"""GPU parity of the decoder support operations (embedding, norms, rotary, attention)
against the oracle's definitions on the same seeded inputs."""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import model as om
from paper_2607_01125_amd import zoact as Z

from gpu_helpers import announce, assert_bf16_close, assert_rel_close, dev, host, t_bf16, t_f32, t_i32

pytestmark = pytest.mark.gpu


def _act(a, bf16):
    return t_bf16(a) if bf16 else t_f32(a)


def _vals(shape, std, seed, *ids, bf16):
    a = synth.normal(shape, std, seed, *ids)
    return synth.bf16_round(a) if bf16 else a


# ------------------------------------------------------------------ embedding
@pytest.mark.parametrize("bf16,with_pos", [(False, False), (True, False), (True, True)])
def test_embed(bf16, with_pos):
    announce("embed", bf16, with_pos)
    V, d, B, S = 300, 192, 3, 37
    table = _vals((V, d), 0.02, 1, 1, bf16=bf16)
    pos = _vals((S + 2, d), 0.02, 1, 2, bf16=bf16) if with_pos else None
    tok = synth.uniform_tokens(B, S, V, 1, 3)
    out = torch.empty(2, B * S, d, dtype=torch.bfloat16 if bf16 else torch.float32, device=dev())
    Z.embed(t_i32(tok.reshape(-1)), _act(table, bf16), out, S, _act(pos, bf16) if with_pos else None,
            pos_offset=2 if with_pos else 0)
    want = table[tok.reshape(-1)].astype(np.float64)
    if with_pos:
        want = want + pos[np.tile(np.arange(S) + 2, B)]
        want = synth.bf16_round(want.astype(np.float32)).astype(np.float64) if bf16 else want
        # the sum of two bf16 values rounded once: at most half an ulp off the exact sum
        got = host(out)
        for h in range(2):
            assert_bf16_close(got[h], want, 0.0, "embed+pos")
    else:
        got = host(out)
        for h in range(2):
            np.testing.assert_array_equal(got[h], want)


# ------------------------------------------------------------------ norms
@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("rows,d", [(7, 128), (300, 4096), (33, 5120)])
def test_rmsnorm(bf16, rows, d):
    announce("rmsnorm", bf16, rows, d)
    x = _vals((rows, d), 1.0, 2, rows, bf16=bf16)
    w = synth.normal((d,), 0.3, 2, d) + np.float32(1.0)
    w = synth.bf16_round(w) if bf16 else w
    y = torch.empty(rows, d, dtype=torch.bfloat16 if bf16 else torch.float32, device=dev())
    Z.rmsnorm(_act(x, bf16), _act(w, bf16), y, 1e-5)
    want = om.rmsnorm(x, w, 1e-5, "bf16" if bf16 else "fp32")
    if bf16:
        assert_bf16_close(host(y), want, 1e-6, "rmsnorm")
    else:
        assert_rel_close(host(y), want, 1e-5, "rmsnorm")


@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("rows,d", [(5, 128), (129, 5120), (7, 2056), (3, 8192), (2, 100)])
def test_layernorm(bf16, rows, d):
    announce("layernorm", bf16, rows, d)
    x = synth.normal((rows, d), 2.0, 3, rows) + np.float32(0.5)
    x = synth.bf16_round(x) if bf16 else x
    w = _vals((d,), 0.2, 3, 1, bf16=bf16)
    b = _vals((d,), 0.1, 3, 2, bf16=bf16)
    y = torch.empty(rows, d, dtype=torch.bfloat16 if bf16 else torch.float32, device=dev())
    Z.layernorm(_act(x, bf16), _act(w, bf16), _act(b, bf16), y, 1e-5)
    want = om.layernorm(x, w, b, 1e-5, "bf16" if bf16 else "fp32")
    if bf16:
        assert_bf16_close(host(y), want, 1e-5, "layernorm")
    else:
        np.testing.assert_allclose(host(y), want, rtol=1e-5, atol=1e-5 * np.sqrt(np.mean(want ** 2)))


# ------------------------------------------------------------------ rotary embedding
@pytest.mark.parametrize("bf16", [False, True])
def test_rope_on_fused_columns(bf16):
    """Rotary embedding applied in place to the q and k column ranges of a fused qkv row."""
    announce("rope", bf16)
    B, S, H, Hkv, hd = 2, 45, 4, 2, 64
    ld = (H + 2 * Hkv) * hd
    x = _vals((B * S, ld), 1.0, 4, 0, bf16=bf16)
    cos, sin = om.rope_tables(S, hd, 5e5)
    xt = _act(x, bf16)
    ct, st = t_f32(cos), t_f32(sin)
    Z.rope(xt, 0, H, hd, S, ct, st)
    Z.rope(xt, H * hd, Hkv, hd, S, ct, st)
    mode = "bf16" if bf16 else "fp32"
    want = x.astype(np.float64).copy()
    want[:, :H * hd] = om.rope(x[:, :H * hd].reshape(B, S, H, hd), cos, sin, mode).reshape(B * S, -1)
    want[:, H * hd:(H + Hkv) * hd] = om.rope(x[:, H * hd:(H + Hkv) * hd].reshape(B, S, Hkv, hd), cos, sin,
                                             mode).reshape(B * S, -1)
    got = host(xt)
    np.testing.assert_array_equal(got[:, (H + Hkv) * hd:], x[:, (H + Hkv) * hd:])   # v untouched
    if bf16:
        assert_bf16_close(got, want, 1e-6, "rope")
    else:
        np.testing.assert_allclose(got, want, rtol=1e-6, atol=1e-6)


# ------------------------------------------------------------------ attention
def _attn_case(bf16, B, S, H, Hkv, hd, seed):
    """(GPU output, oracle output, oracle sum_j p_j |v_j| / l) on a fused qkv buffer."""
    ld = (H + 2 * Hkv) * hd
    qkv = _vals((B * S, ld), 1.0, 5, seed, bf16=bf16)
    q = qkv[:, :H * hd].reshape(B, S, H, hd)
    k = qkv[:, H * hd:(H + Hkv) * hd].reshape(B, S, Hkv, hd)
    v = qkv[:, (H + Hkv) * hd:].reshape(B, S, Hkv, hd)
    mode = "bf16" if bf16 else "fp32"
    want = om.attention(q, k, v, mode).reshape(B * S, H * hd)
    mag = om.attention(q, k, np.abs(v), "fp32").reshape(B * S, H * hd)
    t = _act(qkv, bf16)
    out = torch.empty(B * S, H * hd, dtype=t.dtype, device=dev())
    Z.attention(t[:, :H * hd], t[:, H * hd:(H + Hkv) * hd], t[:, (H + Hkv) * hd:], out, B, S, H, Hkv, hd,
                float(np.float32(1.0 / math.sqrt(hd))))
    return host(out), want, mag


# the last three fill the chip with (sequence, key/value head, four query heads) workgroups,
# which selects the whole-sequence-resident kernel: ragged lengths, both head sizes, and
# eight query heads per key/value head (two workgroups per key/value head)
@pytest.mark.parametrize("B,S,H,Hkv,hd", [(2, 64, 4, 2, 128), (3, 100, 4, 4, 64), (1, 257, 8, 2, 128),
                                          (2, 1, 2, 1, 64), (1, 512, 2, 2, 128), (1, 130, 16, 2, 128),
                                          (1, 70, 6, 2, 64), (2, 256, 32, 8, 128),
                                          (128, 33, 8, 2, 64), (64, 130, 16, 4, 128), (64, 64, 16, 2, 128)])
def test_attention_bf16(B, S, H, Hkv, hd):
    """Bound: the output's own bf16 rounding (2^-7 |o|) plus one bf16 ulp (<= 2^-7 p) on
    every rounded probability, which fp32 scores (GPU) and float64 scores (oracle) can
    round either way: 2^-7 sum_j p_j |v_j| / l."""
    announce("attention bf16", B, S, H, Hkv, hd)
    got, want, mag = _attn_case(True, B, S, H, Hkv, hd, S)
    tol = 2.0 ** -7 * (np.abs(want) + mag) + 1e-6
    bad = np.abs(got - want) > tol
    assert not bad.any(), f"{bad.sum()} outside; first {np.argwhere(bad)[0]}"
    # far inside the bound on average: the rounding differences are rare
    assert np.mean(np.abs(got - want)) <= 0.05 * np.mean(tol)


@pytest.mark.parametrize("B,S,H,Hkv,hd", [(32, 256, 32, 8, 128), (64, 256, 16, 4, 64)])
def test_attention_full_length_sampled(B, S, H, Hkv, hd):
    """Full 256-token sequences on grids that fill the chip (whole-sequence-resident kernel):
    32 sequences with 32 query and 8 key/value heads of 128 (the attention of the Llama-3-8B
    step, both perturbation halves), and head size 64.  The oracle runs on three of the
    sequences; same bound as test_attention_bf16."""
    announce("attention bf16 sampled", B, S, H, Hkv, hd)
    ld = (H + 2 * Hkv) * hd
    qkv = _vals((B * S, ld), 1.0, 5, 4242, bf16=True)
    t = t_bf16(qkv)
    out = torch.empty(B * S, H * hd, dtype=torch.bfloat16, device=dev())
    Z.attention(t[:, :H * hd], t[:, H * hd:(H + Hkv) * hd], t[:, (H + Hkv) * hd:], out, B, S, H, Hkv, hd,
                float(np.float32(1.0 / math.sqrt(hd))))
    got = host(out).reshape(B, S, H * hd)
    x = qkv.reshape(B, S, ld)
    for b in (0, B // 2 + 1, B - 1):
        q = x[b:b + 1, :, :H * hd].reshape(1, S, H, hd)
        k = x[b:b + 1, :, H * hd:(H + Hkv) * hd].reshape(1, S, Hkv, hd)
        v = x[b:b + 1, :, (H + Hkv) * hd:].reshape(1, S, Hkv, hd)
        want = om.attention(q, k, v, "bf16").reshape(S, H * hd)
        mag = om.attention(q, k, np.abs(v), "fp32").reshape(S, H * hd)
        tol = 2.0 ** -7 * (np.abs(want) + mag) + 1e-6
        bad = np.abs(got[b] - want) > tol
        assert not bad.any(), f"sequence {b}: {bad.sum()} outside; first {np.argwhere(bad)[0]}"
        assert np.mean(np.abs(got[b] - want)) <= 0.05 * np.mean(tol)


@pytest.mark.parametrize("B,S,H,Hkv,hd", [(32, 256, 32, 8, 128), (128, 33, 8, 2, 64), (64, 130, 16, 4, 128),
                                          (2, 100, 8, 2, 128), (3, 70, 4, 4, 64)])
def test_attention_rope_equals_rope_then_attention(B, S, H, Hkv, hd):
    """zoact_attention_rope against zoact_rope on q and k followed by zoact_attention, bit
    for bit: on chip-filling grids the rotation happens inside the whole-sequence-resident
    kernel as q and k are read; the last two shapes take the rotary pass first."""
    announce("attention_rope", B, S, H, Hkv, hd)
    ld = (H + 2 * Hkv) * hd
    qkv = t_bf16(_vals((B * S, ld), 1.0, 6, S, bf16=True))
    cos, sin = om.rope_tables(S, hd, 5e5)
    ct, st = t_f32(cos), t_f32(sin)
    scale = float(np.float32(1.0 / math.sqrt(hd)))
    ref_in = qkv.clone()
    Z.rope(ref_in, 0, H + Hkv, hd, S, ct, st)
    ref = torch.empty(B * S, H * hd, dtype=torch.bfloat16, device=dev())
    Z.attention(ref_in[:, :H * hd], ref_in[:, H * hd:(H + Hkv) * hd], ref_in[:, (H + Hkv) * hd:], ref, B, S, H, Hkv,
                hd, scale)
    out = torch.empty_like(ref)
    before = qkv.clone()
    Z.attention_rope(qkv[:, :H * hd], qkv[:, H * hd:(H + Hkv) * hd], qkv[:, (H + Hkv) * hd:], out, B, S, H, Hkv, hd,
                     scale, ct, st)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))
    # the documented post-state of q and k: rotated in place, or untouched
    in_place = Z.attention_rope_in_place(B, S, H, Hkv, hd, Z.BF16)
    assert in_place == (0 if (B, S) in ((32, 256), (128, 33), (64, 130)) else 1)
    want = ref_in if in_place else before
    assert torch.equal(qkv.view(torch.int16), want.view(torch.int16))


@pytest.mark.parametrize("B,S,H,Hkv,hd", [(4, 64, 4, 4, 32), (2, 17, 4, 2, 16), (1, 1, 1, 1, 8)])
def test_attention_f32(B, S, H, Hkv, hd):
    announce("attention f32", B, S, H, Hkv, hd)
    got, want, _ = _attn_case(False, B, S, H, Hkv, hd, S)
    np.testing.assert_allclose(got, want, rtol=2e-5, atol=2e-6)


def test_attention_rejects_bad_grouping():
    t = torch.zeros(8, 3 * 64, dtype=torch.bfloat16, device=dev())
    out = torch.empty(8, 64, dtype=torch.bfloat16, device=dev())
    with pytest.raises(Z.ZoactError):
        Z.attention(t[:, :64], t[:, 64:128], t[:, 128:], out, 1, 8, 3, 2, 64, 0.125)
