"""GPU parity: every hot-path kernel against the CPU oracle on the same seeded inputs.

Bars: Z, indices and the Adam update under teacher forcing bit-exact; bf16
outputs within one bf16 ulp plus an fp32-summation term (gpu_helpers); fp32-mode
outputs and losses within 1e-4 relative; bf16-mode losses within 2e-2 relative.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import adam as oadam
from oracle import basis as obasis
from oracle import linear as olin
from oracle import loss as oloss
from oracle import rng as orng
from oracle.numerics import rne_bf16
from paper_2607_01125_amd import zoact as Z

from gpu_helpers import (announce, assert_bf16_close, assert_rel_close, dev, host, t_bf16, t_f32, t_i32, t_u8)

pytestmark = pytest.mark.gpu


# ------------------------------------------------------------------ Z
@pytest.mark.parametrize("seed,step,query,e0,n", [
    (0, 1, 0, 0, 1 << 22),
    (2024, 7, 3, 5, 1_000_003),
    (2**63 + 11, 2**32 - 1, 1, 2**32 - 1000, 5000),
    (42, 3, 0, 44_040_192 - 4099, 4099),
])
def test_gen_z_bit_exact(seed, step, query, e0, n):
    announce("gen_z", seed, step, query, e0, n)
    out = torch.empty(n, dtype=torch.float32, device=dev())
    Z.gen_z(seed, step, query, e0, n, out)
    got = out.cpu().numpy()
    want = orng.gauss_range(seed, step, query, e0, n)
    np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32))


# 10^8 indices in chunks of 4M: contiguous runs from 0 (the Llama arena and beyond), runs past
# 2^34 (the counter's high word), other seeds, steps and queries; the oracle's chunks are
# computed in worker processes (spawned: they load no GPU runtime)
_Z_CHUNK = 1 << 22
_Z_RUNS = ([(7, 11, 0, i * _Z_CHUNK) for i in range(12)]
           + [(2**64 - 1, 2**32 - 2, 5, (1 << 34) - 3 * _Z_CHUNK // 2 + i * _Z_CHUNK) for i in range(6)]
           + [(1234567, 1 + i, i % 3, (i + 1) * 123_456_789) for i in range(6)]
           + [(0, 0, 0, 44_040_192 - _Z_CHUNK + 8_000_000 - 4_000_000)])   # 25 x 4M >= 10^8


def test_gen_z_bit_exact_1e8():
    import multiprocessing as mp
    from concurrent.futures import ProcessPoolExecutor
    assert len(_Z_RUNS) * _Z_CHUNK >= 10**8
    announce("gen_z 1e8", len(_Z_RUNS), _Z_CHUNK)
    out = torch.empty(_Z_CHUNK, dtype=torch.float32, device=dev())
    cols = list(zip(*_Z_RUNS))
    with ProcessPoolExecutor(max_workers=8, mp_context=mp.get_context("spawn")) as ex:
        wants = ex.map(orng.gauss_range, *cols, [_Z_CHUNK] * len(_Z_RUNS))
        for (seed, step, query, e0), want in zip(_Z_RUNS, wants):
            Z.gen_z(seed, step, query, e0, _Z_CHUNK, out)
            got = out.cpu().numpy()
            bad = np.flatnonzero(got.view(np.uint32) != want.view(np.uint32))
            assert bad.size == 0, f"Z differs at {bad.size} indices from {e0 + bad[0]} (seed {seed}, step {step})"


# ------------------------------------------------------------------ Adam / SGD
@pytest.mark.parametrize("c_bf16", [False, True])
@pytest.mark.parametrize("k", [4, 100_003, 1 << 20])
def test_adam_teacher_forced_bitwise(c_bf16, k):
    announce("adam", c_bf16, k)
    r = np.random.default_rng(k)
    c = r.standard_normal(k).astype(np.float32) * 0.01
    if c_bf16:
        c = rne_bf16(c)
    m = (r.standard_normal(k) * 1e-3).astype(np.float32)
    v = np.abs(r.standard_normal(k) * 1e-5).astype(np.float32)
    lp, lm = np.float32(2.3456), np.float32(2.3441)
    seed, step, eps = 99, 5, 1e-3
    hp = oadam.adam_scalars(5e-5, step)
    g = oadam.projected_grad(lp, lm, eps)
    z = orng.gauss_range(seed, step, 0, 0, k)
    c1, m1, v1, st = oadam.zo_adam(c, m, v, g, z, hp, c_bf16=c_bf16)
    ct = t_bf16(c) if c_bf16 else t_f32(c)
    arena = Z.Arena(ct, t_f32(m), t_f32(v))
    loss = t_f32(np.array([lp, lm]))
    status = torch.zeros(1, dtype=torch.int32, device=dev())
    Z.step(arena, loss, Z.Pert(seed, step, 0, eps), Z.adam_desc(5e-5, step), status)
    np.testing.assert_array_equal(arena.m.cpu().numpy().view(np.uint32), m1.view(np.uint32))
    np.testing.assert_array_equal(arena.v.cpu().numpy().view(np.uint32), v1.view(np.uint32))
    np.testing.assert_array_equal(arena.c.float().cpu().numpy().view(np.uint32), c1.view(np.uint32))
    assert int(status.item()) == 0


def test_adam_nonfinite_guard():
    announce("adam nonfinite")
    k = 1000
    c = np.ones(k, np.float32)
    arena = Z.Arena(t_f32(c), t_f32(c * 0), t_f32(c * 0))
    status = torch.zeros(1, dtype=torch.int32, device=dev())
    Z.step(arena, t_f32(np.array([np.inf, 1.0])), Z.Pert(1, 1, 0, 1e-3), Z.adam_desc(1e-3, 1), status)
    assert int(status.item()) & 1
    np.testing.assert_array_equal(arena.c.cpu().numpy(), c)


def test_sgd_bitwise():
    announce("sgd")
    k = 70_001
    c = (np.random.default_rng(0).standard_normal(k) * 0.01).astype(np.float32)
    arena = Z.Arena(t_f32(c), t_f32(c * 0), t_f32(c * 0))
    lp, lm = np.float32(1.5), np.float32(1.25)
    Z.step_sgd(arena, t_f32(np.array([lp, lm])), Z.Pert(3, 2, 0, 1e-3), 3e-6)
    want, _ = oadam.zo_sgd(c, oadam.projected_grad(lp, lm, 1e-3), orng.gauss_range(3, 2, 0, 0, k), 3e-6)
    np.testing.assert_array_equal(arena.c.cpu().numpy().view(np.uint32), want.view(np.uint32))


# ------------------------------------------------------------------ projection
@pytest.mark.parametrize("n_tok,d,r", [(1000, 512, 32), (77, 256, 8), (2048, 1024, 64), (33, 128, 1),
                                       (1000, 4096, 32), (8200, 4096, 16), (33, 4096, 1)])   # d 4096: the pipelined kernel
def test_project_bf16(n_tok, d, r):
    announce("project bf16", n_tok, d, r)
    x = synth.bf16_round(synth.normal((n_tok, d), 1.0, 1, n_tok))
    ut = synth.bf16_round(synth.normal((r, d), 1.0 / np.sqrt(d), 2, d))
    p = torch.empty(n_tok, r, dtype=torch.bfloat16, device=dev())
    Z.project(t_bf16(x), t_bf16(ut), p)
    assert_bf16_close(host(p), olin.project(x, ut, "bf16"), what="project")


@pytest.mark.parametrize("n_tok,d,r", [(1000, 512, 32), (77, 256, 8), (2048, 1024, 64), (33, 128, 1),
                                       (4100, 4096, 32), (300, 14336, 32), (129, 5120, 64)])
def test_project_bf16_depth_split(n_tok, d, r):
    """The workspace form (depth split over workgroups, partials summed in a fixed order by
    a second pass) against the oracle, and the same bits on a second call."""
    announce("project bf16 split", n_tok, d, r)
    x = synth.bf16_round(synth.normal((n_tok, d), 1.0, 1, n_tok + d))
    ut = synth.bf16_round(synth.normal((r, d), 1.0 / np.sqrt(d), 2, d + r))
    ws = torch.empty(Z.project_workspace_bytes(n_tok, d, r), dtype=torch.uint8, device=dev())
    outs = []
    for _ in range(2):
        p = torch.empty(n_tok, r, dtype=torch.bfloat16, device=dev())
        Z.project(t_bf16(x), t_bf16(ut), p, ws)
        outs.append(host(p))
    assert_bf16_close(outs[0], olin.project(x, ut, "bf16"), what="project split")
    np.testing.assert_array_equal(outs[0], outs[1])


def test_project_f32():
    announce("project f32")
    x = synth.normal((300, 128), 1.0, 1, 1)
    ut = synth.normal((8, 128), 0.1, 2, 2)
    p = torch.empty(300, 8, dtype=torch.float32, device=dev())
    Z.project(t_f32(x), t_f32(ut), p)
    ref = olin.project(x, ut, "fp32")
    assert np.max(np.abs(host(p) - ref)) <= 1e-5 * np.sqrt(np.mean(ref**2))


# ------------------------------------------------------------------ fused +/- linear
def _layer_inputs(T, K, N, r, seed, bias=True, int4=False):
    x = synth.bf16_round(synth.normal((2, T, K), 1.0, seed, 1))
    x[1] = synth.bf16_round(x[0] + synth.normal((T, K), 0.05, seed, 9))  # halves differ slightly
    w = synth.bf16_round(synth.normal((N, K), 0.02, seed, 2))
    b = synth.bf16_round(synth.normal((N,), 0.1, seed, 3)) if bias else None
    ut = synth.bf16_round(np.linalg.qr(synth.normal((K, max(r, 1)), 1.0, seed, 4))[0][:, :r].T.astype(np.float32)) if r else None
    packed = scales = None
    if int4:
        packed, scales = synth.quantize_int4_g128(w)
    return x, w, b, ut, packed, scales


def _run_gpu_linear(x, w, b, ut, c_arena, off, r, eps, seed, step, T, K, N, flags=0, resid=None, packed=None,
                    scales=None, c_bf16=False, out_f32=False, precomputed=False):
    xt = t_bf16(x.reshape(2 * T, K))
    p = None
    if r:
        p = torch.empty(2 * T, r, dtype=torch.bfloat16, device=dev())
        Z.project(xt, t_bf16(ut), p)
    if packed is not None:
        layer = Z.Linear(t_u8(packed), K, N, r, t_bf16(ut) if r else None, off, t_bf16(b) if b is not None else None,
                         t_bf16(scales))
    else:
        layer = Z.Linear(t_bf16(w), K, N, r, t_bf16(ut) if r else None, off, t_bf16(b) if b is not None else None)
    arena = None
    if r:
        ct = t_bf16(c_arena) if c_bf16 else t_f32(c_arena)
        arena = Z.Arena(ct, torch.zeros_like(ct, dtype=torch.float32), torch.zeros_like(ct, dtype=torch.float32))
    if precomputed:
        ch = torch.empty(2 * N * r, dtype=torch.bfloat16, device=dev())
        Z.perturb_coeffs(arena, off, N * r, Z.Pert(seed, step, 0, eps), ch)
        layer.ch, layer.ch_stride = ch, N * r
    nout = N // 2 if flags & Z.EPI_SWIGLU else N
    y = torch.full((2 * T, nout), float("nan"), dtype=torch.float32 if out_f32 else torch.bfloat16, device=dev())
    rt = t_bf16(resid.reshape(2 * T, nout)) if resid is not None else None
    Z.linear_fwd_pm(layer, arena, xt, T, p, y, Z.Pert(seed, step, 0, eps), residual=rt, flags=flags)
    return host(y).reshape(2, T, nout)


def _oracle_linear(x, w, b, ut, c, off, r, eps, seed, step, flags=0, resid=None, round_out=True):
    z = olin.z_block(seed, step, 0, off, w.shape[0], r) if r else None
    outs = []
    for h, sign in ((0, 1), (1, -1)):
        y = olin.adapted_linear(x[h], w, b, ut, c, z, eps, sign, "bf16", round_out=False)
        if flags & Z.EPI_SWIGLU:
            n = w.shape[0]
            f = np.arange(n // 2)
            gi = (f // 16) * 32 + (f % 16)
            g, u = y[:, gi], y[:, gi + 16]
            y = g / (1.0 + np.exp(-g)) * u
        if resid is not None:
            y = y + resid[h]
        if flags & Z.EPI_RELU:
            y = np.maximum(y, 0.0)
        outs.append(rne_bf16(y.astype(np.float32)).astype(np.float64) if round_out else y)
    return np.stack(outs)


@pytest.mark.parametrize("T,K,N,r,off", [
    (300, 512, 336, 32, 0),
    (257, 256, 512, 8, 12),
    (64, 384, 256, 64, 6),
    (500, 256, 272, 80, 3),
    (1, 128, 16, 32, 0),
    (50, 64, 64, 16, 0),
    (300, 1024, 512, 32, 4),
    (513, 2048, 768, 64, 0),
])
def test_linear_pm_bf16(T, K, N, r, off):
    announce("linear_pm bf16", T, K, N, r, off)
    x, w, b, ut, _, _ = _layer_inputs(T, K, N, r, seed=T + K)
    k = off + N * r + 5
    c = synth.normal((k,), 0.01, 7, T)
    eps, seed, step = 1e-3, 1234, 3
    got = _run_gpu_linear(x, w, b, ut, c, off, r, eps, seed, step, T, K, N)
    ref = _oracle_linear(x, w, b, ut, c[off:off + N * r].reshape(N, r), off, r, eps, seed, step)
    assert_bf16_close(got, ref, what="linear_pm")


@pytest.mark.parametrize("c_bf16", [False, True])
@pytest.mark.parametrize("e0,n", [(0, 4096), (3, 1001), (44_040_192 - 777, 777), (8, 1000), (44_040_192 - 4096, 4096)])
def test_perturb_coeffs_bitwise(c_bf16, e0, n):
    """bf16(C + eps Z) and bf16(C - eps Z) over an unaligned arena range, bit for bit."""
    announce("perturb_coeffs", c_bf16, e0, n)
    k = e0 + n + 3
    c = synth.normal((k,), 0.01, 3, k % 1000)
    if c_bf16:
        c = synth.bf16_round(c)
    ct = t_bf16(c) if c_bf16 else t_f32(c)
    arena = Z.Arena(ct, torch.zeros(k, device=dev()), torch.zeros(k, device=dev()))
    out = torch.empty(2 * n, dtype=torch.bfloat16, device=dev())
    Z.perturb_coeffs(arena, e0, n, Z.Pert(77, 5, 0, 1e-3), out)
    z = orng.gauss_range(77, 5, 0, e0, n)
    got = host(out).reshape(2, n)
    for h, sign in ((0, 1), (1, -1)):
        want = olin.perturbed_coeffs(c[e0:e0 + n], z, 1e-3, sign, "bf16")
        np.testing.assert_array_equal(got[h], want)


@pytest.mark.parametrize("T,K,N,r,off,flags", [
    (300, 512, 336, 32, 0, 0),
    (64, 384, 256, 64, 8, 0),
    (513, 2048, 768, 40, 16, 0),
    (257, 256, 512, 32, 0, 1),
])
def test_linear_pm_precomputed_coefficients(T, K, N, r, off, flags):
    """Reading the precomputed C +/- eps Z gives the same bits as forming it in the kernel."""
    announce("linear_pm precomputed", T, K, N, r, off, flags)
    x, w, b, ut, _, _ = _layer_inputs(T, K, N, r, seed=T + 3 * K)
    c = synth.normal((off + N * r + 9,), 0.01, 8, T)
    eps, seed, step = 1e-3, 99, 4
    inline = _run_gpu_linear(x, w, b, ut, c, off, r, eps, seed, step, T, K, N, flags=flags)
    pre = _run_gpu_linear(x, w, b, ut, c, off, r, eps, seed, step, T, K, N, flags=flags, precomputed=True)
    np.testing.assert_array_equal(pre, inline)
    ref = _oracle_linear(x, w, b, ut, c[off:off + N * r].reshape(N, r), off, r, eps, seed, step, flags=flags)
    assert_bf16_close(pre, ref, what="linear_pm precomputed")


@pytest.mark.parametrize("T,K,N,r,off,flags", [
    (300, 512, 336, 1, 3, 0),
    (200, 256, 272, 3, 0, 0),
    (257, 512, 512, 128, 5, 0),
    (130, 1024, 256, 256, 0, 0),
    (200, 512, 512, 128, 0, 1),
    (64, 256, 256, 200, 7, 2),
])
def test_linear_pm_ranks(T, K, N, r, off, flags):
    """Ranks 1, 3, 128, 200 and 256, with C +/- eps Z formed in the kernel and read
    precomputed (the four-wave schedule covers every rank up to 256 from the precomputed
    array; the correction gathers element by element when r % 8 != 0)."""
    announce("linear_pm ranks", T, K, N, r, off, flags)
    x, w, b, ut, _, _ = _layer_inputs(T, K, N, r, seed=T + r)
    c = synth.normal((off + N * r + 3,), 0.01, 8, r)
    eps, seed, step = 1e-3, 42, 6
    ref = _oracle_linear(x, w, b, ut, c[off:off + N * r].reshape(N, r), off, r, eps, seed, step, flags=flags)
    inline = _run_gpu_linear(x, w, b, ut, c, off, r, eps, seed, step, T, K, N, flags=flags)
    assert_bf16_close(inline, ref, what=f"linear_pm r={r}")
    pre = _run_gpu_linear(x, w, b, ut, c, off, r, eps, seed, step, T, K, N, flags=flags, precomputed=True)
    assert_bf16_close(pre, ref, what=f"linear_pm precomputed r={r}")


def test_linear_pm_zero_coeffs_reproduce_base_and_determinism():
    announce("linear_pm base")
    T, K, N, r = 200, 256, 256, 32
    x, w, b, ut, _, _ = _layer_inputs(T, K, N, r, seed=5)
    x[1] = x[0]
    c = np.zeros(N * r, np.float32)
    got = _run_gpu_linear(x, w, b, ut, c, 0, r, 0.0, 1, 1, T, K, N)
    base = _run_gpu_linear(x, w, b, None, None, 0, 0, 0.0, 1, 1, T, K, N)
    np.testing.assert_array_equal(got[0], got[1])
    np.testing.assert_array_equal(got, base)
    ref = rne_bf16((x[0].astype(np.float64) @ w.astype(np.float64).T + b).astype(np.float32))
    assert_bf16_close(got[0], ref, what="base")
    again = _run_gpu_linear(x, w, b, ut, c, 0, r, 0.0, 1, 1, T, K, N)
    np.testing.assert_array_equal(got, again)


@pytest.mark.parametrize("flags", [Z.EPI_SWIGLU, Z.EPI_RELU])
def test_linear_pm_epilogues_with_residual(flags):
    announce("linear_pm epilogue", flags)
    T, K, N, r = 130, 256, 512, 32
    x, w, b, ut, _, _ = _layer_inputs(T, K, N, r, seed=11, bias=False)
    c = synth.normal((N * r,), 0.02, 8, 8)
    nout = N // 2 if flags & Z.EPI_SWIGLU else N
    resid = synth.bf16_round(synth.normal((2, T, nout), 0.5, 9, 9))
    got = _run_gpu_linear(x, w, None, ut, c, 0, r, 1e-2, 5, 2, T, K, N, flags=flags, resid=resid)
    ref = _oracle_linear(x, w, None, ut, c.reshape(N, r), 0, r, 1e-2, 5, 2, flags=flags, resid=resid)
    assert_bf16_close(got, ref, atol_rel_rms=2e-3, what="epilogue")


@pytest.mark.parametrize("c_bf16", [False, True])
def test_linear_pm_int4(c_bf16):
    announce("linear_pm int4", c_bf16)
    T, K, N, r = 200, 512, 384, 32
    x, w, b, ut, packed, scales = _layer_inputs(T, K, N, r, seed=21, bias=False, int4=True)
    c = synth.normal((N * r,), 0.02, 4, 4)
    if c_bf16:
        c = rne_bf16(c)
    got = _run_gpu_linear(x, w, None, ut, c, 0, r, 1e-3, 9, 4, T, K, N, packed=packed, scales=scales, c_bf16=c_bf16)
    wq = olin.dequant_int4(packed, scales)
    ref = _oracle_linear(x, wq, None, ut, c.reshape(N, r), 0, r, 1e-3, 9, 4)
    assert_bf16_close(got, ref, what="int4")


@pytest.mark.parametrize("T,K,N,r,flags,c_bf16", [
    (200, 512, 384, 32, 0, True),      # ragged tokens and features
    (300, 1024, 512, 64, 0, False),
    (257, 256, 512, 32, 1, True),      # SwiGLU epilogue
    (64, 4096, 256, 16, 2, True),      # ReLU epilogue, 32 groups per row
])
def test_linear_pm_int4_precomputed(T, K, N, r, flags, c_bf16):
    """INT4 weights with the precomputed C +/- eps Z (the 64-deep schedule converting the
    packed weights in LDS): against the oracle on the dequantised weights, and bitwise
    against the same layer in bf16 holding those dequantised weights."""
    announce("linear_pm int4 precomputed", T, K, N, r, flags, c_bf16)
    x, w, b, ut, packed, scales = _layer_inputs(T, K, N, r, seed=K + N, bias=True, int4=True)
    c = synth.normal((N * r,), 0.02, 4, 5)
    if c_bf16:
        c = rne_bf16(c)
    wq = olin.dequant_int4(packed, scales).astype(np.float32)
    got = _run_gpu_linear(x, w, b, ut, c, 0, r, 1e-3, 9, 4, T, K, N, flags=flags, packed=packed, scales=scales,
                          c_bf16=c_bf16, precomputed=True)
    same = _run_gpu_linear(x, wq, b, ut, c, 0, r, 1e-3, 9, 4, T, K, N, flags=flags, c_bf16=c_bf16, precomputed=True)
    np.testing.assert_array_equal(got, same)
    ref = _oracle_linear(x, wq, b, ut, c.reshape(N, r), 0, r, 1e-3, 9, 4, flags=flags)
    assert_bf16_close(got, ref, what="int4 precomputed")


@pytest.mark.parametrize("T,K,N,r,flags,out_f32", [
    (2050, 256, 4112, 32, 0, False),              # 306 tiles, four stages per tile
    (4100, 384, 4112, 8, Z.EPI_RELU, False),      # 578 tiles, ragged tokens and features, 3 groups
    (2050, 256, 4128, 16, Z.EPI_SWIGLU, False),   # last feature tile: one gate|up group
    (2050, 512, 4112, 0, 0, True),                # plain layer, fp32 out
])
def test_linear_pm_int4_persistent_tiles(T, K, N, r, flags, out_f32):
    """INT4 weights on more 256 x 256 tiles than the GPU has CUs: the packed-weight ring,
    the conversion into LDS and the x ring run from one tile into the next.  Bitwise equal
    to the bf16 layer holding the dequantised weights, and against the oracle."""
    announce("linear_pm int4 persistent", T, K, N, r, flags, out_f32)
    x, w, b, ut, packed, scales = _layer_inputs(T, K, N, max(r, 1), seed=T + K + N + 1, int4=True)
    if r == 0:
        ut = None
    nout = N // 2 if flags & Z.EPI_SWIGLU else N
    resid = None if out_f32 else synth.bf16_round(synth.normal((2, T, nout), 0.5, 13, T))
    c = synth.normal((N * max(r, 1),), 0.02, 13, 1)
    eps, seed, step = 1e-2, 19, 3
    wq = olin.dequant_int4(packed, scales).astype(np.float32)
    got = _run_gpu_linear(x, w, b, ut, c, 0, r, eps, seed, step, T, K, N, flags=flags, resid=resid,
                          out_f32=out_f32, precomputed=r > 0, packed=packed, scales=scales, c_bf16=True)
    same = _run_gpu_linear(x, wq, b, ut, c, 0, r, eps, seed, step, T, K, N, flags=flags, resid=resid,
                           out_f32=out_f32, precomputed=r > 0, c_bf16=True)
    np.testing.assert_array_equal(got, same)
    if r:
        ref = _oracle_linear(x, wq, b, ut, rne_bf16(c).reshape(N, r), 0, r, eps, seed, step, flags=flags,
                             resid=resid)
        assert_bf16_close(got, ref, atol_rel_rms=2e-3, what="int4 persistent tiles")
    else:
        ref = np.stack([x[h].astype(np.float64) @ wq.astype(np.float64).T + b for h in range(2)])
        assert np.max(np.abs(got - ref)) <= 1e-5 * np.sqrt(np.mean(ref**2)) * 10


def test_linear_pm_r0_fp32_logits():
    announce("linear_pm logits")
    T, K, N = 100, 256, 528
    x, w, _, _, _, _ = _layer_inputs(T, K, N, 0, seed=31, bias=False)
    got = _run_gpu_linear(x, w, None, None, None, 0, 0, 0.0, 1, 1, T, K, N, out_f32=True)
    ref = np.stack([x[h].astype(np.float64) @ w.astype(np.float64).T for h in range(2)])
    assert np.max(np.abs(got - ref)) <= 1e-5 * np.sqrt(np.mean(ref**2)) * 10


def test_linear_pm_fp32_mode():
    announce("linear_pm fp32")
    T, K, N, r = 70, 128, 96, 8
    x = synth.normal((2, T, K), 1.0, 3, 1)
    w = synth.normal((N, K), 0.02, 3, 2)
    b = synth.normal((N,), 0.1, 3, 3)
    ut = np.linalg.qr(synth.normal((K, r), 1.0, 3, 4))[0].T.astype(np.float32)
    c = synth.normal((N * r,), 0.01, 3, 5)
    xt = t_f32(x.reshape(2 * T, K))
    p = torch.empty(2 * T, r, dtype=torch.float32, device=dev())
    Z.project(xt, t_f32(ut), p)
    layer = Z.Linear(t_f32(w), K, N, r, t_f32(ut), 0, t_f32(b))
    ct = t_f32(c)
    arena = Z.Arena(ct, torch.zeros_like(ct), torch.zeros_like(ct))
    y = torch.empty(2 * T, N, dtype=torch.float32, device=dev())
    Z.linear_fwd_pm(layer, arena, xt, T, p, y, Z.Pert(8, 1, 0, 1e-3))
    ref = olin.adapted_linear_pm(x, w, b, ut, c.reshape(N, r), 1e-3, 8, 1, 0, 0, "fp32")
    got = host(y).reshape(2, T, N)
    assert np.max(np.abs(got - ref)) <= 1e-4 * np.max(np.abs(ref))
    # the +/- difference is the rank-r perturbation 2 eps (xU) Z^T (fp32 rounding aside)
    dz = got[0] - got[1] - ((x[0] - x[1]) @ w.T.astype(np.float64))
    zz = olin.z_block(8, 1, 0, 0, N, r).astype(np.float64)
    want = (x[0] @ ut.T.astype(np.float64)) @ (c.reshape(N, r) + 1e-3 * zz).T - \
           (x[1] @ ut.T.astype(np.float64)) @ (c.reshape(N, r) - 1e-3 * zz).T
    assert np.max(np.abs(dz - want)) <= 1e-4 * np.max(np.abs(ref))


# ------------------------------------------------------------------ losses
@pytest.mark.parametrize("bf16", [False, True])
def test_mse_pm(bf16):
    announce("mse", bf16)
    T, N = 1000, 300
    y = synth.normal((2, T, N), 1.0, 1, 1)
    t = synth.normal((T, N), 1.0, 1, 2)
    if bf16:
        y, t = synth.bf16_round(y), synth.bf16_round(t)
    mk = t_bf16 if bf16 else t_f32
    loss = torch.empty(2, dtype=torch.float32, device=dev())
    ws = torch.empty(Z.loss_workspace_bytes(), dtype=torch.uint8, device=dev())
    Z.mse_pm(mk(y.reshape(2 * T, N)), mk(t), loss, ws)
    got = host(loss)
    assert_rel_close(got, [oloss.mse(y[0], t), oloss.mse(y[1], t)], 1e-5, "mse")


def test_xent_pm():
    announce("xent")
    B, S, V = 3, 17, 1000
    lg = synth.normal((2, B, S, V), 2.0, 4, 1)
    tok = synth.uniform_tokens(B, S, V, 4, 2)
    loss = torch.empty(2, dtype=torch.float32, device=dev())
    ws = torch.empty(Z.loss_workspace_bytes(), dtype=torch.uint8, device=dev())
    Z.xent_pm(t_f32(lg.reshape(-1, V)), t_i32(tok), loss, ws)
    assert_rel_close(host(loss), [oloss.next_token_ce(lg[0], tok), oloss.next_token_ce(lg[1], tok)], 1e-5, "xent")
    # uniform logits give ln V
    Z.xent_pm(torch.zeros(2 * B * S, V, device=dev()), t_i32(tok), loss, ws)
    assert_rel_close(host(loss), [np.log(V)] * 2, 1e-6, "xent uniform")


# ------------------------------------------------------------------ basis (Algorithm 1)
def _gapped_x(t, d, r, seed):
    rr = np.random.default_rng(seed)
    q, _ = np.linalg.qr(rr.standard_normal((d, d)))
    sv = np.concatenate([np.linspace(30, 12, r), np.linspace(4, 0.5, d - r)])
    a, _ = np.linalg.qr(rr.standard_normal((t, d)))
    return ((a * sv) @ q.T * np.sqrt(t / d)).astype(np.float32)


@pytest.mark.parametrize("bf16", [False, True])
def test_gram(bf16):
    announce("gram", bf16)
    x = synth.normal((1000, 256), 1.0, 2, 2)
    if bf16:
        x = synth.bf16_round(x)
    g = torch.empty(256, 256, dtype=torch.float32, device=dev())
    Z.gram(t_bf16(x) if bf16 else t_f32(x), g)
    ref = obasis.gram(x)
    assert np.max(np.abs(host(g) - ref)) <= 1e-5 * np.max(np.abs(ref))
    Z.gram(t_bf16(x) if bf16 else t_f32(x), g, accumulate=True)
    assert np.max(np.abs(host(g) - 2 * ref)) <= 2e-5 * np.max(np.abs(ref))


@pytest.mark.parametrize("d,r,bf16", [(128, 8, False), (256, 8, True), (512, 32, True), (2048, 32, True),
                                       (1000, 16, False), (384, 100, False), (640, 64, True)])
def test_basis_init_matches_oracle(d, r, bf16):
    announce("basis", d, r, bf16)
    x = _gapped_x(2 * d, d, r, seed=d + r)
    if bf16:
        x = synth.bf16_round(x)
    u_ref, lam_ref = obasis.basis_init(x, r)
    ut = torch.empty(r, d, dtype=torch.bfloat16 if bf16 else torch.float32, device=dev())
    master = torch.empty(r, d, dtype=torch.float32, device=dev())
    ev = torch.empty(r, dtype=torch.float32, device=dev())
    rep = Z.eig_report_tensor(dev())
    ws = torch.empty(Z.basis_init_workspace_bytes(d, r), dtype=torch.uint8, device=dev())
    assert Z.basis_init(t_bf16(x) if bf16 else t_f32(x), r, ut, ws, ut_master=master, eigvals=ev, report=rep)
    um = host(master).T
    assert np.max(np.abs(um.T @ um - np.eye(r))) <= 1e-5
    assert obasis.overlap(um, u_ref) >= 1 - 1e-6
    assert_rel_close(host(ev), lam_ref, 1e-4, "eigenvalues")
    assert np.max(np.abs(um - u_ref)) <= 1e-4          # same canonical sign
    info = Z.read_eig_report(rep)
    print(f"[parity] basis d={d} r={r}: {info}", flush=True)
    assert info["resid"] <= 1e-5 and info["iters"] == 64 and info["converged"]
    _check_gap(info["gap"], _spectrum(x), r)
    if bf16:
        np.testing.assert_array_equal(host(ut), rne_bf16(host(master)))


def _spectrum(x):
    """Eigenvalues of X^T X, descending (fp64)."""
    return np.linalg.eigvalsh(x.astype(np.float64).T @ x.astype(np.float64))[::-1]


def _check_gap(gap, lam, r):
    """The reported gap is theta_r / theta_{r+1} of the block's Ritz values.  theta_r has
    converged with the basis; theta_{r+1} is a lower bound of lambda_{r+1} (Ritz values
    interlace) that converges only at the rate lambda_{r+p+1} / lambda_{r+1}, so the
    report bounds the true gap from above, and closely on these spectra."""
    true_gap = lam[r - 1] / lam[r]
    assert true_gap * (1 - 1e-4) <= gap <= 1.1 * true_gap, (gap, true_gap)


@pytest.mark.parametrize("d,r", [(512, 32), (640, 64), (384, 100)])
def test_basis_adaptive_stops_early(d, r):
    """Adaptive mode on a spectrum with a gap stops at a check well before max_iter, meets
    the tolerance, and reports a gap consistent with the spectrum's lambda_r / lambda_{r+1}."""
    announce("basis adaptive", d, r)
    x = _gapped_x(2 * d, d, r, seed=3 * d + r)
    u_ref, _ = obasis.basis_init(x, r)
    lam = _spectrum(x)
    ut = torch.empty(r, d, dtype=torch.float32, device=dev())
    rep = Z.eig_report_tensor(dev())
    opts = Z.EigOpts(0, 64, 7, 1e-4, 1, 4)
    ws = torch.empty(Z.basis_init_workspace_bytes(d, r, opts), dtype=torch.uint8, device=dev())
    assert Z.basis_init(t_f32(x), r, ut, ws, opts, report=rep)
    info = Z.read_eig_report(rep)
    print(f"[parity] adaptive d={d} r={r}: {info}", flush=True)
    assert info["converged"] and info["resid"] <= 1e-4
    assert info["iters"] % 4 == 0 and 4 <= info["iters"] < 64
    assert obasis.overlap(host(ut).T, u_ref) >= 1 - 1e-6
    _check_gap(info["gap"], lam, r)


def test_basis_noconverge_keeps_best_effort():
    """One iteration on a flat spectrum cannot meet tol = 1e-7: ZOACT_E_NOCONVERGE, the
    report says so, and the basis written is still orthonormal; a second call on the
    same workspace with a reachable bound converges."""
    announce("basis noconverge")
    d, r = 256, 16
    x = synth.normal((4 * d, d), 1.0, 4, 4)
    ut = torch.empty(r, d, dtype=torch.float32, device=dev())
    rep = Z.eig_report_tensor(dev())
    opts = Z.EigOpts(0, 1, 3, 1e-7, 0, 0)
    ws = torch.empty(Z.basis_init_workspace_bytes(d, r, opts), dtype=torch.uint8, device=dev())
    assert not Z.basis_init(t_f32(x), r, ut, ws, opts, report=rep)
    info = Z.read_eig_report(rep)
    print(f"[parity] noconverge: {info}", flush=True)
    assert not info["converged"] and info["resid"] > 1e-7 and info["iters"] == 1
    u = host(ut).T
    assert np.isfinite(u).all() and np.max(np.abs(u.T @ u - np.eye(r))) <= 1e-5
    # the same flat spectrum, iterated to a bound the fp32 Gram can support
    opts2 = Z.EigOpts(0, 512, 3, 1e-3, 1, 8)
    ok = Z.basis_init(t_f32(x), r, ut, ws, opts2, report=rep)
    info2 = Z.read_eig_report(rep)
    print(f"[parity] flat spectrum adaptive: {info2}", flush=True)
    assert ok and info2["converged"] and info2["resid"] <= 1e-3 and info2["iters"] <= 512


def _gapped_rows_x(t, d, r, seed):
    """t < d rows: X = A diag(sv) Q^T, A [t][t] and Q [d][t] orthonormal, a gap after r."""
    rr = np.random.default_rng(seed)
    q, _ = np.linalg.qr(rr.standard_normal((d, t)))
    a, _ = np.linalg.qr(rr.standard_normal((t, t)))
    sv = np.concatenate([np.linspace(30, 12, r), np.linspace(4, 0.5, t - r)])
    return ((a * sv) @ q.T).astype(np.float32)


@pytest.mark.parametrize("t,d,r", [(256, 512, 16), (512, 1024, 32), (1024, 4096, 32), (300, 1024, 32),
                                    (1000, 2048, 32), (200, 640, 64), (130, 4096, 8), (257, 1024, 16),
                                    (131, 768, 8)])
def test_basis_init_token_side_matches_oracle(t, d, r):
    """bf16 X with fewer rows than features: basis_init solves X X^T (t x t) and maps its
    Ritz vectors back with X^T.  Same bar as the Gram form against the oracle's top-r
    eigenvectors of X^T X, and the Gram form on the GPU (zoact_gram +
    zoact_basis_from_gram) agrees.  X X^T comes from the plain GEMM for t = 256, 512,
    1024 (multiples of 32) and from the triangle kernel for the ragged and odd t (300,
    1000, 200, 130, 257, 131); d = 640 is not a multiple of 128."""
    announce("basis token side", t, d, r)
    x = synth.bf16_round(_gapped_rows_x(t, d, r, seed=t + d + r))
    u_ref, lam_ref = obasis.basis_init(x, r)
    xt = t_bf16(x)
    outs = []
    for form in ("rows", "gram"):
        ut = torch.empty(r, d, dtype=torch.bfloat16, device=dev())
        master = torch.empty(r, d, dtype=torch.float32, device=dev())
        ev = torch.empty(r, dtype=torch.float32, device=dev())
        rep = Z.eig_report_tensor(dev())
        if form == "rows":
            ws = torch.empty(Z.basis_init_workspace_bytes(d, r), dtype=torch.uint8, device=dev())
            assert Z.basis_init(xt, r, ut, ws, ut_master=master, eigvals=ev, report=rep)
        else:
            g = torch.empty(d, d, dtype=torch.float32, device=dev())
            Z.gram(xt, g)
            ws = torch.empty(Z.basis_workspace_bytes(d, r), dtype=torch.uint8, device=dev())
            assert Z.basis_from_gram(g, r, ut, ws, ut_master=master, eigvals=ev, report=rep)
        um = host(master).T
        info = Z.read_eig_report(rep)
        print(f"[parity] basis {form} t={t} d={d} r={r}: {info}", flush=True)
        assert np.max(np.abs(um.T @ um - np.eye(r))) <= 1e-5
        assert obasis.overlap(um, u_ref) >= 1 - 1e-6
        assert_rel_close(host(ev), lam_ref, 1e-4, "eigenvalues")
        assert np.max(np.abs(um - u_ref)) <= 1e-4
        assert info["resid"] <= 1e-5 and info["iters"] == 64 and info["converged"]
        _check_gap(info["gap"], _spectrum(x), r)
        np.testing.assert_array_equal(host(ut), rne_bf16(host(master)))
        outs.append((um, host(ev)))
    assert np.max(np.abs(outs[0][0] - outs[1][0])) <= 1e-4
    assert_rel_close(outs[0][1], outs[1][1], 1e-5, "eigenvalues, token side vs Gram")


def test_basis_init_fp32_fewer_rows_takes_the_gram_form():
    """fp32 X with fewer rows than features keeps the Gram form (X^T X of rank t): same bar
    against the oracle, bitwise equal to zoact_gram + zoact_basis_from_gram on the GPU."""
    announce("basis fp32 fewer rows")
    t, d, r = 200, 512, 16
    x = _gapped_rows_x(t, d, r, seed=21)
    u_ref, lam_ref = obasis.basis_init(x, r)
    xt = t_f32(x)
    ut = torch.empty(r, d, dtype=torch.float32, device=dev())
    ev = torch.empty(r, dtype=torch.float32, device=dev())
    ws = torch.empty(Z.basis_init_workspace_bytes(d, r), dtype=torch.uint8, device=dev())
    assert Z.basis_init(xt, r, ut, ws, eigvals=ev)
    um = host(ut).T
    assert np.max(np.abs(um.T @ um - np.eye(r))) <= 1e-5
    assert np.max(np.abs(um - u_ref)) <= 1e-4
    assert_rel_close(host(ev), lam_ref, 1e-4, "eigenvalues")
    g = torch.empty(d, d, dtype=torch.float32, device=dev())
    Z.gram(xt, g)
    ut2 = torch.empty_like(ut)
    ws2 = torch.empty(Z.basis_workspace_bytes(d, r), dtype=torch.uint8, device=dev())
    assert Z.basis_from_gram(g, r, ut2, ws2)
    np.testing.assert_array_equal(host(ut), host(ut2))


def test_basis_token_side_adaptive_and_noconverge():
    """The token-side form under the adaptive mode stops early and meets tol; with one
    iteration and an unreachable tol it returns ZOACT_E_NOCONVERGE with the residual of
    the basis it wrote against X^T X, and that basis is still orthonormal."""
    announce("basis token side adaptive")
    t, d, r = 512, 2048, 32
    x = synth.bf16_round(_gapped_rows_x(t, d, r, seed=11))
    u_ref, _ = obasis.basis_init(x, r)
    xt = t_bf16(x)
    ut = torch.empty(r, d, dtype=torch.float32, device=dev())
    rep = Z.eig_report_tensor(dev())
    opts = Z.EigOpts(0, 64, 7, 1e-4, 1, 4)
    ws = torch.empty(Z.basis_init_workspace_bytes(d, r, opts), dtype=torch.uint8, device=dev())
    assert Z.basis_init(xt, r, ut, ws, opts, report=rep)
    info = Z.read_eig_report(rep)
    print(f"[parity] token side adaptive: {info}", flush=True)
    assert info["converged"] and info["resid"] <= 1e-4 and 4 <= info["iters"] < 64
    assert obasis.overlap(host(ut).T, u_ref) >= 1 - 1e-6
    # one iteration from the random start: the residual the report gives is the basis's
    # own against X^T X, recomputed here in fp64
    opts1 = Z.EigOpts(0, 1, 3, 1e-9, 0, 0)
    ev = torch.empty(r, dtype=torch.float32, device=dev())
    assert not Z.basis_init(xt, r, ut, ws, opts1, eigvals=ev, report=rep)
    info = Z.read_eig_report(rep)
    u = host(ut).T.astype(np.float64)
    assert np.isfinite(u).all() and np.max(np.abs(u.T @ u - np.eye(r))) <= 1e-5
    x64 = x.astype(np.float64)
    lam = host(ev).astype(np.float64)
    res = np.linalg.norm(x64.T @ (x64 @ u) - u * lam, axis=0).max() / lam[0]
    print(f"[parity] token side one iteration: {info}, fp64 residual {res:.3e}", flush=True)
    assert not info["converged"] and info["iters"] == 1
    assert abs(info["resid"] - res) <= 1e-3 * res + 1e-6


def test_basis_token_side_row_stride():
    """Token-side form on a column slice of a wider matrix (row stride > d: the triangle
    kernel forms X X^T) and on its contiguous copy (the GEMM): both meet the oracle's bar."""
    announce("basis token side row stride")
    t, d, r = 224, 512, 16
    x = synth.bf16_round(_gapped_rows_x(t, d, r, seed=5))
    wide = np.zeros((t, d + 64), dtype=np.float32)
    wide[:, 32:32 + d] = x
    u_ref, lam_ref = obasis.basis_init(x, r)
    view = t_bf16(wide)[:, 32:32 + d]
    assert view.stride(0) == d + 64
    for xx in (view, view.contiguous()):
        ut = torch.empty(r, d, dtype=torch.float32, device=dev())
        ev = torch.empty(r, dtype=torch.float32, device=dev())
        ws = torch.empty(Z.basis_init_workspace_bytes(d, r), dtype=torch.uint8, device=dev())
        assert Z.basis_init(xx, r, ut, ws, eigvals=ev)
        um = host(ut).T
        assert np.max(np.abs(um.T @ um - np.eye(r))) <= 1e-5
        assert np.max(np.abs(um - u_ref)) <= 1e-4
        assert_rel_close(host(ev), lam_ref, 1e-4, "eigenvalues")


def test_basis_init_row_stride():
    """x given as a column slice of a wider matrix (row stride > d) yields the same bits
    as the contiguous copy."""
    announce("basis row stride")
    d, r = 256, 16
    wide = synth.bf16_round(synth.normal((600, d + 64), 1.0, 5, 5))
    x_wide = t_bf16(wide)
    view = x_wide[:, 32:32 + d]
    assert view.stride(0) == d + 64
    outs = []
    for xx in (view, view.contiguous()):
        ut = torch.empty(r, d, dtype=torch.float32, device=dev())
        ws = torch.empty(Z.basis_init_workspace_bytes(d, r), dtype=torch.uint8, device=dev())
        Z.basis_init(xx, r, ut, ws)
        outs.append(host(ut))
    np.testing.assert_array_equal(outs[0], outs[1])


# ------------------------------------------------------------------ full single-layer workload, sampled
def test_single_layer_4096_sampled():
    """d_in = d_out = 4096, r = 32, 8192 tokens per half, planted low-rank x:
    sampled output rows of both halves against the oracle, plus the losses."""
    announce("single layer 4096 sampled")
    T, K, N, r = 8192, 4096, 4096, 32
    x, q = synth.planted_lowrank(T, K, seed=0)
    x = synth.bf16_round(x)
    w = synth.bf16_round(synth.normal((N, K), 0.02, 0, 2))
    ut = synth.bf16_round(q[:, :r].T.copy())
    c = synth.normal((N * r,), 0.01, 0, 3)
    eps, seed, step = 1e-3, 77, 1
    xt = t_bf16(np.stack([x, x]).reshape(2 * T, K))
    p = torch.empty(2 * T, r, dtype=torch.bfloat16, device=dev())
    Z.project(xt, t_bf16(ut), p)
    layer = Z.Linear(t_bf16(w), K, N, r, t_bf16(ut), 0)
    ct = t_f32(c)
    arena = Z.Arena(ct, torch.zeros_like(ct), torch.zeros_like(ct))
    y = torch.empty(2 * T, N, dtype=torch.bfloat16, device=dev())
    Z.linear_fwd_pm(layer, arena, xt, T, p, y, Z.Pert(seed, step, 0, eps))
    rows = np.random.default_rng(0).choice(T, 24, replace=False)
    rows = np.concatenate([rows, [0, T - 1]])
    yh = host(y).reshape(2, T, N)
    xs = x[rows]
    ref = _oracle_linear(np.stack([xs, xs]), w, None, ut, c.reshape(N, r), 0, r, eps, seed, step)
    assert_bf16_close(yh[:, rows], ref, what="single layer sampled")
    # P rows as well
    assert_bf16_close(host(p)[rows], olin.project(xs, ut, "bf16"), what="P sampled")
    # the fused regression loss at full size: the same y, summed in the epilogue
    tgt = t_bf16(synth.normal((T, N), 1.0, 0, 5))
    lpm = torch.zeros(2, dtype=torch.float32, device=dev())
    Z.mse_pm(y, tgt, lpm, torch.empty(Z.loss_workspace_bytes(), dtype=torch.uint8, device=dev()))
    fused = torch.full((2,), float("nan"), dtype=torch.float32, device=dev())
    ws = torch.empty(Z.linear_mse_workspace_bytes(T, N), dtype=torch.uint8, device=dev())
    Z.linear_mse(layer, arena, xt, T, p, Z.Pert(seed, step, 0, eps), tgt, fused, ws)
    np.testing.assert_allclose(host(fused), host(lpm), rtol=2e-6)
    # and with the coefficients precomputed: the 64-deep persistent schedule (1024 tiles,
    # four per workgroup), stored and fused, in the launch configuration the benchmark times
    ch = torch.empty(2 * N * r, dtype=torch.bfloat16, device=dev())
    Z.perturb_coeffs(arena, 0, N * r, Z.Pert(seed, step, 0, eps), ch)
    layer.ch, layer.ch_stride = ch, N * r
    y2 = torch.empty_like(y)
    Z.linear_fwd_pm(layer, arena, xt, T, p, y2, Z.Pert(seed, step, 0, eps))
    assert_bf16_close(host(y2).reshape(2, T, N)[:, rows], ref, what="single layer sampled, 64-deep")
    fused2 = torch.full((2,), float("nan"), dtype=torch.float32, device=dev())
    Z.linear_mse(layer, arena, xt, T, p, Z.Pert(seed, step, 0, eps), tgt, fused2, ws)
    lpm2 = torch.zeros(2, dtype=torch.float32, device=dev())
    Z.mse_pm(y2, tgt, lpm2, torch.empty(Z.loss_workspace_bytes(), dtype=torch.uint8, device=dev()))
    np.testing.assert_allclose(host(fused2), host(lpm2), rtol=2e-6)


# ------------------------------------------------------------------ fused regression loss
@pytest.mark.parametrize("d_out,d_in", [(384, 512), (16, 128), (1000, 4096)])
def test_dequant_int4_bitwise(d_out, d_in):
    """bf16(q * s) of packed INT4 weights, bit for bit against the oracle's dequantisation,
    and the layer on the dequantised weights equals the in-register INT4 layer."""
    announce("dequant int4", d_out, d_in)
    w = synth.bf16_round(synth.normal((d_out, d_in), 0.02, d_out, d_in))
    packed, scales = synth.quantize_int4_g128(w)
    out = torch.empty(d_out, d_in, dtype=torch.bfloat16, device=dev())
    Z.dequant_int4(t_u8(packed), t_bf16(scales), out)
    want = olin.dequant_int4(packed, scales)
    np.testing.assert_array_equal(host(out).astype(np.float32).view(np.uint32),
                                  want.astype(np.float32).view(np.uint32))


@pytest.mark.parametrize("T,K,N,r,mode", [
    (300, 512, 336, 32, "bf16"),       # ragged tokens and features
    (257, 256, 512, 128, "bf16-pre"),  # precomputed coefficients, r > 64
    (200, 512, 384, 32, "int4"),
    (64, 1024, 256, 0, "bf16"),        # plain layer
])
def test_linear_mse_fused(T, K, N, r, mode):
    """The fused loss equals the stored-output path (linear + zoact_mse_pm) up to summation
    order, and the oracle's MSE of its own bf16 outputs within the bf16 bar."""
    announce("linear mse fused", T, K, N, r, mode)
    x, w, b, ut, packed, scales = _layer_inputs(T, K, N, max(r, 1), seed=T + N, int4=(mode == "int4"))
    if r == 0:
        ut = None
    c = synth.normal((N * max(r, 1),), 0.02, 3, 3)
    eps, seed, step = 1e-3, 5, 2
    xt = t_bf16(x.reshape(2 * T, K))
    p = None
    if r:
        p = torch.empty(2 * T, r, dtype=torch.bfloat16, device=dev())
        Z.project(xt, t_bf16(ut), p)
    if mode == "int4":
        layer = Z.Linear(t_u8(packed), K, N, r, t_bf16(ut), 0, t_bf16(b), t_bf16(scales))
    else:
        layer = Z.Linear(t_bf16(w), K, N, r, t_bf16(ut) if r else None, 0, t_bf16(b))
    arena = Z.Arena(t_f32(c), torch.zeros(c.size, device=dev()), torch.zeros(c.size, device=dev())) if r else None
    pert = Z.Pert(seed, step, 0, eps)
    if mode in ("int4", "bf16-pre"):
        ch = torch.empty(2 * N * r, dtype=torch.bfloat16, device=dev())
        Z.perturb_coeffs(arena, 0, N * r, pert, ch)
        layer.ch, layer.ch_stride = ch, N * r
    tgt_np = synth.bf16_round(synth.normal((T, N), 1.0, 4, 4))
    tgt = t_bf16(tgt_np)
    y = torch.empty(2 * T, N, dtype=torch.bfloat16, device=dev())
    Z.linear_fwd_pm(layer, arena, xt, T, p, y, pert)
    lpm = torch.zeros(2, dtype=torch.float32, device=dev())
    Z.mse_pm(y, tgt, lpm, torch.empty(Z.loss_workspace_bytes(), dtype=torch.uint8, device=dev()))
    fused = torch.full((2,), float("nan"), dtype=torch.float32, device=dev())
    ws = torch.empty(Z.linear_mse_workspace_bytes(T, N), dtype=torch.uint8, device=dev())
    Z.linear_mse(layer, arena, xt, T, p, pert, tgt, fused, ws)
    np.testing.assert_allclose(host(fused), host(lpm), rtol=2e-6)
    wq = olin.dequant_int4(packed, scales) if mode == "int4" else w
    if r:
        ref = _oracle_linear(x, wq, b, ut, c.reshape(N, r), 0, r, eps, seed, step)
    else:
        ref = np.stack([rne_bf16((x[h].astype(np.float64) @ wq.astype(np.float64).T + b).astype(np.float32))
                        for h in range(2)]).astype(np.float64)
    want = [oloss.mse(ref[h], tgt_np) for h in range(2)]
    assert_rel_close(host(fused), want, 1e-3, "fused mse vs oracle")


# ------------------------------------------------------------------ more tiles than workgroups
@pytest.mark.parametrize("T,K,N,r,flags,out_f32", [
    (2050, 128, 4112, 32, 0, False),              # 306 tiles, two stages per tile
    (4100, 192, 4112, 8, Z.EPI_RELU, False),      # 578 tiles, ragged tokens and features
    (2050, 256, 4128, 16, Z.EPI_SWIGLU, False),   # last feature tile: one gate|up group
    (2050, 128, 4112, 0, 0, True),                # plain layer, fp32 out
])
def test_linear_pm_persistent_tiles(T, K, N, r, flags, out_f32):
    """More 256 x 256 tiles than the GPU has CUs: each workgroup of the 64-deep schedule
    walks several tiles with its stage ring running from one tile into the next.  Bias and
    residual on, against the oracle element by element."""
    announce("linear_pm persistent", T, K, N, r, flags, out_f32)
    x, w, b, ut, _, _ = _layer_inputs(T, K, N, r, seed=T + K + N)
    nout = N // 2 if flags & Z.EPI_SWIGLU else N
    resid = None if out_f32 else synth.bf16_round(synth.normal((2, T, nout), 0.5, 12, T))
    c = synth.normal((N * max(r, 1),), 0.02, 12, 1)
    eps, seed, step = 1e-2, 17, 3
    got = _run_gpu_linear(x, w, b, ut, c, 0, r, eps, seed, step, T, K, N, flags=flags, resid=resid,
                          out_f32=out_f32, precomputed=r > 0)
    if r:
        ref = _oracle_linear(x, w, b, ut, c.reshape(N, r), 0, r, eps, seed, step, flags=flags, resid=resid)
        assert_bf16_close(got, ref, atol_rel_rms=2e-3, what="persistent tiles")
    else:
        ref = np.stack([x[h].astype(np.float64) @ w.astype(np.float64).T + b for h in range(2)])
        assert np.max(np.abs(got - ref)) <= 1e-5 * np.sqrt(np.mean(ref**2)) * 10


def test_linear_mse_fused_persistent_tiles():
    """The fused regression loss over 578 tiles (ragged both ways) with the precomputed
    coefficients: equal to the stored-output path up to summation order, and to the
    oracle's MSE within the bf16 bar."""
    T, K, N, r = 4100, 192, 4112, 32
    announce("linear mse persistent", T, K, N, r)
    x, w, b, ut, _, _ = _layer_inputs(T, K, N, r, seed=7)
    c = synth.normal((N * r,), 0.02, 7, 7)
    eps, seed, step = 1e-3, 8, 2
    xt = t_bf16(x.reshape(2 * T, K))
    p = torch.empty(2 * T, r, dtype=torch.bfloat16, device=dev())
    Z.project(xt, t_bf16(ut), p)
    layer = Z.Linear(t_bf16(w), K, N, r, t_bf16(ut), 0, t_bf16(b))
    arena = Z.Arena(t_f32(c), torch.zeros(c.size, device=dev()), torch.zeros(c.size, device=dev()))
    pert = Z.Pert(seed, step, 0, eps)
    ch = torch.empty(2 * N * r, dtype=torch.bfloat16, device=dev())
    Z.perturb_coeffs(arena, 0, N * r, pert, ch)
    layer.ch, layer.ch_stride = ch, N * r
    tgt_np = synth.bf16_round(synth.normal((T, N), 1.0, 7, 8))
    tgt = t_bf16(tgt_np)
    y = torch.empty(2 * T, N, dtype=torch.bfloat16, device=dev())
    Z.linear_fwd_pm(layer, arena, xt, T, p, y, pert)
    lpm = torch.zeros(2, dtype=torch.float32, device=dev())
    Z.mse_pm(y, tgt, lpm, torch.empty(Z.loss_workspace_bytes(), dtype=torch.uint8, device=dev()))
    fused = torch.full((2,), float("nan"), dtype=torch.float32, device=dev())
    ws = torch.empty(Z.linear_mse_workspace_bytes(T, N), dtype=torch.uint8, device=dev())
    Z.linear_mse(layer, arena, xt, T, p, pert, tgt, fused, ws)
    np.testing.assert_allclose(host(fused), host(lpm), rtol=2e-6)
    ref = _oracle_linear(x, w, b, ut, c.reshape(N, r), 0, r, eps, seed, step)
    assert_rel_close(host(fused), [oloss.mse(ref[h], tgt_np) for h in range(2)], 1e-3, "persistent mse vs oracle")


@pytest.mark.parametrize("B,S,K,V", [(8, 130, 256, 8000), (3, 7, 128, 50272)])
def test_linear_xent_fused_vs_oracle(B, S, K, V):
    """The LM head with the cross entropy in its epilogue against the oracle's next-token
    cross entropy of the float64 logits: 320 tiles with a ragged last vocabulary tile, and
    a short batch over the OPT vocabulary (197 feature tiles, 50272 = 196 x 256 + 96)."""
    announce("linear xent fused", B, S, K, V)
    T = B * S
    x, w, b, _, _, _ = _layer_inputs(T, K, V, 0, seed=B + S + V, bias=False)
    tok = synth.uniform_tokens(B, S, V, 5, B)
    layer = Z.Linear(t_bf16(w), K, V, 0, None, 0)
    loss = torch.full((2,), float("nan"), dtype=torch.float32, device=dev())
    ws = torch.empty(Z.linear_xent_workspace_bytes(T, V), dtype=torch.uint8, device=dev())
    Z.linear_xent(layer, None, t_bf16(x.reshape(2 * T, K)), t_i32(tok), None, Z.Pert(1, 1, 0, 0.0), loss, ws)
    want = [oloss.next_token_ce((x[h].astype(np.float64) @ w.astype(np.float64).T).reshape(B, S, V), tok)
            for h in range(2)]
    # fp32 logits (summation order) and fp32 exp/log in the per-block partials
    assert_rel_close(host(loss), want, 1e-5, "fused xent vs oracle")


# ------------------------------------------------------------------ shared input (ZOACT_SHARED_X)
def _shared_case(T, K, N, r, seed, bias=True):
    x, w, b, ut, _, _ = _layer_inputs(T, K, N, r, seed=seed, bias=bias)
    x[1] = x[0]   # both halves read the same input
    layer = Z.Linear(t_bf16(w), K, N, r, t_bf16(ut), 0, t_bf16(b) if b is not None else None)
    c = synth.normal((N * r,), 0.02, seed, 5)
    arena = Z.Arena(t_f32(c), torch.zeros(c.size, device=dev()), torch.zeros(c.size, device=dev()))
    pert = Z.Pert(seed, 2, 0, 1e-2)
    ch = torch.empty(2 * N * r, dtype=torch.bfloat16, device=dev())
    Z.perturb_coeffs(arena, 0, N * r, pert, ch)
    layer.ch, layer.ch_stride = ch, N * r
    x1 = t_bf16(x[0])                         # one copy: [T][K]
    x2 = t_bf16(x.reshape(2 * T, K))          # the stacked form: [2][T][K]
    p1 = torch.empty(T, r, dtype=torch.bfloat16, device=dev())
    Z.project(x1, t_bf16(ut), p1)
    p2 = torch.cat([p1, p1])
    return x, w, b, ut, c, layer, arena, pert, x1, x2, p1, p2


@pytest.mark.parametrize("T,K,N,r,flags,out_f32,resid", [
    (300, 512, 336, 32, 0, False, False),          # ragged tokens and features
    (2050, 128, 4112, 16, 0, False, True),         # 153 tiles, two stages, residual
    (4100, 192, 4112, 8, Z.EPI_RELU, False, True),  # 289 tiles: some workgroups take two
    (257, 256, 512, 32, 0, True, False),           # fp32 out
])
def test_linear_pm_shared_x_bitwise(T, K, N, r, flags, out_f32, resid):
    """The base x W^T formed once for both halves gives the same bits as the stacked form
    with the input given twice, for both halves; and the oracle's outputs within the bar."""
    announce("linear_pm shared x", T, K, N, r, flags, out_f32, resid)
    x, w, b, ut, c, layer, arena, pert, x1, x2, p1, p2 = _shared_case(T, K, N, r, T + N + r)
    dt = torch.float32 if out_f32 else torch.bfloat16
    res = t_bf16(synth.bf16_round(synth.normal((2 * T, N), 0.5, 3, T))) if resid else None
    ys = torch.full((2 * T, N), float("nan"), dtype=dt, device=dev())
    yt = torch.full((2 * T, N), float("nan"), dtype=dt, device=dev())
    Z.linear_fwd_pm(layer, arena, x1, T, p1, ys, pert, residual=res, flags=flags | Z.SHARED_X)
    Z.linear_fwd_pm(layer, arena, x2, T, p2, yt, pert, residual=res, flags=flags)
    bits = torch.int32 if out_f32 else torch.int16
    assert torch.equal(ys.view(bits), yt.view(bits)), "shared x differs from the stacked form"
    gs = host(ys)
    if not out_f32 and not resid and flags == 0:
        ref = _oracle_linear(x, w, b, ut, c.reshape(N, r), 0, r, 1e-2, T + N + r, 2)
        assert_bf16_close(gs.reshape(2, T, N), ref, what="shared x vs oracle")


@pytest.mark.parametrize("T,K,dq,dk,dv,r,flags,int4", [
    (1000, 512, 512, 256, 256, 32, 0, False),            # ragged tokens, k between q and v
    (300, 256, 256, 512, 256, 64, Z.EPI_RELU, False),     # k wider than q and v, ReLU
    (4100, 128, 768, 256, 512, 8, 0, False),              # ragged last token tile, 204 tiles
    (1000, 512, 512, 256, 256, 32, 0, True),              # INT4 weights (converted in LDS)
    (300, 256, 256, 512, 256, 64, Z.EPI_RELU, True),
])
def test_linear_plain_range_equals_two_calls(T, K, dq, dk, dv, r, flags, int4):
    """q|k|v in one call with k as the plain feature range (no correction, no coefficient
    rows) gives the same bits as q|v adapted and k plain in two calls."""
    announce("linear plain range", T, K, dq, dk, dv, r, flags, int4)
    N = dq + dk + dv
    x, w, b, ut, packed, scales = _layer_inputs(T, K, N, r, seed=T + N + r, bias=True, int4=int4)

    def weights(rows):   # the layer's weights for a row selection, bf16 or packed INT4 with scales
        if int4:
            return dict(w=t_u8(np.ascontiguousarray(packed[rows])), w_scales=t_bf16(np.ascontiguousarray(scales[rows])))
        return dict(w=t_bf16(np.ascontiguousarray(w[rows])))
    rows = dq + dv
    c = synth.normal((rows * r,), 0.02, N + r, 5)
    arena = Z.Arena(t_f32(c), torch.zeros(c.size, device=dev()), torch.zeros(c.size, device=dev()))
    pert = Z.Pert(N + r, 3, 0, 1e-2)
    ch = torch.empty(2 * rows * r, dtype=torch.bfloat16, device=dev())
    Z.perturb_coeffs(arena, 0, rows * r, pert, ch)
    xt = t_bf16(x.reshape(2 * T, K))
    p = torch.empty(2 * T, r, dtype=torch.bfloat16, device=dev())
    Z.project(xt, t_bf16(ut), p)
    fw = weights(np.s_[:])
    fused = Z.Linear(fw["w"], K, N, r, t_bf16(ut), 0, t_bf16(b), fw.get("w_scales"), ch=ch, ch_stride=rows * r,
                     plain=(dq, dq + dk))
    yf = torch.full((2 * T, N), float("nan"), dtype=torch.bfloat16, device=dev())
    Z.linear_fwd_pm(fused, arena, xt, T, p, yf, pert, flags=flags)
    sel = np.r_[0:dq, dq + dk:N]
    qw, kw = weights(sel), weights(np.s_[dq:dq + dk])
    qv = Z.Linear(qw["w"], K, rows, r, t_bf16(ut), 0, t_bf16(np.ascontiguousarray(b[sel])), qw.get("w_scales"),
                  ch=ch, ch_stride=rows * r)
    kk = Z.Linear(kw["w"], K, dk, 0, None, 0, t_bf16(np.ascontiguousarray(b[dq:dq + dk])), kw.get("w_scales"))
    yqv = torch.empty(2 * T, rows, dtype=torch.bfloat16, device=dev())
    yk = torch.empty(2 * T, dk, dtype=torch.bfloat16, device=dev())
    Z.linear_fwd_pm(qv, arena, xt, T, p, yqv, pert, flags=flags)
    Z.linear_fwd_pm(kk, None, xt, T, None, yk, pert, flags=flags)
    want = torch.cat([yqv[:, :dq], yk, yqv[:, dq:]], dim=1)
    assert torch.equal(yf.view(torch.int16), want.view(torch.int16)), "fused q|k|v differs from the two calls"


@pytest.mark.parametrize("flags,resid,bias", [(0, True, True), (Z.EPI_RELU, False, False)])
def test_linear_split_tail(flags, resid, bias):
    """640 tiles (4096 tokens per half, 5120 features) on a 256-CU grid leave a last round
    of 128 tiles; with a workspace their depth is split over two workgroups.  Against the
    same call without the workspace (the same products, other summation order) and the
    oracle on sampled rows; with equal halves and eps = 0 both halves stay bitwise equal."""
    T, K, N, r = 4096, 512, 5120, 32
    announce("linear split tail", T, K, N, r, flags, resid, bias)
    x, w, b, ut, _, _ = _layer_inputs(T, K, N, r, seed=11, bias=bias)
    x[1] = x[0]
    c = synth.normal((N * r,), 0.02, 11, 5)
    arena = Z.Arena(t_f32(c), torch.zeros(c.size, device=dev()), torch.zeros(c.size, device=dev()))
    pert = Z.Pert(11, 2, 0, 0.0)
    ch = torch.empty(2 * N * r, dtype=torch.bfloat16, device=dev())
    Z.perturb_coeffs(arena, 0, N * r, pert, ch)
    xt = t_bf16(x.reshape(2 * T, K))
    p = torch.empty(2 * T, r, dtype=torch.bfloat16, device=dev())
    Z.project(xt, t_bf16(ut), p)
    res_np = synth.bf16_round(synth.normal((T, N), 0.5, 11, 7)) if resid else None
    res = t_bf16(np.concatenate([res_np, res_np])) if resid else None
    ws = torch.empty(Z.linear_workspace_bytes(), dtype=torch.uint8, device=dev())
    outs = []
    for use_ws in (True, False):
        lay = Z.Linear(t_bf16(w), K, N, r, t_bf16(ut), 0, t_bf16(b) if bias else None, ch=ch, ch_stride=N * r,
                       ws=ws if use_ws else None)
        y = torch.full((2 * T, N), float("nan"), dtype=torch.bfloat16, device=dev())
        Z.linear_fwd_pm(lay, arena, xt, T, p, y, pert, residual=res, flags=flags)
        outs.append(host(y))
    ys, yn = outs
    np.testing.assert_array_equal(ys[:T], ys[T:])   # the pair's halves
    assert_bf16_close(ys, yn, what="split tail vs whole depth")
    rows = np.r_[0:8, 2040:2048, T - 8:T]
    xr = x[0][rows].astype(np.float64)
    pr = synth.bf16_round((xr @ ut.astype(np.float64).T).astype(np.float32)).astype(np.float64)   # P as stored
    cm = synth.bf16_round(c.astype(np.float32)).reshape(N, r).astype(np.float64)                # bf16(C + 0 Z)
    want = xr @ w.astype(np.float64).T + pr @ cm.T
    if bias:
        want = want + b.astype(np.float64)
    if resid:
        want = want + res_np[rows].astype(np.float64)
    if flags == Z.EPI_RELU:
        want = np.maximum(want, 0.0)
    assert_bf16_close(ys[rows], want, what="split tail vs oracle")


def test_linear_plain_range_rejected_where_not_covered():
    """A plain range off the 256-feature tiles, or with fp32 activations: an error, not a
    silent fallback."""
    T, K, N, r = 64, 128, 768, 8
    x, w, b, ut, _, _ = _layer_inputs(T, K, N, r, seed=7, bias=False)
    c = synth.normal((512 * r,), 0.02, 7, 5)
    arena = Z.Arena(t_f32(c), torch.zeros(c.size, device=dev()), torch.zeros(c.size, device=dev()))
    pert = Z.Pert(7, 1, 0, 1e-2)
    ch = torch.empty(2 * 512 * r, dtype=torch.bfloat16, device=dev())
    Z.perturb_coeffs(arena, 0, 512 * r, pert, ch)
    xt = t_bf16(x.reshape(2 * T, K))
    p = torch.zeros(2 * T, r, dtype=torch.bfloat16, device=dev())
    y = torch.empty(2 * T, N, dtype=torch.bfloat16, device=dev())
    bad = Z.Linear(t_bf16(w), K, N, r, t_bf16(ut), 0, None, ch=ch, ch_stride=512 * r, plain=(128, 384))
    with pytest.raises(Z.ZoactError):
        Z.linear_fwd_pm(bad, arena, xt, T, p, y, pert)
    # INT4 weights with a depth the 64-deep INT4 schedule does not cover (K < 256)
    packed, scales = synth.quantize_int4_g128(w)
    bad4 = Z.Linear(t_u8(packed), K, N, r, t_bf16(ut), 0, None, t_bf16(scales), ch=ch, ch_stride=512 * r,
                    plain=(256, 512))
    with pytest.raises(Z.ZoactError):
        Z.linear_fwd_pm(bad4, arena, xt, T, p, y, pert)


def test_linear_mse_shared_x_equals_stacked():
    """The fused regression loss with the shared input: the same per-wave partial sums as the
    stacked form, so the same losses bit for bit (1024 tiles in the stacked form, 512 shared)."""
    T, K, N, r = 8192, 256, 4096, 32
    announce("linear mse shared x", T, K, N, r)
    x, w, b, ut, c, layer, arena, pert, x1, x2, p1, p2 = _shared_case(T, K, N, r, 11)
    tgt = t_bf16(synth.bf16_round(synth.normal((T, N), 1.0, 11, 6)))
    ws = torch.empty(Z.linear_mse_workspace_bytes(T, N), dtype=torch.uint8, device=dev())
    ls = torch.full((2,), float("nan"), dtype=torch.float32, device=dev())
    lt = torch.full((2,), float("nan"), dtype=torch.float32, device=dev())
    Z.linear_mse(layer, arena, x1, T, p1, pert, tgt, ls, ws, flags=Z.SHARED_X)
    Z.linear_mse(layer, arena, x2, T, p2, pert, tgt, lt, ws)
    np.testing.assert_array_equal(host(ls), host(lt))
    assert host(ls)[0] != host(ls)[1]


def test_shared_x_unsupported_cases():
    """Outside the shared form's coverage the call fails with ZOACT_E_UNSUPPORTED (no
    silent fallback): r = 40 (two slices), r = 4 (not a multiple of 8), SwiGLU, no C_h."""
    T, K, N = 64, 128, 256
    x = t_bf16(synth.bf16_round(synth.normal((T, K), 1.0, 1, 1)))
    w = t_bf16(synth.bf16_round(synth.normal((N, K), 0.02, 1, 2)))
    y = torch.empty(2 * T, N, dtype=torch.bfloat16, device=dev())
    for r, flags, with_ch in ((40, 0, True), (4, 0, True), (32, Z.EPI_SWIGLU, True), (32, 0, False)):
        ut = t_bf16(synth.normal((r, K), 0.1, 1, 3))
        c = torch.zeros(N * r, device=dev())
        arena = Z.Arena(c, torch.zeros_like(c), torch.zeros_like(c))
        layer = Z.Linear(w, K, N, r, ut, 0)
        if with_ch:
            ch = torch.zeros(2 * N * r, dtype=torch.bfloat16, device=dev())
            layer.ch, layer.ch_stride = ch, N * r
        p = torch.zeros(T, r, dtype=torch.bfloat16, device=dev())
        yy = torch.empty(2 * T, N // 2 if flags else N, dtype=torch.bfloat16, device=dev())
        with pytest.raises(Z.ZoactError) as e:
            Z.linear_fwd_pm(layer, arena, x, T, p, yy, Z.Pert(1, 1, 0, 1e-3), flags=flags | Z.SHARED_X)
        assert e.value.status == Z.E_UNSUPPORTED, (r, flags, with_ch, e.value)
    del y
