"""Helpers for the GPU parity tests (device transfer and tolerance checks)."""
import sys

import numpy as np
import torch


def dev():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a visible MI355X")
    return torch.device("cuda:0")


def announce(*what):
    """Name the case before a GPU step, flushed, so a crash log says what ran."""
    print("[gpu-case]", *what, flush=True)
    sys.stdout.flush()


def t_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev())


def t_bf16(a):
    """Device bf16 tensor from float32 values (exact when they are bf16 values)."""
    return t_f32(a).to(torch.bfloat16)


def t_u8(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).to(dev())


def t_i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev())


def host(t):
    torch.cuda.synchronize()
    return t.detach().float().cpu().numpy().astype(np.float64)


def assert_bf16_close(got, ref, atol_rel_rms=1e-3, what=""):
    """Element-wise: |got - ref| <= 2^-7 |ref| + atol, atol = atol_rel_rms * rms(ref).

    2^-7 |ref| is at least one bf16 ulp of ref: the two sides round fp32 (GPU) and
    float64 (oracle) accumulations of the same bf16 products, which can land on
    either side of a rounding boundary; the atol term covers the fp32 summation.
    """
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    tol = 2.0 ** -7 * np.abs(ref) + atol_rel_rms * rms + 1e-30
    bad = np.abs(got - ref) > tol
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} outside tolerance; first at {tuple(i)}: "
                             f"got {got[tuple(i)]!r} ref {ref[tuple(i)]!r}")


def assert_rel_close(got, ref, rel, what=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = np.max(np.abs(got - ref) / np.maximum(np.abs(ref), 1e-30))
    assert err <= rel, f"{what}: max relative error {err:.3e} > {rel:.1e}"
