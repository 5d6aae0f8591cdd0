"""The no-allocation form of the fused regression-loss linear (zoact_linear_mse_pair_noalloc):
its losses equal those of zoact_linear_mse_pair with a caller workspace, bit for bit, on two
calls in a row (the second on a smaller problem, so stale partial sums of the first would
show), in the stacked and the shared-input form; a shape beyond the static scratch is
rejected before anything runs."""
import numpy as np
import pytest
import torch

import synth
from paper_2607_01125_amd import zoact as Z

from gpu_helpers import announce, dev, host, t_bf16, t_f32

pytestmark = pytest.mark.gpu


def _case(T, K, N, r, seed):
    x, q = synth.planted_lowrank(T, K, n_dirs=min(64, K), seed=seed)
    x = synth.bf16_round(x)
    w = synth.bf16_round(synth.normal((N, K), 0.02, seed, 2))
    ut = synth.bf16_round(q[:, :r].T.copy())
    c = synth.normal((N * r,), 0.01, seed, 3)
    layer = Z.Linear(t_bf16(w), K, N, r, t_bf16(ut), 0)
    arena = Z.Arena(t_f32(c), torch.zeros(N * r, device=dev()), torch.zeros(N * r, device=dev()))
    pert = Z.Pert(seed, 2, 0, 1e-3)
    ch = torch.empty(2 * N * r, dtype=torch.bfloat16, device=dev())
    Z.perturb_coeffs(arena, 0, N * r, pert, ch)
    layer.ch, layer.ch_stride = ch, N * r
    x1 = t_bf16(x)
    x2 = torch.cat([x1, x1]).contiguous()
    p1 = torch.empty(T, r, dtype=torch.bfloat16, device=dev())
    Z.project(x1, t_bf16(ut), p1)
    p2 = torch.cat([p1, p1]).contiguous()
    tgt = t_bf16(synth.bf16_round(synth.normal((T, N), 1.0, seed, 5)))
    return layer, arena, pert, x1, x2, p1, p2, tgt


@pytest.mark.parametrize("shared", [False, True], ids=["stacked", "shared-x"])
def test_noalloc_matches_workspace_form_twice(shared):
    for T, K, N, r, seed in ((2048, 512, 4096, 32, 1), (300, 256, 1024, 16, 2)):
        announce("linear mse noalloc", "shared" if shared else "stacked", T, K, N, r)
        layer, arena, pert, x1, x2, p1, p2, tgt = _case(T, K, N, r, seed)
        x, p, flags = (x1, p1, Z.SHARED_X) if shared else (x2, p2, 0)
        ws = torch.empty(Z.linear_mse_workspace_bytes(T, N), dtype=torch.uint8, device=dev())
        want = torch.full((2,), float("nan"), dtype=torch.float32, device=dev())
        got = torch.full((2,), float("nan"), dtype=torch.float32, device=dev())
        Z.linear_mse(layer, arena, x, T, p, pert, tgt, want, ws, flags=flags)
        Z.linear_mse_noalloc(layer, arena, x, T, p, pert, tgt, got, flags=flags)
        g, w = host(got), host(want)
        assert np.all(np.isfinite(g)) and g[0] != g[1]
        np.testing.assert_array_equal(g, w)


def test_noalloc_rejects_shapes_beyond_the_scratch():
    """T = 65536 tokens per half and d_out = 16640 need 1.02 MiB of partial sums: E_INVALID,
    with the loss left untouched (nothing was enqueued; every buffer has its full size all
    the same)."""
    announce("linear mse noalloc too large")
    T, K, N, r = 65536, 128, 16640, 8
    assert Z.linear_mse_workspace_bytes(T, N) > Z.MSE_SCRATCH_BYTES
    x = torch.zeros(2 * T, K, dtype=torch.bfloat16, device=dev())
    w = torch.zeros(N, K, dtype=torch.bfloat16, device=dev())
    ut = torch.zeros(r, K, dtype=torch.bfloat16, device=dev())
    layer = Z.Linear(w, K, N, r, ut, 0)
    arena = Z.Arena(torch.zeros(N * r, device=dev()), torch.zeros(N * r, device=dev()), torch.zeros(N * r, device=dev()))
    ch = torch.zeros(2 * N * r, dtype=torch.bfloat16, device=dev())
    layer.ch, layer.ch_stride = ch, N * r
    p = torch.zeros(2 * T, r, dtype=torch.bfloat16, device=dev())
    tgt = torch.zeros(T, N, dtype=torch.bfloat16, device=dev())
    loss = torch.full((2,), 7.0, dtype=torch.float32, device=dev())
    with pytest.raises(Z.ZoactError) as e:
        Z.linear_mse_noalloc(layer, arena, x, T, p, Z.Pert(1, 1, 0, 1e-3), tgt, loss)
    assert e.value.status == Z.E_INVALID
    assert "static scratch" in str(e.value)
    np.testing.assert_array_equal(host(loss), [7.0, 7.0])
