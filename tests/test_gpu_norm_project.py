"""GPU parity of the norm fused with the site's projection (zoact_rmsnorm_project,
zoact_layernorm_project): the norm's output against the oracle's norm, and P against the
oracle's projection of that output (Section 3's X V_r factor), on ragged token counts,
the full model widths and ranks up to 128; shapes outside the fused kernel are refused."""
import numpy as np
import pytest
import torch

import synth
from oracle import linear as olin
from oracle import model as om
from paper_2607_01125_amd import zoact as Z

from gpu_helpers import announce, assert_bf16_close, dev, host, t_bf16

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("ln", [False, True], ids=["rms", "ln"])
@pytest.mark.parametrize("rows,d,r", [(37, 128, 8), (300, 256, 16), (8195, 4096, 32), (500, 5120, 64), (129, 1024, 100),
                                      (64, 2048, 128), (16, 512, 1)])
def test_norm_project_matches_oracle(ln, rows, d, r):
    announce("norm_project", ln, rows, d, r)
    x = synth.bf16_round(synth.normal((rows, d), 1.0, 3, rows, d) + np.float32(0.3))
    w = synth.bf16_round(synth.normal((d,), 0.3, 3, d) + np.float32(1.0))
    b = synth.bf16_round(synth.normal((d,), 0.2, 3, d, 1))
    q, _ = np.linalg.qr(synth.gen(3, d, r).standard_normal((d, r)))
    ut = synth.bf16_round(q.T.astype(np.float32))
    y = torch.full((rows, d), float("nan"), dtype=torch.bfloat16, device=dev())
    p = torch.full((rows, r), float("nan"), dtype=torch.bfloat16, device=dev())
    if ln:
        Z.layernorm_project(t_bf16(x), t_bf16(w), t_bf16(b), y, 1e-5, t_bf16(ut), p)
        want = om.layernorm(x, w, b, 1e-5, "bf16")
    else:
        Z.rmsnorm_project(t_bf16(x), t_bf16(w), y, 1e-5, t_bf16(ut), p)
        want = om.rmsnorm(x, w, 1e-5, "bf16")
    yg = host(y)
    assert_bf16_close(yg, want, 1e-3, "norm output")
    # P from the norm's own (rounded) output: the projection is then exact up to fp32 order
    assert_bf16_close(host(p), olin.project(yg, ut.astype(np.float64), "bf16"), 1e-3, "P")


def test_norm_project_equals_norm_then_project_closely():
    """Against the two separate calls on the Llama width: the same norm output up to
    rounding decisions of the fp32 sums, and P to the same bar."""
    rows, d, r = 4096, 4096, 32
    announce("norm_project vs separate", rows, d, r)
    x = t_bf16(synth.bf16_round(synth.normal((rows, d), 1.0, 5, 1)))
    w = t_bf16(synth.bf16_round(synth.normal((d,), 0.3, 5, 2) + np.float32(1.0)))
    ut = t_bf16(synth.bf16_round(synth.normal((r, d), 1.0 / 64, 5, 3)))
    y1, y2 = (torch.empty(rows, d, dtype=torch.bfloat16, device=dev()) for _ in range(2))
    p1, p2 = (torch.empty(rows, r, dtype=torch.bfloat16, device=dev()) for _ in range(2))
    Z.rmsnorm_project(x, w, y1, 1e-5, ut, p1)
    Z.rmsnorm(x, w, y2, 1e-5)
    Z.project(y2, ut, p2)
    a, b = host(y1), host(y2)
    assert np.mean(a == b) > 0.999
    assert_bf16_close(a, b, 0.0, "norm output vs rmsnorm")
    assert_bf16_close(host(p1), host(p2), 1e-3, "P vs project")


@pytest.mark.parametrize("d,r", [(384, 32), (6144, 32), (256, 129)])
def test_norm_project_unsupported_shapes(d, r):
    announce("norm_project unsupported", d, r)
    x = torch.zeros(16, d, dtype=torch.bfloat16, device=dev())
    w = torch.ones(d, dtype=torch.bfloat16, device=dev())
    ut = torch.zeros(r, d, dtype=torch.bfloat16, device=dev())
    y = torch.empty(16, d, dtype=torch.bfloat16, device=dev())
    p = torch.empty(16, r, dtype=torch.bfloat16, device=dev())
    with pytest.raises(Z.ZoactError) as e:
        Z.rmsnorm_project(x, w, y, 1e-5, ut, p)
    assert e.value.status in (Z.E_UNSUPPORTED, Z.E_INVALID)
