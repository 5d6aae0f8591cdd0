"""Host logic of the GPU model driver: arena layout and fused weight layouts against the
oracle's (independent) definitions.  No GPU needed."""
import numpy as np
import pytest
import torch

import synth
from oracle import model as om
from paper_2607_01125_amd import model as gm

SHAPES = [synth.TINY, synth.LLAMA3_8B, synth.OPT_13B,
          synth.shrink(synth.LLAMA3_8B, n_layers=3, d_model=256, n_heads=4, n_kv_heads=2, d_ff=512, rank=16),
          synth.shrink(synth.TINY, adapted=("q", "v", "o", "gate", "up", "down"))]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s.name}-{s.n_layers}-{len(s.adapted)}")
def test_arena_layout_matches_oracle(shape):
    mine = [(b.layer, b.name, b.rows, b.r, b.offset) for b in gm.arena_layout(shape)]
    theirs = [(b.layer, b.name, b.rows, b.r, b.offset) for b in om.arena_layout(shape)]
    assert mine == theirs


def test_gate_up_interleave_matches_oracle_rows():
    ff, d = 96, 8
    wg = torch.arange(ff * d, dtype=torch.float32).reshape(ff, d)
    wu = -wg - 1
    fused = gm.interleave_gate_up(wg, wu).numpy()
    gr, ur = om.gate_up_rows(ff)
    np.testing.assert_array_equal(fused[gr], wg.numpy())
    np.testing.assert_array_equal(fused[ur], wu.numpy())


def test_site_of_each_block():
    shape = synth.shrink(synth.OPT_13B, n_layers=2)
    sites = {b.name: b.site for b in gm.arena_layout(shape)}
    assert sites == {"qv": "attn", "out": "o", "fc1": "mlp", "fc2": "down"}


def test_unsupported_adaptation_sets_are_rejected():
    with pytest.raises(ValueError):
        gm.arena_layout(synth.shrink(synth.TINY, adapted=("q",)))
    with pytest.raises(ValueError):
        gm.arena_layout(synth.shrink(synth.OPT_13B, adapted=("q", "v")))
