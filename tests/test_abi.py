"""The C-ABI library loads and exports every symbol the headers declare; host-side
argument validation rejects bad calls before anything reaches the GPU (these calls
make no HIP call, so they run without a GPU)."""
import ctypes
import glob
import os
import re

import pytest

from paper_2607_01125_amd import zoact as Z

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        txt = open(h).read()
        txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
        names |= set(re.findall(r"\b(zoact_[a-z0-9_]+)\s*\(", txt))
    return sorted(names)


def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(Z.LIB_PATH)
    names = declared_symbols()
    assert len(names) >= 15
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_covers_header():
    assert set(declared_symbols()) <= set(Z.SIGNATURES)


def test_version_and_status_strings():
    assert Z.version().startswith("zoact-gfx950")
    assert Z.lib().zoact_status_str(Z.E_INVALID) == b"invalid argument"


def _pert():
    return Z.Pert(1, 1, 0, 1e-3)


def test_validation_rejects_before_launch():
    L = Z.lib()
    assert L.zoact_gen_z(1, 1, 0, 0, -5, None, None) == Z.E_INVALID
    assert b"negative" in L.zoact_last_error()
    assert L.zoact_gen_z(1, 1, 0, 0, 10, None, None) == Z.E_INVALID
    # r out of range for the projection
    assert L.zoact_project(ctypes.c_void_p(16), Z.BF16, 8, 64, ctypes.c_void_p(16), 0, ctypes.c_void_p(16), None, 0,
                           None) == Z.E_INVALID
    assert L.zoact_project(ctypes.c_void_p(16), Z.BF16, 8, 64, ctypes.c_void_p(16), 300, ctypes.c_void_p(16), None, 0,
                           None) == Z.E_INVALID
    assert L.zoact_project(ctypes.c_void_p(16), Z.BF16, 8, 64, ctypes.c_void_p(16), 8, ctypes.c_void_p(16),
                           ctypes.c_void_p(24), 1 << 20, None) == Z.E_INVALID        # misaligned workspace
    # INT4 layer with d_in not a multiple of 128
    d = Z.LinearDesc(Z.INT4_G128, 16, 16, None, None, 64, 64, 0, 0)
    st = L.zoact_linear_fwd_pm(ctypes.byref(d), None, ctypes.c_void_p(16), Z.BF16, 4, None, None, 0,
                               ctypes.byref(_pert()), ctypes.c_void_p(16), Z.BF16, None)
    assert st == Z.E_INVALID and b"INT4" in L.zoact_last_error()
    # adapted layer without an arena
    d = Z.LinearDesc(Z.BF16, 16, None, None, 16, 64, 64, 8, 0)
    st = L.zoact_linear_fwd_pm(ctypes.byref(d), None, ctypes.c_void_p(16), Z.BF16, 4, ctypes.c_void_p(16), None, 0,
                               ctypes.byref(_pert()), ctypes.c_void_p(16), Z.BF16, None)
    assert st == Z.E_INVALID
    # coefficient block outside the arena
    a = Z.ArenaDesc(Z.F32, 16, 16, 16, 100)
    d = Z.LinearDesc(Z.BF16, 16, None, None, 16, 64, 64, 8, 0)
    st = L.zoact_linear_fwd_pm(ctypes.byref(d), ctypes.byref(a), ctypes.c_void_p(16), Z.BF16, 4, ctypes.c_void_p(16),
                               None, 0, ctypes.byref(_pert()), ctypes.c_void_p(16), Z.BF16, None)
    assert st == Z.E_INVALID and b"outside the arena" in L.zoact_last_error()
    # misaligned pointer
    d = Z.LinearDesc(Z.BF16, 16, None, None, None, 64, 64, 0, 0)
    st = L.zoact_linear_fwd_pm(ctypes.byref(d), None, ctypes.c_void_p(18), Z.BF16, 4, None, None, 0,
                               ctypes.byref(_pert()), ctypes.c_void_p(16), Z.BF16, None)
    assert st == Z.E_INVALID and b"aligned" in L.zoact_last_error()
    # loss workspace too small
    assert L.zoact_mse_pm(ctypes.c_void_p(16), Z.BF16, ctypes.c_void_p(16), 4, 4, ctypes.c_void_p(16),
                          ctypes.c_void_p(16), 8, None) == Z.E_WORKSPACE
    # basis: fewer tokens than r, oversampled block larger than d
    assert L.zoact_basis_init(ctypes.c_void_p(16), Z.BF16, 4, 64, 64, 8, None, ctypes.c_void_p(16), Z.BF16, None,
                              None, None, ctypes.c_void_p(16), 1 << 30, None) == Z.E_INVALID
    assert L.zoact_basis_from_gram(ctypes.c_void_p(16), 64, 40, None, ctypes.c_void_p(16), Z.F32, None, None, None,
                                   ctypes.c_void_p(16), 1 << 30, None) == Z.E_INVALID
    # basis: adaptive mode without a tolerance, negative tolerance
    for opts in (Z.EigOpts(0, 0, 1, 0.0, 1, 0), Z.EigOpts(0, 0, 1, -1.0, 0, 0)):
        assert L.zoact_basis_from_gram(ctypes.c_void_p(16), 64, 8, ctypes.byref(opts), ctypes.c_void_p(16), Z.F32,
                                       None, None, None, ctypes.c_void_p(16), 1 << 30, None) == Z.E_INVALID
    # Gram: row stride below d, bf16 row stride not a multiple of 8
    assert L.zoact_gram(ctypes.c_void_p(16), Z.F32, 8, 64, 63, ctypes.c_void_p(16), 0, None) == Z.E_INVALID
    assert L.zoact_gram(ctypes.c_void_p(16), Z.BF16, 8, 64, 68, ctypes.c_void_p(16), 0, None) == Z.E_INVALID


def test_attention_rope_post_state_query_rejects_bad_configs():
    L = Z.lib()
    assert L.zoact_attention_rope_in_place(1, 8, 3, 2, 64, Z.BF16) == -1   # 3 query heads over 2 kv heads
    assert L.zoact_attention_rope_in_place(1, 8, 4, 2, 64, 7) == -1        # unknown dtype
    assert L.zoact_attention_rope_in_place(0, 8, 4, 2, 64, Z.BF16) == -1


def test_basis_workspace_grows_with_block():
    a = Z.basis_workspace_bytes(4096, 32)
    b = Z.basis_workspace_bytes(4096, 64)
    assert 0 < a < b


def test_basis_init_workspace_holds_the_gram():
    for d in (129, 4096):
        g = (d * d * 4 + 255) // 256 * 256
        assert Z.basis_init_workspace_bytes(d, 8) == g + Z.basis_workspace_bytes(d, 8)


def test_pair_and_query_step_validation():
    L = Z.lib()
    a = Z.ArenaDesc(Z.F32, 16, 16, 16, 100)
    bad = Z.pert_pair(1, 1, (0, 1), (1, 2), 1e-3)
    d = Z.LinearDesc(Z.BF16, 16, None, None, None, 64, 64, 0, 0)
    st = L.zoact_linear_fwd_pair(ctypes.byref(d), None, ctypes.c_void_p(16), Z.BF16, 4, None, None, 0,
                                 ctypes.byref(bad), ctypes.c_void_p(16), Z.BF16, None)
    assert st == Z.E_INVALID and b"sign" in L.zoact_last_error()
    st = L.zoact_perturb_coeffs_pair(ctypes.byref(a), 0, 10, ctypes.byref(bad), ctypes.c_void_p(16), None)
    assert st == Z.E_INVALID and b"sign" in L.zoact_last_error()
    adam = Z.adam_desc(1e-3, 1)
    for q in (0, 257):
        st = L.zoact_step_q(ctypes.byref(a), ctypes.c_void_p(16), q, 1, 1, 1e-3, ctypes.byref(adam), None, None)
        assert st == Z.E_INVALID and b"q=" in L.zoact_last_error()
        st = L.zoact_step_q_sgd(ctypes.byref(a), ctypes.c_void_p(16), q, 1, 1, 1e-3, 1e-4, None, None)
        assert st == Z.E_INVALID
    st = L.zoact_step_q(ctypes.byref(a), None, 4, 1, 1, 1e-3, ctypes.byref(adam), None, None)
    assert st == Z.E_INVALID
    # the two-sided pair written as a general pair is accepted (fails later only for want of a GPU)
    good = Z.pert_pair(1, 1, (0, 0), (1, -1), 1e-3)
    assert tuple(good.sign) == (1, -1) and tuple(good.query) == (0, 0)
