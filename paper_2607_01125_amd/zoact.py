"""Thin Python binding of libzoact.so (the C ABI declared in include/zoact.h).

Argument marshalling only: every function here checks Python-side types, passes
device pointers of torch tensors and the current HIP stream to the C entry point
of the same name, and raises ZoactError on a non-zero status.  All computation
happens in the library's HIP kernels; nothing falls back to the CPU.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libzoact.so")

F32, BF16, INT4_G128 = 0, 1, 2
EPI_NONE, EPI_SWIGLU, EPI_RELU = 0, 1, 2
SHARED_X = 4   # both halves read one copy of x and p
OK, E_INVALID, E_UNSUPPORTED, E_HIP, E_NOCONVERGE, E_WORKSPACE = range(6)


class ZoactError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"zoact status {status}: {msg}")
        self.status = status


class Pert(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("step", ctypes.c_uint32), ("query", ctypes.c_uint32),
                ("eps", ctypes.c_float)]


class PertPair(ctypes.Structure):
    """General pair: half h evaluates C + sign[h] eps Z(seed, step, query[h]), sign in {-1, 0, 1}."""
    _fields_ = [("seed", ctypes.c_uint64), ("step", ctypes.c_uint32), ("query", ctypes.c_uint32 * 2),
                ("sign", ctypes.c_int32 * 2), ("eps", ctypes.c_float)]


def pert_pair(seed: int, step: int, queries, signs, eps: float) -> PertPair:
    return PertPair(seed, step, (ctypes.c_uint32 * 2)(*queries), (ctypes.c_int32 * 2)(*signs), eps)


class LinearDesc(ctypes.Structure):
    _fields_ = [("w_dtype", ctypes.c_int32), ("w", ctypes.c_void_p), ("w_scales", ctypes.c_void_p),
                ("bias", ctypes.c_void_p), ("ut", ctypes.c_void_p), ("d_in", ctypes.c_int64),
                ("d_out", ctypes.c_int64), ("r", ctypes.c_int32), ("coef_offset", ctypes.c_int64),
                ("ch", ctypes.c_void_p), ("ch_half_stride", ctypes.c_int64), ("plain_begin", ctypes.c_int64),
                ("plain_end", ctypes.c_int64), ("ws", ctypes.c_void_p), ("ws_bytes", ctypes.c_size_t)]


class ArenaDesc(ctypes.Structure):
    _fields_ = [("c_dtype", ctypes.c_int32), ("c", ctypes.c_void_p), ("m", ctypes.c_void_p),
                ("v", ctypes.c_void_p), ("k", ctypes.c_int64)]


class AdamDesc(ctypes.Structure):
    _fields_ = [("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("weight_decay", ctypes.c_float), ("step_size", ctypes.c_float),
                ("inv_sqrt_bc2", ctypes.c_float), ("one_minus_beta1", ctypes.c_float),
                ("one_minus_beta2", ctypes.c_float)]


class EigOpts(ctypes.Structure):
    _fields_ = [("oversample", ctypes.c_int32), ("max_iter", ctypes.c_int32), ("seed", ctypes.c_uint64),
                ("tol", ctypes.c_float), ("adaptive", ctypes.c_int32), ("check_every", ctypes.c_int32)]


def eig_report_tensor(device) -> torch.Tensor:
    """Device buffer for one zoact_eig_report (resid f32, gap f32, iters i32, converged i32)."""
    return torch.zeros(4, dtype=torch.int32, device=device)


def read_eig_report(t: torch.Tensor) -> dict:
    h = t.cpu()
    f = h.view(torch.float32)
    return {"resid": float(f[0]), "gap": float(f[1]), "iters": int(h[2]), "converged": bool(h[3])}


_P = ctypes.c_void_p
_I32, _I64, _U32, _U64, _F = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_float
_SZ = ctypes.c_size_t

SIGNATURES = {
    "zoact_version": ([], ctypes.c_char_p),
    "zoact_status_str": ([_I32], ctypes.c_char_p),
    "zoact_last_error": ([], ctypes.c_char_p),
    "zoact_gen_z": ([_U64, _U32, _U32, _I64, _I64, _P, _P], _I32),
    "zoact_project_workspace_bytes": ([_I64, _I64, _I32], _SZ),
    "zoact_project": ([_P, _I32, _I64, _I64, _P, _I32, _P, _P, _SZ, _P], _I32),
    "zoact_rmsnorm_project": ([_P, _P, _I64, _I64, _F, _P, _I32, _P, _P, _P], _I32),
    "zoact_layernorm_project": ([_P, _P, _P, _I64, _I64, _F, _P, _I32, _P, _P, _P], _I32),
    "zoact_linear_fwd_pm": ([ctypes.POINTER(LinearDesc), ctypes.POINTER(ArenaDesc), _P, _I32, _I64, _P, _P, _U32,
                             ctypes.POINTER(Pert), _P, _I32, _P], _I32),
    "zoact_perturb_coeffs": ([ctypes.POINTER(ArenaDesc), _I64, _I64, ctypes.POINTER(Pert), _P, _P], _I32),
    "zoact_linear_workspace_bytes": ([], _SZ),
    "zoact_dequant_int4": ([_P, _P, _I64, _I64, _P, _P], _I32),
    "zoact_linear_fwd_pair": ([ctypes.POINTER(LinearDesc), ctypes.POINTER(ArenaDesc), _P, _I32, _I64, _P, _P, _U32,
                               ctypes.POINTER(PertPair), _P, _I32, _P], _I32),
    "zoact_perturb_coeffs_pair": ([ctypes.POINTER(ArenaDesc), _I64, _I64, ctypes.POINTER(PertPair), _P, _P], _I32),
    "zoact_step_q": ([ctypes.POINTER(ArenaDesc), _P, _I32, _U64, _U32, _F, ctypes.POINTER(AdamDesc), _P, _P], _I32),
    "zoact_step_q_sgd": ([ctypes.POINTER(ArenaDesc), _P, _I32, _U64, _U32, _F, _F, _P, _P], _I32),
    "zoact_loss_workspace_bytes": ([], _SZ),
    "zoact_linear_xent_workspace_bytes": ([_I64, _I64], _SZ),
    "zoact_linear_xent_pair": ([ctypes.POINTER(LinearDesc), ctypes.POINTER(ArenaDesc), _P, _I64, _I64, _P,
                                ctypes.POINTER(PertPair), _P, _P, _P, _SZ, _P], _I32),
    "zoact_linear_mse_workspace_bytes": ([_I64, _I64], _SZ),
    "zoact_linear_mse_pair": ([ctypes.POINTER(LinearDesc), ctypes.POINTER(ArenaDesc), _P, _I64, _U32, _P,
                               ctypes.POINTER(PertPair), _P, _P, _P, _SZ, _P], _I32),
    "zoact_linear_mse_pair_noalloc": ([ctypes.POINTER(LinearDesc), ctypes.POINTER(ArenaDesc), _P, _I64, _U32, _P,
                                       ctypes.POINTER(PertPair), _P, _P, _P], _I32),
    "zoact_mse_pm": ([_P, _I32, _P, _I64, _I64, _P, _P, _SZ, _P], _I32),
    "zoact_xent_pm": ([_P, _P, _I64, _I64, _I64, _P, _P, _SZ, _P], _I32),
    "zoact_step": ([ctypes.POINTER(ArenaDesc), _P, ctypes.POINTER(Pert), ctypes.POINTER(AdamDesc), _P, _P], _I32),
    "zoact_step_perturb": ([ctypes.POINTER(ArenaDesc), _P, ctypes.POINTER(Pert), ctypes.POINTER(AdamDesc), _P,
                            ctypes.POINTER(Pert), _P, _P], _I32),
    "zoact_step_sgd": ([ctypes.POINTER(ArenaDesc), _P, ctypes.POINTER(Pert), _F, _P, _P], _I32),
    "zoact_basis_workspace_bytes": ([_I64, _I32, ctypes.POINTER(EigOpts)], _SZ),
    "zoact_basis_init_workspace_bytes": ([_I64, _I32, ctypes.POINTER(EigOpts)], _SZ),
    "zoact_gram": ([_P, _I32, _I64, _I64, _I64, _P, _I32, _P], _I32),
    "zoact_basis_from_gram": ([_P, _I64, _I32, ctypes.POINTER(EigOpts), _P, _I32, _P, _P, _P, _P, _SZ, _P], _I32),
    "zoact_basis_init": ([_P, _I32, _I64, _I64, _I64, _I32, ctypes.POINTER(EigOpts), _P, _I32, _P, _P, _P, _P, _SZ,
                          _P],
                         _I32),
    "zoact_embed": ([_P, _I64, _I32, _I64, _P, _P, _I64, _I32, _I64, _I64, _I32, _P, _P], _I32),
    "zoact_rmsnorm": ([_P, _P, _I64, _I64, _F, _I32, _P, _P], _I32),
    "zoact_layernorm": ([_P, _P, _P, _I64, _I64, _F, _I32, _P, _P], _I32),
    "zoact_rope": ([_P, _I32, _I64, _I64, _I64, _I32, _I32, _I64, _P, _P, _P], _I32),
    "zoact_attention": ([_P, _I64, _P, _I64, _P, _I64, _I64, _I64, _I32, _I32, _I32, _F, _I32, _P, _P], _I32),
    "zoact_attention_rope_in_place": ([_I64, _I64, _I32, _I32, _I32, _I32], _I32),
    "zoact_attention_rope": ([_P, _I64, _P, _I64, _P, _I64, _I64, _I64, _I32, _I32, _I32, _F, _I32, _P, _P, _P, _P],
                             _I32),
}

_lib = None


def lib():
    """The loaded library; raises if it has not been built (no CPU fallback exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_01125_amd.build`")
        h = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in SIGNATURES.items():
            f = getattr(h, name)
            f.argtypes = args
            f.restype = res
        _lib = h
    return _lib


def _check(st: int):
    if st != OK:
        raise ZoactError(st, lib().zoact_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise ValueError(f"unsupported activation dtype {t.dtype}")


@dataclass
class Linear:
    """Device tensors of one adapted layer (w: [d_out][d_in] or packed int4 [d_out][d_in/2])."""
    w: torch.Tensor
    d_in: int
    d_out: int
    r: int = 0
    ut: torch.Tensor | None = None
    coef_offset: int = 0
    bias: torch.Tensor | None = None
    w_scales: torch.Tensor | None = None
    ch: torch.Tensor | None = None      # precomputed bf16(C +/- eps Z): half 0 at ch, half 1 at ch + ch_stride
    ch_stride: int = 0
    plain: tuple = (0, 0)               # output features [begin, end) not adapted (no coefficient rows)
    ws: torch.Tensor | None = None      # optional workspace (linear_workspace_bytes)

    def desc(self) -> LinearDesc:
        wd = INT4_G128 if self.w.dtype == torch.uint8 else dtype_code(self.w)
        return LinearDesc(wd, self.w.data_ptr(), self.w_scales.data_ptr() if self.w_scales is not None else None,
                          self.bias.data_ptr() if self.bias is not None else None,
                          self.ut.data_ptr() if self.ut is not None else None, self.d_in, self.d_out, self.r,
                          self.coef_offset, self.ch.data_ptr() if self.ch is not None else None, self.ch_stride,
                          self.plain[0], self.plain[1], self.ws.data_ptr() if self.ws is not None else None,
                          self.ws.numel() * self.ws.element_size() if self.ws is not None else 0)


@dataclass
class Arena:
    """Flat coefficient arena C and Adam moments m, v (all [k])."""
    c: torch.Tensor
    m: torch.Tensor
    v: torch.Tensor

    @property
    def k(self) -> int:
        return self.c.numel()

    def desc(self) -> ArenaDesc:
        return ArenaDesc(dtype_code(self.c), self.c.data_ptr(), self.m.data_ptr(), self.v.data_ptr(), self.k)


def version() -> str:
    return lib().zoact_version().decode()


def gen_z(seed: int, step: int, query: int, e0: int, n: int, out: torch.Tensor, stream=None):
    _check(lib().zoact_gen_z(seed, step, query, e0, n, _ptr(out), _stream(stream)))


def linear_workspace_bytes() -> int:
    return int(lib().zoact_linear_workspace_bytes())


def project_workspace_bytes(n_tok: int, d_in: int, r: int) -> int:
    return int(lib().zoact_project_workspace_bytes(n_tok, d_in, r))


def project(x: torch.Tensor, ut: torch.Tensor, p: torch.Tensor, ws: torch.Tensor | None = None, stream=None):
    """p = x U; with a workspace `ws` (project_workspace_bytes) the depth-split form."""
    d_in = x.shape[-1]
    n_tok = x.numel() // d_in
    nb = ws.numel() * ws.element_size() if ws is not None else 0
    _check(lib().zoact_project(_ptr(x), dtype_code(x), n_tok, d_in, _ptr(ut), ut.shape[0], _ptr(p), _ptr(ws), nb,
                               _stream(stream)))


def rmsnorm_project(x: torch.Tensor, w: torch.Tensor, y: torch.Tensor, eps: float, ut: torch.Tensor, p: torch.Tensor,
                    stream=None):
    """y = RMSNorm(x) * w and p = y U in one pass (bf16); raises ZoactError(E_UNSUPPORTED)
    outside the fused kernel's shapes."""
    d = x.shape[-1]
    _check(lib().zoact_rmsnorm_project(_ptr(x), _ptr(w), x.numel() // d, d, eps, _ptr(ut), ut.shape[0], _ptr(y),
                                       _ptr(p), _stream(stream)))


def layernorm_project(x: torch.Tensor, w: torch.Tensor, b: torch.Tensor, y: torch.Tensor, eps: float,
                      ut: torch.Tensor, p: torch.Tensor, stream=None):
    """y = LayerNorm(x) * w + b and p = y U in one pass (bf16)."""
    d = x.shape[-1]
    _check(lib().zoact_layernorm_project(_ptr(x), _ptr(w), _ptr(b), x.numel() // d, d, eps, _ptr(ut), ut.shape[0],
                                         _ptr(y), _ptr(p), _stream(stream)))


def linear_fwd_pm(layer: Linear, arena: Arena | None, x: torch.Tensor, T: int, p: torch.Tensor | None,
                  y: torch.Tensor, pert: Pert | PertPair, residual: torch.Tensor | None = None, flags: int = 0,
                  stream=None):
    """Both halves of the adapted linear: the +/- pair for a Pert (zoact_linear_fwd_pm), the
    general pair for a PertPair (zoact_linear_fwd_pair)."""
    d = layer.desc()
    a = arena.desc() if arena is not None else None
    fn = lib().zoact_linear_fwd_pair if isinstance(pert, PertPair) else lib().zoact_linear_fwd_pm
    _check(fn(ctypes.byref(d), ctypes.byref(a) if a is not None else None, _ptr(x), dtype_code(x), T, _ptr(p),
              _ptr(residual), flags, ctypes.byref(pert), _ptr(y), dtype_code(y), _stream(stream)))


def perturb_coeffs(arena: Arena, e0: int, n: int, pert: Pert | PertPair, out: torch.Tensor, stream=None):
    """out bf16 [2][n]: bf16(C[e] + s_h eps Z(e)) for arena indices e0 .. e0 + n - 1 (s = (+1, -1)
    for a Pert; the pair's signs and queries for a PertPair)."""
    a = arena.desc()
    fn = lib().zoact_perturb_coeffs_pair if isinstance(pert, PertPair) else lib().zoact_perturb_coeffs
    _check(fn(ctypes.byref(a), e0, n, ctypes.byref(pert), _ptr(out), _stream(stream)))


def dequant_int4(w: torch.Tensor, scales: torch.Tensor, out: torch.Tensor, stream=None):
    """bf16 [d_out][d_in] = bf16(q * s) of INT4 weights (packed uint8 [d_out][d_in/2])."""
    d_out, d_in = w.shape[0], w.shape[1] * 2
    _check(lib().zoact_dequant_int4(_ptr(w), _ptr(scales), d_out, d_in, _ptr(out), _stream(stream)))


def as_pair(pert: Pert | PertPair) -> PertPair:
    """The general pair of a perturbation (the +/- pair for a Pert)."""
    if isinstance(pert, PertPair):
        return pert
    return pert_pair(pert.seed, pert.step, (pert.query, pert.query), (1, -1), pert.eps)


def linear_xent_workspace_bytes(T: int, d_out: int) -> int:
    return int(lib().zoact_linear_xent_workspace_bytes(T, d_out))


def linear_xent(layer: Linear, arena: Arena | None, x: torch.Tensor, tokens: torch.Tensor, p: torch.Tensor | None,
                pert: Pert | PertPair, loss_pm: torch.Tensor, ws: torch.Tensor, stream=None):
    """LM head of both halves with the next-token cross entropy in its epilogue:
    loss_pm[h] = mean over B (S - 1) positions, logits not stored (tokens int32 [B][S])."""
    d = layer.desc()
    a = arena.desc() if arena is not None else None
    B, S = tokens.shape
    pp = as_pair(pert)
    _check(lib().zoact_linear_xent_pair(ctypes.byref(d), ctypes.byref(a) if a is not None else None, _ptr(x), B, S,
                                        _ptr(p), ctypes.byref(pp), _ptr(tokens), _ptr(loss_pm), _ptr(ws),
                                        ws.numel() * ws.element_size(), _stream(stream)))


def linear_mse_workspace_bytes(T: int, d_out: int) -> int:
    return int(lib().zoact_linear_mse_workspace_bytes(T, d_out))


def linear_mse(layer: Linear, arena: Arena | None, x: torch.Tensor, T: int, p: torch.Tensor | None,
               pert: Pert | PertPair, target: torch.Tensor, loss_pm: torch.Tensor, ws: torch.Tensor, stream=None,
               flags: int = 0):
    """Adapted linear of both halves with the regression loss fused into its epilogue:
    loss_pm[h] = mean (bf16(y[h]) - target)^2, y not stored.  flags: SHARED_X when x and p
    hold one copy read by both halves."""
    d = layer.desc()
    a = arena.desc() if arena is not None else None
    pp = as_pair(pert)
    _check(lib().zoact_linear_mse_pair(ctypes.byref(d), ctypes.byref(a) if a is not None else None, _ptr(x), T,
                                       flags, _ptr(p), ctypes.byref(pp), _ptr(target), _ptr(loss_pm), _ptr(ws),
                                       ws.numel() * ws.element_size(), _stream(stream)))


MSE_SCRATCH_BYTES = 1 << 20   # ZOACT_MSE_SCRATCH_BYTES


def linear_mse_noalloc(layer: Linear, arena: Arena | None, x: torch.Tensor, T: int, p: torch.Tensor | None,
                       pert: Pert | PertPair, target: torch.Tensor, loss_pm: torch.Tensor, stream=None,
                       flags: int = 0):
    """linear_mse() with the partial sums in the library's static device scratch (no workspace)."""
    d = layer.desc()
    a = arena.desc() if arena is not None else None
    pp = as_pair(pert)
    _check(lib().zoact_linear_mse_pair_noalloc(ctypes.byref(d), ctypes.byref(a) if a is not None else None, _ptr(x),
                                               T, flags, _ptr(p), ctypes.byref(pp), _ptr(target), _ptr(loss_pm),
                                               _stream(stream)))


def loss_workspace_bytes() -> int:
    return int(lib().zoact_loss_workspace_bytes())


def mse_pm(y: torch.Tensor, target: torch.Tensor, loss_pm: torch.Tensor, ws: torch.Tensor, stream=None):
    T, N = target.shape
    _check(lib().zoact_mse_pm(_ptr(y), dtype_code(y), _ptr(target), T, N, _ptr(loss_pm), _ptr(ws), ws.numel() *
                              ws.element_size(), _stream(stream)))


def xent_pm(logits: torch.Tensor, tokens: torch.Tensor, loss_pm: torch.Tensor, ws: torch.Tensor, stream=None):
    B, S = tokens.shape
    V = logits.shape[-1]
    _check(lib().zoact_xent_pm(_ptr(logits), _ptr(tokens), B, S, V, _ptr(loss_pm), _ptr(ws),
                               ws.numel() * ws.element_size(), _stream(stream)))


def step(arena: Arena, loss_pm: torch.Tensor, pert: Pert, adam: AdamDesc, status: torch.Tensor | None = None,
         stream=None):
    a = arena.desc()
    _check(lib().zoact_step(ctypes.byref(a), _ptr(loss_pm), ctypes.byref(pert), ctypes.byref(adam), _ptr(status),
                            _stream(stream)))


def step_perturb(arena: Arena, loss_pm: torch.Tensor, pert: Pert, adam: AdamDesc, next_pert: Pert,
                 ch_next: torch.Tensor, status: torch.Tensor | None = None, stream=None):
    """step(), then perturb_coeffs(arena, 0, k, next_pert, ch_next), in one pass."""
    a = arena.desc()
    _check(lib().zoact_step_perturb(ctypes.byref(a), _ptr(loss_pm), ctypes.byref(pert), ctypes.byref(adam),
                                    _ptr(status), ctypes.byref(next_pert), _ptr(ch_next), _stream(stream)))


def step_sgd(arena: Arena, loss_pm: torch.Tensor, pert: Pert, lr: float, status: torch.Tensor | None = None,
             stream=None):
    a = arena.desc()
    _check(lib().zoact_step_sgd(ctypes.byref(a), _ptr(loss_pm), ctypes.byref(pert), lr, _ptr(status),
                                _stream(stream)))


def step_q(arena: Arena, losses: torch.Tensor, q: int, seed: int, step: int, eps: float, adam: AdamDesc,
           status: torch.Tensor | None = None, stream=None):
    """One-sided q-query update (Adam): losses fp32 [q + 1] = (L, L_1 .. L_q) on the device."""
    a = arena.desc()
    _check(lib().zoact_step_q(ctypes.byref(a), _ptr(losses), q, seed, step, eps, ctypes.byref(adam), _ptr(status),
                              _stream(stream)))


def step_q_sgd(arena: Arena, losses: torch.Tensor, q: int, seed: int, step: int, eps: float, lr: float,
               status: torch.Tensor | None = None, stream=None):
    a = arena.desc()
    _check(lib().zoact_step_q_sgd(ctypes.byref(a), _ptr(losses), q, seed, step, eps, lr, _ptr(status),
                                  _stream(stream)))


def basis_workspace_bytes(d: int, r: int, opts: EigOpts | None = None) -> int:
    """Workspace of basis_from_gram."""
    return int(lib().zoact_basis_workspace_bytes(d, r, ctypes.byref(opts) if opts is not None else None))


def basis_init_workspace_bytes(d: int, r: int, opts: EigOpts | None = None) -> int:
    """Workspace of basis_init (the Gram plus basis_from_gram's)."""
    return int(lib().zoact_basis_init_workspace_bytes(d, r, ctypes.byref(opts) if opts is not None else None))


def _rows(x: torch.Tensor):
    """(n_tok, d, row stride) of a 2-D activation matrix with unit column stride."""
    if x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be 2-D with contiguous rows")
    return x.shape[0], x.shape[1], x.stride(0)


def _check_basis(st: int) -> bool:
    """True on success, False when the residual bound was not met (outputs written)."""
    if st == E_NOCONVERGE:
        return False
    _check(st)
    return True


def gram(x: torch.Tensor, g: torch.Tensor, accumulate: bool = False, stream=None):
    n_tok, d, ld = _rows(x)
    _check(lib().zoact_gram(_ptr(x), dtype_code(x), n_tok, d, ld, _ptr(g), int(accumulate), _stream(stream)))


def basis_from_gram(g: torch.Tensor, r: int, ut: torch.Tensor, ws: torch.Tensor, opts: EigOpts | None = None,
                    ut_master=None, eigvals=None, report=None, stream=None) -> bool:
    """Returns False when opts.tol was not met (ZOACT_E_NOCONVERGE; the basis is still written)."""
    d = g.shape[0]
    return _check_basis(lib().zoact_basis_from_gram(
        _ptr(g), d, r, ctypes.byref(opts) if opts is not None else None, _ptr(ut), dtype_code(ut), _ptr(ut_master),
        _ptr(eigvals), _ptr(report), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def basis_init(x: torch.Tensor, r: int, ut: torch.Tensor, ws: torch.Tensor, opts: EigOpts | None = None,
               ut_master=None, eigvals=None, report=None, stream=None) -> bool:
    """Returns False when opts.tol was not met (ZOACT_E_NOCONVERGE; the basis is still written)."""
    n_tok, d, ld = _rows(x)
    return _check_basis(lib().zoact_basis_init(
        _ptr(x), dtype_code(x), n_tok, d, ld, r, ctypes.byref(opts) if opts is not None else None, _ptr(ut),
        dtype_code(ut), _ptr(ut_master), _ptr(eigvals), _ptr(report), _ptr(ws), ws.numel() * ws.element_size(),
        _stream(stream)))


def adam_desc(lr: float, t: int, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
              weight_decay: float = 0.0) -> AdamDesc:
    """Host-side Adam scalars for step t (float64, then one rounding to fp32 by ctypes)."""
    if t < 1:
        raise ValueError("Adam step t starts at 1")
    return AdamDesc(beta1, beta2, eps, weight_decay, lr / (1.0 - beta1 ** t), 1.0 / math.sqrt(1.0 - beta2 ** t),
                    1.0 - beta1, 1.0 - beta2)


# ---------------------------------------------------------------- model support ops (zoact_model.h)
def embed(tokens: torch.Tensor, table: torch.Tensor, out: torch.Tensor, seq: int, pos: torch.Tensor | None = None,
          pos_offset: int = 0, distinct_halves: bool = False, stream=None):
    """out [2][n_tok][d]; with distinct_halves, tokens holds [2][n_tok] (one set per half)."""
    n_tok = tokens.numel() // (2 if distinct_halves else 1)
    vocab, d = table.shape
    _check(lib().zoact_embed(_ptr(tokens), n_tok, int(distinct_halves), vocab, _ptr(table), _ptr(pos),
                             pos.shape[0] if pos is not None else 0, pos_offset, seq, d, dtype_code(table), _ptr(out),
                             _stream(stream)))


def rmsnorm(x: torch.Tensor, w: torch.Tensor, y: torch.Tensor, eps: float, stream=None):
    d = x.shape[-1]
    _check(lib().zoact_rmsnorm(_ptr(x), _ptr(w), x.numel() // d, d, eps, dtype_code(x), _ptr(y), _stream(stream)))


def layernorm(x: torch.Tensor, w: torch.Tensor, b: torch.Tensor, y: torch.Tensor, eps: float, stream=None):
    d = x.shape[-1]
    _check(lib().zoact_layernorm(_ptr(x), _ptr(w), _ptr(b), x.numel() // d, d, eps, dtype_code(x), _ptr(y),
                                 _stream(stream)))


def rope(x: torch.Tensor, col0: int, n_heads: int, head_dim: int, seq: int, cos_t: torch.Tensor, sin_t: torch.Tensor,
         stream=None):
    ld = x.shape[-1]
    _check(lib().zoact_rope(_ptr(x), dtype_code(x), x.numel() // ld, ld, col0, n_heads, head_dim, seq, _ptr(cos_t),
                            _ptr(sin_t), _stream(stream)))


def attention_rope_in_place(n_seq: int, seq: int, n_heads: int, n_kv_heads: int, head_dim: int, dtype: int) -> int:
    """1 if attention_rope rotates q and k in place for this configuration, 0 if it leaves them."""
    return int(lib().zoact_attention_rope_in_place(n_seq, seq, n_heads, n_kv_heads, head_dim, dtype))


def attention_rope(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, out: torch.Tensor, n_seq: int, seq: int,
                   n_heads: int, n_kv_heads: int, head_dim: int, scale: float, cos_t: torch.Tensor,
                   sin_t: torch.Tensor, stream=None):
    """Rotary on q and k, then attention; q and k are consumed (left rotated or not)."""
    _check(lib().zoact_attention_rope(_ptr(q), q.stride(0), _ptr(k), k.stride(0), _ptr(v), v.stride(0), n_seq, seq,
                                      n_heads, n_kv_heads, head_dim, scale, dtype_code(out), _ptr(cos_t), _ptr(sin_t),
                                      _ptr(out), _stream(stream)))


def attention(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, out: torch.Tensor, n_seq: int, seq: int, n_heads: int,
              n_kv_heads: int, head_dim: int, scale: float, stream=None):
    """q, k, v may be column slices (views) of wider row-major buffers."""
    _check(lib().zoact_attention(_ptr(q), q.stride(0), _ptr(k), k.stride(0), _ptr(v), v.stride(0), n_seq, seq, n_heads,
                                 n_kv_heads, head_dim, scale, dtype_code(out), _ptr(out), _stream(stream)))
