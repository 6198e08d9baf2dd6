"""Batched 4x4 Birkhoff projection on MI355X: Python binding of libbirkhoff4.so.

Argument marshalling only. Every step of the projection and of its gradient
runs in the HIP kernels of ``csrc/birkhoff4.hip`` behind the C ABI declared in
``include/birkhoff4.h``; PyTorch supplies device memory and the current stream.
There is no CPU fallback: if the library is missing or the tensors are not on
a GPU, the calls raise.

    P, dual = fwd(H)                  # eq. birkhoff_projection via Newton (Sec. 3)
    dH = bwd(P, dP)                   # implicit differentiation (Sec. 4, eq. derivative)
    P = project(H)                    # autograd-aware: backward calls bwd
    P, dual, hess, _ = fwd_hess(H); dH = bwd_hess(P, hess, dP)   # saved-Hessian variant (Sec. 4.2)
    P = sk_fwd(H, 20); dH = sk_bwd(H, dP, 20)   # Sinkhorn-Knopp baseline
    P, dual = fwd8(H); dH = bwd8(P, dP); P = project8(H)   # the same for 8 x 8 matrices
    T, dual = ot_fwd(M, a, b, eta); dM = ot_bwd(T, a, dT, eta)  # general entropic OT, 4 x 4
    T, dual = ot8_fwd(M, a, b, eta); dM = ot8_bwd(T, a, dT, eta)  # the same for 8 x 8
    Y, P, _, _ = mix_fwd(H, X); dX, dH = mix_bwd(P, X, dY)  # residual mixing Y = P X (Sec. 2.1)
    Y = mix(H, X)                     # autograd-aware, gradients for H and X (4 or 8 streams)
    Y, P, _, _ = mix8_fwd(H8, X8); dX, dH = mix8_bwd(P, X8, dY)  # 8 streams per token
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbirkhoff4.so")

F32, BF16 = 0, 1
AUTO, THROUGHPUT, LATENCY = 0, 1, 2
NOT_CONVERGED, NON_FINITE = -1, -2
DEFAULT_TOL = 1e-6
DEFAULT_MAX_ITER = 64

_lib = None


class Birkhoff4Error(RuntimeError):
    pass


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise Birkhoff4Error(
            f"{LIB_PATH} is missing: build it with `python -m paper_2606_07574_amd.build` "
            "(or __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, f32, i32, st = ctypes.c_void_p, ctypes.c_int64, ctypes.c_float, ctypes.c_int, ctypes.c_void_p
    sigs = {
        "birkhoff4_fwd": [vp, vp, vp, i64, f32, i32, st],
        "birkhoff4_bwd": [vp, vp, vp, vp, i64, st],
        "birkhoff4_fwd_ex": [vp, i32, vp, vp, vp, i64, f32, i32, st],
        "birkhoff4_fwd_ex2": [vp, i32, vp, vp, vp, i64, f32, i32, i32, st],
        "birkhoff4_bwd_ex": [vp, vp, i32, vp, i64, st],
        "birkhoff4_fwd_hess": [vp, i32, vp, vp, vp, vp, i64, f32, i32, st],
        "birkhoff4_bwd_hess": [vp, vp, vp, i32, vp, i64, st],
        "birkhoff4_sk_fwd": [vp, i32, vp, i64, i32, st],
        "birkhoff4_sk_bwd": [vp, i32, vp, i32, vp, i64, i32, st],
        "birkhoff8_fwd": [vp, i32, vp, vp, vp, i64, f32, i32, st],
        "birkhoff4_ot_fwd": [vp, vp, vp, f32, vp, vp, vp, i64, f32, i32, st],
        "birkhoff4_ot_bwd": [vp, vp, vp, f32, vp, i64, st],
        "birkhoff8_bwd": [vp, vp, i32, vp, i64, st],
        "birkhoff8_ot_fwd": [vp, vp, vp, f32, vp, vp, vp, i64, f32, i32, st],
        "birkhoff8_ot_bwd": [vp, vp, vp, f32, vp, i64, st],
        "birkhoff4_mix_fwd": [vp, i32, vp, i32, vp, vp, vp, vp, i64, i64, f32, i32, st],
        "birkhoff4_mix_bwd": [vp, vp, vp, i32, vp, vp, i64, i64, st],
        "birkhoff8_mix_fwd": [vp, i32, vp, i32, vp, vp, vp, vp, i64, i64, f32, i32, st],
        "birkhoff8_mix_bwd": [vp, vp, vp, i32, vp, vp, i64, i64, st],
        "birkhoff4_version": [],
    }
    for name, args in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.birkhoff4_strerror.argtypes = [ctypes.c_int]
    lib.birkhoff4_strerror.restype = ctypes.c_char_p
    _lib = lib
    return lib


def lib():
    """The loaded ctypes library (raises if it is not built)."""
    return _load()


def _check(code: int) -> None:
    if code != 0:
        msg = _load().birkhoff4_strerror(code).decode()
        raise Birkhoff4Error(f"birkhoff4 error {code}: {msg}")


def _stream(t: torch.Tensor) -> int:
    return torch.cuda.current_stream(t.device).cuda_stream


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")


def _batch(t: torch.Tensor, name: str, n: int = 4) -> int:
    if not t.is_cuda:
        raise Birkhoff4Error(f"{name} must be a GPU tensor (no CPU path)")
    if t.dim() < 2 or tuple(t.shape[-2:]) != (n, n):
        raise ValueError(f"{name} must have shape [..., {n}, {n}], got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.numel() // (n * n)


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


def _same_device(first: torch.Tensor, *others: torch.Tensor) -> None:
    for t in others:
        if t.device != first.device:
            raise ValueError(f"all tensors must be on {first.device}, got one on {t.device}")


def _out(out: torch.Tensor | None, shape, device, name: str = "out") -> torch.Tensor:
    """A new float32 tensor of the given shape, or the caller's after checking that the
    kernel may write exactly that many float32 values into it."""
    if out is None:
        return torch.empty(shape, dtype=torch.float32, device=device)
    if (tuple(out.shape) != tuple(shape) or out.dtype != torch.float32 or out.device != device
            or not out.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous float32 tensor of shape {tuple(shape)} on {device}")
    return out


def fwd(H: torch.Tensor, tol: float = DEFAULT_TOL, max_iter: int = DEFAULT_MAX_ITER,
        want_dual: bool = True, want_iters: bool = False, out: torch.Tensor | None = None,
        variant: int = AUTO):
    """Project exp(H) onto the Birkhoff polytope, per trailing 4x4 matrix.

    H: float32 or bfloat16 [..., 4, 4] on the GPU. Returns (P, dual, iters):
    P float32 like H, dual float32 [..., 8] or None, iters int32 [...] or None.
    variant: AUTO, THROUGHPUT (one problem per lane) or LATENCY (four lanes per problem).
    """
    B = _batch(H, "H")
    lead = H.shape[:-2]
    P = _out(out, H.shape, H.device)
    dual = torch.empty(*lead, 8, dtype=torch.float32, device=H.device) if want_dual else None
    iters = torch.empty(lead, dtype=torch.int32, device=H.device) if want_iters else None
    with torch.cuda.device(H.device):
        _check(_load().birkhoff4_fwd_ex2(_ptr(H), _dtype_code(H), _ptr(P), _ptr(dual), _ptr(iters),
                                         B, float(tol), int(max_iter), int(variant), _stream(H)))
    return P, dual, iters


def bwd(P: torch.Tensor, dP: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
    """dL/dH from P (the forward output) and dL/dP (float32 or bfloat16)."""
    B = _batch(P, "P")
    if _batch(dP, "dP") != B:
        raise ValueError("P and dP batch sizes differ")
    if P.dtype != torch.float32:
        raise TypeError("P must be float32")
    _same_device(P, dP)
    dH = _out(out, P.shape, P.device)
    with torch.cuda.device(P.device):
        _check(_load().birkhoff4_bwd_ex(_ptr(P), _ptr(dP), _dtype_code(dP), _ptr(dH), B, _stream(P)))
    return dH


def fwd_hess(H: torch.Tensor, tol: float = DEFAULT_TOL, max_iter: int = DEFAULT_MAX_ITER,
             want_dual: bool = True, want_iters: bool = False):
    """fwd that also returns the column weights of P (the Hessian at the solution, Sec. 4.2):
    (P, dual or None, hess float32 [..., 8] = (W12, W13, W14, W23, W24, W34, 0, 0), iters or None)."""
    B = _batch(H, "H")
    lead = H.shape[:-2]
    P = torch.empty(H.shape, dtype=torch.float32, device=H.device)
    dual = torch.empty(*lead, 8, dtype=torch.float32, device=H.device) if want_dual else None
    hess = torch.empty(*lead, 8, dtype=torch.float32, device=H.device)
    iters = torch.empty(lead, dtype=torch.int32, device=H.device) if want_iters else None
    with torch.cuda.device(H.device):
        _check(_load().birkhoff4_fwd_hess(_ptr(H), _dtype_code(H), _ptr(P), _ptr(dual), _ptr(hess), _ptr(iters),
                                          B, float(tol), int(max_iter), _stream(H)))
    return P, dual, hess, iters


def bwd_hess(P: torch.Tensor, hess: torch.Tensor, dP: torch.Tensor) -> torch.Tensor:
    """bwd taking the column weights saved by fwd_hess instead of recomputing them from P."""
    B = _batch(P, "P")
    if _batch(dP, "dP") != B:
        raise ValueError("P and dP batch sizes differ")
    if P.dtype != torch.float32:
        raise TypeError("P must be float32")
    if (tuple(hess.shape) != (*P.shape[:-2], 8) or hess.dtype != torch.float32 or not hess.is_contiguous()):
        raise ValueError(f"hess must be a contiguous float32 tensor of shape {(*P.shape[:-2], 8)}")
    _same_device(P, hess, dP)
    dH = torch.empty(P.shape, dtype=torch.float32, device=P.device)
    with torch.cuda.device(P.device):
        _check(_load().birkhoff4_bwd_hess(_ptr(P), _ptr(hess), _ptr(dP), _dtype_code(dP), _ptr(dH), B, _stream(P)))
    return dH


def sk_fwd(H: torch.Tensor, n_steps: int = 20) -> torch.Tensor:
    """n_steps Sinkhorn-Knopp iterations (baseline)."""
    B = _batch(H, "H")
    P = torch.empty(H.shape, dtype=torch.float32, device=H.device)
    with torch.cuda.device(H.device):
        _check(_load().birkhoff4_sk_fwd(_ptr(H), _dtype_code(H), _ptr(P), B, int(n_steps), _stream(H)))
    return P


def sk_bwd(H: torch.Tensor, dP: torch.Tensor, n_steps: int = 20) -> torch.Tensor:
    """Gradient of the n_steps Sinkhorn-Knopp map at H, applied to dP (baseline)."""
    B = _batch(H, "H")
    if _batch(dP, "dP") != B:
        raise ValueError("H and dP batch sizes differ")
    _same_device(H, dP)
    dH = torch.empty(H.shape, dtype=torch.float32, device=H.device)
    with torch.cuda.device(H.device):
        _check(_load().birkhoff4_sk_bwd(_ptr(H), _dtype_code(H), _ptr(dP), _dtype_code(dP), _ptr(dH),
                                        B, int(n_steps), _stream(H)))
    return dH


class Birkhoff4Fn(torch.autograd.Function):
    """P = proj(exp(H)); the backward is the implicit-differentiation kernel and
    needs only the saved P (no iterates, no Hessian)."""

    @staticmethod
    def forward(ctx, H, tol=DEFAULT_TOL, max_iter=DEFAULT_MAX_ITER):
        P, _, _ = fwd(H.contiguous(), tol, max_iter, want_dual=False)
        ctx.save_for_backward(P)
        ctx.in_dtype = H.dtype
        return P

    @staticmethod
    def backward(ctx, dP):
        (P,) = ctx.saved_tensors
        dH = bwd(P, dP.contiguous())
        return dH.to(ctx.in_dtype), None, None


def project(H: torch.Tensor, tol: float = DEFAULT_TOL, max_iter: int = DEFAULT_MAX_ITER) -> torch.Tensor:
    return Birkhoff4Fn.apply(H, tol, max_iter)


def fwd8(H: torch.Tensor, tol: float = DEFAULT_TOL, max_iter: int = DEFAULT_MAX_ITER,
         want_dual: bool = True, want_iters: bool = False, out: torch.Tensor | None = None):
    """fwd for trailing 8x8 matrices: returns (P, dual [..., 16] or None, iters or None)."""
    B = _batch(H, "H", 8)
    lead = H.shape[:-2]
    P = _out(out, H.shape, H.device)
    dual = torch.empty(*lead, 16, dtype=torch.float32, device=H.device) if want_dual else None
    iters = torch.empty(lead, dtype=torch.int32, device=H.device) if want_iters else None
    with torch.cuda.device(H.device):
        _check(_load().birkhoff8_fwd(_ptr(H), _dtype_code(H), _ptr(P), _ptr(dual), _ptr(iters),
                                     B, float(tol), int(max_iter), _stream(H)))
    return P, dual, iters


def bwd8(P: torch.Tensor, dP: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
    """bwd for trailing 8x8 matrices."""
    B = _batch(P, "P", 8)
    if _batch(dP, "dP", 8) != B:
        raise ValueError("P and dP batch sizes differ")
    if P.dtype != torch.float32:
        raise TypeError("P must be float32")
    _same_device(P, dP)
    dH = _out(out, P.shape, P.device)
    with torch.cuda.device(P.device):
        _check(_load().birkhoff8_bwd(_ptr(P), _ptr(dP), _dtype_code(dP), _ptr(dH), B, _stream(P)))
    return dH


class Birkhoff8Fn(torch.autograd.Function):
    """Birkhoff4Fn for 8x8 matrices."""

    @staticmethod
    def forward(ctx, H, tol=DEFAULT_TOL, max_iter=DEFAULT_MAX_ITER):
        P, _, _ = fwd8(H.contiguous(), tol, max_iter, want_dual=False)
        ctx.save_for_backward(P)
        ctx.in_dtype = H.dtype
        return P

    @staticmethod
    def backward(ctx, dP):
        (P,) = ctx.saved_tensors
        dH = bwd8(P, dP.contiguous())
        return dH.to(ctx.in_dtype), None, None


def project8(H: torch.Tensor, tol: float = DEFAULT_TOL, max_iter: int = DEFAULT_MAX_ITER) -> torch.Tensor:
    return Birkhoff8Fn.apply(H, tol, max_iter)


def _marginals(x: torch.Tensor, lead, name: str, n: int = 4) -> None:
    if not x.is_cuda or x.dtype != torch.float32 or not x.is_contiguous():
        raise ValueError(f"{name} must be a contiguous float32 GPU tensor")
    if tuple(x.shape) != (*lead, n):
        raise ValueError(f"{name} must have shape {(*lead, n)}, got {tuple(x.shape)}")


def ot_fwd(M: torch.Tensor, a: torch.Tensor, b: torch.Tensor, eta: float = 1.0, tol: float = DEFAULT_TOL,
           max_iter: int = DEFAULT_MAX_ITER, want_dual: bool = True, want_iters: bool = False):
    """Entropic OT per trailing 4x4 cost matrix M (float32) with marginals a, b [..., 4]
    (positive, equal sums) and regulariser eta. Returns (T, dual [..., 8] or None, iters or None)."""
    B = _batch(M, "M")
    if M.dtype != torch.float32:
        raise TypeError("M must be float32")
    lead = M.shape[:-2]
    _marginals(a, lead, "a")
    _marginals(b, lead, "b")
    _same_device(M, a, b)
    T = torch.empty(M.shape, dtype=torch.float32, device=M.device)
    dual = torch.empty(*lead, 8, dtype=torch.float32, device=M.device) if want_dual else None
    iters = torch.empty(lead, dtype=torch.int32, device=M.device) if want_iters else None
    with torch.cuda.device(M.device):
        _check(_load().birkhoff4_ot_fwd(_ptr(M), _ptr(a), _ptr(b), float(eta), _ptr(T), _ptr(dual), _ptr(iters),
                                        B, float(tol), int(max_iter), _stream(M)))
    return T, dual, iters


def ot_bwd(T: torch.Tensor, a: torch.Tensor, dT: torch.Tensor, eta: float = 1.0) -> torch.Tensor:
    """dL/dM of the OT solution T from dL/dT (float32)."""
    B = _batch(T, "T")
    if _batch(dT, "dT") != B:
        raise ValueError("T and dT batch sizes differ")
    if T.dtype != torch.float32 or dT.dtype != torch.float32:
        raise TypeError("T and dT must be float32")
    _marginals(a, T.shape[:-2], "a")
    _same_device(T, a, dT)
    dM = torch.empty(T.shape, dtype=torch.float32, device=T.device)
    with torch.cuda.device(T.device):
        _check(_load().birkhoff4_ot_bwd(_ptr(T), _ptr(a), _ptr(dT), float(eta), _ptr(dM), B, _stream(T)))
    return dM


class OTFn(torch.autograd.Function):
    """T = OT(M; a, b, eta); gradient with respect to M only (eq. derivative)."""

    @staticmethod
    def forward(ctx, M, a, b, eta=1.0, tol=DEFAULT_TOL, max_iter=DEFAULT_MAX_ITER):
        a = a.contiguous()
        T, _, _ = ot_fwd(M.contiguous(), a, b.contiguous(), eta, tol, max_iter, want_dual=False)
        ctx.save_for_backward(T, a)
        ctx.eta = eta
        return T

    @staticmethod
    def backward(ctx, dT):
        T, a = ctx.saved_tensors
        return ot_bwd(T, a, dT.contiguous().float(), ctx.eta), None, None, None, None, None


def ot(M: torch.Tensor, a: torch.Tensor, b: torch.Tensor, eta: float = 1.0, tol: float = DEFAULT_TOL,
       max_iter: int = DEFAULT_MAX_ITER) -> torch.Tensor:
    return OTFn.apply(M, a, b, eta, tol, max_iter)


def ot8_fwd(M: torch.Tensor, a: torch.Tensor, b: torch.Tensor, eta: float = 1.0, tol: float = DEFAULT_TOL,
            max_iter: int = DEFAULT_MAX_ITER, want_dual: bool = True, want_iters: bool = False):
    """ot_fwd for trailing 8x8 cost matrices and marginals [..., 8]: (T, dual [..., 16] or None, iters)."""
    B = _batch(M, "M", 8)
    if M.dtype != torch.float32:
        raise TypeError("M must be float32")
    lead = M.shape[:-2]
    _marginals(a, lead, "a", 8)
    _marginals(b, lead, "b", 8)
    _same_device(M, a, b)
    T = torch.empty(M.shape, dtype=torch.float32, device=M.device)
    dual = torch.empty(*lead, 16, dtype=torch.float32, device=M.device) if want_dual else None
    iters = torch.empty(lead, dtype=torch.int32, device=M.device) if want_iters else None
    with torch.cuda.device(M.device):
        _check(_load().birkhoff8_ot_fwd(_ptr(M), _ptr(a), _ptr(b), float(eta), _ptr(T), _ptr(dual), _ptr(iters),
                                        B, float(tol), int(max_iter), _stream(M)))
    return T, dual, iters


def ot8_bwd(T: torch.Tensor, a: torch.Tensor, dT: torch.Tensor, eta: float = 1.0) -> torch.Tensor:
    """ot_bwd for trailing 8x8 problems."""
    B = _batch(T, "T", 8)
    if _batch(dT, "dT", 8) != B:
        raise ValueError("T and dT batch sizes differ")
    if T.dtype != torch.float32 or dT.dtype != torch.float32:
        raise TypeError("T and dT must be float32")
    _marginals(a, T.shape[:-2], "a", 8)
    _same_device(T, a, dT)
    dM = torch.empty(T.shape, dtype=torch.float32, device=T.device)
    with torch.cuda.device(T.device):
        _check(_load().birkhoff8_ot_bwd(_ptr(T), _ptr(a), _ptr(dT), float(eta), _ptr(dM), B, _stream(T)))
    return dM


class OT8Fn(torch.autograd.Function):
    """OTFn for 8x8 problems."""

    @staticmethod
    def forward(ctx, M, a, b, eta=1.0, tol=DEFAULT_TOL, max_iter=DEFAULT_MAX_ITER):
        a = a.contiguous()
        T, _, _ = ot8_fwd(M.contiguous(), a, b.contiguous(), eta, tol, max_iter, want_dual=False)
        ctx.save_for_backward(T, a)
        ctx.eta = eta
        return T

    @staticmethod
    def backward(ctx, dT):
        T, a = ctx.saved_tensors
        return ot8_bwd(T, a, dT.contiguous().float(), ctx.eta), None, None, None, None, None


def ot8(M: torch.Tensor, a: torch.Tensor, b: torch.Tensor, eta: float = 1.0, tol: float = DEFAULT_TOL,
        max_iter: int = DEFAULT_MAX_ITER) -> torch.Tensor:
    return OT8Fn.apply(M, a, b, eta, tol, max_iter)


def _streams(X: torch.Tensor, lead, name: str, n: int = 4) -> int:
    """Checks X as [..., n, C] streams matching the leading dims; returns C."""
    if not X.is_cuda:
        raise Birkhoff4Error(f"{name} must be a GPU tensor (no CPU path)")
    if X.dim() < 2 or tuple(X.shape[:-2]) != tuple(lead) or X.shape[-2] != n:
        raise ValueError(f"{name} must have shape {(*lead, n, 'C')}, got {tuple(X.shape)}")
    if not X.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return X.shape[-1]


def _mix_fwd(n, H, X, tol, max_iter, want_dual, want_iters):
    B = _batch(H, "H", n)
    lead = H.shape[:-2]
    C = _streams(X, lead, "X", n)
    _same_device(H, X)
    Y = torch.empty_like(X)
    P = torch.empty(H.shape, dtype=torch.float32, device=H.device)
    dual = torch.empty(*lead, 2 * n, dtype=torch.float32, device=H.device) if want_dual else None
    iters = torch.empty(lead, dtype=torch.int32, device=H.device) if want_iters else None
    fn = _load().birkhoff4_mix_fwd if n == 4 else _load().birkhoff8_mix_fwd
    with torch.cuda.device(H.device):
        _check(fn(_ptr(H), _dtype_code(H), _ptr(X), _dtype_code(X), _ptr(Y), _ptr(P), _ptr(dual), _ptr(iters), B, C,
                  float(tol), int(max_iter), _stream(H)))
    return Y, P, dual, iters


def _mix_bwd(n, P, X, dY):
    B = _batch(P, "P", n)
    if P.dtype != torch.float32:
        raise TypeError("P must be float32")
    lead = P.shape[:-2]
    C = _streams(X, lead, "X", n)
    if _streams(dY, lead, "dY", n) != C or dY.dtype != X.dtype:
        raise ValueError("dY must have the shape and dtype of X")
    _same_device(P, X, dY)
    dX = torch.empty_like(X)
    dH = torch.empty(P.shape, dtype=torch.float32, device=P.device)
    fn = _load().birkhoff4_mix_bwd if n == 4 else _load().birkhoff8_mix_bwd
    with torch.cuda.device(P.device):
        _check(fn(_ptr(P), _ptr(X), _ptr(dY), _dtype_code(X), _ptr(dX), _ptr(dH), B, C, _stream(P)))
    return dX, dH


def mix_fwd(H: torch.Tensor, X: torch.Tensor, tol: float = DEFAULT_TOL, max_iter: int = DEFAULT_MAX_ITER,
            want_dual: bool = False, want_iters: bool = False):
    """Residual mixing of the mHC layer: P = proj(exp(H)) per token and Y = P X.

    H: [..., 4, 4] float32 or bfloat16 logits; X: [..., 4, C] float32 or bfloat16 streams
    (C a multiple of 8 for bfloat16, of 4 for float32). Returns (Y like X, P float32,
    dual or None, iters or None)."""
    return _mix_fwd(4, H, X, tol, max_iter, want_dual, want_iters)


def mix_bwd(P: torch.Tensor, X: torch.Tensor, dY: torch.Tensor):
    """Backward of mix_fwd: (dX = P^T dY like X, dH float32) from P, X and dY (dtype of X)."""
    return _mix_bwd(4, P, X, dY)


def mix8_fwd(H: torch.Tensor, X: torch.Tensor, tol: float = DEFAULT_TOL, max_iter: int = DEFAULT_MAX_ITER,
             want_dual: bool = False, want_iters: bool = False):
    """mix_fwd for 8 streams per token: H [..., 8, 8], X [..., 8, C]."""
    return _mix_fwd(8, H, X, tol, max_iter, want_dual, want_iters)


def mix8_bwd(P: torch.Tensor, X: torch.Tensor, dY: torch.Tensor):
    """Backward of mix8_fwd."""
    return _mix_bwd(8, P, X, dY)


class MixFn(torch.autograd.Function):
    """Y = proj(exp(H)) X per token (4 or 8 streams, from H's shape); the backward is one
    pass over X and dY."""

    @staticmethod
    def forward(ctx, H, X, tol=DEFAULT_TOL, max_iter=DEFAULT_MAX_ITER):
        X = X.contiguous()
        n = H.shape[-1]
        Y, P, _, _ = _mix_fwd(n, H.contiguous(), X, tol, max_iter, False, False)
        ctx.save_for_backward(P, X)
        ctx.h_dtype = H.dtype
        ctx.n = n
        return Y

    @staticmethod
    def backward(ctx, dY):
        P, X = ctx.saved_tensors
        dX, dH = _mix_bwd(ctx.n, P, X, dY.contiguous().to(X.dtype))
        return dH.to(ctx.h_dtype), dX, None, None


def mix(H: torch.Tensor, X: torch.Tensor, tol: float = DEFAULT_TOL, max_iter: int = DEFAULT_MAX_ITER) -> torch.Tensor:
    """Y = proj(exp(H)) X per token with gradients for H and X; H [..., n, n] with n = 4 or 8."""
    if H.dim() < 2 or H.shape[-1] not in (4, 8):
        raise ValueError(f"H must have shape [..., 4, 4] or [..., 8, 8], got {tuple(H.shape)}")
    return MixFn.apply(H, X, tol, max_iter)


def version() -> int:
    return _load().birkhoff4_version()
