"""Host-side checks of the C ABI (no GPU needed).

The library must load, export every entry point that include/birkhoff4.h
declares, and reject bad arguments on the host before touching the device.
The calls below use fake device addresses: every one of them fails validation
and returns before any HIP call, so nothing is dereferenced.
"""
import ctypes
import os
import re

import pytest

import paper_2606_07574_amd as b4

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "birkhoff4.h")

OK, ERR_NULL, ERR_SIZE, ERR_TOL, ERR_MAX_ITER, ERR_DTYPE, ERR_ALIGN, ERR_OVERLAP, ERR_STEPS = (
    0, -1, -2, -3, -4, -5, -6, -7, -8)
ERR_VARIANT = -11
ERR_ETA = -12
ERR_CHANNELS = -13
E = 0x50000000
F = 0x60000000

A = 0x10000000        # fake, 16-byte aligned device addresses far apart
Bp = 0x20000000
C = 0x30000000
D = 0x40000000


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(birkhoff[48]_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(b4.LIB_PATH)
    names = declared_functions()
    assert {"birkhoff4_fwd", "birkhoff4_bwd", "birkhoff4_fwd_ex", "birkhoff4_bwd_ex",
            "birkhoff4_sk_fwd", "birkhoff4_sk_bwd", "birkhoff8_fwd", "birkhoff8_bwd"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_version_and_strerror():
    lib = b4.lib()
    assert lib.birkhoff4_version() >= 100
    for code in range(-12, 1):
        assert lib.birkhoff4_strerror(code)
    assert lib.birkhoff4_strerror(-999) == b"unknown error"


def test_forward_argument_errors():
    lib = b4.lib()
    f = lib.birkhoff4_fwd
    assert f(A, Bp, C, 0, 1e-6, 20, None) == OK              # B = 0 is a no-op
    assert f(None, None, None, 0, 1e-6, 20, None) == OK
    assert f(A, Bp, C, -1, 1e-6, 20, None) == ERR_SIZE
    assert f(None, Bp, C, 10, 1e-6, 20, None) == ERR_NULL
    assert f(A, None, C, 10, 1e-6, 20, None) == ERR_NULL
    assert f(A, Bp, C, 10, -1.0, 20, None) == ERR_TOL
    assert f(A, Bp, C, 10, float("nan"), 20, None) == ERR_TOL
    assert f(A, Bp, C, 10, 1e-6, -1, None) == ERR_MAX_ITER
    assert f(A, Bp, C, 10, 1e-6, 10001, None) == ERR_MAX_ITER
    assert f(A + 4, Bp, C, 10, 1e-6, 20, None) == ERR_ALIGN
    assert f(A, Bp + 8, C, 10, 1e-6, 20, None) == ERR_ALIGN
    assert f(A, A + 64 * 5, C, 10, 1e-6, 20, None) == ERR_OVERLAP   # P inside H
    assert f(A, Bp, Bp + 64 * 9, 10, 1e-6, 20, None) == ERR_OVERLAP  # dual inside P
    fx = lib.birkhoff4_fwd_ex
    assert fx(A, 7, Bp, C, None, 10, 1e-6, 20, None) == ERR_DTYPE
    assert fx(A, 1, Bp, C, D + 4, 10, 1e-6, 20, None) == ERR_ALIGN
    assert fx(A, 1, Bp, C, C + 32 * 3, 10, 1e-6, 20, None) == ERR_OVERLAP  # iters inside dual
    # bf16 H occupies 32 B per matrix: P 32 B too early does overlap
    assert fx(A, 1, A + 32 * 9, None, None, 10, 1e-6, 20, None) == ERR_OVERLAP
    f2 = lib.birkhoff4_fwd_ex2
    for variant in (0, 1, 2):
        assert f2(A, 0, Bp, C, None, 0, 1e-6, 20, variant, None) == OK
        assert f2(A, 0, Bp, C, None, 10, -1.0, 20, variant, None) == ERR_TOL
        assert f2(A, 0, A + 64 * 5, C, None, 10, 1e-6, 20, variant, None) == ERR_OVERLAP
    assert f2(A, 0, Bp, C, None, 10, 1e-6, 20, 3, None) == ERR_VARIANT
    assert f2(A, 0, Bp, C, None, 10, 1e-6, 20, -1, None) == ERR_VARIANT


def test_n8_argument_errors():
    lib = b4.lib()
    f = lib.birkhoff8_fwd
    assert f(A, 0, Bp, C, None, 0, 1e-6, 20, None) == OK
    assert f(A, 0, Bp, C, None, -1, 1e-6, 20, None) == ERR_SIZE
    assert f(None, 0, Bp, C, None, 10, 1e-6, 20, None) == ERR_NULL
    assert f(A, 2, Bp, C, None, 10, 1e-6, 20, None) == ERR_DTYPE
    assert f(A, 0, Bp, C, None, 10, -1.0, 20, None) == ERR_TOL
    assert f(A, 0, Bp, C, None, 10, 1e-6, 10001, None) == ERR_MAX_ITER
    assert f(A, 0, Bp + 4, C, None, 10, 1e-6, 20, None) == ERR_ALIGN
    assert f(A, 0, A + 256 * 9, C, None, 10, 1e-6, 20, None) == ERR_OVERLAP   # P inside H
    assert f(A, 1, A + 128 * 9, None, None, 10, 1e-6, 20, None) == ERR_OVERLAP  # bf16 H: 128 B each
    assert f(A, 0, Bp, Bp + 256 * 9, None, 10, 1e-6, 20, None) == ERR_OVERLAP  # dual inside P
    g = lib.birkhoff8_bwd
    assert g(A, Bp, 0, C, 0, None) == OK
    assert g(A, Bp, 0, C, -3, None) == ERR_SIZE
    assert g(A, None, 0, C, 3, None) == ERR_NULL
    assert g(A, Bp, 5, C, 3, None) == ERR_DTYPE
    assert g(A, Bp, 0, A + 256, 3, None) == ERR_OVERLAP


def test_ot_argument_errors():
    lib = b4.lib()
    f = lib.birkhoff4_ot_fwd
    E = 0x50000000
    assert f(A, Bp, C, 1.0, D, None, None, 0, 1e-6, 20, None) == OK
    assert f(A, Bp, C, 0.0, D, None, None, 5, 1e-6, 20, None) == ERR_ETA
    assert f(A, Bp, C, -1.0, D, None, None, 5, 1e-6, 20, None) == ERR_ETA
    assert f(A, Bp, C, float("inf"), D, None, None, 5, 1e-6, 20, None) == ERR_ETA
    assert f(A, Bp, C, float("nan"), D, None, None, 5, 1e-6, 20, None) == ERR_ETA
    assert f(A, None, C, 1.0, D, None, None, 5, 1e-6, 20, None) == ERR_NULL
    assert f(A, Bp, C, 1.0, D, None, None, 5, -1.0, 20, None) == ERR_TOL
    assert f(A, Bp + 8, C, 1.0, D, None, None, 5, 1e-6, 20, None) == ERR_ALIGN
    assert f(A, Bp, C, 1.0, A + 64 * 2, None, None, 5, 1e-6, 20, None) == ERR_OVERLAP  # T inside M
    assert f(A, Bp, C, 1.0, D, Bp + 16, None, 5, 1e-6, 20, None) == ERR_OVERLAP  # dual inside a
    assert f(A, Bp, C, 1.0, D, E, D + 64, 5, 1e-6, 20, None) == ERR_OVERLAP      # iters inside T
    g = lib.birkhoff4_ot_bwd
    assert g(A, Bp, C, 1.0, D, 0, None) == OK
    assert g(A, Bp, C, 0.0, D, 5, None) == ERR_ETA
    assert g(A, Bp, None, 1.0, D, 5, None) == ERR_NULL
    assert g(A, Bp, C, 1.0, C + 16, 5, None) == ERR_OVERLAP


def test_backward_and_baseline_argument_errors():
    lib = b4.lib()
    g = lib.birkhoff4_bwd
    assert g(A, None, Bp, C, 0, None) == OK
    assert g(A, None, Bp, C, -5, None) == ERR_SIZE
    assert g(None, None, Bp, C, 5, None) == ERR_NULL
    assert g(A, None, None, C, 5, None) == ERR_NULL
    assert g(A, None, Bp, None, 5, None) == ERR_NULL
    assert g(A, None, Bp, A + 16, 5, None) in (ERR_ALIGN, ERR_OVERLAP)
    assert g(A, None, Bp, Bp + 64, 5, None) == ERR_OVERLAP
    assert lib.birkhoff4_bwd_ex(A, Bp, 3, C, 5, None) == ERR_DTYPE
    s = lib.birkhoff4_sk_fwd
    assert s(A, 0, Bp, 5, 0, None) == ERR_STEPS
    assert s(A, 0, Bp, 5, 49, None) == ERR_STEPS
    assert s(A, 0, Bp, 0, 20, None) == OK
    assert s(A, 5, Bp, 5, 20, None) == ERR_DTYPE
    sb = lib.birkhoff4_sk_bwd
    assert sb(A, 0, Bp, 0, C, 5, 0, None) == ERR_STEPS
    assert sb(A, 0, Bp, 9, C, 5, 20, None) == ERR_DTYPE
    assert sb(A, 0, Bp, 0, A + 64, 5, 20, None) == ERR_OVERLAP


def test_binding_refuses_cpu_tensors():
    import torch
    H = torch.zeros(3, 4, 4)
    with pytest.raises(b4.Birkhoff4Error):
        b4.fwd(H)
    with pytest.raises(b4.Birkhoff4Error):
        b4.bwd(H, H)


def test_binding_output_and_device_checks():
    import torch
    dev = torch.device("cpu")
    assert b4._out(None, (3, 4, 4), dev).shape == (3, 4, 4)
    good = torch.empty(3, 4, 4)
    assert b4._out(good, (3, 4, 4), dev) is good
    for bad in (torch.empty(3, 4, 5), torch.empty(2, 4, 4), torch.empty(3, 4, 4, dtype=torch.float64),
                torch.empty(3, 4, 8)[..., ::2]):
        with pytest.raises(ValueError):
            b4._out(bad, (3, 4, 4), dev)
    b4._same_device(good, torch.empty(1))
    with pytest.raises(ValueError):
        b4._same_device(good, torch.empty(1, device="meta"))


def test_saved_hessian_argument_errors():
    lib = b4.lib()
    f = lib.birkhoff4_fwd_hess  # (H, h_dtype, P, dual, hess, iters, B, tol, max_iter, stream)
    assert f(A, 0, Bp, None, C, None, 0, 1e-6, 20, None) == OK
    assert f(A, 0, Bp, None, C, None, -1, 1e-6, 20, None) == ERR_SIZE
    assert f(A, 0, Bp, None, None, None, 10, 1e-6, 20, None) == ERR_NULL
    assert f(A, 3, Bp, None, C, None, 10, 1e-6, 20, None) == ERR_DTYPE
    assert f(A, 0, Bp, None, C, None, 10, -1.0, 20, None) == ERR_TOL
    assert f(A, 0, Bp, None, C, None, 10, 1e-6, -2, None) == ERR_MAX_ITER
    assert f(A, 0, Bp, None, C + 4, None, 10, 1e-6, 20, None) == ERR_ALIGN
    assert f(A, 0, Bp, None, Bp + 64 * 5, None, 10, 1e-6, 20, None) == ERR_OVERLAP  # hess inside P
    assert f(A, 0, Bp, D, D + 32 * 3, None, 10, 1e-6, 20, None) == ERR_OVERLAP    # hess inside dual
    g = lib.birkhoff4_bwd_hess  # (P, hess, dP, dp_dtype, dH, B, stream)
    assert g(A, Bp, C, 0, D, 0, None) == OK
    assert g(A, Bp, C, 0, D, -5, None) == ERR_SIZE
    assert g(A, None, C, 0, D, 5, None) == ERR_NULL
    assert g(A, Bp, C, 7, D, 5, None) == ERR_DTYPE
    assert g(A, Bp + 8, C, 0, D, 5, None) == ERR_ALIGN
    assert g(A, Bp, C, 0, Bp + 32, 5, None) == ERR_OVERLAP  # dH over hess


def test_ot8_argument_errors():
    lib = b4.lib()
    f = lib.birkhoff8_ot_fwd  # (M, a, b, eta, T, dual, iters, B, tol, max_iter, stream)
    assert f(A, Bp, C, 1.0, D, None, None, 0, 1e-6, 20, None) == OK
    assert f(A, Bp, C, 1.0, D, None, None, -1, 1e-6, 20, None) == ERR_SIZE
    assert f(A, Bp, C, 0.0, D, None, None, 5, 1e-6, 20, None) == ERR_ETA
    assert f(A, Bp, C, float("nan"), D, None, None, 5, 1e-6, 20, None) == ERR_ETA
    assert f(A, Bp, C, 1.0, D, None, None, 5, -1.0, 20, None) == ERR_TOL
    assert f(A, None, C, 1.0, D, None, None, 5, 1e-6, 20, None) == ERR_NULL
    assert f(A, Bp + 4, C, 1.0, D, None, None, 5, 1e-6, 20, None) == ERR_ALIGN
    assert f(A, Bp, C, 1.0, A + 256 * 3, None, None, 5, 1e-6, 20, None) == ERR_OVERLAP  # T inside M
    assert f(A, Bp, C, 1.0, D, Bp + 32 * 2, None, 5, 1e-6, 20, None) == ERR_OVERLAP    # dual inside a
    g = lib.birkhoff8_ot_bwd  # (T, a, dT, eta, dM, B, stream)
    assert g(A, Bp, C, 1.0, D, 0, None) == OK
    assert g(A, Bp, C, -1.0, D, 5, None) == ERR_ETA
    assert g(A, None, C, 1.0, D, 5, None) == ERR_NULL
    assert g(A, Bp, C, 1.0, A + 256, 5, None) == ERR_OVERLAP


def test_mix_argument_errors():
    lib = b4.lib()
    f = lib.birkhoff4_mix_fwd  # (H, h_dtype, X, x_dtype, Y, P, dual, iters, B, C, tol, max_iter, stream)
    BF, F32 = b4.BF16, b4.F32
    assert f(A, F32, Bp, BF, C, D, None, None, 0, 64, 1e-6, 20, None) == OK
    assert f(A, F32, Bp, BF, C, D, None, None, -1, 64, 1e-6, 20, None) == ERR_SIZE
    assert f(A, F32, Bp, 7, C, D, None, None, 5, 64, 1e-6, 20, None) == ERR_DTYPE
    assert f(A, 7, Bp, BF, C, D, None, None, 5, 64, 1e-6, 20, None) == ERR_DTYPE
    assert f(A, F32, Bp, BF, C, D, None, None, 5, 12, 1e-6, 20, None) == ERR_CHANNELS  # bf16: C % 8
    assert f(A, F32, Bp, F32, C, D, None, None, 5, 6, 1e-6, 20, None) == ERR_CHANNELS  # fp32: C % 4
    assert f(A, F32, Bp, F32, C, D, None, None, 5, -4, 1e-6, 20, None) == ERR_CHANNELS
    assert f(A, F32, Bp, BF, C, D, None, None, 1 << 40, 1 << 30, 1e-6, 20, None) == ERR_SIZE
    assert f(A, F32, Bp, BF, C, D, None, None, 5, 64, -1.0, 20, None) == ERR_TOL
    assert f(A, F32, Bp, BF, C, D, None, None, 5, 64, 1e-6, -1, None) == ERR_MAX_ITER
    assert f(A, F32, None, BF, C, D, None, None, 5, 64, 1e-6, 20, None) == ERR_NULL
    assert f(A, F32, Bp, BF, None, D, None, None, 5, 64, 1e-6, 20, None) == ERR_NULL
    assert f(A, F32, Bp, BF, C, None, None, None, 5, 64, 1e-6, 20, None) == ERR_NULL
    assert f(A, F32, Bp + 8, BF, C, D, None, None, 5, 64, 1e-6, 20, None) == ERR_ALIGN
    assert f(A, F32, Bp, BF, Bp + 16, D, None, None, 5, 64, 1e-6, 20, None) == ERR_OVERLAP   # Y inside X
    assert f(A, F32, Bp, BF, C, Bp + 64, None, None, 5, 64, 1e-6, 20, None) == ERR_OVERLAP   # P inside X
    assert f(A, F32, Bp, BF, C, D, C + 32, None, 5, 64, 1e-6, 20, None) == ERR_OVERLAP      # dual inside Y
    assert f(A, F32, Bp, BF, C, D, D + 32, None, 5, 64, 1e-6, 20, None) == ERR_OVERLAP      # dual inside P
    assert f(A, F32, Bp, BF, C, A + 16, None, None, 5, 64, 1e-6, 20, None) == ERR_OVERLAP   # P inside H
    g = lib.birkhoff4_mix_bwd  # (P, X, dY, x_dtype, dX, dH, B, C, stream)
    assert g(A, Bp, C, BF, D, E, 0, 64, None) == OK
    assert g(A, Bp, C, BF, D, E, 5, 60, None) == ERR_CHANNELS
    assert g(A, Bp, C, 9, D, E, 5, 64, None) == ERR_DTYPE
    assert g(A, Bp, C, BF, D, None, 5, 64, None) == ERR_NULL
    assert g(A, Bp, None, BF, D, E, 5, 64, None) == ERR_NULL
    assert g(A, Bp, C, BF, D + 4, E, 5, 64, None) == ERR_ALIGN
    assert g(A, Bp, C, BF, C + 256, E, 5, 64, None) == ERR_OVERLAP    # dX inside dY
    assert g(A, Bp, C, BF, D, A + 64, 5, 64, None) == ERR_OVERLAP     # dH inside P
    assert g(A, Bp, C, BF, D, Bp + 128, 5, 64, None) == ERR_OVERLAP   # dH inside X


def test_mix8_argument_errors():
    lib = b4.lib()
    f = lib.birkhoff8_mix_fwd
    BF, F32 = b4.BF16, b4.F32
    assert f(A, F32, Bp, BF, C, D, None, None, 0, 64, 1e-6, 20, None) == OK
    assert f(A, F32, Bp, BF, C, D, None, None, 5, 12, 1e-6, 20, None) == ERR_CHANNELS
    assert f(A, F32, None, BF, C, D, None, None, 5, 64, 1e-6, 20, None) == ERR_NULL
    assert f(A, F32, Bp, BF, Bp + 128 * 8, D, None, None, 5, 64, 1e-6, 20, None) == ERR_OVERLAP  # Y inside X
    assert f(A, F32, Bp, BF, C, D, D + 256, None, 5, 64, 1e-6, 20, None) == ERR_OVERLAP           # dual inside P
    g = lib.birkhoff8_mix_bwd
    assert g(A, Bp, C, BF, D, E, 0, 64, None) == OK
    assert g(A, Bp, C, BF, D, E, 5, 4, None) == ERR_CHANNELS
    assert g(A, Bp, C, BF, D, A + 256, 5, 64, None) == ERR_OVERLAP    # dH inside P
    assert g(A, Bp, C, BF, D + 4, E, 5, 64, None) == ERR_ALIGN
