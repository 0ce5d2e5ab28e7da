"""CPU oracle for the fused W8A8 linear -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may import
this package. The product (the HIP library and its Python binding) never imports,
loads or calls it, and shares no code with it.

This is a thin numpy/ctypes wrapper over ``oracle.c`` (plain C loops, built with
``gcc -O2 -ffp-contract=off -fopenmp``). Every function takes and returns numpy
arrays: bf16 tensors travel as their raw uint16 bits.

Functions and the passages they follow (Section 3 of the paper, "The quantization
recipe (reused)" and "The fused kernel"):
  quantize_rows(v_bits)            per-row absmax int8 codes and float32 scales
  gemm_acc(xq, wq)                 exact int32 accumulator of Xq @ Wq^T
  epilogue(acc, sx, sw, b_bits)    bf16(fmaf(float(acc), sx*sw, b))
  epilogue_f64(...)                diagnostic: same in double, rounded once
  linear(x_bits, wq, sw, b_bits)   quantize X per token, product, epilogue
  quantize_rows(v_bits, act=, col_mul=)
                                   the row rule on T(x) * c[k] (T identity or GELU,
                                   c the SmoothQuant runtime multiplier)
  gelu_f64(x)                      x * Phi(x) in double (via erfc)
  col_absmax(v_bits, act=)         per-column max |T(x)| (calibration)
  smooth_factors(ax, aw, alpha)    SmoothQuant factors s and 1/s per input channel
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared"]

_lib = None


class OracleError(RuntimeError):
    pass


_ERRORS = {1: "non-finite input", 2: "rounding mode is not round-to-nearest",
           3: "accumulator does not fit int32", 4: "bad argument"}


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so next to it (gcc, no GPU needed)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.run(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build(force=True)
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    INT = ctypes.c_int
    lib.orc_quantize_rows.argtypes = [P, I64, I64, P, P, INT]
    lib.orc_quantize_rows_ex.argtypes = [P, I64, I64, INT, P, P, P, INT]
    lib.orc_col_absmax.argtypes = [P, I64, I64, INT, P]
    lib.orc_smooth_factors.argtypes = [P, P, I64, ctypes.c_float, P, P]
    lib.orc_gelu_f64_array.argtypes = [P, I64, P]
    lib.orc_gemm_acc.argtypes = [P, P, I64, I64, I64, P, INT]
    lib.orc_epilogue.argtypes = [P, P, P, P, I64, I64, P, INT]
    lib.orc_epilogue_f64.argtypes = [P, P, P, P, I64, I64, P, INT]
    lib.orc_linear.argtypes = [P, P, P, P, I64, I64, I64, P, P, P, P, INT]
    lib.orc_f32_to_bf16.argtypes = [ctypes.c_float]
    lib.orc_f32_to_bf16.restype = ctypes.c_uint16
    lib.orc_f64_to_bf16.argtypes = [ctypes.c_double]
    lib.orc_f64_to_bf16.restype = ctypes.c_uint16
    lib.orc_bf16_to_f32.argtypes = [ctypes.c_uint16]
    lib.orc_bf16_to_f32.restype = ctypes.c_float
    lib.orc_max_threads.restype = ctypes.c_int
    lib.orc_f32_to_bf16_array.argtypes = [P, I64, P]
    lib.orc_f64_to_bf16_array.argtypes = [P, I64, P]
    for f in ("orc_quantize_rows", "orc_gemm_acc", "orc_epilogue", "orc_epilogue_f64",
              "orc_linear", "orc_quantize_rows_ex", "orc_col_absmax", "orc_smooth_factors"):
        getattr(lib, f).restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int):
    if rc != 0:
        raise OracleError(_ERRORS.get(rc, f"error {rc}"))


def _c(a, dtype):
    a = np.asarray(a)
    if a.dtype != dtype:
        raise TypeError(f"expected {np.dtype(dtype)}, got {a.dtype}")
    return np.ascontiguousarray(a)


def max_threads() -> int:
    return int(_load().orc_max_threads())


def f32_to_bf16(values) -> np.ndarray:
    """bf16 bits of float32 values, round-to-nearest-even (the oracle's own rounding)."""
    v = np.ascontiguousarray(values, dtype=np.float32).ravel()
    out = np.empty(v.size, np.uint16)
    _load().orc_f32_to_bf16_array(_ptr(v), v.size, _ptr(out))
    return out


def f64_to_bf16(values) -> np.ndarray:
    v = np.ascontiguousarray(values, dtype=np.float64).ravel()
    out = np.empty(v.size, np.uint16)
    _load().orc_f64_to_bf16_array(_ptr(v), v.size, _ptr(out))
    return out


def bf16_to_f32(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


ACTS = {"none": 0, "gelu": 1}


def quantize_rows(v_bits, nthreads: int = 0, *, act: str = "none", col_mul=None):
    """Per-row absmax quantization of v = T(x) * col_mul[k]: returns (q int8 [R,K],
    scale float32 [R]). act "none" is the plain rule on the bf16 values."""
    v = _c(v_bits, np.uint16)
    R, K = v.shape
    q = np.empty((R, K), np.int8)
    s = np.empty(R, np.float32)
    if act == "none" and col_mul is None:
        _check(_load().orc_quantize_rows(_ptr(v), R, K, _ptr(q), _ptr(s), nthreads))
        return q, s
    cm = None if col_mul is None else _c(col_mul, np.float32)
    if cm is not None and cm.shape != (K,):
        raise ValueError("col_mul must be [K]")
    _check(_load().orc_quantize_rows_ex(_ptr(v), R, K, ACTS[act], _ptr(cm), _ptr(q), _ptr(s),
                                        nthreads))
    return q, s


def gelu_f64(x) -> np.ndarray:
    """GELU(x) = x * Phi(x) in double precision."""
    v = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty_like(v)
    _load().orc_gelu_f64_array(_ptr(v), v.size, _ptr(out))
    return out


def col_absmax(v_bits, *, act: str = "none") -> np.ndarray:
    """amax[k] = max_r |T(x[r, k])| as float32."""
    v = _c(v_bits, np.uint16)
    R, K = v.shape
    out = np.empty(K, np.float32)
    _check(_load().orc_col_absmax(_ptr(v), R, K, ACTS[act], _ptr(out)))
    return out


def smooth_factors(ax, aw, alpha: float = 0.5):
    """SmoothQuant factors: (s, s_inv) float32 [K], s = ax^alpha / aw^(1 - alpha)."""
    ax = _c(ax, np.float32)
    aw = _c(aw, np.float32)
    if ax.shape != aw.shape or ax.ndim != 1:
        raise ValueError("ax and aw must be matching [K] vectors")
    s = np.empty_like(ax)
    si = np.empty_like(ax)
    _check(_load().orc_smooth_factors(_ptr(ax), _ptr(aw), ax.size, float(alpha), _ptr(s),
                                      _ptr(si)))
    return s, si


def gemm_acc(xq, wq, nthreads: int = 0):
    """Exact int32 acc[m,n] = sum_k xq[m,k] * wq[n,k]."""
    xq = _c(xq, np.int8)
    wq = _c(wq, np.int8)
    M, K = xq.shape
    N, K2 = wq.shape
    if K != K2:
        raise ValueError("K mismatch")
    acc = np.empty((M, N), np.int32)
    _check(_load().orc_gemm_acc(_ptr(xq), _ptr(wq), M, N, K, _ptr(acc), nthreads))
    return acc


def epilogue(acc, sx, sw, b_bits=None, nthreads: int = 0):
    """bf16 bits of fmaf(float(acc), sx[m]*sw[n], b[n]) (b = +0 without bias)."""
    acc = _c(acc, np.int32)
    sx = _c(sx, np.float32)
    sw = _c(sw, np.float32)
    b = None if b_bits is None else _c(b_bits, np.uint16)
    M, N = acc.shape
    y = np.empty((M, N), np.uint16)
    _check(_load().orc_epilogue(_ptr(acc), _ptr(sx), _ptr(sw), _ptr(b), M, N, _ptr(y),
                                nthreads))
    return y


def epilogue_f64(acc, sx, sw, b_bits=None, nthreads: int = 0):
    acc = _c(acc, np.int32)
    sx = _c(sx, np.float32)
    sw = _c(sw, np.float32)
    b = None if b_bits is None else _c(b_bits, np.uint16)
    M, N = acc.shape
    y = np.empty((M, N), np.uint16)
    _check(_load().orc_epilogue_f64(_ptr(acc), _ptr(sx), _ptr(sw), _ptr(b), M, N,
                                    _ptr(y), nthreads))
    return y


def linear(x_bits, wq, sw, b_bits=None, nthreads: int = 0):
    """Whole linear on pre-quantized weights: returns (y bits, xq, sx, acc)."""
    x = _c(x_bits, np.uint16)
    wq = _c(wq, np.int8)
    sw = _c(sw, np.float32)
    b = None if b_bits is None else _c(b_bits, np.uint16)
    M, K = x.shape
    N = wq.shape[0]
    xq = np.empty((M, K), np.int8)
    sx = np.empty(M, np.float32)
    acc = np.empty((M, N), np.int32)
    y = np.empty((M, N), np.uint16)
    _check(_load().orc_linear(_ptr(x), _ptr(wq), _ptr(sw), _ptr(b), M, N, K, _ptr(xq),
                              _ptr(sx), _ptr(acc), _ptr(y), nthreads))
    return y, xq, sx, acc
