"""NumPy-facing wrapper around the plain C oracle (``oracle/oracle.c``).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the CPU-baseline
leg of the benchmark are the only callers.  The HIP library never imports,
loads or calls anything here, and this module never imports the HIP library.

Each function takes and returns NumPy arrays; the arithmetic lives in the C
file, whose definitions cite the paper (Methodology; Tables 1 and 2).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile liboracle.so with gcc and OpenMP (no HIP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
             "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        p = ctypes.c_void_p
        i64 = ctypes.c_int64
        for name in ("oracle_gemm_i16i32", "oracle_gemm_i32_s24"):
            getattr(lib, name).argtypes = [p, p, p, i64, i64, i64, i64]
        for name in ("oracle_conv2d_direct", "oracle_conv2d_im2col", "oracle_conv2d_s24_direct",
                     "oracle_conv2d_f64_direct"):
            getattr(lib, name).argtypes = [p, p, p] + [i64] * 9
        for name in ("oracle_attn_i32", "oracle_attn_i32_assoc", "oracle_attn_f64",
                     "oracle_attn_f64_assoc", "oracle_attn_f32"):
            getattr(lib, name).argtypes = [p, p, p, p, i64, i64]
        lib.oracle_sdpa_f64.argtypes = [p, p, p, p, i64, i64, i64, ctypes.c_double, ctypes.c_int32]
        lib.oracle_minmax_i32.argtypes = [p, i64, p]
        lib.oracle_minmax_i16.argtypes = [p, i64, p]
        for name in ("oracle_avgpool2_i32", "oracle_maxpool2_f32"):
            getattr(lib, name).argtypes = [p, p, i64, i64, i64, i64]
        _lib = lib
    return _lib


def set_threads(n: int) -> None:
    """Number of OpenMP threads the oracle's loops use from now on (the CPU
    baseline times it on all host cores and on one)."""
    _load()
    ctypes.CDLL("libgomp.so.1").omp_set_num_threads(int(n))


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def _c(a, dtype):
    a = np.asarray(a)
    if a.dtype != dtype:
        raise TypeError(f"expected {np.dtype(dtype)}, got {a.dtype}")
    return np.ascontiguousarray(a)


def gemm_i16i32(A, B):
    """C = A @ B (mod 2^32), A [batch][M][K] or [M][K] int16, B [..][K][N] int16."""
    A = _c(A, np.int16)
    B = _c(B, np.int16)
    squeeze = A.ndim == 2
    if squeeze:
        A, B = A[None], B[None]
    batch, M, K = A.shape
    assert B.shape[0] == batch and B.shape[1] == K
    N = B.shape[2]
    C = np.empty((batch, M, N), np.int32)
    _load().oracle_gemm_i16i32(_ptr(A), _ptr(B), _ptr(C), M, N, K, batch)
    return C[0] if squeeze else C


def gemm_i32_s24(A, B):
    """C = sext24(A) @ sext24(B) (mod 2^32); shapes as gemm_i16i32, int32."""
    A = _c(A, np.int32)
    B = _c(B, np.int32)
    squeeze = A.ndim == 2
    if squeeze:
        A, B = A[None], B[None]
    batch, M, K = A.shape
    assert B.shape[0] == batch and B.shape[1] == K
    N = B.shape[2]
    C = np.empty((batch, M, N), np.int32)
    _load().oracle_gemm_i32_s24(_ptr(A), _ptr(B), _ptr(C), M, N, K, batch)
    return C[0] if squeeze else C


def conv_out_shape(N, Ci, H, W, Co, KH, KW, stride, pad):
    Ho = (H + 2 * pad - KH) // stride + 1
    Wo = (W + 2 * pad - KW) // stride + 1
    return (N, Co, Ho, Wo)


def _conv(fn, x, w, stride, pad, in_dtype=np.int16, out_dtype=np.int32):
    x = _c(x, in_dtype)
    w = _c(w, in_dtype)
    N, Ci, H, W = x.shape
    Co, Ci2, KH, KW = w.shape
    assert Ci == Ci2
    y = np.empty(conv_out_shape(N, Ci, H, W, Co, KH, KW, stride, pad), out_dtype)
    fn(_ptr(x), _ptr(w), _ptr(y), N, Ci, H, W, Co, KH, KW, stride, pad)
    return y


def conv2d_direct(x, w, stride=1, pad=0):
    """Direct 7-loop cross-correlation, zero padding, NCHW/OIHW -> NCHW int32."""
    return _conv(_load().oracle_conv2d_direct, x, w, stride, pad)


def conv2d_im2col(x, w, stride=1, pad=0):
    """The same convolution via explicit im2col and the GEMM oracle."""
    return _conv(_load().oracle_conv2d_im2col, x, w, stride, pad)


def conv2d_s24(x, w, stride=1, pad=0):
    """INT32 convolution under the smul24 contract: operands read as sext24 of
    their low 24 bits, int32 result mod 2^32 (Table 2, Conv2D INT32 row)."""
    return _conv(_load().oracle_conv2d_s24_direct, x, w, stride, pad, np.int32, np.int32)


def conv2d_f64(x, w, stride=1, pad=0):
    """FP32 convolution's reference: float32 inputs, float64 products and sums
    (Table 2, Conv2D FP32 row)."""
    return _conv(_load().oracle_conv2d_f64_direct, x, w, stride, pad, np.float32, np.float64)


def _attn(fn, Q, K, V, dtype, out_dtype):
    Q, K, V = (_c(t, dtype) for t in (Q, K, V))
    L, d = Q.shape
    assert K.shape == (L, d) and V.shape == (L, d)
    O = np.empty((L, d), out_dtype)
    fn(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), L, d)
    return O


def attn_i32(Q, K, V):
    """O = (Q K^T) V (mod 2^32), [L][d] int32."""
    return _attn(_load().oracle_attn_i32, Q, K, V, np.int32, np.int32)


def attn_i32_assoc(Q, K, V):
    """O = Q (K^T V) (mod 2^32): an invariant, equal bit for bit to attn_i32."""
    return _attn(_load().oracle_attn_i32_assoc, Q, K, V, np.int32, np.int32)


def attn_f64(Q, K, V):
    """float64 reference R = (Q K^T) V from float32 inputs."""
    return _attn(_load().oracle_attn_f64, Q, K, V, np.float32, np.float64)


def attn_f64_assoc(Q, K, V):
    """float64 Q (K^T V) from float32 inputs (cross-check of attn_f64)."""
    return _attn(_load().oracle_attn_f64_assoc, Q, K, V, np.float32, np.float64)


def attn_f32(Q, K, V):
    """plain float32, sequential summation order."""
    return _attn(_load().oracle_attn_f32, Q, K, V, np.float32, np.float32)


def minmax(x):
    """(min, max) of a non-empty int32 or int16 array (Table 2, Min/max rows)."""
    x = np.asarray(x)
    if x.dtype == np.int16:
        x = _c(x, np.int16)
        out = np.empty(2, np.int16)
        _load().oracle_minmax_i16(_ptr(x), x.size, _ptr(out))
    else:
        x = _c(x, np.int32)
        out = np.empty(2, np.int32)
        _load().oracle_minmax_i32(_ptr(x), x.size, _ptr(out))
    return out


def _pool(fn, x, dtype):
    x = _c(x, dtype)
    N, C, H, W = x.shape
    y = np.empty((N, C, H // 2, W // 2), dtype)
    fn(_ptr(x), _ptr(y), N, C, H, W)
    return y


def avgpool2_i32(x):
    """2x2 / stride 2 average of int32 NCHW: floor(sum of 4 / 4) (Table 2, AvgPool row)."""
    return _pool(_load().oracle_avgpool2_i32, x, np.int32)


def maxpool2_f32(x):
    """2x2 / stride 2 maximum of float32 NCHW (Table 2, MaxPool row)."""
    return _pool(_load().oracle_maxpool2_f32, x, np.float32)


def lenet_i32(x, w1, w2, f1, f2, f3):
    """LeNet-5-shaped INT32 pipeline (Results: end-to-end CNN), composed of
    the functions above: conv (smul24) -> ReLU -> 2x2 floor average -> conv
    -> ReLU -> 2x2 average -> FC -> ReLU -> FC -> ReLU -> FC, every layer
    int32 mod 2^32 with its operands read under the smul24 contract.
    x [B][1][32][32]; FC weights [in][out]; returns [B][10] int32."""
    B = x.shape[0]
    a = conv2d_s24(x, w1, 1, 0)
    a = avgpool2_i32(np.maximum(a, 0))
    a = conv2d_s24(a, w2, 1, 0)
    a = avgpool2_i32(np.maximum(a, 0)).reshape(1, B, 400)
    h = np.maximum(gemm_i32_s24(a, np.asarray(f1, np.int32)[None]), 0)
    h = np.maximum(gemm_i32_s24(h, np.asarray(f2, np.int32)[None]), 0)
    return gemm_i32_s24(h, np.asarray(f3, np.int32)[None])[0]


def sdpa_f64(Q, K, V, scale=1.0, causal=False):
    """softmax(scale Q K^T [causal mask]) V per head, float64 from float32
    inputs [BH][L][d] (the softmax attention of Table 2's FP32 baseline)."""
    Q, K, V = (_c(t, np.float32) for t in (Q, K, V))
    BH, L, d = Q.shape
    O = np.empty((BH, L, d), np.float64)
    _load().oracle_sdpa_f64(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), BH, L, d, float(scale), 1 if causal else 0)
    return O
