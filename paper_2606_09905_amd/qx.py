"""Thin Python binding of libqx (the C ABI in include/qx.h).

Argument marshalling only: every step of every operation runs in the HIP
kernels of libqx.so.  torch supplies device memory and the current stream.
If the library is missing, every call raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import math
import os
import re

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libqx.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "qx.h")

# qx_status
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_RANGE, ERR_OUT_OF_MEMORY, ERR_DEVICE = range(6)
STATUS_NAMES = ["OK", "INVALID_ARG", "UNSUPPORTED", "RANGE", "OUT_OF_MEMORY", "DEVICE"]

# qx_attn_dtype
DT_F32, DT_I32 = 0, 1
# qx_pool_kind
POOL_AVG_I32, POOL_MAX_F32 = 0, 1

# qx_route
ROUTE = {
    "auto": 0, "i8_direct": 1, "f16_exact": 2, "i8_karatsuba": 3, "i8_offset4": 4,
    "valu_dot2": 5, "s24_valu": 6, "s24_i8limb": 7,
    "attn_f32_mfma": 8, "attn_i32_mfma": 9, "attn_i32_valu": 10, "attn_f32_valu": 11,
    "f32_mfma": 12, "f32_valu": 13,
}
ROUTE_NAME = {v: k for k, v in ROUTE.items()}


class QxError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        name = STATUS_NAMES[status] if 0 <= status < len(STATUS_NAMES) else str(status)
        super().__init__(f"qx {name}: {message}")


class PlanInfo(ctypes.Structure):
    _fields_ = [
        ("route", ctypes.c_int32), ("chunk", ctypes.c_int32), ("products", ctypes.c_int32),
        ("tile_m", ctypes.c_int32), ("tile_n", ctypes.c_int32), ("tile_k", ctypes.c_int32),
        ("kernels", ctypes.c_int32), ("exact_no_wrap", ctypes.c_int32),
        ("operand_format", ctypes.c_int32), ("k_splits", ctypes.c_int32),
        ("workspace_bytes", ctypes.c_int64),
    ]

    def as_dict(self) -> dict:
        d = {f: getattr(self, f) for f, _ in self._fields_}
        d["route_name"] = ROUTE_NAME.get(self.route, str(self.route))
        return d


_lib = None
_i64, _i32, _p, _f32 = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_float


def lib() -> ctypes.CDLL:
    """Load libqx.so (built in-tree); raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2606_09905_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        sig = {
            "qgemm_i16i32": [_p, _p, _p, _i64, _i64, _i64, _i64, _i32, _i32, _p],
            "qgemm_i32_s24": [_p, _p, _p, _i64, _i64, _i64, _i64, _p],
            "qgemm_i16i32_noalloc": [_p, _p, _p, _i64, _i64, _i64, _i64, _i32, _i32, _p],
            "conv2d_gemm": [_p, _p, _p] + [_i64] * 9 + [_i32, _i32, _p],
            "conv2d_gemm_t": [_i32, _p, _p, _p] + [_i64] * 9 + [_p],
            "attn_core": [_i32, _p, _p, _p, _p, _i64, _i64, _i32, _p],
            "qx_exec_create_gemm_i16i32": [_p, _i64, _i64, _i64, _i64, _i32, _i32],
            "qx_exec_create_gemm_i32_s24": [_p, _i64, _i64, _i64, _i64],
            "qx_exec_create_conv2d": [_p] + [_i64] * 9 + [_i32, _i32],
            "qx_exec_create_attn": [_p, _i32, _i64, _i64, _i32],
            "qx_exec_create_gemm_i16i32_route": [_p, _i64, _i64, _i64, _i64, _i32, _i32, _i32],
            "qx_exec_create_gemm_i32_s24_route": [_p, _i64, _i64, _i64, _i64, _i32],
            "qx_exec_create_conv2d_route": [_p] + [_i64] * 9 + [_i32, _i32, _i32],
            "qx_exec_create_attn_route": [_p, _i32, _i64, _i64, _i32, _i32],
            "qx_exec_create_conv2d_t": [_p, _i32] + [_i64] * 9 + [_i32],
            "qx_testing_host_double": [_i32],
            "qx_exec_run": [_p, _p, _p, _p],
            "qx_exec_plan": [_p, _p],
            "qx_exec_profile": [_p, _p, _p, _p, _i32, _p, _p, _i32],
            "qx_exec_destroy": [_p],
            "qx_plan_gemm_i16i32": [_p, _i64, _i64, _i64, _i64, _i32, _i32, _i32],
            "qx_plan_gemm_i32_s24": [_p, _i64, _i64, _i64, _i64, _i32],
            "qx_plan_conv2d": [_p] + [_i64] * 9 + [_i32, _i32, _i32],
            "qx_plan_conv2d_t": [_p, _i32] + [_i64] * 9 + [_i32],
            "qx_plan_attn": [_p, _i32, _i64, _i64, _i32, _i32],
            "minmax": [_p, _i64, _i32, _p, _p],
            "pool2x2": [_i32, _p, _p, _i64, _i64, _i64, _i64, _p],
            "qx_exec_create_minmax": [_p, _i64, _i32],
            "qx_exec_create_pool2x2": [_p, _i32, _i64, _i64, _i64, _i64],
            "qx_plan_minmax": [_p, _i64, _i32],
            "qx_plan_lenet_i32": [_p, _i64],
            "qx_exec_create_lenet_i32": [_p, _i64],
            "qx_plan_pool2x2": [_p, _i32, _i64, _i64, _i64, _i64],
            "sdpa_f32": [_p, _p, _p, _p, _i64, _i64, _i64, _f32, _i32, _p],
            "qx_exec_create_sdpa_f32": [_p, _i64, _i64, _i64, _f32, _i32],
            "qx_plan_sdpa_f32": [_p, _i64, _i64, _i64, _f32, _i32],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        L.qx_last_error.argtypes = []
        L.qx_last_error.restype = ctypes.c_char_p
        L.qx_release_cache.argtypes = []
        L.qx_release_cache.restype = None
        L.qx_testing_counters.argtypes = [_p, _i32]
        L.qx_testing_counters.restype = None
        _lib = L
    return _lib


def header_functions(path: str = HEADER_PATH) -> list[str]:
    """Names of every function a header (default include/qx.h) declares."""
    with open(path) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"^\s*#.*$", "", text, flags=re.M)     # preprocessor lines
    return sorted(set(re.findall(r"\b([A-Za-z_]\w*)\s*\(", text)) -
                  {"if", "defined", "sizeof"})


def check(status: int) -> None:
    if status != OK:
        msg = lib().qx_last_error()
        raise QxError(status, msg.decode() if msg else "")


# ---------------------------------------------------------------------------
# torch marshalling
# ---------------------------------------------------------------------------
def _torch():
    import torch
    return torch


def _stream(stream):
    """The HIP stream handle (an int) of a torch stream, a raw handle, or
    None for torch's current stream."""
    if stream is None:
        return _torch().cuda.current_stream().cuda_stream
    handle = getattr(stream, "cuda_stream", None)
    return handle if handle is not None else int(stream)


def _dev_tensor(t, dtype, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a GPU device")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _gemm_shapes(A, B):
    if A.dim() == 2 and B.dim() == 2:
        (M, K), (K2, N) = A.shape, B.shape
        batch, out_shape = 1, (M, N)
    elif A.dim() == 3 and B.dim() == 3:
        (batch, M, K), (b2, K2, N) = A.shape, B.shape
        if b2 != batch:
            raise ValueError("batch mismatch")
        out_shape = (batch, M, N)
    else:
        raise ValueError("A and B must both be 2-D or both 3-D")
    if K2 != K:
        raise ValueError(f"inner dimensions differ: {K} vs {K2}")
    return batch, M, N, K, out_shape


def qgemm_i16i32(A, B, bound_a: int = 0, bound_b: int = 0, out=None, stream=None):
    """C = A @ B, int16 in, int32 out (exact mod 2^32); [M,K]@[K,N] or batched."""
    torch = _torch()
    batch, M, N, K, shape = _gemm_shapes(A, B)
    if out is None:
        out = torch.empty(shape, dtype=torch.int32, device=A.device)
    check(lib().qgemm_i16i32(_dev_tensor(A, torch.int16, "A"), _dev_tensor(B, torch.int16, "B"),
                             _dev_tensor(out, torch.int32, "C"), M, N, K, batch,
                             int(bound_a), int(bound_b), _stream(stream)))
    return out


def qgemm_i16i32_noalloc(A, B, out, bound_a: int = 0, bound_b: int = 0, stream=None):
    """qgemm_i16i32 into a caller-provided `out`, with no device allocation
    (the library's fixed per-device scratch serves as workspace)."""
    torch = _torch()
    batch, M, N, K, shape = _gemm_shapes(A, B)
    if tuple(out.shape) != tuple(shape):
        raise ValueError(f"out must have shape {shape}")
    check(lib().qgemm_i16i32_noalloc(_dev_tensor(A, torch.int16, "A"), _dev_tensor(B, torch.int16, "B"),
                                     _dev_tensor(out, torch.int32, "C"), M, N, K, batch,
                                     int(bound_a), int(bound_b), _stream(stream)))
    return out


def qgemm_i32_s24(A, B, out=None, stream=None):
    """C = sext24(A) @ sext24(B) mod 2^32, int32 in and out."""
    torch = _torch()
    batch, M, N, K, shape = _gemm_shapes(A, B)
    if out is None:
        out = torch.empty(shape, dtype=torch.int32, device=A.device)
    check(lib().qgemm_i32_s24(_dev_tensor(A, torch.int32, "A"), _dev_tensor(B, torch.int32, "B"),
                              _dev_tensor(out, torch.int32, "C"), M, N, K, batch, _stream(stream)))
    return out


def conv_out_hw(H, W, KH, KW, stride, pad):
    return (H + 2 * pad - KH) // stride + 1, (W + 2 * pad - KW) // stride + 1


def conv2d_gemm(x, w, stride: int = 1, pad: int = 0, bound_x: int = 0, bound_w: int = 0,
                out=None, stream=None):
    """NCHW int16 x, OIHW int16 w -> NCHW int32 y (cross-correlation, zero padding)."""
    torch = _torch()
    N, Ci, H, W = x.shape
    Co, Ci2, KH, KW = w.shape
    if Ci2 != Ci:
        raise ValueError("channel mismatch")
    Ho, Wo = conv_out_hw(H, W, KH, KW, stride, pad)
    if out is None:
        out = torch.empty((N, Co, max(Ho, 0), max(Wo, 0)), dtype=torch.int32, device=x.device)
    check(lib().conv2d_gemm(_dev_tensor(x, torch.int16, "x"), _dev_tensor(w, torch.int16, "w"),
                            _dev_tensor(out, torch.int32, "y"), N, Ci, H, W, Co, KH, KW,
                            stride, pad, int(bound_x), int(bound_w), _stream(stream)))
    return out


def conv2d_gemm_t(x, w, stride: int = 1, pad: int = 0, out=None, stream=None):
    """Conv2D on float32 (fp32 sum) or int32 (smul24 contract, exact mod 2^32)
    NCHW x and OIHW w -> NCHW y of the same dtype."""
    torch = _torch()
    if x.dtype == torch.float32:
        dt = DT_F32
    elif x.dtype == torch.int32:
        dt = DT_I32
    else:
        raise TypeError("x must be float32 or int32")
    N, Ci, H, W = x.shape
    Co, Ci2, KH, KW = w.shape
    if Ci2 != Ci:
        raise ValueError("channel mismatch")
    Ho, Wo = conv_out_hw(H, W, KH, KW, stride, pad)
    if out is None:
        out = torch.empty((N, Co, max(Ho, 0), max(Wo, 0)), dtype=x.dtype, device=x.device)
    check(lib().conv2d_gemm_t(dt, _dev_tensor(x, x.dtype, "x"), _dev_tensor(w, x.dtype, "w"),
                              _dev_tensor(out, x.dtype, "y"), N, Ci, H, W, Co, KH, KW, stride, pad,
                              _stream(stream)))
    return out


def attn_core(Q, K, V, bound: int = 0, out=None, stream=None):
    """O = (Q K^T) V for [L, d] float32 or int32 tensors."""
    torch = _torch()
    if Q.dtype == torch.float32:
        dt = DT_F32
    elif Q.dtype == torch.int32:
        dt = DT_I32
    else:
        raise TypeError("Q must be float32 or int32")
    L, d = Q.shape
    if out is None:
        out = torch.empty((L, d), dtype=Q.dtype, device=Q.device)
    check(lib().attn_core(dt, _dev_tensor(Q, Q.dtype, "Q"), _dev_tensor(K, Q.dtype, "K"),
                          _dev_tensor(V, Q.dtype, "V"), _dev_tensor(out, Q.dtype, "O"), L, d,
                          int(bound), _stream(stream)))
    return out


def sdpa_f32(Q, K, V, scale: float = 1.0, causal: bool = False, out=None, stream=None):
    """softmax(scale Q K^T [causal mask]) V per head for float32 [..., L, d]
    tensors; leading dimensions are flattened into heads."""
    torch = _torch()
    if Q.dtype != torch.float32:
        raise TypeError("Q must be float32")
    if Q.dim() < 2 or K.shape != Q.shape or V.shape != Q.shape:
        raise ValueError("Q, K, V must share one shape [..., L, d]")
    L, d = Q.shape[-2], Q.shape[-1]
    BH = math.prod(Q.shape[:-2])
    if out is None:
        out = torch.empty(Q.shape, dtype=Q.dtype, device=Q.device)
    check(lib().sdpa_f32(_dev_tensor(Q, Q.dtype, "Q"), _dev_tensor(K, Q.dtype, "K"),
                         _dev_tensor(V, Q.dtype, "V"), _dev_tensor(out, Q.dtype, "O"), BH, L, d,
                         float(scale), 1 if causal else 0, _stream(stream)))
    return out


def minmax(x, out=None, stream=None):
    """(min, max) of a non-empty int32 or int16 tensor, as a 2-element tensor."""
    torch = _torch()
    if x.dtype not in (torch.int32, torch.int16):
        raise TypeError("x must be int32 or int16")
    if out is None:
        out = torch.empty(2, dtype=x.dtype, device=x.device)
    check(lib().minmax(_dev_tensor(x, x.dtype, "x"), x.numel(), x.element_size(),
                       _dev_tensor(out, x.dtype, "out"), _stream(stream)))
    return out


def pool2x2(x, out=None, stream=None):
    """2x2 / stride 2 pooling of an NCHW tensor: int32 -> floor average, float32 -> maximum."""
    torch = _torch()
    if x.dtype == torch.int32:
        kind = POOL_AVG_I32
    elif x.dtype == torch.float32:
        kind = POOL_MAX_F32
    else:
        raise TypeError("x must be int32 (average) or float32 (maximum)")
    N, C, H, W = x.shape
    if out is None:
        out = torch.empty((N, C, H // 2, W // 2), dtype=x.dtype, device=x.device)
    check(lib().pool2x2(kind, _dev_tensor(x, x.dtype, "x"), _dev_tensor(out, x.dtype, "y"),
                        N, C, H, W, _stream(stream)))
    return out


# ---------------------------------------------------------------------------
# planner queries (host only)
# ---------------------------------------------------------------------------
def _route(route) -> int:
    return ROUTE[route] if isinstance(route, str) else int(route)


def plan_gemm_i16i32(M, N, K, batch=1, bound_a=0, bound_b=0, route="auto") -> dict:
    info = PlanInfo()
    check(lib().qx_plan_gemm_i16i32(ctypes.byref(info), M, N, K, batch, bound_a, bound_b, _route(route)))
    return info.as_dict()


def plan_gemm_i32_s24(M, N, K, batch=1, route="auto") -> dict:
    info = PlanInfo()
    check(lib().qx_plan_gemm_i32_s24(ctypes.byref(info), M, N, K, batch, _route(route)))
    return info.as_dict()


def plan_conv2d(N, Ci, H, W, Co, KH, KW, stride=1, pad=0, bound_x=0, bound_w=0, route="auto") -> dict:
    info = PlanInfo()
    check(lib().qx_plan_conv2d(ctypes.byref(info), N, Ci, H, W, Co, KH, KW, stride, pad,
                               bound_x, bound_w, _route(route)))
    return info.as_dict()


def plan_conv2d_t(dtype: str, N, Ci, H, W, Co, KH, KW, stride=1, pad=0, route="auto") -> dict:
    info = PlanInfo()
    check(lib().qx_plan_conv2d_t(ctypes.byref(info), DT_F32 if dtype == "f32" else DT_I32, N, Ci, H, W,
                                 Co, KH, KW, stride, pad, _route(route)))
    return info.as_dict()


def plan_minmax(n, elem_bytes) -> dict:
    info = PlanInfo()
    check(lib().qx_plan_minmax(ctypes.byref(info), n, elem_bytes))
    return info.as_dict()


def plan_pool2x2(kind: str, N, C, H, W) -> dict:
    info = PlanInfo()
    check(lib().qx_plan_pool2x2(ctypes.byref(info), POOL_AVG_I32 if kind == "avg_i32" else POOL_MAX_F32,
                                N, C, H, W))
    return info.as_dict()


def plan_lenet_i32(batch) -> dict:
    info = PlanInfo()
    check(lib().qx_plan_lenet_i32(ctypes.byref(info), batch))
    return info.as_dict()


def plan_sdpa_f32(BH, L, d, scale=1.0, causal=False) -> dict:
    info = PlanInfo()
    check(lib().qx_plan_sdpa_f32(ctypes.byref(info), BH, L, d, float(scale), 1 if causal else 0))
    return info.as_dict()


def plan_attn(dtype: str, L, d, bound=0, route="auto") -> dict:
    info = PlanInfo()
    check(lib().qx_plan_attn(ctypes.byref(info), DT_F32 if dtype == "f32" else DT_I32, L, d,
                             bound, _route(route)))
    return info.as_dict()


# ---------------------------------------------------------------------------
# persistent executor
# ---------------------------------------------------------------------------
class Executor:
    """Owns a qx_exec handle: planned and allocated once, re-dispatched by run()."""

    def __init__(self, handle: ctypes.c_void_p, out_shape, out_dtype, n_inputs: int):
        self._h = handle
        self.out_shape = tuple(out_shape)
        self.out_dtype = out_dtype
        self.n_inputs = n_inputs

    @classmethod
    def gemm_i16i32(cls, M, N, K, batch=1, bound_a=0, bound_b=0, route="auto"):
        torch = _torch()
        h = ctypes.c_void_p()
        if _route(route) == 0:
            check(lib().qx_exec_create_gemm_i16i32(ctypes.byref(h), M, N, K, batch, bound_a, bound_b))
        else:
            check(lib().qx_exec_create_gemm_i16i32_route(ctypes.byref(h), M, N, K, batch, bound_a, bound_b,
                                                         _route(route)))
        return cls(h, (batch, M, N), torch.int32, 2)

    @classmethod
    def gemm_i32_s24(cls, M, N, K, batch=1, route="auto"):
        torch = _torch()
        h = ctypes.c_void_p()
        if _route(route) == 0:
            check(lib().qx_exec_create_gemm_i32_s24(ctypes.byref(h), M, N, K, batch))
        else:
            check(lib().qx_exec_create_gemm_i32_s24_route(ctypes.byref(h), M, N, K, batch, _route(route)))
        return cls(h, (batch, M, N), torch.int32, 2)

    @classmethod
    def conv2d(cls, N, Ci, H, W, Co, KH, KW, stride=1, pad=0, bound_x=0, bound_w=0, route="auto"):
        torch = _torch()
        h = ctypes.c_void_p()
        if _route(route) == 0:
            check(lib().qx_exec_create_conv2d(ctypes.byref(h), N, Ci, H, W, Co, KH, KW, stride, pad,
                                              bound_x, bound_w))
        else:
            check(lib().qx_exec_create_conv2d_route(ctypes.byref(h), N, Ci, H, W, Co, KH, KW, stride, pad,
                                                    bound_x, bound_w, _route(route)))
        Ho, Wo = conv_out_hw(H, W, KH, KW, stride, pad)
        return cls(h, (N, Co, Ho, Wo), torch.int32, 2)

    @classmethod
    def conv2d_t(cls, dtype: str, N, Ci, H, W, Co, KH, KW, stride=1, pad=0, route="auto"):
        torch = _torch()
        h = ctypes.c_void_p()
        dt = DT_F32 if dtype == "f32" else DT_I32
        check(lib().qx_exec_create_conv2d_t(ctypes.byref(h), dt, N, Ci, H, W, Co, KH, KW, stride, pad,
                                            _route(route)))
        Ho, Wo = conv_out_hw(H, W, KH, KW, stride, pad)
        return cls(h, (N, Co, Ho, Wo), torch.float32 if dtype == "f32" else torch.int32, 2)

    @classmethod
    def minmax(cls, n, dtype: str):
        """dtype "i32" or "i16"; the output is 2 elements (min, max)."""
        torch = _torch()
        h = ctypes.c_void_p()
        check(lib().qx_exec_create_minmax(ctypes.byref(h), n, 4 if dtype == "i32" else 2))
        return cls(h, (2,), torch.int32 if dtype == "i32" else torch.int16, 1)

    @classmethod
    def pool2x2(cls, kind: str, N, C, H, W):
        """kind "avg_i32" or "max_f32"."""
        torch = _torch()
        h = ctypes.c_void_p()
        k = POOL_AVG_I32 if kind == "avg_i32" else POOL_MAX_F32
        check(lib().qx_exec_create_pool2x2(ctypes.byref(h), k, N, C, H, W))
        return cls(h, (N, C, H // 2, W // 2), torch.int32 if k == POOL_AVG_I32 else torch.float32, 1)

    @classmethod
    def lenet_i32(cls, batch):
        """inputs (x, w1, w2, f1, f2, f3) int32; output [batch][10] int32."""
        torch = _torch()
        h = ctypes.c_void_p()
        check(lib().qx_exec_create_lenet_i32(ctypes.byref(h), batch))
        return cls(h, (batch, 10), torch.int32, 6)

    @classmethod
    def attn(cls, dtype: str, L, d, bound=0, route="auto"):
        torch = _torch()
        h = ctypes.c_void_p()
        dt = DT_F32 if dtype == "f32" else DT_I32
        if _route(route) == 0:
            check(lib().qx_exec_create_attn(ctypes.byref(h), dt, L, d, bound))
        else:
            check(lib().qx_exec_create_attn_route(ctypes.byref(h), dt, L, d, bound, _route(route)))
        return cls(h, (L, d), torch.float32 if dtype == "f32" else torch.int32, 3)

    @classmethod
    def sdpa_f32(cls, BH, L, d, scale=1.0, causal=False):
        """inputs (Q, K, V) float32 [BH][L][d]; output [BH][L][d]."""
        torch = _torch()
        h = ctypes.c_void_p()
        check(lib().qx_exec_create_sdpa_f32(ctypes.byref(h), BH, L, d, float(scale), 1 if causal else 0))
        return cls(h, (BH, L, d), torch.float32, 3)

    def plan(self) -> dict:
        info = PlanInfo()
        check(lib().qx_exec_plan(self._h, ctypes.byref(info)))
        return info.as_dict()

    def run_ptrs(self, in_ptrs, out_ptr: int, stream=None) -> None:
        """Enqueue with raw device pointers (ints).  Kept lean: for small
        problems the host's cost per call is what bounds back-to-back runs."""
        arr = (ctypes.c_void_p * len(in_ptrs))(*in_ptrs)
        st = lib().qx_exec_run(self._h, arr, out_ptr, _stream(stream))
        if st != OK:
            check(st)

    def run(self, inputs, out=None, stream=None):
        torch = _torch()
        if len(inputs) != self.n_inputs:
            raise ValueError(f"expected {self.n_inputs} inputs")
        if out is None:
            out = torch.empty(self.out_shape, dtype=self.out_dtype, device=inputs[0].device)
        ptrs = []
        for i, t in enumerate(inputs):
            if t.device.type != "cuda" or not t.is_contiguous():
                raise ValueError(f"input {i} must be a contiguous GPU tensor")
            ptrs.append(t.data_ptr())
        if not out.is_contiguous() or out.dtype != self.out_dtype:
            raise ValueError("bad output tensor")
        self.run_ptrs(ptrs, out.data_ptr(), stream)
        return out

    def profile(self, inputs, out, reps: int = 10, stream=None) -> list:
        """Mean execute-only duration (ms) of every launch: [(kernel, ms), ...]."""
        nk = self.plan()["kernels"]
        ms = (ctypes.c_float * max(nk, 1))()
        names = (ctypes.c_char_p * max(nk, 1))()
        arr = (ctypes.c_void_p * len(inputs))(*[ctypes.c_void_p(t.data_ptr()) for t in inputs])
        check(lib().qx_exec_profile(self._h, arr, ctypes.c_void_p(out.data_ptr()), _stream(stream),
                                    int(reps), ms, names, nk))
        return [(names[i].decode(), float(ms[i])) for i in range(nk)]

    def close(self) -> None:
        if self._h:
            check(lib().qx_exec_destroy(self._h))
            self._h = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            if self._h:
                lib().qx_exec_destroy(self._h)
        except Exception:
            pass


# ---------------------------------------------------------------------------
# test seams (include/qx_testing.h): no result is computed under the double
# ---------------------------------------------------------------------------
COUNTERS = ("allocs", "frees", "events", "events_freed", "launches", "live_handles")


def testing_host_double(on: bool) -> None:
    """Switch executor creation to the host-only runtime double (or back)."""
    check(lib().qx_testing_host_double(1 if on else 0))


def testing_counters() -> dict:
    vals = (ctypes.c_int64 * len(COUNTERS))()
    lib().qx_testing_counters(vals, len(COUNTERS))
    return dict(zip(COUNTERS, list(vals)))


class HostTensor:
    """Stand-in for a device tensor under the host double: a pointer, a
    shape and a dtype (nothing is ever read or written through it)."""

    def __init__(self, ptr: int, shape, dtype=None):
        self.ptr, self.shape, self.dtype = ptr, tuple(shape), dtype

    def data_ptr(self) -> int:
        return self.ptr
