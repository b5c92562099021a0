"""Seeded synthetic inputs for the integer GEMM substrate.

This module only draws random numbers; it holds none of the method's
arithmetic, so both the HIP path and the CPU oracle can take their inputs from
it.  The paper gives no shapes for its operator table and uses no dataset, so
the workloads below are synthetic by definition: a small INT16 GEMM (values in
[-1024, 1023]), smul24 INT32 GEMMs over the full signed 24-bit range, an INT16
3x3 convolution, the FP32 and INT32 attention cores, the large INT16 GEMMs
(values in [-256, 255]), and the same 3x3 convolution on FP32 and on smul24
INT32 operands, and the HBM-bound rows: min/max over INT32 and INT16 arrays,
2x2 INT32 average pooling and FP32 max pooling, and a LeNet-5-shaped INT32
pipeline with synthetic weights (images in [0, 255], weights in [-3, 3]),
and multi-head softmax attention (32 heads of 4096 x 64, plain and causal).
Integers are uniform over a
closed range; FP32 attention-core inputs are N(0, 1) / sqrt(d), FP32
convolution inputs N(0, 1) with weights N(0, 1) / sqrt(C_in KH KW), pooling
inputs N(0, 1), softmax-attention inputs N(0, 1) * d^(-1/4), so that at
scale 1 the scores have unit variance.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


def ints(rng: np.random.Generator, shape, lo: int, hi: int, dtype) -> np.ndarray:
    """Uniform integers in the closed range [lo, hi]."""
    return rng.integers(lo, hi, size=shape, dtype=dtype, endpoint=True)


def normal_f32(rng: np.random.Generator, shape, scale: float) -> np.ndarray:
    """float32 samples of N(0, 1) * scale (drawn in float64, then rounded)."""
    return (rng.standard_normal(shape) * scale).astype(np.float32)


@dataclass(frozen=True)
class Workload:
    name: str
    op: str            # "gemm_i16i32" | "gemm_i32_s24" | "conv2d" | "conv2d_f32" | "conv2d_i32"
                       # | "attn_f32" | "attn_i32" | "sdpa_f32" | ...
    seed: int
    dims: dict = field(default_factory=dict)
    lo: int = 0
    hi: int = 0
    bound: int = 0     # operand-range contract: max |x|

    @property
    def ops(self) -> float:
        """Algorithmic operations (2 per multiply-add) of one evaluation."""
        d = self.dims
        if self.op in ("gemm_i16i32", "gemm_i32_s24"):
            return 2.0 * d["M"] * d["N"] * d["K"] * d["batch"]
        if self.op in ("conv2d", "conv2d_f32", "conv2d_i32"):
            ho = (d["H"] + 2 * d["pad"] - d["KH"]) // d["stride"] + 1
            wo = (d["W"] + 2 * d["pad"] - d["KW"]) // d["stride"] + 1
            return 2.0 * d["N"] * d["Co"] * ho * wo * d["Ci"] * d["KH"] * d["KW"]
        if self.op in ("attn_f32", "attn_i32"):
            return 4.0 * d["L"] * d["L"] * d["d"]
        if self.op == "sdpa_f32":
            # two products per (query, key) pair seen: all L^2, or L(L+1)/2 under the mask
            pairs = d["L"] * (d["L"] + 1) / 2 if d["causal"] else d["L"] * d["L"]
            return 4.0 * d["BH"] * pairs * d["d"]
        if self.op in ("minmax_i32", "minmax_i16", "avgpool_i32", "maxpool_f32"):
            return 0.0      # measured in bytes per second (see in_bytes)
        if self.op == "lenet_i32":
            # conv 6@5x5 on 32x32, conv 16@5x5 on 14x14, FC 400-120-84-10
            per_image = 2 * (6 * 28 * 28 * 25 + 16 * 10 * 10 * 150 + 400 * 120 + 120 * 84 + 84 * 10)
            return float(per_image) * d["B"]
        raise ValueError(self.op)

    @property
    def in_bytes(self) -> int:
        """Bytes of input one evaluation reads (the GiB/s metric of the
        min/max and pooling rows)."""
        d = self.dims
        if self.op == "minmax_i32":
            return 4 * d["n"]
        if self.op == "minmax_i16":
            return 2 * d["n"]
        if self.op in ("avgpool_i32", "maxpool_f32"):
            return 4 * d["N"] * d["C"] * d["H"] * d["W"]
        return 0

    def generate(self):
        """Inputs as NumPy arrays, drawn in a fixed order from default_rng(seed)."""
        rng = np.random.default_rng(self.seed)
        d = self.dims
        if self.op == "gemm_i16i32":
            a_shape = (d["batch"], d["M"], d["K"])
            b_shape = (d["batch"], d["K"], d["N"])
            A = ints(rng, a_shape, self.lo, self.hi, np.int16)
            B = ints(rng, b_shape, self.lo, self.hi, np.int16)
            return A, B
        if self.op == "gemm_i32_s24":
            A = ints(rng, (d["batch"], d["M"], d["K"]), self.lo, self.hi, np.int32)
            B = ints(rng, (d["batch"], d["K"], d["N"]), self.lo, self.hi, np.int32)
            return A, B
        if self.op == "conv2d":
            x = ints(rng, (d["N"], d["Ci"], d["H"], d["W"]), self.lo, self.hi, np.int16)
            w = ints(rng, (d["Co"], d["Ci"], d["KH"], d["KW"]), self.lo, self.hi, np.int16)
            return x, w
        if self.op == "conv2d_f32":
            x = normal_f32(rng, (d["N"], d["Ci"], d["H"], d["W"]), 1.0)
            w = normal_f32(rng, (d["Co"], d["Ci"], d["KH"], d["KW"]), 1.0 / np.sqrt(d["Ci"] * d["KH"] * d["KW"]))
            return x, w
        if self.op == "conv2d_i32":
            x = ints(rng, (d["N"], d["Ci"], d["H"], d["W"]), self.lo, self.hi, np.int32)
            w = ints(rng, (d["Co"], d["Ci"], d["KH"], d["KW"]), self.lo, self.hi, np.int32)
            return x, w
        if self.op == "lenet_i32":
            x = ints(rng, (d["B"], 1, 32, 32), 0, 255, np.int32)
            shapes = ((6, 1, 5, 5), (16, 6, 5, 5), (400, 120), (120, 84), (84, 10))
            return (x,) + tuple(ints(rng, s, self.lo, self.hi, np.int32) for s in shapes)
        if self.op == "minmax_i32":
            return (ints(rng, (d["n"],), self.lo, self.hi, np.int32),)
        if self.op == "minmax_i16":
            return (ints(rng, (d["n"],), self.lo, self.hi, np.int16),)
        if self.op == "avgpool_i32":
            return (ints(rng, (d["N"], d["C"], d["H"], d["W"]), self.lo, self.hi, np.int32),)
        if self.op == "maxpool_f32":
            return (normal_f32(rng, (d["N"], d["C"], d["H"], d["W"]), 1.0),)
        if self.op == "attn_f32":
            s = 1.0 / np.sqrt(d["d"])
            return tuple(normal_f32(rng, (d["L"], d["d"]), s) for _ in range(3))
        if self.op == "attn_i32":
            return tuple(ints(rng, (d["L"], d["d"]), self.lo, self.hi, np.int32) for _ in range(3))
        if self.op == "sdpa_f32":
            s = d["d"] ** -0.25
            return tuple(normal_f32(rng, (d["BH"], d["L"], d["d"]), s) for _ in range(3))
        raise ValueError(self.op)


def _gemm(name, op, seed, M, N, K, batch, lo, hi):
    return Workload(name, op, seed, dict(M=M, N=N, K=K, batch=batch), lo, hi, max(-lo, hi))


WORKLOADS = {w.name: w for w in [
    _gemm("gemm_i16_256", "gemm_i16i32", 1, 256, 256, 256, 1, -1024, 1023),
    _gemm("gemm_s24_1024", "gemm_i32_s24", 2, 1024, 1024, 1024, 1, -(1 << 23), (1 << 23) - 1),
    _gemm("gemm_s24_16x512", "gemm_i32_s24", 3, 512, 512, 512, 16, -(1 << 23), (1 << 23) - 1),
    Workload("conv_8x64x56x56_128_3x3", "conv2d", 4,
             dict(N=8, Ci=64, H=56, W=56, Co=128, KH=3, KW=3, stride=1, pad=1), -256, 255, 256),
    Workload("attn_f32_4096x64", "attn_f32", 5, dict(L=4096, d=64)),
    Workload("attn_i32_4096x64", "attn_i32", 6, dict(L=4096, d=64), -64, 63, 64),
    _gemm("gemm_i16_8192", "gemm_i16i32", 7, 8192, 8192, 8192, 1, -256, 255),
    _gemm("gemm_i16_64x2048", "gemm_i16i32", 8, 2048, 2048, 2048, 64, -256, 255),
    Workload("conv_f32_8x64x56x56_128_3x3", "conv2d_f32", 9,
             dict(N=8, Ci=64, H=56, W=56, Co=128, KH=3, KW=3, stride=1, pad=1)),
    Workload("conv_i32_8x64x56x56_128_3x3", "conv2d_i32", 10,
             dict(N=8, Ci=64, H=56, W=56, Co=128, KH=3, KW=3, stride=1, pad=1),
             -(1 << 23), (1 << 23) - 1, 1 << 23),
    Workload("minmax_i32_128Mi", "minmax_i32", 11, dict(n=1 << 27), -(1 << 31), (1 << 31) - 1),
    Workload("minmax_i16_256Mi", "minmax_i16", 12, dict(n=1 << 28), -32768, 32767),
    Workload("avgpool_i32_16x64x224x224", "avgpool_i32", 13, dict(N=16, C=64, H=224, W=224),
             -(1 << 31), (1 << 31) - 1),
    Workload("maxpool_f32_16x64x224x224", "maxpool_f32", 14, dict(N=16, C=64, H=224, W=224)),
    Workload("lenet_i32_b4096", "lenet_i32", 15, dict(B=4096), -3, 3, 3),
    Workload("sdpa_f32_32x4096x64", "sdpa_f32", 16, dict(BH=32, L=4096, d=64, scale=1.0, causal=0)),
    Workload("sdpa_f32_causal_32x4096x64", "sdpa_f32", 17, dict(BH=32, L=4096, d=64, scale=1.0, causal=1)),
]}
