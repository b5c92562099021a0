"""Definitional brute force in Python integers (and exact rationals).

Independent of the C oracle: used by the CPU tests to pin the oracle on tiny
inputs.  Every function is the textbook definition with arbitrary-precision
Python arithmetic, reduced to two's-complement 32 bits at the very end.
"""
from __future__ import annotations

from fractions import Fraction


def wrap32(v: int) -> int:
    v &= 0xFFFFFFFF
    return v - (1 << 32) if v >= (1 << 31) else v


def sext24(x: int) -> int:
    u = x & 0xFFFFFF
    return u - (1 << 24) if u >= (1 << 23) else u


def gemm(A, B, f=lambda v: v):
    """A: list of rows (M x K), B: (K x N); f maps each operand first."""
    M, K = len(A), len(A[0]) if A else 0
    N = len(B[0]) if B else 0
    return [[wrap32(sum(f(int(A[i][k])) * f(int(B[k][j])) for k in range(K)))
             for j in range(N)] for i in range(M)]


def conv2d(x, w, stride, pad, f=int, wrap=True):
    """x [N][Ci][H][W], w [Co][Ci][KH][KW] nested lists -> y [N][Co][Ho][Wo].
    f maps each operand first (int, sext24 of an int word, or Fraction for
    exact real arithmetic); wrap reduces the exact sum mod 2^32."""
    N, Ci, H, W = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    Co, KH, KW = len(w), len(w[0][0]), len(w[0][0][0])
    Ho = (H + 2 * pad - KH) // stride + 1
    Wo = (W + 2 * pad - KW) // stride + 1
    y = [[[[0] * Wo for _ in range(Ho)] for _ in range(Co)] for _ in range(N)]
    for n in range(N):
        for co in range(Co):
            for oh in range(Ho):
                for ow in range(Wo):
                    s = 0
                    for ci in range(Ci):
                        for kh in range(KH):
                            for kw in range(KW):
                                ih, iw = oh * stride - pad + kh, ow * stride - pad + kw
                                if 0 <= ih < H and 0 <= iw < W:
                                    s += f(x[n][ci][ih][iw]) * f(w[co][ci][kh][kw])
                    y[n][co][oh][ow] = wrap32(s) if wrap else s
    return y


def attn_int(Q, K, V):
    """(Q K^T) V in exact integers, reduced mod 2^32."""
    L, d = len(Q), len(Q[0])
    S = [[sum(int(Q[i][t]) * int(K[j][t]) for t in range(d)) for j in range(L)] for i in range(L)]
    return [[wrap32(sum(S[i][j] * int(V[j][t]) for j in range(L))) for t in range(d)]
            for i in range(L)]


def attn_exact(Q, K, V):
    """(Q K^T) V as exact rationals of the float inputs."""
    L, d = len(Q), len(Q[0])
    q = [[Fraction(float(v)) for v in r] for r in Q]
    k = [[Fraction(float(v)) for v in r] for r in K]
    v = [[Fraction(float(x)) for x in r] for r in V]
    S = [[sum(q[i][t] * k[j][t] for t in range(d)) for j in range(L)] for i in range(L)]
    return [[sum(S[i][j] * v[j][t] for j in range(L)) for t in range(d)] for i in range(L)]


def lenet_i32(x, w1, w2, f1, f2, f3):
    """The LeNet-5-shaped INT32 pipeline for one image, layer by layer in
    Python integers: smul24 operand reading, wrap to int32 after every
    layer, ReLU, floor average of 2x2 windows."""
    s24 = lambda v: sext24(int(v))

    def relu_pool(y):
        C, H, W = len(y), len(y[0]), len(y[0][0])
        return [[[(max(y[c][2 * i][2 * j], 0) + max(y[c][2 * i][2 * j + 1], 0) +
                   max(y[c][2 * i + 1][2 * j], 0) + max(y[c][2 * i + 1][2 * j + 1], 0)) // 4
                  for j in range(W // 2)] for i in range(H // 2)] for c in range(C)]

    a = conv2d([x], w1, 1, 0, f=s24)[0]
    a = relu_pool(a)
    a = conv2d([a], w2, 1, 0, f=s24)[0]
    a = relu_pool(a)
    v = [a[c][i][j] for c in range(16) for i in range(5) for j in range(5)]
    for f, last in ((f1, False), (f2, False), (f3, True)):
        v = [wrap32(sum(s24(v[k]) * s24(f[k][n]) for k in range(len(v)))) for n in range(len(f[0]))]
        if not last:
            v = [max(t, 0) for t in v]
    return v
