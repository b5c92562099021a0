"""Pins of the CPU oracle against things other than itself.

Brute force in Python integers / exact rationals on tiny inputs, closed forms,
the smul24 extremes (tests/golden), a library special case (NumPy int64
matmul), algebraic invariants, and exact associativity of the integer
attention core.  A plausible slip in the oracle (a dropped term, a sign, a
swapped index, a transposed operand, a missing wrap or mask) fails at least
one of these.
"""
import os

import numpy as np
import pytest

import brute
from oracle import oracle as orc

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _np_gemm_wrap(A, B):
    """NumPy int64 matmul (exact integer loops, no BLAS), low 32 bits."""
    full = np.matmul(A.astype(np.int64), B.astype(np.int64))
    return (full & 0xFFFFFFFF).astype(np.uint32).view(np.int32)


# ----------------------------------------------------------------------------
# packed INT16 -> INT32 GEMM
# ----------------------------------------------------------------------------
TINY = [1, 2, 3, 5, 7, 9]


@pytest.mark.parametrize("M", TINY)
@pytest.mark.parametrize("N", [1, 4, 9])
@pytest.mark.parametrize("K", [1, 3, 8])
def test_gemm_i16_bruteforce_tiny(M, N, K):
    rng = np.random.default_rng(M * 100 + N * 10 + K)
    A = rng.integers(-32768, 32767, (M, K), dtype=np.int16, endpoint=True)
    B = rng.integers(-32768, 32767, (K, N), dtype=np.int16, endpoint=True)
    assert orc.gemm_i16i32(A, B).tolist() == brute.gemm(A.tolist(), B.tolist())


@pytest.mark.parametrize("shape", [(15, 17, 16), (16, 31, 33), (33, 15, 63), (2, 65, 64)])
@pytest.mark.parametrize("batch", [1, 2, 3])
def test_gemm_i16_bruteforce_batched(shape, batch):
    M, N, K = shape
    rng = np.random.default_rng(batch * 7 + M)
    A = rng.integers(-32768, 32767, (batch, M, K), dtype=np.int16, endpoint=True)
    B = rng.integers(-32768, 32767, (batch, K, N), dtype=np.int16, endpoint=True)
    C = orc.gemm_i16i32(A, B)
    for b in range(batch):
        assert C[b].tolist() == brute.gemm(A[b].tolist(), B[b].tolist())


def test_gemm_i16_wraps_mod_2_32():
    # 9 products of (-32768)^2 = 2^30 sum to 9 * 2^30, which wraps.
    A = np.full((1, 9), -32768, np.int16)
    B = np.full((9, 1), -32768, np.int16)
    assert orc.gemm_i16i32(A, B)[0, 0] == brute.wrap32(9 << 30) == 1073741824
    A = np.full((1, 4), -32768, np.int16)
    B = np.full((4, 1), 32767, np.int16)
    assert orc.gemm_i16i32(A, B)[0, 0] == brute.wrap32(-4 * 32768 * 32767)


def test_gemm_i16_closed_forms():
    rng = np.random.default_rng(11)
    K, M, N = 37, 5, 6
    ones_a = np.ones((M, K), np.int16)
    ones_b = np.ones((K, N), np.int16)
    assert (orc.gemm_i16i32(ones_a, ones_b) == K).all()
    B = rng.integers(-300, 300, (K, N), dtype=np.int16)
    c = -7
    A = np.full((M, K), c, np.int16)
    expect = c * B.astype(np.int64).sum(axis=0)
    assert (orc.gemm_i16i32(A, B) == expect[None, :]).all()
    A = rng.integers(-300, 300, (M, K), dtype=np.int16)
    assert (orc.gemm_i16i32(A, np.eye(K, dtype=np.int16)) == A).all()
    assert (orc.gemm_i16i32(np.eye(K, dtype=np.int16), B) == B).all()
    # K = 1: outer product
    a = rng.integers(-1000, 1000, (M, 1), dtype=np.int16)
    b = rng.integers(-1000, 1000, (1, N), dtype=np.int16)
    assert (orc.gemm_i16i32(a, b) == a.astype(np.int64) * b.astype(np.int64)).all()
    assert (orc.gemm_i16i32(np.zeros((M, K), np.int16), B) == 0).all()


def test_gemm_i16_matches_numpy_int64():
    rng = np.random.default_rng(5)
    for (M, N, K) in [(96, 80, 112), (129, 65, 257), (64, 64, 1024)]:
        A = rng.integers(-32768, 32767, (M, K), dtype=np.int16, endpoint=True)
        B = rng.integers(-32768, 32767, (K, N), dtype=np.int16, endpoint=True)
        assert (orc.gemm_i16i32(A, B) == _np_gemm_wrap(A, B)).all()


def test_gemm_i16_invariants():
    rng = np.random.default_rng(9)
    M, N, K = 23, 19, 41
    A1 = rng.integers(-200, 200, (M, K), dtype=np.int16)
    A2 = rng.integers(-200, 200, (M, K), dtype=np.int16)
    B = rng.integers(-200, 200, (K, N), dtype=np.int16)
    lhs = orc.gemm_i16i32((A1 + A2).astype(np.int16), B).astype(np.int64)
    rhs = orc.gemm_i16i32(A1, B).astype(np.int64) + orc.gemm_i16i32(A2, B).astype(np.int64)
    assert ((lhs - rhs) % (1 << 32) == 0).all()
    # (AB)^T = B^T A^T
    assert (orc.gemm_i16i32(A1, B).T == orc.gemm_i16i32(np.ascontiguousarray(B.T),
                                                        np.ascontiguousarray(A1.T))).all()
    # row permutation equivariance
    p = rng.permutation(M)
    assert (orc.gemm_i16i32(A1[p], B) == orc.gemm_i16i32(A1, B)[p]).all()
    # column permutation of B
    q = rng.permutation(N)
    assert (orc.gemm_i16i32(A1, B[:, q]) == orc.gemm_i16i32(A1, B)[:, q]).all()
    # batched == loop of singles
    Ab = rng.integers(-32768, 32767, (3, M, K), dtype=np.int16)
    Bb = rng.integers(-32768, 32767, (3, K, N), dtype=np.int16)
    Cb = orc.gemm_i16i32(Ab, Bb)
    for b in range(3):
        assert (Cb[b] == orc.gemm_i16i32(Ab[b], Bb[b])).all()


# ----------------------------------------------------------------------------
# smul24 INT32 GEMM
# ----------------------------------------------------------------------------
def _golden_smul24():
    rows = []
    with open(os.path.join(GOLDEN, "smul24_extremes.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(tuple(int(t) for t in line.split()))
    return rows


def test_smul24_golden_extremes():
    rows = _golden_smul24()
    assert len(rows) == 7
    for a, b, expect in rows:
        A = np.array([[a]], np.int32)
        B = np.array([[b]], np.int32)
        assert orc.gemm_i32_s24(A, B)[0, 0] == expect, (a, b)
        assert brute.wrap32(brute.sext24(a) * brute.sext24(b)) == expect


@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (3, 5, 7), (9, 4, 16), (17, 15, 33)])
def test_smul24_bruteforce_full_int32_words(M, N, K):
    # Operands use all 32 bits: the contract must ignore bits 24..31.
    rng = np.random.default_rng(M + N + K)
    A = rng.integers(-(1 << 31), (1 << 31) - 1, (M, K), dtype=np.int32, endpoint=True)
    B = rng.integers(-(1 << 31), (1 << 31) - 1, (K, N), dtype=np.int32, endpoint=True)
    assert orc.gemm_i32_s24(A, B).tolist() == brute.gemm(A.tolist(), B.tolist(), brute.sext24)


def test_smul24_masking_and_wrap_numpy():
    rng = np.random.default_rng(3)
    M, N, K = 40, 33, 300
    A = rng.integers(-(1 << 23), (1 << 23) - 1, (2, M, K), dtype=np.int32, endpoint=True)
    B = rng.integers(-(1 << 23), (1 << 23) - 1, (2, K, N), dtype=np.int32, endpoint=True)
    # adding multiples of 2^24 must not change the result
    hi = rng.integers(-64, 63, A.shape, dtype=np.int64) << 24
    A2 = (A.astype(np.int64) + hi).astype(np.int32)
    C = orc.gemm_i32_s24(A, B)
    assert (orc.gemm_i32_s24(A2, B) == C).all()
    # wrapping int64 matmul (products < 2^46, K*2^46 < 2^63)
    for b in range(2):
        ref = (np.matmul(A[b].astype(np.int64), B[b].astype(np.int64)) & 0xFFFFFFFF)
        assert (C[b] == ref.astype(np.uint32).view(np.int32)).all()


# ----------------------------------------------------------------------------
# Conv2D
# ----------------------------------------------------------------------------
CONV_TINY = [
    # N, Ci, H, W, Co, KH, KW, stride, pad
    (1, 1, 3, 3, 1, 3, 3, 1, 1),
    (2, 3, 5, 4, 2, 3, 3, 1, 1),
    (1, 2, 6, 7, 3, 3, 2, 2, 0),
    (2, 2, 5, 5, 2, 1, 1, 1, 0),
    (1, 3, 4, 6, 2, 3, 3, 2, 2),
    (1, 1, 2, 2, 1, 3, 3, 1, 1),
]


@pytest.mark.parametrize("cfg", CONV_TINY)
def test_conv_bruteforce(cfg):
    N, Ci, H, W, Co, KH, KW, s, p = cfg
    rng = np.random.default_rng(sum(cfg))
    x = rng.integers(-32768, 32767, (N, Ci, H, W), dtype=np.int16, endpoint=True)
    w = rng.integers(-32768, 32767, (Co, Ci, KH, KW), dtype=np.int16, endpoint=True)
    ref = brute.conv2d(x.tolist(), w.tolist(), s, p)
    assert orc.conv2d_direct(x, w, s, p).tolist() == ref
    assert orc.conv2d_im2col(x, w, s, p).tolist() == ref


@pytest.mark.parametrize("cfg", [(2, 16, 13, 11, 8, 3, 3, 1, 1), (3, 5, 17, 9, 7, 3, 3, 2, 1),
                                 (1, 8, 12, 12, 4, 5, 5, 1, 2), (2, 4, 9, 10, 6, 2, 3, 3, 0)])
def test_conv_direct_equals_im2col(cfg):
    N, Ci, H, W, Co, KH, KW, s, p = cfg
    rng = np.random.default_rng(len(cfg) + N)
    x = rng.integers(-32768, 32767, (N, Ci, H, W), dtype=np.int16, endpoint=True)
    w = rng.integers(-32768, 32767, (Co, Ci, KH, KW), dtype=np.int16, endpoint=True)
    assert (orc.conv2d_direct(x, w, s, p) == orc.conv2d_im2col(x, w, s, p)).all()


def test_conv_closed_forms():
    rng = np.random.default_rng(1)
    N, C, H, W = 2, 5, 7, 6
    x = rng.integers(-500, 500, (N, C, H, W), dtype=np.int16)
    # centre-delta kernel with pad 1 is the identity
    w = np.zeros((C, C, 3, 3), np.int16)
    for c in range(C):
        w[c, c, 1, 1] = 1
    assert (orc.conv2d_direct(x, w, 1, 1) == x).all()
    # 1x1, pad 0 == per-image GEMM W[Co][Ci] . x[n][Ci][HW]
    Co = 4
    w1 = rng.integers(-500, 500, (Co, C, 1, 1), dtype=np.int16)
    y = orc.conv2d_direct(x, w1, 1, 0)
    for n in range(N):
        ref = w1[:, :, 0, 0].astype(np.int64) @ x[n].reshape(C, -1).astype(np.int64)
        assert (y[n].reshape(Co, -1) == ref).all()
    # all-ones 3x3, pad 1: interior 9*Ci, edges 6*Ci, corners 4*Ci
    ones_x = np.ones((1, C, H, W), np.int16)
    ones_w = np.ones((1, C, 3, 3), np.int16)
    y = orc.conv2d_direct(ones_x, ones_w, 1, 1)[0, 0]
    assert y[0, 0] == y[0, -1] == y[-1, 0] == y[-1, -1] == 4 * C
    assert (y[0, 1:-1] == 6 * C).all() and (y[1:-1, 0] == 6 * C).all()
    assert (y[1:-1, 1:-1] == 9 * C).all()


# ----------------------------------------------------------------------------
# Conv2D on INT32 operands under the smul24 contract, and on FP32 operands
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("cfg", CONV_TINY)
def test_conv_s24_bruteforce_full_int32_words(cfg):
    # every bit of the words is random: bits 24..31 must be ignored
    N, Ci, H, W, Co, KH, KW, s, p = cfg
    rng = np.random.default_rng(sum(cfg) + 7)
    x = rng.integers(-(1 << 31), (1 << 31) - 1, (N, Ci, H, W), dtype=np.int32, endpoint=True)
    w = rng.integers(-(1 << 31), (1 << 31) - 1, (Co, Ci, KH, KW), dtype=np.int32, endpoint=True)
    ref = brute.conv2d(x.tolist(), w.tolist(), s, p, f=lambda v: brute.sext24(int(v)))
    assert orc.conv2d_s24(x, w, s, p).tolist() == ref


def test_conv_s24_contract_invariants():
    rng = np.random.default_rng(5)
    x = rng.integers(-32768, 32767, (2, 6, 9, 8), dtype=np.int16, endpoint=True)
    w = rng.integers(-32768, 32767, (5, 6, 3, 3), dtype=np.int16, endpoint=True)
    # int16 values are their own sext24: equals the INT16 convolution
    y16 = orc.conv2d_direct(x, w, 1, 1)
    y24 = orc.conv2d_s24(x.astype(np.int32), w.astype(np.int32), 1, 1)
    assert (y16 == y24).all()
    # adding multiples of 2^24 to the words changes nothing
    hi = rng.integers(-128, 127, x.shape, endpoint=True).astype(np.int64) << 24
    xm = ((x.astype(np.int64) + hi + (1 << 31)) % (1 << 32) - (1 << 31)).astype(np.int32)
    assert (orc.conv2d_s24(xm, w.astype(np.int32), 1, 1) == y24).all()
    # closed form: all operands 2^23 - 1, 1x1 kernel: Ci * (2^46 - 2^24 + 1) mod 2^32
    Ci = 3
    top = (1 << 23) - 1
    y = orc.conv2d_s24(np.full((1, Ci, 2, 2), top, np.int32), np.full((1, Ci, 1, 1), top, np.int32), 1, 0)
    assert (y == brute.wrap32(Ci * ((1 << 46) - (1 << 24) + 1))).all()
    assert brute.wrap32(Ci * ((1 << 46) - (1 << 24) + 1)) == -3 * 16777215
    # -2^23 everywhere: each product is 2^46 = 0 mod 2^32
    bot = -(1 << 23)
    y = orc.conv2d_s24(np.full((1, 4, 3, 3), bot, np.int32), np.full((2, 4, 3, 3), bot, np.int32), 1, 1)
    assert (y == 0).all()


@pytest.mark.parametrize("cfg", CONV_TINY[:4])
def test_conv_f64_exact_rationals(cfg):
    from fractions import Fraction
    N, Ci, H, W, Co, KH, KW, s, p = cfg
    rng = np.random.default_rng(sum(cfg) + 11)
    x = rng.standard_normal((N, Ci, H, W)).astype(np.float32)
    w = rng.standard_normal((Co, Ci, KH, KW)).astype(np.float32)
    exact = brute.conv2d(x.tolist(), w.tolist(), s, p, f=lambda v: Fraction(float(v)), wrap=False)
    y = orc.conv2d_f64(x, w, s, p)
    # float64 products of float32 inputs are exact; the sums round at most
    # (terms - 1) times by 2^-53 relative to the sum of |products|
    absx = np.abs(x).astype(np.float64)
    absw = np.abs(w).astype(np.float64)
    bound_sum = orc.conv2d_f64(absx.astype(np.float32), absw.astype(np.float32), s, p)
    terms = Ci * KH * KW
    err = np.abs(y - np.array([[[[float(v) for v in r] for r in c] for c in im] for im in exact]))
    assert (err <= terms * 2.0 ** -52 * bound_sum + 1e-300).all()


def test_conv_f64_integer_values_and_numpy():
    rng = np.random.default_rng(9)
    xi = rng.integers(-100, 100, (2, 7, 10, 9), dtype=np.int16, endpoint=True)
    wi = rng.integers(-100, 100, (4, 7, 3, 2), dtype=np.int16, endpoint=True)
    # integer-valued floats: every partial sum is an exact small integer
    y = orc.conv2d_f64(xi.astype(np.float32), wi.astype(np.float32), 2, 1)
    assert (y == orc.conv2d_direct(xi, wi, 2, 1)).all()
    # independent library route: zero-pad, gather windows, float64 tensordot
    x = rng.standard_normal((2, 7, 10, 9)).astype(np.float32)
    w = rng.standard_normal((4, 7, 3, 2)).astype(np.float32)
    s, p = 2, 1
    xp = np.pad(x.astype(np.float64), ((0, 0), (0, 0), (p, p), (p, p)))
    win = np.lib.stride_tricks.sliding_window_view(xp, (3, 2), axis=(2, 3))[:, :, ::s, ::s]
    ref = np.tensordot(win, w.astype(np.float64), axes=([1, 4, 5], [1, 2, 3])).transpose(0, 3, 1, 2)
    y = orc.conv2d_f64(x, w, s, p)
    assert y.shape == ref.shape
    assert np.max(np.abs(y - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_conv_output_shape():
    assert orc.conv_out_shape(8, 64, 56, 56, 128, 3, 3, 1, 1) == (8, 128, 56, 56)
    assert orc.conv_out_shape(1, 1, 7, 6, 1, 3, 2, 2, 0) == (1, 1, 3, 3)


# ----------------------------------------------------------------------------
# Attention core
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("L,d", [(1, 1), (1, 5), (3, 2), (5, 7), (9, 4), (17, 3)])
def test_attn_i32_bruteforce(L, d):
    rng = np.random.default_rng(L * 31 + d)
    Q, K, V = (rng.integers(-(1 << 31), (1 << 31) - 1, (L, d), dtype=np.int32, endpoint=True)
               for _ in range(3))
    ref = brute.attn_int(Q.tolist(), K.tolist(), V.tolist())
    assert orc.attn_i32(Q, K, V).tolist() == ref
    assert orc.attn_i32_assoc(Q, K, V).tolist() == ref


def test_attn_i32_associativity_and_L1():
    rng = np.random.default_rng(2)
    L, d = 257, 64
    Q, K, V = (rng.integers(-64, 63, (L, d), dtype=np.int32, endpoint=True) for _ in range(3))
    assert (orc.attn_i32(Q, K, V) == orc.attn_i32_assoc(Q, K, V)).all()
    # exact int64 reference: |S| <= 64*64*64 = 2^18, |O| <= 257 * 2^18 * 64 < 2^31
    S = Q.astype(np.int64) @ K.astype(np.int64).T
    assert (orc.attn_i32(Q, K, V) == S @ V.astype(np.int64)).all()
    q, k, v = Q[:1], K[:1], V[:1]
    s = int((q.astype(np.int64) * k.astype(np.int64)).sum())
    assert (orc.attn_i32(q, k, v)[0] == s * v[0].astype(np.int64)).all()


@pytest.mark.parametrize("L,d", [(1, 1), (2, 3), (4, 4), (7, 5), (9, 2)])
def test_attn_f64_exact_rational(L, d):
    rng = np.random.default_rng(L + 10 * d)
    Q, K, V = (rng.standard_normal((L, d)).astype(np.float32) for _ in range(3))
    exact = brute.attn_exact(Q.tolist(), K.tolist(), V.tolist())
    R = orc.attn_f64(Q, K, V)
    R2 = orc.attn_f64_assoc(Q, K, V)
    scale = max(abs(float(v)) for row in exact for v in row) or 1.0
    for i in range(L):
        for t in range(d):
            assert abs(R[i, t] - float(exact[i][t])) <= 1e-13 * scale
            assert abs(R2[i, t] - float(exact[i][t])) <= 1e-13 * scale


def test_attn_f64_orders_and_numpy_agree():
    rng = np.random.default_rng(4)
    L, d = 300, 64
    Q, K, V = ((rng.standard_normal((L, d)) / 8).astype(np.float32) for _ in range(3))
    R = orc.attn_f64(Q, K, V)
    R2 = orc.attn_f64_assoc(Q, K, V)
    Rn = (Q.astype(np.float64) @ K.astype(np.float64).T) @ V.astype(np.float64)
    scale = np.abs(R).max()
    assert np.abs(R - R2).max() <= 1e-12 * scale
    assert np.abs(R - Rn).max() <= 1e-12 * scale
    # textbook float32 evaluation stays within its a-priori bound (d + L) u
    F = orc.attn_f32(Q, K, V).astype(np.float64)
    absref = (np.abs(Q).astype(np.float64) @ np.abs(K).astype(np.float64).T) @ np.abs(V)
    u = 2.0 ** -24
    assert (np.abs(F - R) <= (d + L) * u * absref + 1e-30).all()


# ----------------------------------------------------------------------------
# Softmax attention (the SDPA baseline of Table 2's footnote; Discussion)
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("BH,L,d,scale,causal", [(1, 1, 1, 1.0, False), (2, 5, 3, 0.7, True),
                                                 (3, 17, 8, 1.0, False), (2, 33, 16, 0.25, True),
                                                 (1, 64, 64, -0.5, False)])
def test_sdpa_f64_matches_torch_float64(BH, L, d, scale, causal):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(BH + L + d)
    Q, K, V = (rng.standard_normal((BH, L, d)).astype(np.float32) for _ in range(3))
    R = orc.sdpa_f64(Q, K, V, scale, causal)
    T = torch.nn.functional.scaled_dot_product_attention(
        *(torch.from_numpy(a.astype(np.float64)) for a in (Q, K, V)), is_causal=causal, scale=scale).numpy()
    assert np.abs(R - T).max() <= 1e-13 * max(np.abs(T).max(), 1.0)


def test_sdpa_f64_closed_forms():
    rng = np.random.default_rng(7)
    L, d = 9, 4
    Q, K, V = (rng.standard_normal((1, L, d)).astype(np.float32) for _ in range(3))
    V64 = V[0].astype(np.float64)
    # scale 0: uniform weights over the keys a query sees (all keys, or the prefix)
    R = orc.sdpa_f64(Q, K, V, 0.0, False)[0]
    assert np.abs(R - V64.mean(axis=0)).max() <= 1e-14
    R = orc.sdpa_f64(Q, K, V, 0.0, True)[0]
    prefix = np.cumsum(V64, axis=0) / np.arange(1, L + 1)[:, None]
    assert np.abs(R - prefix).max() <= 1e-14
    # the first query under the mask sees only key 0; one key is the identity
    assert (orc.sdpa_f64(Q, K, V, 3.0, True)[0, 0] == V64[0]).all()
    assert (orc.sdpa_f64(Q[:, :1], K[:, :1], V[:, :1], 3.0, False)[0, 0] == V64[0]).all()
    # Q = t I and K a permutation matrix: the score of query i is t on key
    # pi(i) and 0 elsewhere, so O[i] = (e^t V[pi(i)] + sum_{j != pi(i)} V[j]) / (e^t + L - 1)
    n, t = 6, 2.5
    perm = np.array([3, 0, 5, 1, 4, 2])
    Qm = (t * np.eye(n)).astype(np.float32)[None]
    Km = np.eye(n, dtype=np.float32)[perm][None]        # row i of K is e_perm(i)
    Vm = rng.standard_normal((1, n, n)).astype(np.float32)
    R = orc.sdpa_f64(Qm, Km, Vm, 1.0, False)[0]
    Vd = Vm[0].astype(np.float64)
    inv = np.argsort(perm)                               # key j carries e_perm(j); query i matches j = inv[i]
    for i in range(n):
        j = inv[i]
        want = (np.exp(t) * Vd[j] + (Vd.sum(axis=0) - Vd[j])) / (np.exp(t) + n - 1)
        assert np.abs(R[i] - want).max() <= 1e-14


def test_sdpa_f64_invariants():
    rng = np.random.default_rng(8)
    BH, L, d = 3, 20, 6
    Q, K, V = (rng.standard_normal((BH, L, d)).astype(np.float32) for _ in range(3))
    for causal in (False, True):
        R = orc.sdpa_f64(Q, K, V, 0.8, causal)
        # heads are independent
        for b in range(BH):
            assert np.array_equal(R[b], orc.sdpa_f64(Q[b:b + 1], K[b:b + 1], V[b:b + 1], 0.8, causal)[0])
        # a shift of every key by u adds q.u to every score of a query: no change
        u = np.float32(0.5) * np.ones(d, np.float32)
        Rs = orc.sdpa_f64(Q, K + u, V, 0.8, causal)
        assert np.abs(R - Rs).max() <= 1e-5 * np.abs(R).max()
        # the weights are a convex combination: each output within V's column range
        for b in range(BH):
            for i in range(L):
                seen = V[b, : i + 1] if causal else V[b]
                assert (R[b, i] >= seen.min(axis=0) - 1e-12).all() and (R[b, i] <= seen.max(axis=0) + 1e-12).all()
    # without the mask, permuting keys and values together changes nothing
    perm = rng.permutation(L)
    R = orc.sdpa_f64(Q, K, V, 0.8, False)
    Rp = orc.sdpa_f64(Q, K[:, perm], V[:, perm], 0.8, False)
    assert np.abs(R - Rp).max() <= 1e-13 * np.abs(R).max()
    # under the mask, query i ignores keys after it: changing the last key
    # and value changes the last row only
    K2, V2 = K.copy(), V.copy()
    K2[:, -1] += 3.0
    V2[:, -1] -= 2.0
    R1 = orc.sdpa_f64(Q, K, V, 0.8, True)
    R2 = orc.sdpa_f64(Q, K2, V2, 0.8, True)
    assert np.array_equal(R1[:, :-1], R2[:, :-1])
    assert not np.array_equal(R1[:, -1], R2[:, -1])


# ----------------------------------------------------------------------------
# Min/max, 2x2 average and max pooling (Table 2 rows)
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("n", [1, 2, 7, 1000, 65537])
def test_minmax_against_numpy(n):
    rng = np.random.default_rng(n)
    for dt, lo, hi in ((np.int32, -(1 << 31), (1 << 31) - 1), (np.int16, -32768, 32767)):
        x = rng.integers(lo, hi, n, dtype=dt, endpoint=True)
        assert orc.minmax(x).tolist() == [int(x.min()), int(x.max())]
    # the extremes sit anywhere, including first and last
    x = np.zeros(9, np.int32)
    x[0], x[-1] = -(1 << 31), (1 << 31) - 1
    assert orc.minmax(x).tolist() == [-(1 << 31), (1 << 31) - 1]
    x = np.full(5, -3, np.int16)
    assert orc.minmax(x).tolist() == [-3, -3]


@pytest.mark.parametrize("shape", [(1, 1, 2, 2), (2, 3, 6, 8), (1, 2, 7, 9), (3, 1, 5, 4)])
def test_pools_against_numpy(shape):
    N, C, H, W = shape
    rng = np.random.default_rng(H * W + C)
    x = rng.integers(-(1 << 31), (1 << 31) - 1, shape, dtype=np.int32, endpoint=True)
    Ho, Wo = H // 2, W // 2
    win = x[:, :, :2 * Ho, :2 * Wo].astype(np.int64).reshape(N, C, Ho, 2, Wo, 2)
    assert (orc.avgpool2_i32(x) == win.sum(axis=(3, 5)) // 4).all()   # numpy floor division
    xf = rng.standard_normal(shape).astype(np.float32)
    winf = xf[:, :, :2 * Ho, :2 * Wo].reshape(N, C, Ho, 2, Wo, 2)
    assert (orc.maxpool2_f32(xf) == winf.max(axis=(3, 5))).all()


def test_pool_closed_forms():
    # constant input: the average and the maximum are the constant
    x = np.full((1, 2, 4, 6), -123456789, np.int32)
    assert (orc.avgpool2_i32(x) == -123456789).all()
    assert (orc.maxpool2_f32(np.full((1, 1, 4, 4), 2.5, np.float32)) == 2.5).all()
    # floor of a negative quarter, exact sum beyond int32
    x = np.array([[[[1, 2], [3, -7]]]], np.int32)
    assert orc.avgpool2_i32(x)[0, 0, 0, 0] == -1
    big = (1 << 31) - 1
    assert orc.avgpool2_i32(np.full((1, 1, 2, 2), big, np.int32))[0, 0, 0, 0] == big
    assert orc.avgpool2_i32(np.full((1, 1, 2, 2), -big - 1, np.int32))[0, 0, 0, 0] == -big - 1
    # the maximum of one window picks each position in turn
    for pos in range(4):
        v = np.zeros(4, np.float32)
        v[pos] = 1.0
        assert orc.maxpool2_f32(v.reshape(1, 1, 2, 2))[0, 0, 0, 0] == 1.0


# ----------------------------------------------------------------------------
# LeNet-5-shaped INT32 pipeline (Results: end-to-end CNN)
# ----------------------------------------------------------------------------
def _lenet_inputs(rng, B, lo=-300, hi=300):
    x = rng.integers(0, 255, (B, 1, 32, 32), dtype=np.int32, endpoint=True)
    ws = [rng.integers(lo, hi, s, dtype=np.int32, endpoint=True)
          for s in ((6, 1, 5, 5), (16, 6, 5, 5), (400, 120), (120, 84), (84, 10))]
    return x, ws


def test_lenet_bruteforce_single_images():
    # layer-by-layer Python integers; the weights are large enough that the
    # FC sums wrap mod 2^32 and later layers read only the low 24 bits
    rng = np.random.default_rng(21)
    x, ws = _lenet_inputs(rng, 2)
    got = orc.lenet_i32(x, *ws)
    for b in range(2):
        ref = brute.lenet_i32(x[b].tolist(), ws[0].tolist(), ws[1].tolist(),
                              ws[2].tolist(), ws[3].tolist(), ws[4].tolist())
        assert got[b].tolist() == ref


def test_lenet_batch_is_per_image():
    rng = np.random.default_rng(22)
    x, ws = _lenet_inputs(rng, 5, -3, 3)
    full = orc.lenet_i32(x, *ws)
    for b in range(5):
        assert (orc.lenet_i32(x[b:b + 1], *ws)[0] == full[b]).all()
