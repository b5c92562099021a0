"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Integer results must match bit for bit; FP32 attention must satisfy
max|O - R| / max|R| <= 1e-4 against the float64 reference R.  Small shapes
span several tiles and ragged tails on every route; the full-size workloads
are checked on oracle-computed sampled rows and with Freivalds' check
C r == A (B r), exact in int64, which covers every output element.
"""
import sys
import zlib

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2606_09905_amd import qx
from paper_2606_09905_amd.workloads import WORKLOADS

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def dev(a: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t) -> np.ndarray:
    torch.cuda.synchronize()
    return t.cpu().numpy()


def run_exec(ex, inputs):
    out = ex.run([dev(a) for a in inputs])
    return host(out)


def same(got, ref, what=""):
    """Bit-exact comparison that reports a short summary instead of arrays."""
    got, ref = np.asarray(got), np.asarray(ref)
    assert got.shape == ref.shape, f"{what} shape {got.shape} != {ref.shape}"
    bad = np.flatnonzero(got.reshape(-1) != ref.reshape(-1))
    if bad.size:
        i = np.unravel_index(bad[0], got.shape)
        raise AssertionError(f"{what} {bad.size} of {got.size} elements differ; first at {i}: "
                             f"got {got[i]} expected {ref[i]}")


def rand_int(rng, shape, b, dtype):
    return rng.integers(-b, b, size=shape, dtype=np.int64, endpoint=True).astype(dtype)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    qx.lib()
    yield
    qx.lib().qx_release_cache()


# ---------------------------------------------------------------------------
# INT16 GEMM, every route
# ---------------------------------------------------------------------------
GEMM_SHAPES = [  # M, N, K, batch
    (1, 1, 1, 1), (3, 5, 7, 1), (15, 17, 16, 2), (33, 65, 127, 1), (128, 128, 64, 1),
    (129, 257, 200, 3), (256, 256, 256, 1), (200, 136, 64, 2), (64, 72, 520, 1),
    (100, 200, 600, 3),   # vector-ALU routes: 4 K slices per batch (grid z = batch x slices)
]
I16_ROUTES = [  # route, bound
    ("i8_direct", 127), ("f16_exact", 256), ("f16_exact", 1024), ("f16_exact", 2048),
    ("i8_karatsuba", 8127), ("i8_offset4", 32768), ("valu_dot2", 32768),
]


@pytest.mark.parametrize("route,bound", I16_ROUTES)
@pytest.mark.parametrize("shape", GEMM_SHAPES)
def test_gemm_i16_routes(route, bound, shape):
    M, N, K, batch = shape
    b_eff = bound if route != "f16_exact" or bound != 2048 else 2048
    bb = 16 if (route == "f16_exact" and bound == 2048) else bound  # keep chunk >= 16
    rng = np.random.default_rng(zlib.crc32(repr((route, bound, shape)).encode()))
    A = rand_int(rng, (batch, M, K), min(b_eff, 32767), np.int16)
    B = rand_int(rng, (batch, K, N), min(bb, 32767), np.int16)
    with qx.Executor.gemm_i16i32(M, N, K, batch, bound, bb, route) as ex:
        assert ex.plan()["route_name"] == route
        got = run_exec(ex, (A, B))
    ref = orc.gemm_i16i32(A, B)
    same(got, ref)


@pytest.mark.parametrize("route,bound", I16_ROUTES)
def test_gemm_i16_extremes(route, bound):
    # All operands at the contract's most negative value: largest products,
    # fp16 partial sums exactly at chunk * bound^2, wrap-around for full int16.
    b = min(bound, 32768)
    bb = 16 if (route == "f16_exact" and bound == 2048) else b
    for K in (64, 1000, 4096):
        A = np.full((1, 64, K), -b, np.int16)
        B = np.full((1, K, 64), -bb, np.int16)
        A[0, ::3, ::2] = min(b, 32767)          # mix in the most positive value
        with qx.Executor.gemm_i16i32(64, 64, K, 1, bound, bb, route) as ex:
            got = run_exec(ex, (A, B))
        same(got, orc.gemm_i16i32(A, B), str((route, K)))


@pytest.mark.parametrize("shape,bound", [
    ((300, 520, 200, 2), 256), ((1000, 300, 136, 1), 128), ((257, 129, 1000, 1), 300),
    ((64, 1024, 4096, 1), 256), ((513, 2000, 520, 3), 512), ((128, 25088, 576, 1), 256),
])
def test_gemm_i16_encode_nt_path(shape, bound):
    # Large enough for the encode + direct-to-LDS route; ragged in M, N, K;
    # chunks of 256, 1024, 128 (bound 300) and 64 (bound 512) K elements.
    M, N, K, batch = shape
    rng = np.random.default_rng(zlib.crc32(repr((shape, bound)).encode()))
    A = rand_int(rng, (batch, M, K), bound, np.int16)
    B = rand_int(rng, (batch, K, N), bound, np.int16)
    A[0, 0, :] = -bound
    B[0, :, 0] = -bound
    with qx.Executor.gemm_i16i32(M, N, K, batch, bound, bound) as ex:
        plan = ex.plan()
        assert plan["route_name"] == "f16_exact" and plan["kernels"] == 3, plan
        got = run_exec(ex, (A, B))
    same(got, orc.gemm_i16i32(A, B))


I8NT_SHAPES = [  # M, N, K, batch: large enough for the limb-plane encode + NT route
    (300, 520, 200, 2), (257, 129, 1000, 1), (64, 1024, 4096, 1), (513, 2000, 520, 3),
    (1024, 1024, 1024, 1), (33, 700, 999, 2), (700, 900, 1000, 1),
]


@pytest.mark.parametrize("route,bound", [("i8_direct", 127), ("i8_karatsuba", 8127),
                                         ("i8_offset4", 32768)])
@pytest.mark.parametrize("shape", I8NT_SHAPES)
def test_gemm_i16_limb_encode_nt_path(route, bound, shape):
    # Ragged M, N and K (odd K also takes the encoders' element-wise loads);
    # for offset4 the encoders also produce the sums of the rank-1 correction.
    M, N, K, batch = shape
    rng = np.random.default_rng(zlib.crc32(repr((route, shape)).encode()))
    A = rand_int(rng, (batch, M, K), min(bound, 32767), np.int16)
    B = rand_int(rng, (batch, K, N), min(bound, 32767), np.int16)
    A[0, 0, :] = -min(bound, 32768)
    B[0, :, 0] = -min(bound, 32768)
    with qx.Executor.gemm_i16i32(M, N, K, batch, bound, bound, route) as ex:
        plan = ex.plan()
        assert plan["route_name"] == route
        # K sliced over workgroups: a clearing launch comes first
        assert plan["kernels"] == (3 if plan["k_splits"] else 2), plan
        got = run_exec(ex, (A, B))
    same(got, orc.gemm_i16i32(A, B), str((route, shape)))


@pytest.mark.parametrize("shape", I8NT_SHAPES + [(512, 512, 512, 16), (300, 200, 5000, 1), (64, 64, 8448, 1)])
def test_gemm_s24_encode_nt_path(shape):
    # The last two slice K over workgroups: 12 slices of 7 K tiles with 2 in
    # the last, and 15 slices of 9 with 6 in the last.
    M, N, K, batch = shape
    rng = np.random.default_rng(zlib.crc32(repr(("s24", shape)).encode()))
    A = rng.integers(-(1 << 31), (1 << 31) - 1, (batch, M, K), dtype=np.int32, endpoint=True)
    B = rng.integers(-(1 << 31), (1 << 31) - 1, (batch, K, N), dtype=np.int32, endpoint=True)
    A[0, 0, :] = -(1 << 23)
    B[0, :, 0] = (1 << 23) - 1
    with qx.Executor.gemm_i32_s24(M, N, K, batch) as ex:
        plan = ex.plan()
        assert plan["route_name"] == "s24_i8limb", plan
        assert plan["kernels"] == (3 if plan["k_splits"] else 2), plan
        got = run_exec(ex, (A, B))
    same(got, orc.gemm_i32_s24(A, B), str(shape))


@pytest.mark.parametrize("shape,groups", [((2048, 2048, 2048, 17), [9, 8]), ((3000, 2900, 3000, 9), [5, 4])])
def test_gemm_batch_groups(shape, groups):
    # Encoded operands beyond 256 MiB: the batches run in groups (the last
    # one short), each encoded and then contracted.  Sampled rows of the
    # batches at every group boundary against the oracle, Freivalds' check
    # on every batch, and a second run of the same executor.
    M, N, K, batch = shape
    rng = np.random.default_rng(zlib.crc32(repr(("groups", shape)).encode()))
    A = rand_int(rng, (batch, M, K), 256, np.int16)
    B = rand_int(rng, (batch, K, N), 256, np.int16)
    A[0, 0, :] = -256
    B[-1, :, -1] = -256
    with qx.Executor.gemm_i16i32(M, N, K, batch, 256, 256) as ex:
        plan = ex.plan()
        assert plan["kernels"] == 3 * len(groups), plan
        C = run_exec(ex, (A, B))
        C2 = run_exec(ex, (A, B))
    same(C2, C, "second run")
    edges = sorted({0, groups[0] - 1, groups[0], batch - 1})
    for b in edges:
        rows = np.unique(np.concatenate([np.sort(rng.choice(M, size=6, replace=False)), [0, M - 1]]))
        same(C[b, rows], orc.gemm_i16i32(np.ascontiguousarray(A[b, rows]), B[b]), f"batch {b}")
    assert freivalds(A, B, C, trials=2)


def test_f16_exact_mixed_magnitudes():
    # Products alternating between 2^16 and 1 inside one fp32 partial sum:
    # a narrow internal adder would lose the small terms.
    K = 8192
    A = np.ones((1, 64, K), np.int16)
    B = np.ones((1, K, 64), np.int16)
    A[0, :, ::2] = -256
    B[0, ::2, :] = -256
    A[0, 5, 1::4] = 255
    with qx.Executor.gemm_i16i32(64, 64, K, 1, 256, 256, "f16_exact") as ex:
        got = run_exec(ex, (A, B))
    same(got, orc.gemm_i16i32(A, B))


@pytest.mark.parametrize("K", [256, 4096, 4100])
def test_bf16_operands_extremes(K):
    # bf16-encoded operands (bounds <= 256): +-256, +-255 and +-1 in patterns
    # that make full 256-element partial sums reach 2^24 exactly and mix
    # 2^16-sized products with unit ones.
    M = N = 64 if K >= 4096 else 1024
    vals = np.array([-256, 256, -255, 255, -1, 1], np.int16)
    rng = np.random.default_rng(K)
    A = vals[rng.integers(0, 6, (1, M, K))]
    B = vals[rng.integers(0, 6, (1, K, N))]
    A[0, 0, :] = -256
    B[0, :, 0] = -256
    A[0, 1, :] = 256
    B[0, :, 1] = -256
    with qx.Executor.gemm_i16i32(M, N, K, 1, 256, 256) as ex:
        plan = ex.plan()
        assert plan["route_name"] == "f16_exact" and plan["operand_format"] == 1, plan
        got = run_exec(ex, (A, B))
    want = orc.gemm_i16i32(A, B)
    assert want[0, 0, 0] == K * 65536 and want[0, 1, 1] == -K * 65536
    same(got, want)


def test_gemm_i16_oneshot_and_empty():
    rng = np.random.default_rng(3)
    A = rand_int(rng, (96, 80), 1024, np.int16)
    B = rand_int(rng, (80, 112), 1024, np.int16)
    C = host(qx.qgemm_i16i32(dev(A), dev(B), 1024, 1024))
    same(C, orc.gemm_i16i32(A, B))
    # K == 0 -> zeros; M == 0 -> empty
    Z = qx.qgemm_i16i32(torch.empty((5, 0), dtype=torch.int16, device="cuda"),
                        torch.empty((0, 7), dtype=torch.int16, device="cuda"))
    assert Z.shape == (5, 7) and int(Z.abs().sum()) == 0
    E = qx.qgemm_i16i32(torch.empty((0, 9), dtype=torch.int16, device="cuda"),
                        torch.ones((9, 4), dtype=torch.int16, device="cuda"))
    assert E.shape == (0, 4)


# ---------------------------------------------------------------------------
# smul24 GEMM
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("route", ["s24_i8limb", "s24_valu"])
@pytest.mark.parametrize("shape", GEMM_SHAPES)
def test_gemm_s24_routes(route, shape):
    M, N, K, batch = shape
    rng = np.random.default_rng(M * 7 + N + K)
    # full 32-bit words: bits 24..31 must be ignored
    A = rng.integers(-(1 << 31), (1 << 31) - 1, (batch, M, K), dtype=np.int32, endpoint=True)
    B = rng.integers(-(1 << 31), (1 << 31) - 1, (batch, K, N), dtype=np.int32, endpoint=True)
    with qx.Executor.gemm_i32_s24(M, N, K, batch, route) as ex:
        got = run_exec(ex, (A, B))
    same(got, orc.gemm_i32_s24(A, B))


@pytest.mark.parametrize("route", ["s24_i8limb", "s24_valu"])
def test_gemm_s24_extremes_and_accumulator_wrap(route):
    # -2^23 everywhere: all limbs -128, each limb product 2^14; with K = 2^17
    # the int32 accumulators of the matrix cores pass 2^31 and must wrap.
    K = 1 << 17
    A = np.full((1, 32, K), -(1 << 23), np.int32)
    B = np.full((1, K, 32), -(1 << 23), np.int32)
    A[0, 1, :] = (1 << 23) - 1
    B[0, :, 2] = 0x01000005
    with qx.Executor.gemm_i32_s24(32, 32, K, 1, route) as ex:
        got = run_exec(ex, (A, B))
    same(got, orc.gemm_i32_s24(A, B))


SKINNY_S24_SHAPES = [  # M, N, K, batch: at most 128 columns, at least 1024 rows over the batch
    (4096, 120, 400, 1), (4096, 10, 84, 1), (1100, 84, 120, 1), (1030, 127, 37, 2),
    (2000, 9, 130, 1), (1500, 128, 1, 1), (1024, 128, 4096, 1), (600, 65, 64, 3),
    # fewer than 8 columns: 4, 2 or 1 column per workgroup, the last group
    # shifted left over the previous one
    (1500, 7, 37, 1), (1100, 5, 64, 2), (1024, 3, 100, 1), (1030, 2, 33, 1), (2048, 1, 96, 1),
]


@pytest.mark.parametrize("route", ["auto", "s24_valu"])
@pytest.mark.parametrize("shape", SKINNY_S24_SHAPES)
def test_gemm_s24_skinny(route, shape):
    # One row per thread, eight columns per workgroup: ragged rows (M not a
    # multiple of 256), ragged column groups, K not a multiple of 4 (the
    # element-wise A loads) or of 64 (a short last B stage), batches.
    M, N, K, batch = shape
    rng = np.random.default_rng(zlib.crc32(repr(("skinny", shape)).encode()))
    A = rng.integers(-(1 << 31), (1 << 31) - 1, (batch, M, K), dtype=np.int32, endpoint=True)
    B = rng.integers(-(1 << 31), (1 << 31) - 1, (batch, K, N), dtype=np.int32, endpoint=True)
    A[0, 0, :] = -(1 << 23)
    B[0, :, 0] = -(1 << 23)
    with qx.Executor.gemm_i32_s24(M, N, K, batch, route) as ex:
        plan = ex.plan()
        if route == "s24_valu" or M * N * K * batch <= 1 << 26:
            assert plan["route_name"] == "s24_valu" and plan["tile_n"] == 8, plan
        got = run_exec(ex, (A, B))
    same(got, orc.gemm_i32_s24(A, B), str(shape))


# ---------------------------------------------------------------------------
# Conv2D
# ---------------------------------------------------------------------------
CONV_CASES = [  # N, Ci, H, W, Co, KH, KW, stride, pad, bound
    (1, 1, 3, 3, 1, 3, 3, 1, 1, 256), (2, 3, 9, 7, 5, 3, 3, 1, 1, 256),
    (1, 16, 13, 11, 40, 3, 3, 2, 1, 1024), (2, 8, 12, 12, 4, 5, 5, 1, 2, 127),
    (3, 5, 17, 9, 7, 3, 2, 3, 0, 0), (1, 64, 20, 20, 130, 1, 1, 1, 0, 8000),
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv(case):
    N, Ci, H, W, Co, KH, KW, s, p, b = case
    rng = np.random.default_rng(sum(case))
    bx = b if b else 32767
    x = rand_int(rng, (N, Ci, H, W), bx, np.int16)
    w = rand_int(rng, (Co, Ci, KH, KW), bx, np.int16)
    y = host(qx.conv2d_gemm(dev(x), dev(w), s, p, b, b))
    same(y, orc.conv2d_direct(x, w, s, p))


CONV_NT_CASES = [  # large enough for the encode + NT route
    (2, 32, 30, 28, 64, 3, 3, 1, 1, 256), (4, 32, 40, 36, 128, 3, 3, 2, 1, 128),
    (2, 16, 24, 20, 64, 5, 5, 1, 2, 256), (4, 12, 30, 30, 64, 3, 3, 1, 1, 256),
    (8, 64, 20, 20, 96, 1, 1, 1, 0, 256),
]


@pytest.mark.parametrize("case", CONV_NT_CASES)
def test_conv_encode_nt_path(case):
    N, Ci, H, W, Co, KH, KW, s, p, b = case
    rng = np.random.default_rng(zlib.crc32(repr(case).encode()))
    x = rand_int(rng, (N, Ci, H, W), b, np.int16)
    w = rand_int(rng, (Co, Ci, KH, KW), b, np.int16)
    x[0, :, 0, 0] = -b
    w[0, :, 0, 0] = -b
    with qx.Executor.conv2d(N, Ci, H, W, Co, KH, KW, s, p, b, b) as ex:
        plan = ex.plan()
        assert plan["route_name"] == "f16_exact", plan
        assert plan["kernels"] == (2 if Ci % 64 == 0 else 3), plan
        y = run_exec(ex, (x, w))
    same(y, orc.conv2d_direct(x, w, s, p))


CONV_IMPLICIT_CASES = [  # C_in a multiple of 64: implicit lowering from the NHWC copy
    (2, 64, 30, 26, 100, 3, 3, 1, 1, 256), (3, 128, 17, 19, 64, 3, 3, 2, 1, 256),
    (2, 64, 23, 23, 64, 7, 7, 2, 3, 128), (1, 192, 14, 14, 256, 3, 3, 1, 0, 256),
    (4, 64, 9, 33, 48, 5, 3, 1, 2, 255), (8, 256, 32, 32, 64, 1, 1, 2, 0, 256),
    # 128 channels (two K tiles per tap), stride 2, 1x1 and 5x5 kernels,
    # pixel tiles ending mid-row and short images
    (2, 128, 12, 10, 70, 3, 3, 1, 1, 256), (8, 64, 9, 24, 64, 3, 3, 2, 1, 256),
    (12, 64, 16, 16, 130, 1, 1, 1, 0, 256), (1, 64, 19, 23, 64, 5, 5, 1, 2, 255),
]


@pytest.mark.parametrize("case", CONV_IMPLICIT_CASES)
def test_conv_implicit_lowering(case):
    # Ragged C_out and pixel counts, strides 1 and 2, pads 0..3, square and
    # rectangular kernels; extreme values on the image border and in every tap.
    N, Ci, H, W, Co, KH, KW, s, p, b = case
    rng = np.random.default_rng(zlib.crc32(repr(("impl", case)).encode()))
    x = rand_int(rng, (N, Ci, H, W), b, np.int16)
    w = rand_int(rng, (Co, Ci, KH, KW), b, np.int16)
    x[0, :, 0, :] = -b
    x[-1, :, :, -1] = -b
    w[0] = -b
    with qx.Executor.conv2d(N, Ci, H, W, Co, KH, KW, s, p, b, b) as ex:
        plan = ex.plan()
        assert plan["route_name"] == "f16_exact" and plan["kernels"] == 2, plan
        y = run_exec(ex, (x, w))
        y2 = run_exec(ex, (x, w))
    ref = orc.conv2d_direct(x, w, s, p)
    same(y, ref, str(case))
    same(y2, ref, "second run " + str(case))


# ---------------------------------------------------------------------------
# Attention core
# ---------------------------------------------------------------------------
def normwise(O, R):
    return float(np.abs(O.astype(np.float64) - R).max() / max(np.abs(R).max(), 1e-300))


@pytest.mark.parametrize("L,d", [(1, 32), (31, 64), (32, 64), (100, 64), (257, 32), (300, 128),
                                 (1024, 64), (77, 96), (100, 48)])
def test_attn_f32(L, d):
    rng = np.random.default_rng(L + d)
    Q, K, V = ((rng.standard_normal((L, d)) / np.sqrt(d)).astype(np.float32) for _ in range(3))
    O = host(qx.attn_core(dev(Q), dev(K), dev(V)))
    R = orc.attn_f64(Q, K, V)
    assert normwise(O, R) <= 1e-4
    # elementwise a-priori bound of fp32 evaluation in any order: (d + L) u |Q||K|^T|V|
    absref = (np.abs(Q).astype(np.float64) @ np.abs(K).astype(np.float64).T) @ np.abs(V)
    assert (np.abs(O - R) <= (d + L) * 2.0 ** -24 * absref + 1e-30).all()


@pytest.mark.parametrize("L,d,b", [(1, 32, 64), (33, 64, 64), (128, 64, 127), (300, 32, 100),
                                   (1024, 128, 127), (257, 96, 64), (1000, 64, 64), (4100, 128, 100),
                                   (5000, 32, 127), (2049, 64, 127), (4096, 64, 127), (63, 32, 127),
                                   (64, 64, 1), (65, 64, 127), (8191, 64, 64)])
def test_attn_i32_mfma(L, d, b):
    # d in {32, 64}: the prep launch plus the streaming kernel (eight
    # waves: two query tiles x four key parts per split, joined in LDS;
    # query tiles past L, ragged last split, zero-padded keys; one split ->
    # plain stores); d = 128: the
    # prep plus the LDS-resident splits; d = 96: the LDS-staged loop kernel
    rng = np.random.default_rng(L * 3 + d + b)
    Q, K, V = (rand_int(rng, (L, d), b, np.int32) for _ in range(3))
    O = host(qx.attn_core(dev(Q), dev(K), dev(V), bound=b))
    same(O, orc.attn_i32(Q, K, V))


@pytest.mark.parametrize("L,d", [(1, 5), (40, 64), (129, 17)])
def test_attn_i32_valu_full_range(L, d):
    rng = np.random.default_rng(L + 11 * d)
    Q, K, V = (rng.integers(-(1 << 31), (1 << 31) - 1, (L, d), dtype=np.int32, endpoint=True)
               for _ in range(3))
    O = host(qx.attn_core(dev(Q), dev(K), dev(V), bound=0))
    same(O, orc.attn_i32(Q, K, V))


@pytest.mark.parametrize("L,d", [(512, 64), (700, 128), (333, 32)])
def test_attn_i32_extremes(L, d):
    b = 127
    Q = np.full((L, d), -b, np.int32)
    K = np.full((L, d), -b, np.int32)
    V = np.full((L, d), b, np.int32)
    K[::2] = b
    O = host(qx.attn_core(dev(Q), dev(K), dev(V), bound=b))
    same(O, orc.attn_i32(Q, K, V))


# ---------------------------------------------------------------------------
# Determinism and the executor
# ---------------------------------------------------------------------------
def test_repeatable_bit_identical():
    rng = np.random.default_rng(0)
    L, d = 2048, 64
    Q, K, V = ((rng.standard_normal((L, d)) / 8).astype(np.float32) for _ in range(3))
    tq, tk, tv = dev(Q), dev(K), dev(V)
    first = host(qx.attn_core(tq, tk, tv))
    for _ in range(5):
        same(host(qx.attn_core(tq, tk, tv)), first)
    A = rand_int(rng, (512, 768), 256, np.int16)
    B = rand_int(rng, (768, 640), 256, np.int16)
    ta, tb = dev(A), dev(B)
    with qx.Executor.gemm_i16i32(512, 640, 768, 1, 256, 256) as ex:
        outs = [host(ex.run([ta, tb])) for _ in range(5)]
    assert all(np.array_equal(o, outs[0]) for o in outs)
    same(outs[0][0], orc.gemm_i16i32(A, B))


def test_executor_profile_times_every_launch():
    rng = np.random.default_rng(8)
    A = rand_int(rng, (1, 512, 1024), 256, np.int16)
    B = rand_int(rng, (1, 1024, 768), 256, np.int16)
    ta, tb = dev(A), dev(B)
    out = torch.empty((1, 512, 768), dtype=torch.int32, device="cuda")
    with qx.Executor.gemm_i16i32(512, 768, 1024, 1, 256, 256) as ex:
        prof = ex.profile([ta, tb], out, reps=3)
    names = [n for n, _ in prof]
    # operands within [-256, 256]: the encoders write bf16
    assert names[:2] == ["enc_a_bf16", "enc_bt_bf16"] and names[2].startswith("gemm_nt_bf16_")
    assert all(ms > 0 for _, ms in prof)
    same(host(out), orc.gemm_i16i32(A, B))


def test_validate_scan_refuses_out_of_contract_operands(monkeypatch):
    # QX_VALIDATE=1: every bounded operand is scanned first; one element past
    # its declared bound gives QX_ERR_RANGE naming the operand, and the
    # output is left untouched.
    monkeypatch.setenv("QX_VALIDATE", "1")
    rng = np.random.default_rng(11)

    def refused(ex, inputs, which, shape):
        out = torch.full(shape, 7, dtype=ex.out_dtype, device="cuda")
        with pytest.raises(qx.QxError) as e:
            ex.run([dev(a) for a in inputs], out=out)
        assert e.value.status == qx.ERR_RANGE and f"input {which}" in str(e.value), str(e.value)
        assert bool((out == 7).all())

    A = rand_int(rng, (2, 70, 90), 256, np.int16)
    B = rand_int(rng, (2, 90, 50), 300, np.int16)
    with qx.Executor.gemm_i16i32(70, 50, 90, 2, 256, 300) as ex:
        same(run_exec(ex, (A, B)), orc.gemm_i16i32(A, B))       # at the bounds: runs
        A2 = A.copy()
        A2[1, 69, 89] = 257
        refused(ex, (A2, B), 0, (2, 70, 50))
        B2 = B.copy()
        B2[0, 0, 0] = -301
        refused(ex, (A, B2), 1, (2, 70, 50))
    x = rand_int(rng, (2, 8, 9, 9), 100, np.int16)
    w = rand_int(rng, (4, 8, 3, 3), 50, np.int16)
    with qx.Executor.conv2d(2, 8, 9, 9, 4, 3, 3, 1, 1, 100, 50) as ex:
        same(run_exec(ex, (x, w)), orc.conv2d_direct(x, w, 1, 1))
        x2 = x.copy()
        x2[1, 7, 8, 8] = 101
        refused(ex, (x2, w), 0, (2, 4, 9, 9))
    Q, K, V = (rand_int(rng, (64, 32), 64, np.int32) for _ in range(3))
    with qx.Executor.attn("i32", 64, 32, 64) as ex:
        same(run_exec(ex, (Q, K, V)), orc.attn_i32(Q, K, V))
        V2 = V.copy()
        V2[63, 31] = -65
        refused(ex, (Q, K, V2), 2, (64, 32))
    # without the variable nothing is scanned: the same call is enqueued
    monkeypatch.delenv("QX_VALIDATE")
    with qx.Executor.gemm_i16i32(70, 50, 90, 2, 256, 300) as ex:
        run_exec(ex, (A2, B))


def test_executor_reuse_and_errors():
    rng = np.random.default_rng(5)
    with qx.Executor.gemm_i32_s24(100, 90, 80, 2) as ex:
        for _ in range(3):
            A = rng.integers(-(1 << 23), (1 << 23) - 1, (2, 100, 80), dtype=np.int32)
            B = rng.integers(-(1 << 23), (1 << 23) - 1, (2, 80, 90), dtype=np.int32)
            same(run_exec(ex, (A, B)), orc.gemm_i32_s24(A, B))
        t = torch.zeros(2 * 100 * 80 + 1, dtype=torch.int32, device="cuda")
        with pytest.raises(qx.QxError) as e:          # misaligned input pointer
            ex.run_ptrs([t.data_ptr() + 4, t.data_ptr()], t.data_ptr())
        assert e.value.status == qx.ERR_INVALID_ARG


def test_size_limits():
    # the largest batch the grid takes (65535 in grid z), a grid of 2^14
    # row tiles, and the one-element and one-row degenerate shapes
    rng = np.random.default_rng(6)
    A = rand_int(rng, (65535, 2, 3), 127, np.int16)
    B = rand_int(rng, (65535, 3, 2), 127, np.int16)
    with qx.Executor.gemm_i16i32(2, 2, 3, 65535, 127, 127) as ex:
        same(run_exec(ex, (A, B)), orc.gemm_i16i32(A, B))
    A = rand_int(rng, (1, 1 << 20, 5), 2048, np.int16)
    B = rand_int(rng, (1, 5, 3), 16, np.int16)
    with qx.Executor.gemm_i16i32(1 << 20, 3, 5, 1, 2048, 16) as ex:
        same(run_exec(ex, (A, B)), orc.gemm_i16i32(A, B))
    A = rng.integers(-(1 << 31), (1 << 31) - 1, (3, 1, 1), dtype=np.int32, endpoint=True)
    B = rng.integers(-(1 << 31), (1 << 31) - 1, (3, 1, 1), dtype=np.int32, endpoint=True)
    with qx.Executor.gemm_i32_s24(1, 1, 1, 3) as ex:
        same(run_exec(ex, (A, B)), orc.gemm_i32_s24(A, B))
    x = rand_int(rng, (1, 1, 1, 1), 256, np.int16)
    w = rand_int(rng, (1, 1, 1, 1), 256, np.int16)
    same(host(qx.conv2d_gemm(dev(x), dev(w), 1, 0, 256, 256)), orc.conv2d_direct(x, w, 1, 0))


# ---------------------------------------------------------------------------
# Full-size workloads (the benchmark's launch configuration)
# ---------------------------------------------------------------------------
def freivalds(A, B, C, trials=3, seed=0):
    """C[b] == A[b] B[b] exactly (int64), all elements covered w.h.p."""
    rng = np.random.default_rng(seed)
    for b in range(A.shape[0]):
        for _ in range(trials):
            r = rng.integers(0, 1 << 20, size=(C.shape[2],), dtype=np.int64)
            lhs = C[b].astype(np.int64) @ r
            rhs = A[b].astype(np.int64) @ (B[b].astype(np.int64) @ r)
            if not np.array_equal(lhs, rhs):
                return False
    return True


@pytest.mark.parametrize("name", ["gemm_i16_256", "gemm_s24_1024", "gemm_s24_16x512"])
def test_workload_small_full_oracle(name):
    w = WORKLOADS[name]
    A, B = w.generate()
    d = w.dims
    _say(f"[{name}] full oracle")
    if w.op == "gemm_i16i32":
        ex = qx.Executor.gemm_i16i32(d["M"], d["N"], d["K"], d["batch"], w.bound, w.bound)
        ref = orc.gemm_i16i32(A, B)
    else:
        ex = qx.Executor.gemm_i32_s24(d["M"], d["N"], d["K"], d["batch"])
        ref = orc.gemm_i32_s24(A, B)
    with ex:
        got = run_exec(ex, (A, B))
    same(got, ref)


def test_workload_conv_full_oracle():
    w = WORKLOADS["conv_8x64x56x56_128_3x3"]
    x, wt = w.generate()
    d = w.dims
    with qx.Executor.conv2d(d["N"], d["Ci"], d["H"], d["W"], d["Co"], d["KH"], d["KW"],
                            d["stride"], d["pad"], w.bound, w.bound) as ex:
        y = run_exec(ex, (x, wt))
    same(y, orc.conv2d_direct(x, wt, d["stride"], d["pad"]))


CONV_T_CASES = [  # N, Ci, H, W, Co, KH, KW, stride, pad: fp32 MFMA needs C_in % 32 == 0
    (1, 32, 8, 8, 16, 3, 3, 1, 1), (2, 64, 30, 26, 100, 3, 3, 1, 1), (3, 96, 17, 19, 40, 3, 3, 2, 1),
    (2, 32, 23, 23, 64, 7, 7, 2, 3), (4, 64, 9, 33, 48, 5, 3, 1, 2), (1, 3, 20, 20, 8, 3, 3, 1, 1),
    (2, 5, 9, 7, 5, 3, 3, 1, 1), (3, 12, 17, 9, 7, 3, 2, 3, 0),
]


@pytest.mark.parametrize("case", CONV_T_CASES)
def test_conv_f32(case):
    # FP32 conv (Table 2, Conv2D FP32 row): normwise 1e-4 against the float64
    # sum, and the elementwise a-priori bound Kd * 2^-24 * (|x| conv |w|) of an
    # fp32 sum in any order; repeated runs are bit-identical.
    N, Ci, H, W, Co, KH, KW, s, p = case
    rng = np.random.default_rng(zlib.crc32(repr(("f32", case)).encode()))
    x = rng.standard_normal((N, Ci, H, W)).astype(np.float32)
    w = (rng.standard_normal((Co, Ci, KH, KW)) / np.sqrt(Ci * KH * KW)).astype(np.float32)
    with qx.Executor.conv2d_t("f32", N, Ci, H, W, Co, KH, KW, s, p) as ex:
        plan = ex.plan()
        assert plan["route_name"] == ("f32_mfma" if Ci % 32 == 0 else "f32_valu"), plan
        y = run_exec(ex, (x, w))
        y2 = run_exec(ex, (x, w))
    R = orc.conv2d_f64(x, w, s, p)
    assert normwise(y, R) <= 1e-4
    absref = orc.conv2d_f64(np.abs(x), np.abs(w), s, p)
    assert (np.abs(y - R) <= Ci * KH * KW * 2.0 ** -24 * absref + 1e-30).all()
    assert np.array_equal(y, y2)
    if Ci % 32 == 0:   # the vector-ALU route on the same data meets the same bar
        with qx.Executor.conv2d_t("f32", N, Ci, H, W, Co, KH, KW, s, p, "f32_valu") as ex:
            yv = run_exec(ex, (x, w))
        assert normwise(yv, R) <= 1e-4


@pytest.mark.parametrize("route", ["s24_i8limb", "s24_valu"])
@pytest.mark.parametrize("case", CONV_T_CASES[:5] + [(8, 64, 20, 20, 96, 3, 3, 1, 1), (3, 6, 14, 14, 16, 5, 5, 1, 0),
                                                     (2, 5, 11, 9, 3, 3, 2, 2, 1), (2, 150, 6, 6, 16, 1, 1, 1, 0),
                                                     (7, 6, 14, 14, 16, 5, 5, 1, 0), (1, 16, 40, 40, 4, 3, 3, 1, 0),
                                                     (2, 3, 70, 70, 6, 5, 5, 2, 2), (2, 3, 12, 12, 8, 5, 5, 1, 0),
                                                     (3, 4, 9, 10, 5, 4, 4, 1, 0), (2, 2, 8, 14, 16, 2, 7, 1, 0),
                                                     (1, 3, 50, 50, 6, 3, 3, 1, 0), (2, 2, 9, 9, 3, 3, 3, 1, 0),
                                                     (2, 3, 6, 6, 1100, 3, 3, 1, 1)])
def test_conv_i32_smul24(route, case):
    # INT32 conv under the smul24 contract: full 32-bit words (bits 24..31
    # ignored), bit-exact mod 2^32 against the oracle.  On the vector-ALU
    # route the direct kernel stages whole images in LDS when they fit
    # (7 images of 14x14x6 in groups of 5 leave a partial group) and reads
    # the windows from global memory when an image has more output pixels
    # than a workgroup's threads cover (40x40, 50x50 and 70x70 inputs).
    # Stride 1 without padding takes unguarded window reads shared between
    # a thread's pixels: 4, 2 and 1 pixels per thread, kernel widths 3 and 5
    # and the generic width path (1, 4, 7).  1100 output channels over 72
    # positions lower explicitly onto the skinny vector-ALU GEMM, whose
    # stores scatter into NCHW.
    N, Ci, H, W, Co, KH, KW, s, p = case
    rng = np.random.default_rng(zlib.crc32(repr(("i32", route, case)).encode()))
    x = rng.integers(-(1 << 31), (1 << 31) - 1, (N, Ci, H, W), dtype=np.int32, endpoint=True)
    w = rng.integers(-(1 << 31), (1 << 31) - 1, (Co, Ci, KH, KW), dtype=np.int32, endpoint=True)
    x[0, :, 0, :] = -(1 << 23)
    w[0] = (1 << 23) - 1
    with qx.Executor.conv2d_t("i32", N, Ci, H, W, Co, KH, KW, s, p, route) as ex:
        assert ex.plan()["route_name"] == route
        y = run_exec(ex, (x, w))
    same(y, orc.conv2d_s24(x, w, s, p), str((route, case)))


def test_conv_t_oneshot_and_empty():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((1, 32, 6, 5)).astype(np.float32)
    w = rng.standard_normal((3, 32, 3, 3)).astype(np.float32)
    y = host(qx.conv2d_gemm_t(dev(x), dev(w), 1, 1))
    assert normwise(y, orc.conv2d_f64(x, w, 1, 1)) <= 1e-4
    xi = rng.integers(-(1 << 23), (1 << 23) - 1, (2, 3, 5, 5), dtype=np.int32)
    wi = rng.integers(-(1 << 23), (1 << 23) - 1, (4, 3, 2, 2), dtype=np.int32)
    same(host(qx.conv2d_gemm_t(dev(xi), dev(wi), 2, 0)), orc.conv2d_s24(xi, wi, 2, 0))
    # C_in == 0 -> zeros
    z = qx.conv2d_gemm_t(torch.empty((1, 0, 4, 4), dtype=torch.float32, device="cuda"),
                         torch.empty((2, 0, 3, 3), dtype=torch.float32, device="cuda"), 1, 1)
    assert z.shape == (1, 2, 4, 4) and float(z.abs().sum()) == 0.0


@pytest.mark.parametrize("case", CONV_IMPLICIT_CASES)
def test_conv_i32_implicit_lowering(case):
    # INT32 conv with C_in a multiple of 64 on the int8 limb route: one
    # launch writes the bordered NHWC limb planes (border = the limbs of 0),
    # the per-chunk position sums and the (kh, kw, ci)-ordered weight planes;
    # the contraction gathers its column tiles from the planes, so the
    # workspace holds about the image, not the 9x larger column matrix.
    # Strides 1-2, pads 0-3, 1x1 to 7x7 and rectangular kernels, 64-192
    # channels, pixel tiles ending mid-row; bit-exact mod 2^32.
    N, Ci, H, W, Co, KH, KW, s, p, _ = case
    rng = np.random.default_rng(zlib.crc32(repr(("i32 implicit", case)).encode()))
    x = rng.integers(-(1 << 31), (1 << 31) - 1, (N, Ci, H, W), dtype=np.int32, endpoint=True)
    w = rng.integers(-(1 << 31), (1 << 31) - 1, (Co, Ci, KH, KW), dtype=np.int32, endpoint=True)
    x[0, :, 0, :] = -(1 << 23)
    x[-1, :, -1, :] = (1 << 23) - 1
    w[0] = (1 << 23) - 1
    w[-1] = -(1 << 23)
    Ho, Wo = (H + 2 * p - KH) // s + 1, (W + 2 * p - KW) // s + 1
    with qx.Executor.conv2d_t("i32", N, Ci, H, W, Co, KH, KW, s, p, "s24_i8limb") as ex:
        plan = ex.plan()
        assert plan["kernels"] == 2, plan
        planes = 3 * N * (H + 2 * p) * (W + 2 * p) * Ci
        assert plan["workspace_bytes"] < planes + 3 * (Co + 128) * KH * KW * Ci + 4 * N * (H + 2 * p) * (W + 2 * p) * Ci // 64 + 4 * Co + 4096, plan
        y = run_exec(ex, (x, w))
    assert y.shape == (N, Co, Ho, Wo)
    same(y, orc.conv2d_s24(x, w, s, p), str(case))


def test_workload_conv_t_full_oracle():
    wf = WORKLOADS["conv_f32_8x64x56x56_128_3x3"]
    x, w = wf.generate()
    d = wf.dims
    with qx.Executor.conv2d_t("f32", d["N"], d["Ci"], d["H"], d["W"], d["Co"], d["KH"], d["KW"],
                              d["stride"], d["pad"]) as ex:
        y = run_exec(ex, (x, w))
    err = normwise(y, orc.conv2d_f64(x, w, d["stride"], d["pad"]))
    _say(f"[conv_f32] normwise error {err:.3e}")
    assert err <= 1e-4
    wi = WORKLOADS["conv_i32_8x64x56x56_128_3x3"]
    x, w = wi.generate()
    with qx.Executor.conv2d_t("i32", d["N"], d["Ci"], d["H"], d["W"], d["Co"], d["KH"], d["KW"],
                              d["stride"], d["pad"]) as ex:
        y = run_exec(ex, (x, w))
    same(y, orc.conv2d_s24(x, w, d["stride"], d["pad"]))


# ---------------------------------------------------------------------------
# Min/max and 2x2 pooling (Table 2 rows)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("n", [1, 5, 63, 64, 1000, 65537, 3 * (1 << 20) + 7])
def test_minmax(n):
    rng = np.random.default_rng(n)
    for dt, lo, hi in ((np.int32, -(1 << 31), (1 << 31) - 1), (np.int16, -32768, 32767)):
        x = rng.integers(lo // 2, hi // 2, n, dtype=dt, endpoint=True)
        # the extremes at random positions, including the very last element
        x[rng.integers(0, n)] = lo
        x[-1] = hi
        got = host(qx.minmax(dev(x)))
        same(got, orc.minmax(x), f"{dt.__name__} n={n}")


@pytest.mark.parametrize("shape", [(1, 1, 2, 2), (2, 3, 6, 8), (1, 2, 7, 9), (3, 1, 5, 4), (2, 4, 16, 40),
                                   (1, 8, 33, 64), (4, 3, 224, 224)])
def test_pools(shape):
    rng = np.random.default_rng(sum(shape))
    x = rng.integers(-(1 << 31), (1 << 31) - 1, shape, dtype=np.int32, endpoint=True)
    same(host(qx.pool2x2(dev(x))), orc.avgpool2_i32(x), f"avg {shape}")
    xf = rng.standard_normal(shape).astype(np.float32)
    xf.reshape(-1)[::7] = -0.0          # signed zeros and ties take the oracle's order
    same(host(qx.pool2x2(dev(xf))).view(np.uint32), orc.maxpool2_f32(xf).view(np.uint32), f"max {shape}")


def test_minmax_pool_executors_and_errors():
    with pytest.raises(qx.QxError) as e:
        qx.plan_minmax(0, 4)
    assert e.value.status == qx.ERR_INVALID_ARG
    x = np.arange(-50, 50, dtype=np.int32)
    with qx.Executor.minmax(100, "i32") as ex:
        assert ex.plan()["kernels"] == 2
        same(run_exec(ex, (x,)), np.array([-50, 49], np.int32))
        same(run_exec(ex, (x[::-1].copy(),)), np.array([-50, 49], np.int32))
    with qx.Executor.pool2x2("max_f32", 1, 1, 4, 8) as ex:
        xf = np.arange(32, dtype=np.float32).reshape(1, 1, 4, 8)
        same(run_exec(ex, (xf,)), orc.maxpool2_f32(xf))
    # H or W below 2: empty output, nothing launched
    assert qx.plan_pool2x2("avg_i32", 2, 3, 1, 8)["kernels"] == 0


@pytest.mark.parametrize("name", ["minmax_i32_128Mi", "minmax_i16_256Mi", "avgpool_i32_16x64x224x224",
                                  "maxpool_f32_16x64x224x224"])
def test_workload_hbm_rows_full_oracle(name):
    w = WORKLOADS[name]
    (x,) = w.generate()
    d = w.dims
    if w.op.startswith("minmax"):
        with qx.Executor.minmax(d["n"], w.op[-3:]) as ex:
            same(run_exec(ex, (x,)), orc.minmax(x))
        return
    kind = "avg_i32" if w.op == "avgpool_i32" else "max_f32"
    with qx.Executor.pool2x2(kind, d["N"], d["C"], d["H"], d["W"]) as ex:
        y = run_exec(ex, (x,))
    ref = orc.avgpool2_i32(x) if kind == "avg_i32" else orc.maxpool2_f32(x)
    same(y.view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("B,wb", [(1, 3), (7, 300), (64, 3), (300, 300)])
def test_lenet_pipeline(B, wb):
    # every layer chained through the executor's workspace; weights of 300
    # make the sums wrap and later layers read only the low 24 bits
    rng = np.random.default_rng(B * 1000 + wb)
    x = rng.integers(0, 255, (B, 1, 32, 32), dtype=np.int32, endpoint=True)
    ws = [rng.integers(-wb, wb, s, dtype=np.int32, endpoint=True)
          for s in ((6, 1, 5, 5), (16, 6, 5, 5), (400, 120), (120, 84), (84, 10))]
    with qx.Executor.lenet_i32(B) as ex:
        y = run_exec(ex, (x, *ws))
        y2 = run_exec(ex, (x, *ws))
    ref = orc.lenet_i32(x, *ws)
    same(y, ref)
    same(y2, ref, "second run")


def test_workload_lenet_full_oracle():
    w = WORKLOADS["lenet_i32_b4096"]
    inputs = w.generate()
    with qx.Executor.lenet_i32(w.dims["B"]) as ex:
        y = run_exec(ex, inputs)
    same(y, orc.lenet_i32(*inputs))


def test_workload_attn_full_oracle():
    wf = WORKLOADS["attn_f32_4096x64"]
    Q, K, V = wf.generate()
    with qx.Executor.attn("f32", 4096, 64) as ex:
        O = run_exec(ex, (Q, K, V))
    R = orc.attn_f64(Q, K, V)
    err = normwise(O, R)
    _say(f"[attn_f32_4096x64] normwise error {err:.3e}")
    assert err <= 1e-4
    wi = WORKLOADS["attn_i32_4096x64"]
    Q, K, V = wi.generate()
    with qx.Executor.attn("i32", 4096, 64, wi.bound) as ex:
        O = run_exec(ex, (Q, K, V))
    same(O, orc.attn_i32(Q, K, V))


# ---------------------------------------------------------------------------
# Softmax attention over heads (FP32): normwise 1e-4 against the float64 oracle
# ---------------------------------------------------------------------------
SDPA_CASES = [  # BH, L, d, scale, causal, input sigma (None: d^-1/4, unit-variance scores)
    (1, 1, 64, 1.0, False, None), (1, 1, 64, 1.0, True, None), (2, 31, 32, 1.0, False, None),
    (3, 100, 64, 0.125, True, 1.0), (2, 257, 64, 1.0, False, 1.0), (4, 300, 128, 0.088, True, None),
    (2, 77, 96, 0.5, False, None), (2, 100, 40, 0.3, True, None), (1, 50, 1, 2.0, False, 1.0),
    (3, 129, 17, -0.7, True, None), (1, 4096, 64, 1.0, True, None), (1, 2000, 128, 0.1, False, 1.0),
    (40, 130, 64, 1.0, True, None), (2, 64, 64, 0.0, False, 1.0), (5, 33, 100, 0.1, False, None),
]


def sdpa_inputs(BH, L, d, sigma, seed):
    rng = np.random.default_rng(seed)
    s = d ** -0.25 if sigma is None else sigma
    return tuple((rng.standard_normal((BH, L, d)) * s).astype(np.float32) for _ in range(3))


@pytest.mark.parametrize("case", SDPA_CASES)
def test_sdpa_f32(case):
    BH, L, d, scale, causal, sigma = case
    _say(f"[sdpa] BH={BH} L={L} d={d} scale={scale} causal={causal}")
    Q, K, V = sdpa_inputs(BH, L, d, sigma, BH * 1000 + L + d)
    plan = qx.plan_sdpa_f32(BH, L, d, scale, causal)
    O = host(qx.sdpa_f32(dev(Q), dev(K), dev(V), scale, causal))
    R = orc.sdpa_f64(Q, K, V, scale, causal)
    err = normwise(O, R)
    assert err <= 1e-4, (err, plan)
    # key splits merge in a fixed order: a second run is bit-identical
    O2 = host(qx.sdpa_f32(dev(Q), dev(K), dev(V), scale, causal))
    assert np.array_equal(O, O2)


def test_sdpa_executor_oneshot_and_errors():
    BH, L, d = 3, 200, 64
    Q, K, V = sdpa_inputs(BH, L, d, None, 5)
    with qx.Executor.sdpa_f32(BH, L, d, 1.0, True) as ex:
        assert ex.plan()["kernels"] == 2
        O = run_exec(ex, (Q, K, V))
    assert np.array_equal(O, host(qx.sdpa_f32(dev(Q), dev(K), dev(V), 1.0, True)))
    # [B][H][L][d] is BH = B*H heads
    O4 = host(qx.sdpa_f32(*(dev(a.reshape(1, BH, L, d)) for a in (Q, K, V)), 1.0, True))
    assert np.array_equal(O4.reshape(BH, L, d), O)
    # empty sizes are no-ops; a NULL operand of a non-empty call is refused
    e = torch.empty((0, 5, 64), dtype=torch.float32, device="cuda")
    assert qx.sdpa_f32(e, e, e).shape == (0, 5, 64)
    assert qx.lib().sdpa_f32(None, None, None, None, 1, 4, 64, 1.0, 0, None) == qx.ERR_INVALID_ARG
    assert qx.lib().sdpa_f32(None, None, None, None, 0, 4, 64, 1.0, 0, None) == 0


@pytest.mark.parametrize("name,heads", [("sdpa_f32_32x4096x64", (0, 13, 31)),
                                        ("sdpa_f32_causal_32x4096x64", (0, 31))])
def test_workload_sdpa_sampled_heads(name, heads):
    w = WORKLOADS[name]
    d = w.dims
    _say(f"[{name}] generate")
    Q, K, V = w.generate()
    with qx.Executor.sdpa_f32(d["BH"], d["L"], d["d"], d["scale"], bool(d["causal"])) as ex:
        O = run_exec(ex, (Q, K, V))
    _say(f"[{name}] heads {heads} against the oracle")
    hs = list(heads)
    R = orc.sdpa_f64(Q[hs], K[hs], V[hs], d["scale"], bool(d["causal"]))
    err = normwise(O[hs], R)
    _say(f"[{name}] normwise error {err:.3e}")
    assert err <= 1e-4
    assert np.isfinite(O).all()


@pytest.mark.parametrize("name", ["gemm_i16_8192", "gemm_i16_64x2048"])
def test_workload_large_gemm(name):
    w = WORKLOADS[name]
    d = w.dims
    _say(f"[{name}] generate")
    A, B = w.generate()
    with qx.Executor.gemm_i16i32(d["M"], d["N"], d["K"], d["batch"], w.bound, w.bound) as ex:
        C = run_exec(ex, (A, B))
    _say(f"[{name}] sampled rows against the oracle")
    rng = np.random.default_rng(1)
    batches = [0] if d["batch"] == 1 else [0, d["batch"] // 2, d["batch"] - 1]
    for b in batches:
        rows = np.sort(rng.choice(d["M"], size=16 if d["batch"] == 1 else 8, replace=False))
        rows = np.unique(np.concatenate([rows, [0, d["M"] - 1]]))
        ref = orc.gemm_i16i32(np.ascontiguousarray(A[b, rows]), B[b])
        same(C[b, rows], ref)
    _say(f"[{name}] Freivalds over every batch")
    sel = range(d["batch"]) if d["batch"] <= 64 else range(0, d["batch"], 8)
    sel = list(sel)
    assert freivalds(A[sel], B[sel], C[sel], trials=2)
