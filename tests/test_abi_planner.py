"""Host-only checks of libqx: it loads, exports every declared symbol, and
its planner picks exact routes from the operand-range contract.  No device
call is made here (validation and planning run before any HIP call)."""
import ctypes

import pytest

from paper_2606_09905_amd import qx
from paper_2606_09905_amd.workloads import WORKLOADS


def test_library_exports_every_header_symbol():
    L = qx.lib()
    names = qx.header_functions()
    assert len(names) >= 17
    for n in names:
        assert hasattr(L, n), n


def test_auto_routes_for_the_workloads():
    w = WORKLOADS
    d = w["gemm_i16_256"].dims
    p = qx.plan_gemm_i16i32(d["M"], d["N"], d["K"], 1, 1024, 1024)
    assert p["route_name"] == "f16_exact" and p["chunk"] == 16 and p["exact_no_wrap"] == 1
    for name in ("gemm_i16_8192", "gemm_i16_64x2048"):
        d = w[name].dims
        p = qx.plan_gemm_i16i32(d["M"], d["N"], d["K"], d["batch"], 256, 256)
        assert p["route_name"] == "f16_exact" and p["chunk"] == 256 and p["exact_no_wrap"] == 1
        # encode A, encode B^T, contract: the fp16 copies live in the workspace.
        # 64 x 2048^3 runs as 4 groups of 16 batches (256 MiB of encoded
        # operands each), one after the other
        assert p["kernels"] == (3 if d["batch"] == 1 else 3 * 4)
        assert p["workspace_bytes"] == 2 * 2 * d["M"] * d["K"] * d["batch"]
    p = qx.plan_gemm_i32_s24(1024, 1024, 1024, 1)
    assert p["route_name"] == "s24_i8limb" and p["products"] == 8 and p["exact_no_wrap"] == 0
    assert p["workspace_bytes"] >= 4 * 2048
    # few columns, many rows, at most 2^26 multiply-adds: one skinny
    # vector-ALU launch, no workspace
    for M, N, K in ((4096, 84, 120), (4096, 10, 84), (4096, 64, 120)):
        p = qx.plan_gemm_i32_s24(M, N, K, 1)
        assert p["route_name"] == "s24_valu" and p["kernels"] == 1 and p["workspace_bytes"] == 0, p
        assert (p["tile_m"], p["tile_n"]) == (64, 8)
    # more work (or few rows) keeps the matrix cores
    assert qx.plan_gemm_i32_s24(4096, 120, 400, 1)["route_name"] == "s24_i8limb"
    assert qx.plan_gemm_i32_s24(64, 64, 8448, 1)["route_name"] == "s24_i8limb"
    # the vector-ALU route asked for by name takes the skinny kernel too
    assert qx.plan_gemm_i32_s24(4096, 120, 400, 1, "s24_valu")["tile_n"] == 8
    # its 64x64 tiles slice K when they give under 1024 workgroups: the
    # output is cleared, then the slices add into it
    p = qx.plan_gemm_i32_s24(1024, 1024, 1024, 1, "s24_valu")
    assert p["k_splits"] == 4 and p["kernels"] == 2, p
    assert qx.plan_gemm_i32_s24(512, 512, 512, 16, "s24_valu")["k_splits"] == 0
    assert qx.plan_gemm_i16i32(256, 256, 256, 1, 0, 0, "valu_dot2")["k_splits"] == 2
    assert qx.plan_gemm_i32_s24(0, 1024, 1024, 1, "s24_valu")["kernels"] == 0
    d = w["conv_8x64x56x56_128_3x3"].dims
    p = qx.plan_conv2d(d["N"], d["Ci"], d["H"], d["W"], d["Co"], d["KH"], d["KW"], 1, 1, 256, 256)
    # one launch writes the bordered NHWC fp16 image and the fp16 weights,
    # then the contraction gathers its column tiles from that image
    assert p["route_name"] == "f16_exact" and p["kernels"] == 2
    assert p["workspace_bytes"] >= 2 * 8 * 58 * 58 * 64 + 2 * 128 * 576
    assert p["workspace_bytes"] < 2 * 576 * 8 * 56 * 56   # no explicit column matrix
    # C_in not a multiple of 64: explicit transposed column matrix
    p = qx.plan_conv2d(8, 32, 56, 56, 128, 3, 3, 1, 1, 256, 256)
    assert p["kernels"] == 3 and p["workspace_bytes"] >= 2 * 288 * 8 * 56 * 56
    assert qx.plan_attn("f32", 4096, 64)["route_name"] == "attn_f32_mfma"
    p = qx.plan_attn("i32", 4096, 64, 64)
    assert p["route_name"] == "attn_i32_mfma" and p["products"] == 3


def test_limb_routes_take_the_encode_nt_structure_when_large():
    # smul24, 1024^3: one launch encodes A and B^T into limb planes (and
    # produces the row and column sums of the offset correction), then the
    # NT int8 contraction runs on 64x64 tiles (64 tiles of 128x128 would
    # leave most of the chip idle).
    p = qx.plan_gemm_i32_s24(1024, 1024, 1024, 1)
    assert p["kernels"] == 2 and (p["tile_m"], p["tile_n"]) == (64, 64) and p["k_splits"] == 0, p
    # three int8 planes of each operand (padded to 64) after the sums
    assert p["workspace_bytes"] >= 2 * 3 * 1024 * 1024
    # 16 x 512^3: 256 tiles of 128x128 (at least 128 of them), run by eight
    # waves of 64x32 each
    p = qx.plan_gemm_i32_s24(512, 512, 512, 16)
    assert p["kernels"] == 2 and (p["tile_m"], p["tile_n"]) == (128, 128) and p["k_splits"] == 0
    p = qx.plan_gemm_i32_s24(4096, 4096, 512, 1)
    assert p["kernels"] == 2 and (p["tile_m"], p["tile_n"]) == (128, 128) and p["k_splits"] == 0
    for route, b, kernels in (("i8_direct", 127, 2), ("i8_karatsuba", 8127, 2), ("i8_offset4", 0, 2)):
        p = qx.plan_gemm_i16i32(2048, 2048, 2048, 1, b, b, route)
        assert p["kernels"] == kernels and p["tile_m"] == 128, (route, p)
    # K slices when there are at most 128 tiles: enough slices to give each
    # CU one workgroup, at most 16, each of at least four 64-wide K tiles,
    # none empty (132 K tiles: 16 slices of 9 would leave the last empty,
    # so 15; 79 K tiles in 12 slices of 7 leave 2 for the last)
    for (M, N, K, b), splits in (((300, 200, 5000, 1), 12), ((64, 1024, 4096, 1), 16),
                                 ((33, 700, 999, 2), 4), ((640, 640, 640, 1), 2),
                                 ((640, 640, 448, 1), 0), ((700, 900, 1000, 1), 0),
                                 ((64, 64, 8448, 1), 15), ((1024, 1024, 256, 1), 0),
                                 ((2048, 1024, 4096, 1), 0)):
        p = qx.plan_gemm_i32_s24(M, N, K, b)
        assert p["k_splits"] == splits and p["kernels"] == (3 if splits else 2), ((M, N, K, b), p)
    p = qx.plan_gemm_i16i32(257, 129, 1000, 1, 32768, 32768, "i8_offset4")
    assert p["k_splits"] == 4 and p["kernels"] == 3, p
    # small problems keep the single-pass register-staged kernel
    assert qx.plan_gemm_i32_s24(64, 64, 64, 1)["kernels"] == 2
    assert qx.plan_gemm_i16i32(64, 64, 64, 1, 127, 127)["kernels"] == 1


def test_conv_f32_i32_plans():
    # FP32: the fp32 matrix cores when C_in % 32 == 0 (prep launch + gathering
    # NT GEMM), else explicit lowering + vector-ALU fp32 GEMM
    p = qx.plan_conv2d_t("f32", 8, 64, 56, 56, 128, 3, 3, 1, 1)
    assert p["route_name"] == "f32_mfma" and p["kernels"] == 2
    assert p["workspace_bytes"] >= 4 * 8 * 58 * 58 * 64 + 4 * 128 * 576
    p = qx.plan_conv2d_t("f32", 2, 3, 20, 20, 8, 3, 3, 1, 1)
    assert p["route_name"] == "f32_valu" and p["kernels"] == 2
    with pytest.raises(qx.QxError) as e:
        qx.plan_conv2d_t("f32", 2, 3, 20, 20, 8, 3, 3, 1, 1, "f32_mfma")
    assert e.value.status == qx.ERR_UNSUPPORTED
    with pytest.raises(qx.QxError) as e:
        qx.plan_conv2d_t("f32", 2, 32, 20, 20, 8, 3, 3, 1, 1, "f16_exact")
    assert e.value.status == qx.ERR_INVALID_ARG
    # INT32 (smul24): large problems with C_in a multiple of 64 write the
    # image once as bordered NHWC limb planes and the contraction gathers its
    # column tiles from them (workspace about 3 bytes per bordered image
    # element); other C_in gather the im2col columns inside the limb-plane
    # encoder (3 bytes per column-matrix element); small ones lower
    # explicitly and run the register-staged smul24 GEMM
    p = qx.plan_conv2d_t("i32", 8, 64, 56, 56, 128, 3, 3, 1, 1)
    assert p["route_name"] == "s24_i8limb" and p["kernels"] == 2
    assert p["workspace_bytes"] < 3 * 8 * 58 * 58 * 64 + 3 * 128 * 576 + 4 * 8 * 58 * 58 + 4 * 128 + 4096
    p = qx.plan_conv2d_t("i32", 8, 48, 56, 56, 128, 3, 3, 1, 1)
    assert p["route_name"] == "s24_i8limb" and p["kernels"] == 2
    assert p["workspace_bytes"] > 3 * 432 * 8 * 56 * 56
    p = qx.plan_conv2d_t("i32", 1, 4, 8, 8, 40, 3, 3, 1, 1)
    assert p["route_name"] == "s24_i8limb" and p["kernels"] == 3   # im2col, sums, GEMM
    # few output channels: one direct vector-ALU kernel
    p = qx.plan_conv2d_t("i32", 1, 4, 8, 8, 4, 3, 3, 1, 1)
    assert p["route_name"] == "s24_valu" and p["kernels"] == 1 and p["workspace_bytes"] == 0
    assert qx.plan_conv2d_t("i32", 1, 4, 8, 8, 4, 3, 3, 1, 1, "s24_i8limb")["kernels"] == 3
    assert qx.plan_conv2d_t("i32", 1, 2, 5, 5, 3, 3, 3, 1, 1, "s24_valu")["route_name"] == "s24_valu"
    with pytest.raises(qx.QxError) as e:
        qx.plan_conv2d_t("i32", 1, 2, 5, 5, 3, 3, 3, 1, 1, "f32_mfma")
    assert e.value.status == qx.ERR_INVALID_ARG
    assert qx.plan_conv2d_t("f32", 0, 32, 5, 5, 3, 3, 3, 1, 1)["kernels"] == 0
    assert qx.plan_conv2d_t("i32", 1, 0, 5, 5, 3, 3, 3, 1, 1)["kernels"] == 1


def test_lenet_plan_chains_the_operators():
    p = qx.plan_lenet_i32(4096)
    # both convs: one direct launch each with ReLU and the 2x2 average fused
    # (only the pooled maps reach the workspace); then 3 FC GEMMs: the first
    # through its limb encoder and the int8 contraction, the other two one
    # skinny vector-ALU launch each; the first two store through their ReLU.
    # A small batch runs every FC layer through the limb planes and their
    # sums, with the two ReLUs as launches of their own: 4 launches more.
    assert p["kernels"] == 6, p
    assert qx.plan_lenet_i32(7)["kernels"] == 10
    assert 4 * 4096 * (6 * 14 * 14 + 400) <= p["workspace_bytes"] < 4 * 4096 * 6 * 28 * 28
    assert qx.plan_lenet_i32(0)["kernels"] == 0
    with pytest.raises(qx.QxError):
        qx.plan_lenet_i32(-1)


def test_minmax_pool_plans():
    p = qx.plan_minmax(1 << 27, 4)
    assert p["kernels"] == 2 and p["workspace_bytes"] == 8 * 2048
    assert qx.plan_minmax(1, 2)["kernels"] == 2
    for bad in ((0, 4), (10, 3), (-1, 2)):
        with pytest.raises(qx.QxError) as e:
            qx.plan_minmax(*bad)
        assert e.value.status == qx.ERR_INVALID_ARG
    assert qx.plan_pool2x2("avg_i32", 16, 64, 224, 224)["kernels"] == 1
    assert qx.plan_pool2x2("max_f32", 1, 1, 3, 3)["kernels"] == 1
    assert qx.plan_pool2x2("max_f32", 1, 1, 1, 3)["kernels"] == 0
    with pytest.raises(qx.QxError):
        qx.plan_pool2x2("avg_i32", -1, 1, 4, 4)


@pytest.mark.parametrize("b,route", [
    (1, "i8_direct"), (127, "i8_direct"), (128, "f16_exact"), (256, "f16_exact"),
    (1024, "f16_exact"), (2048, "i8_karatsuba"), (8127, "i8_karatsuba"),
    (8128, "i8_offset4"), (0, "i8_offset4"), (32768, "i8_offset4"),
])
def test_route_boundaries(b, route):
    assert qx.plan_gemm_i16i32(64, 64, 64, 1, b, b)["route_name"] == route


@pytest.mark.parametrize("ba,bb,chunk", [
    (128, 128, 1024), (256, 256, 256), (255, 255, 256), (300, 300, 176), (512, 512, 64),
    (724, 724, 32), (1024, 1024, 16), (2048, 512, 16), (1, 2048, 8192),
])
def test_f16_chunk_rule(ba, bb, chunk):
    # chunk: largest multiple of 16 with chunk * ba * bb <= 2^24; the kernel
    # flushes every 64 K (one tile) or every 16 K (one MFMA step) within it.
    p = qx.plan_gemm_i16i32(64, 64, 64, 1, ba, bb, "f16_exact")
    largest = (2 ** 24 // (ba * bb)) // 16 * 16
    assert largest >= 16
    expect = largest // 64 * 64 if largest >= 64 else 16
    assert p["chunk"] == expect == (chunk // 64 * 64 if chunk >= 64 else 16)
    assert p["chunk"] * ba * bb <= 2 ** 24


def test_f16_infeasible_and_forced_routes():
    with pytest.raises(qx.QxError) as e:
        qx.plan_gemm_i16i32(64, 64, 64, 1, 2049, 16, "f16_exact")
    assert e.value.status == qx.ERR_RANGE
    with pytest.raises(qx.QxError) as e:
        qx.plan_gemm_i16i32(64, 64, 64, 1, 1448, 1448, "f16_exact")  # chunk < 16
    assert e.value.status == qx.ERR_RANGE
    with pytest.raises(qx.QxError) as e:
        qx.plan_gemm_i16i32(64, 64, 64, 1, 128, 5, "i8_direct")
    assert e.value.status == qx.ERR_RANGE
    with pytest.raises(qx.QxError) as e:
        qx.plan_gemm_i16i32(64, 64, 64, 1, 8128, 5, "i8_karatsuba")
    assert e.value.status == qx.ERR_RANGE
    with pytest.raises(qx.QxError) as e:
        qx.plan_gemm_i16i32(64, 64, 64, 1, 0, 0, "s24_valu")
    assert e.value.status == qx.ERR_INVALID_ARG
    with pytest.raises(qx.QxError) as e:
        qx.plan_gemm_i32_s24(64, 64, 64, 1, "f16_exact")
    assert e.value.status == qx.ERR_INVALID_ARG
    for r in ("i8_offset4", "valu_dot2"):
        assert qx.plan_gemm_i16i32(5, 5, 5, 1, 0, 0, r)["route_name"] == r
    assert qx.plan_gemm_i32_s24(5, 5, 5, 1, "s24_valu")["route_name"] == "s24_valu"


@pytest.mark.parametrize("args", [
    (-1, 4, 4, 1), (4, -1, 4, 1), (4, 4, -1, 1), (4, 4, 4, -1),
])
def test_negative_dims_rejected(args):
    with pytest.raises(qx.QxError) as e:
        qx.plan_gemm_i16i32(*args)
    assert e.value.status == qx.ERR_INVALID_ARG
    assert "must be >= 0" in str(e.value)


def test_size_limits_and_bad_bounds():
    with pytest.raises(qx.QxError) as e:
        qx.plan_gemm_i16i32(1 << 31, 4, 4)
    assert e.value.status == qx.ERR_UNSUPPORTED
    with pytest.raises(qx.QxError) as e:
        qx.plan_gemm_i16i32(1 << 21, 1 << 21, 4)
    assert e.value.status == qx.ERR_UNSUPPORTED
    with pytest.raises(qx.QxError) as e:
        qx.plan_gemm_i16i32(4, 4, 4, 70000)
    assert e.value.status == qx.ERR_UNSUPPORTED
    for bad in (-1, 32769):
        with pytest.raises(qx.QxError) as e:
            qx.plan_gemm_i16i32(4, 4, 4, 1, bad, 1)
        assert e.value.status == qx.ERR_INVALID_ARG
    with pytest.raises(qx.QxError) as e:
        qx.plan_gemm_i16i32(4, 4, 4, 1, 1, 1, 99)
    assert e.value.status == qx.ERR_INVALID_ARG


def test_empty_and_degenerate_plans():
    p = qx.plan_gemm_i16i32(0, 5, 5)
    assert p["kernels"] == 0 and p["workspace_bytes"] == 0
    p = qx.plan_gemm_i16i32(5, 5, 0)
    assert p["kernels"] == 1  # K == 0: the output is filled with zeros
    p = qx.plan_gemm_i32_s24(3, 0, 9, 2)
    assert p["kernels"] == 0
    assert qx.plan_attn("f32", 0, 64)["kernels"] == 0
    assert qx.plan_conv2d(0, 3, 5, 5, 2, 3, 3, 1, 1)["kernels"] == 0
    assert qx.plan_conv2d(1, 0, 5, 5, 2, 3, 3, 1, 1)["kernels"] == 1


def test_conv_validation():
    with pytest.raises(qx.QxError) as e:
        qx.plan_conv2d(1, 1, 2, 2, 1, 5, 5, 1, 0)   # kernel larger than the input
    assert e.value.status == qx.ERR_INVALID_ARG
    with pytest.raises(qx.QxError) as e:
        qx.plan_conv2d(1, 1, 8, 8, 1, 3, 3, 0, 1)   # stride 0
    assert e.value.status == qx.ERR_INVALID_ARG
    with pytest.raises(qx.QxError) as e:
        qx.plan_conv2d(1, 1, 8, 8, 1, 0, 3, 1, 1)   # empty kernel
    assert e.value.status == qx.ERR_INVALID_ARG
    p = qx.plan_conv2d(2, 3, 7, 9, 4, 3, 2, 2, 1, 0, 0)
    assert p["route_name"] == "i8_offset4"


def test_attention_plans():
    assert qx.plan_attn("f32", 100, 48)["route_name"] == "attn_f32_valu"
    assert qx.plan_attn("i32", 100, 64, 0)["route_name"] == "attn_i32_valu"
    assert qx.plan_attn("i32", 100, 64, 127)["route_name"] == "attn_i32_mfma"
    assert qx.plan_attn("i32", 100, 128, 127)["route_name"] == "attn_i32_mfma"
    with pytest.raises(qx.QxError) as e:
        qx.plan_attn("i32", 100, 64, 128, "attn_i32_mfma")
    assert e.value.status == qx.ERR_RANGE
    with pytest.raises(qx.QxError) as e:
        qx.plan_attn("f32", 100, 48, 0, "attn_f32_mfma")
    assert e.value.status == qx.ERR_UNSUPPORTED
    with pytest.raises(qx.QxError) as e:
        qx.plan_attn("f32", 100, 300)
    assert e.value.status == qx.ERR_UNSUPPORTED
    # key splits: every split boundary on a 32-key block, one workgroup per
    # CU (32 query blocks x 8 splits of 512 keys)
    p = qx.plan_attn("f32", 4096, 64)
    assert p["tile_k"] % 32 == 0 and (4096 // 128) * (4096 // p["tile_k"]) >= 256
    assert p["tile_k"] == 512
    # INT32, d = 32 and 64: the streaming kernel (64 queries per workgroup,
    # four key parts of whole 64-key pairs of blocks) fills the chip with 64
    # query groups x 4 splits of 1024 keys; short sequences round the split
    # up to 256 keys; d = 128 keeps the LDS-resident splits, both int8
    # tiles within 48 KiB of LDS (192 keys)
    assert qx.plan_attn("i32", 4096, 64, 64)["tile_k"] == 1024
    assert qx.plan_attn("i32", 4096, 32, 64)["tile_k"] == 1024
    for L in (1, 63, 65, 300, 2049, 8191):
        kps = qx.plan_attn("i32", L, 64, 64)["tile_k"]
        assert kps % 256 == 0 and kps >= 256
    assert qx.plan_attn("i32", 4096, 128, 64)["tile_k"] == 192


def test_sdpa_plans():
    # 32 heads x 32 query blocks fill the chip: one launch, no workspace
    p = qx.plan_sdpa_f32(32, 4096, 64, 1.0, False)
    assert p["kernels"] == 1 and p["workspace_bytes"] == 0 and p["tile_k"] == 4096
    # one head: key splits on 32-key boundaries, merged by a second launch;
    # the workspace holds unnormalised outputs plus (max, sum) per row
    p = qx.plan_sdpa_f32(1, 4096, 64, 0.125, True)
    splits = 4096 // p["tile_k"]
    assert p["kernels"] == 2 and p["tile_k"] % 32 == 0 and 32 * splits >= 512
    assert p["workspace_bytes"] >= splits * 4096 * (64 + 2) * 4
    # any d up to 128 (ragged d pads to the next multiple of 32 on chip)
    for d in (1, 17, 40, 100, 128):
        assert qx.plan_sdpa_f32(2, 100, d)["kernels"] >= 1
    for args, status in (((1, 10, 129), qx.ERR_UNSUPPORTED), ((65536, 10, 64), qx.ERR_UNSUPPORTED),
                         ((1, (1 << 20) + 1, 64), qx.ERR_UNSUPPORTED), ((-1, 10, 64), qx.ERR_INVALID_ARG),
                         ((1, 10, 64, float("nan")), qx.ERR_INVALID_ARG),
                         ((1, 10, 64, float("inf")), qx.ERR_INVALID_ARG)):
        with pytest.raises(qx.QxError) as e:
            qx.plan_sdpa_f32(*args)
        assert e.value.status == status, args
    info = qx.PlanInfo()
    assert qx.lib().qx_plan_sdpa_f32(qx.ctypes.byref(info), 1, 10, 64, 1.0, 2) == qx.ERR_INVALID_ARG
    assert qx.lib().qx_plan_sdpa_f32(None, 1, 10, 64, 1.0, 0) == qx.ERR_INVALID_ARG
    for args in ((0, 10, 64), (2, 0, 64), (2, 10, 0)):
        assert qx.plan_sdpa_f32(*args)["kernels"] == 0


def test_null_pointer_validation_before_device():
    # Validation returns before any HIP call, so this runs without a GPU.
    L = qx.lib()
    st = L.qgemm_i16i32(None, None, None, 4, 4, 4, 1, 0, 0, None)
    assert st == qx.ERR_INVALID_ARG
    assert b"NULL" in L.qx_last_error()
    st = L.qgemm_i16i32(None, None, None, -4, 4, 4, 1, 0, 0, None)
    assert st == qx.ERR_INVALID_ARG
    # empty problems are a no-op and need no pointers
    assert L.qgemm_i16i32(None, None, None, 0, 0, 4, 1, 0, 0, None) == qx.OK
    assert L.qgemm_i16i32(None, None, None, 0, 4, 4, 1, 0, 0, None) == qx.ERR_INVALID_ARG  # B non-empty
    assert L.attn_core(0, None, None, None, None, 0, 64, 0, None) == qx.OK
    assert L.attn_core(7, None, None, None, None, 4, 64, 0, None) == qx.ERR_INVALID_ARG
    assert L.qx_exec_run(None, None, None, None) == qx.ERR_INVALID_ARG
    assert L.qx_exec_destroy(None) == qx.OK
    info = qx.PlanInfo()
    assert L.qx_exec_plan(None, ctypes.byref(info)) == qx.ERR_INVALID_ARG


def test_bf16_operand_format_for_small_bounds():
    # Large fp16-exact problems whose bounds are both <= 256 encode the
    # operands as bf16 (integers up to 256 need eight significant bits);
    # wider bounds, the register-staged small-problem kernel and the conv
    # image copy stay fp16.
    for ba, bb, fmt in ((256, 256, 1), (128, 256, 1), (1, 200, 1), (257, 256, 0), (300, 300, 0), (1024, 16, 0)):
        p = qx.plan_gemm_i16i32(4096, 4096, 4096, 1, ba, bb)
        assert p["route_name"] == "f16_exact" and p["operand_format"] == fmt, (ba, bb, p)
    assert qx.plan_gemm_i16i32(64, 64, 64, 1, 256, 256)["operand_format"] == 0
    assert qx.plan_conv2d(8, 64, 56, 56, 128, 3, 3, 1, 1, 256, 256)["operand_format"] == 0
    # the chunk rule does not depend on the operand format
    assert qx.plan_gemm_i16i32(4096, 4096, 4096, 1, 256, 256)["chunk"] == 256


def test_nt_route_holds_32_bit_panel_offsets():
    # The encode + NT kernel addresses a 256-row operand panel with 32-bit
    # offsets; from Kp = 2^22 on the register-staged kernel (64-bit
    # addressing, no workspace) takes over.
    below = qx.plan_gemm_i16i32(256, 256, (1 << 22) - 64, 1, 256, 256)
    assert below["kernels"] == 3 and below["workspace_bytes"] > 0
    for K in ((1 << 22) - 63, 1 << 22, 1 << 24):
        p = qx.plan_gemm_i16i32(256, 256, K, 1, 256, 256)
        assert p["route_name"] == "f16_exact" and p["kernels"] == 1 and p["workspace_bytes"] == 0, (K, p)


def test_fill_grid_is_capped_for_huge_outputs():
    # K == 0 clears the output; from 2^32 words the launch must still fit
    # the grid limits (checked by the host double's launch check).
    qx.lib().qx_release_cache()
    qx.testing_host_double(True)
    try:
        for M, N, batch in ((1 << 16, 1 << 16, 1), (1 << 16, 1 << 16, 3), (1 << 20, 1 << 13, 1)):
            with qx.Executor.gemm_i16i32(M, N, 0, batch, 256, 256) as ex:
                assert ex.plan()["kernels"] == 1
                ex.run_ptrs([1 << 40, 1 << 41], 1 << 44, 0)
    finally:
        qx.testing_host_double(False)
