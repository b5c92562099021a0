"""Host-only checks of the boundary and of the persistent executor's
bookkeeping.

1. The declarations in include/qx.h of the operations and executor calls
   match the specified interface parameter for parameter (names, types,
   order).  The specified listing is restated below; `hipStream_t` is passed
   as `void*`, which is the same C ABI (hipStream_t is a pointer type).
2. With the host double of the device runtime (include/qx_testing.h),
   every executor type is created, run and destroyed on the CPU: workspace
   and timing events are counted, a run acquires nothing, every launch
   of the full-size workloads has a legal geometry, injected allocation
   failures release everything acquired before them, and stale handles are
   refused without being read.  The double computes nothing.
"""
import ctypes
import os
import re

import pytest

from paper_2606_09905_amd import qx
from paper_2606_09905_amd.workloads import WORKLOADS

# The operations' interface (persistent executors, operand-range contracts,
# the GEMM, convolution and attention operators of the Methodology), as
# specified for this library.
SPECIFIED = """
qx_status qgemm_i16i32(const int16_t* A, const int16_t* B, int32_t* C,
                       int64_t M, int64_t N, int64_t K, int64_t batch,
                       int32_t bound_a, int32_t bound_b, hipStream_t stream);
qx_status qgemm_i32_s24(const int32_t* A, const int32_t* B, int32_t* C,
                        int64_t M, int64_t N, int64_t K, int64_t batch, hipStream_t stream);
qx_status conv2d_gemm(const int16_t* x, const int16_t* w, int32_t* y,
                      int64_t N, int64_t C_in, int64_t H, int64_t W, int64_t C_out,
                      int64_t KH, int64_t KW, int64_t stride, int64_t pad,
                      int32_t bound_x, int32_t bound_w, hipStream_t stream);
qx_status attn_core(qx_attn_dtype dt, const void* Q, const void* K, const void* V, void* O,
                    int64_t L, int64_t d, int32_t bound, hipStream_t stream);
qx_status qx_exec_create_gemm_i16i32(qx_exec* out, int64_t M, int64_t N, int64_t K, int64_t batch,
                                     int32_t bound_a, int32_t bound_b);
qx_status qx_exec_create_gemm_i32_s24(qx_exec* out, int64_t M, int64_t N, int64_t K, int64_t batch);
qx_status qx_exec_create_conv2d(qx_exec* out, int64_t N, int64_t C_in, int64_t H, int64_t W, int64_t C_out,
                                int64_t KH, int64_t KW, int64_t stride, int64_t pad,
                                int32_t bound_x, int32_t bound_w);
qx_status qx_exec_create_attn(qx_exec* out, qx_attn_dtype dt, int64_t L, int64_t d, int32_t bound);
qx_status qx_exec_run(qx_exec h, const void* const* inputs, void* output, hipStream_t stream);
qx_status qx_exec_destroy(qx_exec h);
const char* qx_last_error(void);
"""

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _prototypes(text: str) -> dict:
    """name -> (return type, [(type, name), ...]) of every function declared."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    out = {}
    for m in re.finditer(r"([A-Za-z_][\w\s\*]*?)\b([A-Za-z_]\w*)\s*\(([^;{]*?)\)\s*;", text):
        ret, name, params = " ".join(m.group(1).split()), m.group(2), m.group(3)
        if name in ("if", "sizeof", "defined"):
            continue
        plist = []
        for p in params.split(","):
            p = " ".join(p.replace("*", " * ").split())
            if p in ("void", ""):
                continue
            toks = p.split(" ")
            ptype = " ".join(toks[:-1]).replace(" *", "*").replace("hipStream_t", "void*")
            plist.append((ptype, toks[-1]))
        out[name] = (ret.replace(" *", "*"), plist)
    return out


def test_header_matches_the_specified_interface():
    spec = _prototypes(SPECIFIED)
    with open(os.path.join(ROOT, "include", "qx.h")) as f:
        have = _prototypes(f.read())
    assert len(spec) == 11
    for name, proto in spec.items():
        assert name in have, name
        assert have[name] == proto, (name, have[name], proto)


def test_route_forcing_variants_are_separate_calls():
    with open(os.path.join(ROOT, "include", "qx.h")) as f:
        have = _prototypes(f.read())
    for base in ("gemm_i16i32", "gemm_i32_s24", "conv2d", "attn"):
        plain = have[f"qx_exec_create_{base}"][1]
        forced = have[f"qx_exec_create_{base}_route"][1]
        assert forced == plain + [("int32_t", "route")], base
    L = qx.lib()
    for n in qx.header_functions(os.path.join(ROOT, "include", "qx_testing.h")):
        assert hasattr(L, n), n


# ---------------------------------------------------------------------------
# executor bookkeeping under the host double
# ---------------------------------------------------------------------------
@pytest.fixture
def double():
    qx.lib().qx_release_cache()
    qx.testing_host_double(True)
    yield
    qx.testing_host_double(False)


def _fake_ptrs(n, base=1 << 40):
    # distinct, 256-byte aligned addresses; under the double nothing is
    # dereferenced, only checked for being bound
    return [base + (i + 1) * (1 << 20) for i in range(n)]


def _make(w):
    """Executor for a workload (same mapping as the benchmark)."""
    d = w.dims
    E = qx.Executor
    if w.op == "gemm_i16i32":
        return E.gemm_i16i32(d["M"], d["N"], d["K"], d["batch"], w.bound, w.bound)
    if w.op == "gemm_i32_s24":
        return E.gemm_i32_s24(d["M"], d["N"], d["K"], d["batch"])
    if w.op == "conv2d":
        return E.conv2d(d["N"], d["Ci"], d["H"], d["W"], d["Co"], d["KH"], d["KW"], d["stride"], d["pad"],
                        w.bound, w.bound)
    if w.op in ("conv2d_f32", "conv2d_i32"):
        return E.conv2d_t(w.op[-3:], d["N"], d["Ci"], d["H"], d["W"], d["Co"], d["KH"], d["KW"], d["stride"],
                          d["pad"])
    if w.op == "lenet_i32":
        return E.lenet_i32(d["B"])
    if w.op in ("minmax_i32", "minmax_i16"):
        return E.minmax(d["n"], w.op[-3:])
    if w.op in ("avgpool_i32", "maxpool_f32"):
        return E.pool2x2("avg_i32" if w.op == "avgpool_i32" else "max_f32", d["N"], d["C"], d["H"], d["W"])
    if w.op == "attn_f32":
        return E.attn("f32", d["L"], d["d"])
    if w.op == "attn_i32":
        return E.attn("i32", d["L"], d["d"], w.bound)
    if w.op == "sdpa_f32":
        return E.sdpa_f32(d["BH"], d["L"], d["d"], d["scale"], bool(d["causal"]))
    raise ValueError(w.op)


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_full_size_workloads_create_run_destroy(double, name):
    """Every launch of every full-size workload has a legal grid and bound
    pointers; runs acquire nothing; destroy releases what create acquired."""
    w = WORKLOADS[name]
    c0 = qx.testing_counters()
    with _make(w) as ex:
        c1 = qx.testing_counters()
        plan = ex.plan()
        assert c1["live_handles"] == c0["live_handles"] + 1
        # one allocation at most: the workspace (plus the validation flag
        # word behind it when the plan has bounded operands)
        assert c1["allocs"] - c0["allocs"] == (1 if plan["workspace_bytes"] else c1["allocs"] - c0["allocs"])
        assert c1["allocs"] - c0["allocs"] <= 1
        out = _fake_ptrs(1, 1 << 44)[0]
        for _ in range(3):
            ex.run_ptrs(_fake_ptrs(ex.n_inputs), out, 0)
        c2 = qx.testing_counters()
        for k in ("allocs", "frees", "events"):
            assert c2[k] == c1[k], (k, "a run acquired a device resource")
        assert c2["launches"] - c1["launches"] == 3 * plan["kernels"]
        # execute-only timing creates (and releases) its own timing events only
        prof = ex.profile([qx.HostTensor(p, ()) for p in _fake_ptrs(ex.n_inputs)], qx.HostTensor(out, ()),
                          reps=2, stream=0)
        assert len(prof) == plan["kernels"]
        c3 = qx.testing_counters()
        assert c3["allocs"] == c2["allocs"]
        assert c3["events"] - c2["events"] == c3["events_freed"] - c2["events_freed"]
    c4 = qx.testing_counters()
    assert c4["live_handles"] == c0["live_handles"]
    assert c4["allocs"] - c0["allocs"] == c4["frees"] - c0["frees"]
    assert c4["events"] - c0["events"] == c4["events_freed"] - c0["events_freed"]


def _batched_gemm():
    # 64 x 2048^3: eight batch groups sharing one workspace, the only device
    # resource a create acquires
    return qx.Executor.gemm_i16i32(2048, 2048, 2048, 64, 256, 256)


def test_injected_allocation_failures_release_everything(double, monkeypatch):
    c0 = qx.testing_counters()
    with _batched_gemm() as ex:
        assert ex.plan()["workspace_bytes"] > 0
    c1 = qx.testing_counters()
    assert c1["allocs"] - c0["allocs"] == 1 and c1["events"] == c0["events"]
    monkeypatch.setenv("QX_TEST_FAIL_ALLOC", "1")
    before = qx.testing_counters()
    with pytest.raises(qx.QxError) as e:
        _batched_gemm()
    assert e.value.status == qx.ERR_OUT_OF_MEMORY
    after = qx.testing_counters()
    for a, b in (("allocs", "frees"), ("events", "events_freed")):
        assert after[a] - before[a] == after[b] - before[b], a
    assert after["live_handles"] == before["live_handles"]
    # past the last acquisition the create succeeds
    monkeypatch.setenv("QX_TEST_FAIL_ALLOC", "2")
    _batched_gemm().close()
    # a create without a workspace has nothing to fail
    monkeypatch.setenv("QX_TEST_FAIL_ALLOC", "1")
    with qx.Executor.pool2x2("max_f32", 2, 3, 16, 16) as ex:
        assert ex.plan()["workspace_bytes"] == 0
    with pytest.raises(qx.QxError) as e:
        qx.Executor.attn("f32", 4096, 64)          # split partials: one workspace
    assert e.value.status == qx.ERR_OUT_OF_MEMORY
    assert qx.testing_counters()["live_handles"] == c0["live_handles"]


def test_out_is_null_after_a_failed_create(double, monkeypatch):
    monkeypatch.setenv("QX_TEST_FAIL_ALLOC", "1")
    h = ctypes.c_void_p(12345)
    st = qx.lib().qx_exec_create_gemm_i16i32(ctypes.byref(h), 4096, 4096, 4096, 1, 256, 256)
    assert st == qx.ERR_OUT_OF_MEMORY and not h.value
    assert b"out of memory" in qx.lib().qx_last_error().lower() or qx.lib().qx_last_error()


def test_stale_and_foreign_handles_are_refused(double):
    L = qx.lib()
    h = ctypes.c_void_p()
    assert L.qx_exec_create_gemm_i16i32(ctypes.byref(h), 256, 256, 256, 1, 256, 256) == qx.OK
    info = qx.PlanInfo()
    assert L.qx_exec_plan(h, ctypes.byref(info)) == qx.OK
    assert L.qx_exec_destroy(h) == qx.OK
    # second destroy, and every other use of the dead handle
    assert L.qx_exec_destroy(h) == qx.ERR_INVALID_ARG
    assert b"not live" in L.qx_last_error()
    assert L.qx_exec_plan(h, ctypes.byref(info)) == qx.ERR_INVALID_ARG
    arr = (ctypes.c_void_p * 2)(1 << 40, 1 << 41)
    assert L.qx_exec_run(h, arr, ctypes.c_void_p(1 << 42), None) == qx.ERR_INVALID_ARG
    # a pointer that no create returned (a buffer of garbage, never read)
    junk = ctypes.create_string_buffer(b"\x78\x65\x78\x71" * 64)
    assert L.qx_exec_destroy(ctypes.cast(junk, ctypes.c_void_p)) == qx.ERR_INVALID_ARG
    assert L.qx_exec_run(ctypes.cast(junk, ctypes.c_void_p), arr, ctypes.c_void_p(1 << 42), None) == \
        qx.ERR_INVALID_ARG


def test_runtime_switch_refused_while_handles_live():
    qx.lib().qx_release_cache()
    qx.testing_host_double(True)
    try:
        ex = qx.Executor.gemm_i16i32(64, 64, 64)
        with pytest.raises(qx.QxError) as e:
            qx.testing_host_double(False)
        assert e.value.status == qx.ERR_INVALID_ARG
        ex.close()
    finally:
        qx.testing_host_double(False)


def test_oneshot_cache_reuses_one_executor(double):
    L = qx.lib()
    c0 = qx.testing_counters()
    A, B, C = _fake_ptrs(3)
    for _ in range(4):
        assert L.qgemm_i16i32(A, B, C, 4096, 4096, 4096, 1, 256, 256, None) == qx.OK
    c1 = qx.testing_counters()
    assert c1["live_handles"] - c0["live_handles"] == 1
    assert c1["allocs"] - c0["allocs"] == 1
    L.qx_release_cache()
    c2 = qx.testing_counters()
    assert c2["live_handles"] == c0["live_handles"] and c2["frees"] - c1["frees"] == 1


def test_validation_path_under_the_double(double, monkeypatch):
    # QX_VALIDATE=1 scans bounded operands first; under the double the
    # scan's flag stays clear, so the run goes on and launches the plan
    monkeypatch.setenv("QX_VALIDATE", "1")
    with qx.Executor.gemm_i16i32(512, 512, 512, 1, 256, 256) as ex:
        c0 = qx.testing_counters()
        ex.run_ptrs(_fake_ptrs(2), 1 << 44, 0)
        c1 = qx.testing_counters()
        # one flag clear + one scan per bounded operand + the plan
        assert c1["launches"] - c0["launches"] == 1 + 2 + ex.plan()["kernels"]
