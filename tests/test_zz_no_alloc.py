"""The allocation-free GEMM entry point against the allocating one.

qgemm_i16i32_noalloc must give, bit for bit, what qgemm_i16i32 gives on the
same inputs, call after call, with the scratch left over from the previous
call (always a larger problem first, then a smaller one), on every structure
its plans take: the encoded-operand path, batch groups run in order on one
stream, the register-staged kernels when the encoded operands would not fit
the scratch, and the offset limb route with its row and column sums.  Both
sides go through the C ABI.
"""
import sys
import zlib

import numpy as np
import pytest

from paper_2606_09905_amd import qx

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SCRATCH = 64 << 20


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    qx.lib()
    yield
    qx.lib().qx_release_cache()


def _operands(shape, bound, seed):
    batch, M, N, K = shape
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    A = torch.randint(-bound, bound + 1, (batch, M, K), dtype=torch.int32, device="cuda", generator=g)
    B = torch.randint(-bound, bound + 1, (batch, K, N), dtype=torch.int32, device="cuda", generator=g)
    return A.to(torch.int16).contiguous(), B.to(torch.int16).contiguous()


def _check_pair(shape, bound):
    """One call of each entry point on the same inputs; returns the plan
    route the allocating side took."""
    batch, M, N, K = shape
    _say(f"[no_alloc] shape {shape} bound {bound}")
    A, B = _operands(shape, bound, zlib.crc32(repr((shape, bound)).encode()))
    ref = qx.qgemm_i16i32(A, B, bound, bound)
    out = torch.full((batch, M, N), 0x5A5A5A5A, dtype=torch.int32, device="cuda")
    qx.qgemm_i16i32_noalloc(A, B, out, bound, bound)
    torch.cuda.synchronize()
    got, want = out.cpu().numpy(), ref.cpu().numpy()
    bad = np.flatnonzero(got.reshape(-1) != want.reshape(-1))
    assert bad.size == 0, f"{shape}: {bad.size} elements differ (first flat index {bad[0]})"


# (batch, M, N, K), bound.  Each list runs larger first, then smaller, so the
# second call reads a scratch the first one filled.
SEQUENCES = [
    # encoded operands (bf16): 2048 x 1536 x 1024 fits the scratch; then a
    # ragged small problem (register-staged, no scratch at all)
    [((1, 2048, 1536, 1024), 256), ((1, 300, 200, 136), 256)],
    # batch groups (2^33 multiply-adds) in plan order on one stream, then
    # a single smaller encoded problem with ragged tiles
    [((8, 1024, 1024, 1024), 256), ((1, 1000, 520, 700), 255)],
    # 4096^3 would need 64 MiB of encoded operands plus the validation word:
    # the register-staged kernels run instead; then a fitting encoded one
    [((1, 4096, 4096, 4096), 256), ((2, 1024, 768, 512), 200)],
    # full int16 range: offset limb route (limb planes + row / column sums),
    # then a smaller one of the same route
    [((1, 1536, 1024, 1024), 0), ((3, 333, 257, 190), 0)],
]


@pytest.mark.parametrize("seq", SEQUENCES, ids=[f"seq{i}" for i in range(len(SEQUENCES))])
def test_noalloc_matches_the_allocating_entry_point(seq):
    for shape, bound in seq:
        _check_pair(shape, bound)


def test_noalloc_plans_fit_the_scratch():
    # what the plans above ask for: encoded paths fit, the 4096^3 one does not
    p = qx.plan_gemm_i16i32(2048, 1536, 1024, 1, 256, 256)
    assert p["kernels"] == 3 and p["workspace_bytes"] + 256 <= SCRATCH
    p = qx.plan_gemm_i16i32(4096, 4096, 4096, 1, 256, 256)
    assert p["workspace_bytes"] + 256 > SCRATCH


def test_noalloc_rejects_oversized_requests_before_launching():
    # full-range int16 with a huge N: even the register-staged offset route
    # needs per-slice column sums beyond the scratch
    L = qx.lib()
    st = L.qgemm_i16i32_noalloc(None, None, None, 64, 1 << 17, 1 << 14, 1, 0, 0, None)
    assert st == qx.ERR_UNSUPPORTED, st
    assert b"allocation-free" in L.qx_last_error()
