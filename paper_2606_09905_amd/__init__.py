"""MI355X (gfx950) tiled integer matrix-multiplication substrate.

The C ABI lives in include/qx.h and libqx.so; this package is its thin
binding (qx.py), the in-tree build (build.py) and the seeded synthetic
workloads (workloads.py).
"""
from . import qx  # noqa: F401
from .qx import (Executor, QxError, attn_core, conv2d_gemm, qgemm_i16i32,  # noqa: F401
                 qgemm_i32_s24)
