/*
 * qx_testing.h -- test seams of libqx.  Not part of the operations'
 * interface (include/qx.h); meant for the library's own tests of the
 * executor's bookkeeping, which must also run on machines without a GPU.
 *
 * Nothing here computes a result: while the host double is on, operations
 * are planned, their resources counted and their launches checked, but no
 * kernel runs and no output is written.
 */
#ifndef QX_TESTING_H
#define QX_TESTING_H

#include <stdint.h>

#include "qx.h"

#ifdef __cplusplus
extern "C" {
#endif

/* on = 1: every later executor create (and one-shot call) uses a host-only
 * double of the device runtime: it reports one gfx950 device, gives
 * workspaces host memory, creates dummy timing events, and for every
 * launch checks the grid against the hardware limits (x * block <= 2^32 - 1,
 * y, z <= 65535, 1..1024 threads per workgroup, <= 160 KiB of LDS) and that
 * every pointer slot of the parameter block is bound, instead of enqueueing
 * it; a failed check is QX_ERR_DEVICE.  on = 0 returns to the HIP runtime.
 * Switching releases the one-shot cache first and returns
 * QX_ERR_INVALID_ARG if other handles are still live.  Handles keep the
 * runtime they were created with. */
qx_status qx_testing_host_double(int32_t on);

/* Counters since the library was loaded, both runtimes together:
 * out[0] workspace allocations, out[1] workspace frees, out[2] timing events
 * created (qx_exec_profile), out[3] timing events destroyed, out[4] kernel
 * launches enqueued (or checked, under the double), out[5] live executor
 * handles.  Writes min(n, 6) values.
 *
 * Fault injection: with the environment variable QX_TEST_FAIL_ALLOC=k
 * (read at every executor create), the k-th device resource that create
 * acquires (counted from 1; a create acquires at most one, its workspace)
 * fails as if the device were out of memory: the create returns
 * QX_ERR_OUT_OF_MEMORY, *out is NULL, and nothing stays allocated. */
void qx_testing_counters(int64_t* out, int32_t n);

#ifdef __cplusplus
}
#endif

#endif /* QX_TESTING_H */
