// Runs the host side of libqx -- argument validation, the planner of every
// operation, and the executor's create / run / destroy bookkeeping through
// the host double of the device runtime -- under AddressSanitizer and
// UndefinedBehaviorSanitizer.  No kernel runs (the double only checks each
// launch's geometry).  Prints "ok" and exits 0 when every call returned what
// it should; any sanitizer report aborts the run.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <initializer_list>
#include <vector>

#include "../../include/qx.h"
#include "../../include/qx_testing.h"

static int failures = 0;
#define CHECK(c, ...)                               \
    do {                                            \
        if (!(c)) {                                 \
            fprintf(stderr, "FAIL: " __VA_ARGS__);  \
            fprintf(stderr, " (%s)\n", qx_last_error()); \
            ++failures;                             \
        }                                           \
    } while (0)

static void planner() {
    qx_plan_info info;
    const int64_t dims[] = {0, 1, 2, 15, 31, 63, 64, 65, 127, 129, 255, 511, 1023, 4097};
    const int32_t bounds[] = {0, 1, 127, 128, 255, 256, 383, 724, 725, 1024, 2048, 8127, 8128, 32768};
    for (int64_t M : dims)
        for (int64_t N : {1, 64, 300})
            for (int64_t K : {0, 1, 64, 1000, 9000})
                for (int32_t b : bounds)
                    for (int32_t r = 0; r <= 7; ++r) {
                        const qx_status st = qx_plan_gemm_i16i32(&info, M, N, K, 3, b, b, r);
                        CHECK(st == QX_OK || st == QX_ERR_RANGE || st == QX_ERR_INVALID_ARG, "plan gemm");
                        if (r == 0) CHECK(st == QX_OK, "plan gemm auto");
                    }
    for (int64_t M : dims) {
        CHECK(qx_plan_gemm_i32_s24(&info, M, M + 3, 2 * M + 1, 2, 0) == QX_OK, "plan s24");
        CHECK(qx_plan_gemm_i32_s24(&info, M, 17, M, 1, 6) == QX_OK, "plan s24 valu");
    }
    // edges: negative sizes, overflowing products, bad enums and pointers
    CHECK(qx_plan_gemm_i16i32(&info, -1, 4, 4, 1, 0, 0, 0) == QX_ERR_INVALID_ARG, "negative M");
    CHECK(qx_plan_gemm_i16i32(&info, 1LL << 30, 1LL << 30, 1LL << 30, 1, 0, 0, 0) == QX_ERR_UNSUPPORTED, "2^90");
    CHECK(qx_plan_gemm_i16i32(&info, 4, 4, 4, 1, -3, 0, 0) == QX_ERR_INVALID_ARG, "bound < 0");
    CHECK(qx_plan_gemm_i16i32(&info, 4, 4, 4, 1, 0, 0, 99) == QX_ERR_INVALID_ARG, "route 99");
    CHECK(qx_plan_gemm_i16i32(nullptr, 4, 4, 4, 1, 0, 0, 0) == QX_ERR_INVALID_ARG, "null out");
    CHECK(qx_plan_gemm_i16i32(&info, 4, 4, 4, 70000, 0, 0, 0) == QX_ERR_UNSUPPORTED, "batch");
    for (int64_t s = 1; s <= 3; ++s)
        for (int64_t p = 0; p <= 2; ++p)
            for (int64_t ci : {1, 3, 64, 96})
                for (int32_t b : {0, 255, 256, 1024}) {
                    CHECK(qx_plan_conv2d(&info, 2, ci, 13, 11, 5, 3, 3, s, p, b, b, 0) == QX_OK, "plan conv");
                    CHECK(qx_plan_conv2d_t(&info, QX_DT_F32, 2, ci, 13, 11, 5, 3, 3, s, p, 0) == QX_OK, "conv f32");
                    CHECK(qx_plan_conv2d_t(&info, QX_DT_I32, 2, ci, 13, 11, 5, 3, 3, s, p, 0) == QX_OK, "conv i32");
                }
    CHECK(qx_plan_conv2d(&info, 1, 1, 2, 2, 1, 5, 5, 1, 0, 0, 0, 0) != QX_OK, "kernel larger than the image");
    CHECK(qx_plan_conv2d(&info, 1, 1, 8, 8, 1, 3, 3, 0, 0, 0, 0, 0) == QX_ERR_INVALID_ARG, "stride 0");
    for (int64_t L : {0, 1, 31, 100, 4096})
        for (int64_t d : {0, 1, 32, 48, 64, 96, 128, 256}) {
            for (int32_t r = 0; r <= 11; ++r) (void)qx_plan_attn(&info, QX_DT_F32, L, d, 0, r);
            for (int32_t b : {0, 63, 64, 127, 128})
                for (int32_t r = 0; r <= 11; ++r) (void)qx_plan_attn(&info, QX_DT_I32, L, d, b, r);
            CHECK(qx_plan_attn(&info, QX_DT_I32, L, d, 64, 0) == (d <= 256 ? QX_OK : QX_ERR_UNSUPPORTED),
                  "plan attn");
            CHECK(qx_plan_sdpa_f32(&info, 3, L, d, 0.125f, 1) == (d <= 128 ? QX_OK : QX_ERR_UNSUPPORTED),
                  "plan sdpa");
        }
    CHECK(qx_plan_attn(&info, (qx_attn_dtype)7, 4, 4, 0, 0) == QX_ERR_INVALID_ARG, "attn dtype");
    for (int64_t n : {(int64_t)1, (int64_t)63, (int64_t)64, (int64_t)1000, (int64_t)1 << 27}) {
        CHECK(qx_plan_minmax(&info, n, 4) == QX_OK, "plan minmax");
        CHECK(qx_plan_minmax(&info, n, 2) == QX_OK, "plan minmax i16");
    }
    CHECK(qx_plan_minmax(&info, 0, 4) == QX_ERR_INVALID_ARG, "minmax n = 0");
    CHECK(qx_plan_minmax(&info, 10, 3) == QX_ERR_INVALID_ARG, "minmax element size");
    for (int32_t k : {0, 1})
        for (int64_t h : {1, 2, 7, 224}) CHECK(qx_plan_pool2x2(&info, k, 2, 3, h, h + 1) == QX_OK, "plan pool");
    for (int64_t b : {0, 1, 7, 4096}) CHECK(qx_plan_lenet_i32(&info, b) == QX_OK, "plan lenet");
}

static void executors() {
    CHECK(qx_testing_host_double(1) == QX_OK, "host double on");
    std::vector<void*> in(6);
    for (int i = 0; i < 6; ++i) in[i] = (void*)(uintptr_t)((uint64_t)(i + 1) << 32);
    void* out = (void*)(uintptr_t)((uint64_t)64 << 32);
    auto cycle = [&](qx_status st, qx_exec h, const char* what) {
        CHECK(st == QX_OK && h, "create %s", what);
        if (st != QX_OK) return;
        for (int r = 0; r < 2; ++r) CHECK(qx_exec_run(h, in.data(), out, nullptr) == QX_OK, "run %s", what);
        float ms[64];
        const char* names[64];
        CHECK(qx_exec_profile(h, in.data(), out, nullptr, 2, ms, names, 64) == QX_OK, "profile %s", what);
        CHECK(qx_exec_destroy(h) == QX_OK, "destroy %s", what);
        CHECK(qx_exec_destroy(h) == QX_ERR_INVALID_ARG, "second destroy %s", what);
    };
    qx_exec h = nullptr;
    cycle(qx_exec_create_gemm_i16i32(&h, 8192, 8192, 8192, 1, 256, 256), h, "gemm 8192");
    cycle(qx_exec_create_gemm_i16i32(&h, 2048, 2048, 2048, 64, 256, 256), h, "gemm 64x2048");
    cycle(qx_exec_create_gemm_i16i32(&h, 300, 200, 5000, 3, 0, 0), h, "gemm offset");
    cycle(qx_exec_create_gemm_i16i32_route(&h, 1000, 1000, 1000, 1, 8127, 8127, 3), h, "gemm karatsuba");
    cycle(qx_exec_create_gemm_i32_s24(&h, 1024, 1024, 1024, 1), h, "s24");
    cycle(qx_exec_create_gemm_i32_s24_route(&h, 512, 512, 512, 16, 6), h, "s24 valu");
    cycle(qx_exec_create_conv2d(&h, 8, 64, 56, 56, 128, 3, 3, 1, 1, 256, 256), h, "conv");
    cycle(qx_exec_create_conv2d_t(&h, QX_DT_I32, 8, 64, 56, 56, 128, 3, 3, 1, 1, 0), h, "conv i32");
    cycle(qx_exec_create_conv2d_t(&h, QX_DT_F32, 8, 64, 56, 56, 128, 3, 3, 1, 1, 0), h, "conv f32");
    cycle(qx_exec_create_attn(&h, QX_DT_F32, 4096, 64, 0), h, "attn f32");
    cycle(qx_exec_create_attn(&h, QX_DT_I32, 4096, 64, 64), h, "attn i32");
    cycle(qx_exec_create_sdpa_f32(&h, 32, 4096, 64, 1.0f, 1), h, "sdpa");
    cycle(qx_exec_create_lenet_i32(&h, 4096), h, "lenet");
    cycle(qx_exec_create_minmax(&h, 1 << 27, 4), h, "minmax");
    cycle(qx_exec_create_pool2x2(&h, 0, 16, 64, 224, 224), h, "pool");
    // an injected failure of the one acquisition (the workspace), then past it
    setenv("QX_TEST_FAIL_ALLOC", "1", 1);
    qx_exec f = (qx_exec)(uintptr_t)1;
    CHECK(qx_exec_create_gemm_i16i32(&f, 2048, 2048, 2048, 64, 256, 256) == QX_ERR_OUT_OF_MEMORY && f == nullptr,
          "injected failure");
    setenv("QX_TEST_FAIL_ALLOC", "2", 1);
    cycle(qx_exec_create_gemm_i16i32(&f, 2048, 2048, 2048, 64, 256, 256), f, "past the injected failure");
    unsetenv("QX_TEST_FAIL_ALLOC");
    int64_t c[6];
    qx_testing_counters(c, 6);
    CHECK(c[0] == c[1] && c[2] == c[3] && c[5] == 0, "every resource released");
    // one-shot calls under the double
    for (int r = 0; r < 3; ++r)
        CHECK(qgemm_i16i32((const int16_t*)in[0], (const int16_t*)in[1], (int32_t*)out, 512, 512, 512, 1, 256, 256,
                           nullptr) == QX_OK, "one-shot");
    qx_release_cache();
    CHECK(qx_testing_host_double(0) == QX_OK, "host double off");
}

int main() {
    planner();
    executors();
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("ok\n");
    return 0;
}
