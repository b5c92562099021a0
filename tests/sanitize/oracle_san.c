/* Runs every function of the CPU oracle (oracle/oracle.c) on small, ragged
 * and empty shapes under AddressSanitizer and UndefinedBehaviorSanitizer
 * (signed overflow, shifts, out-of-bounds), and checks each against an
 * independent plain loop written here or against the oracle's own second
 * form (conv direct vs im2col, (Q K^T) V vs Q (K^T V)).  Prints "ok" and
 * exits 0 when every check holds; any sanitizer report aborts the run. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void oracle_gemm_i16i32(const int16_t*, const int16_t*, int32_t*, int64_t, int64_t, int64_t, int64_t);
void oracle_gemm_i32_s24(const int32_t*, const int32_t*, int32_t*, int64_t, int64_t, int64_t, int64_t);
void oracle_conv2d_direct(const int16_t*, const int16_t*, int32_t*, int64_t, int64_t, int64_t, int64_t, int64_t,
                          int64_t, int64_t, int64_t, int64_t);
void oracle_conv2d_im2col(const int16_t*, const int16_t*, int32_t*, int64_t, int64_t, int64_t, int64_t, int64_t,
                          int64_t, int64_t, int64_t, int64_t);
void oracle_conv2d_s24_direct(const int32_t*, const int32_t*, int32_t*, int64_t, int64_t, int64_t, int64_t,
                              int64_t, int64_t, int64_t, int64_t, int64_t);
void oracle_conv2d_f64_direct(const float*, const float*, double*, int64_t, int64_t, int64_t, int64_t, int64_t,
                              int64_t, int64_t, int64_t, int64_t);
void oracle_minmax_i32(const int32_t*, int64_t, int32_t*);
void oracle_minmax_i16(const int16_t*, int64_t, int16_t*);
void oracle_avgpool2_i32(const int32_t*, int32_t*, int64_t, int64_t, int64_t, int64_t);
void oracle_maxpool2_f32(const float*, float*, int64_t, int64_t, int64_t, int64_t);
void oracle_sdpa_f64(const float*, const float*, const float*, double*, int64_t, int64_t, int64_t, double, int32_t);
void oracle_attn_i32(const int32_t*, const int32_t*, const int32_t*, int32_t*, int64_t, int64_t);
void oracle_attn_i32_assoc(const int32_t*, const int32_t*, const int32_t*, int32_t*, int64_t, int64_t);
void oracle_attn_f64(const float*, const float*, const float*, double*, int64_t, int64_t);
void oracle_attn_f64_assoc(const float*, const float*, const float*, double*, int64_t, int64_t);
void oracle_attn_f32(const float*, const float*, const float*, float*, int64_t, int64_t);

static uint64_t g_state = 0x9E3779B97F4A7C15ull;
static uint32_t next32(void) {            /* xorshift64*, high half */
    g_state ^= g_state >> 12;
    g_state ^= g_state << 25;
    g_state ^= g_state >> 27;
    return (uint32_t)((g_state * 0x2545F4914F6CDD1Dull) >> 32);
}
static int64_t rnd(int64_t lo, int64_t hi) { return lo + (int64_t)(next32() % (uint64_t)(hi - lo + 1)); }

static int failures = 0;
#define CHECK(c, ...)                                  \
    do {                                               \
        if (!(c)) {                                    \
            fprintf(stderr, "FAIL: " __VA_ARGS__);     \
            fputc('\n', stderr);                       \
            ++failures;                                \
        }                                              \
    } while (0)

static void* xmalloc(size_t n) { return malloc(n ? n : 1); }

static int32_t wrap32(uint64_t v) {
    uint32_t u = (uint32_t)v;
    int32_t r;
    memcpy(&r, &u, 4);
    return r;
}
static int64_t s24(int32_t x) {
    int64_t u = (int64_t)((uint32_t)x & 0xFFFFFFu);
    return u >= 0x800000 ? u - 0x1000000 : u;
}

static void gemms(void) {
    const int64_t shapes[][4] = {{1, 1, 1, 1}, {3, 5, 7, 2}, {17, 9, 33, 1}, {0, 4, 4, 1}, {4, 0, 4, 2},
                                 {4, 4, 0, 1}, {2, 3, 4, 0}, {31, 2, 65, 3}};
    for (size_t s = 0; s < sizeof shapes / sizeof shapes[0]; ++s) {
        const int64_t M = shapes[s][0], N = shapes[s][1], K = shapes[s][2], B = shapes[s][3];
        int16_t* a = xmalloc(sizeof(int16_t) * B * M * K);
        int16_t* b = xmalloc(sizeof(int16_t) * B * K * N);
        int32_t* a32 = xmalloc(sizeof(int32_t) * B * M * K);
        int32_t* b32 = xmalloc(sizeof(int32_t) * B * K * N);
        int32_t* c = xmalloc(sizeof(int32_t) * B * M * N);
        for (int64_t i = 0; i < B * M * K; ++i) {
            a[i] = (int16_t)rnd(-32768, 32767);
            a32[i] = (int32_t)(int64_t)(int32_t)next32();
        }
        for (int64_t i = 0; i < B * K * N; ++i) {
            b[i] = (int16_t)rnd(-32768, 32767);
            b32[i] = (int32_t)next32();
        }
        oracle_gemm_i16i32(a, b, c, M, N, K, B);
        for (int64_t z = 0; z < B; ++z)
            for (int64_t i = 0; i < M; ++i)
                for (int64_t j = 0; j < N; ++j) {
                    uint64_t acc = 0;
                    for (int64_t k = 0; k < K; ++k)
                        acc += (uint64_t)((int64_t)a[(z * M + i) * K + k] * b[(z * K + k) * N + j]);
                    CHECK(c[(z * M + i) * N + j] == wrap32(acc), "gemm_i16i32 %lld %lld %lld", (long long)M,
                          (long long)N, (long long)K);
                }
        oracle_gemm_i32_s24(a32, b32, c, M, N, K, B);
        for (int64_t z = 0; z < B; ++z)
            for (int64_t i = 0; i < M; ++i)
                for (int64_t j = 0; j < N; ++j) {
                    uint64_t acc = 0;
                    for (int64_t k = 0; k < K; ++k)
                        acc += (uint64_t)(s24(a32[(z * M + i) * K + k]) * s24(b32[(z * K + k) * N + j]));
                    CHECK(c[(z * M + i) * N + j] == wrap32(acc), "gemm_i32_s24");
                }
        free(a); free(b); free(a32); free(b32); free(c);
    }
    /* smul24 extremes of the contract */
    int32_t x[2] = {(1 << 23) - 1, -(1 << 23)}, y[2] = {(1 << 23) - 1, -(1 << 23)}, r = 0;
    oracle_gemm_i32_s24(&x[0], &y[0], &r, 1, 1, 1, 1);
    CHECK(r == -16777215, "smul24 (2^23-1)^2");
    oracle_gemm_i32_s24(&x[1], &y[1], &r, 1, 1, 1, 1);
    CHECK(r == 0, "smul24 (-2^23)^2");
    oracle_gemm_i32_s24(&x[1], &y[0], &r, 1, 1, 1, 1);
    CHECK(r == 8388608, "smul24 -2^23 (2^23-1)");
}

static void convs(void) {
    const int64_t cs[][9] = {{1, 1, 5, 5, 1, 3, 3, 1, 1}, {2, 3, 7, 6, 4, 3, 2, 2, 1}, {1, 2, 4, 4, 3, 1, 1, 1, 0},
                             {2, 1, 9, 5, 2, 5, 3, 3, 2}, {0, 2, 4, 4, 2, 3, 3, 1, 1}, {1, 0, 4, 4, 2, 3, 3, 1, 1}};
    for (size_t s = 0; s < sizeof cs / sizeof cs[0]; ++s) {
        const int64_t N = cs[s][0], Ci = cs[s][1], H = cs[s][2], W = cs[s][3], Co = cs[s][4], KH = cs[s][5],
                      KW = cs[s][6], st = cs[s][7], p = cs[s][8];
        const int64_t Ho = (H + 2 * p - KH) / st + 1, Wo = (W + 2 * p - KW) / st + 1;
        const int64_t nx = N * Ci * H * W, nw = Co * Ci * KH * KW, ny = N * Co * Ho * Wo;
        int16_t* x = xmalloc(2 * nx);
        int16_t* w = xmalloc(2 * nw);
        int32_t* x32 = xmalloc(4 * nx);
        int32_t* w32 = xmalloc(4 * nw);
        float* xf = xmalloc(4 * nx);
        float* wf = xmalloc(4 * nw);
        int32_t* y1 = xmalloc(4 * ny);
        int32_t* y2 = xmalloc(4 * ny);
        double* yd = xmalloc(8 * ny);
        for (int64_t i = 0; i < nx; ++i) {
            x[i] = (int16_t)rnd(-32768, 32767);
            x32[i] = (int32_t)next32();
            xf[i] = (float)rnd(-100, 100) / 8.0f;
        }
        for (int64_t i = 0; i < nw; ++i) {
            w[i] = (int16_t)rnd(-32768, 32767);
            w32[i] = (int32_t)next32();
            wf[i] = (float)rnd(-100, 100) / 16.0f;
        }
        oracle_conv2d_direct(x, w, y1, N, Ci, H, W, Co, KH, KW, st, p);
        oracle_conv2d_im2col(x, w, y2, N, Ci, H, W, Co, KH, KW, st, p);
        CHECK(memcmp(y1, y2, 4 * ny) == 0, "conv direct vs im2col case %zu", s);
        oracle_conv2d_s24_direct(x32, w32, y1, N, Ci, H, W, Co, KH, KW, st, p);
        oracle_conv2d_f64_direct(xf, wf, yd, N, Ci, H, W, Co, KH, KW, st, p);
        /* one element of each against a plain sum (the values are small
         * dyadic rationals, so the float64 sum is exact) */
        if (ny > 0) {
            const int64_t n = N - 1, co = Co - 1, oh = Ho / 2, ow = Wo - 1;
            uint64_t acc = 0;
            double accd = 0.0;
            for (int64_t ci = 0; ci < Ci; ++ci)
                for (int64_t kh = 0; kh < KH; ++kh)
                    for (int64_t kw = 0; kw < KW; ++kw) {
                        const int64_t ih = oh * st - p + kh, iw = ow * st - p + kw;
                        if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
                        const int64_t xi = ((n * Ci + ci) * H + ih) * W + iw, wi = ((co * Ci + ci) * KH + kh) * KW + kw;
                        acc += (uint64_t)(s24(x32[xi]) * s24(w32[wi]));
                        accd += (double)xf[xi] * (double)wf[wi];
                    }
            const int64_t yi = ((n * Co + co) * Ho + oh) * Wo + ow;
            CHECK(y1[yi] == wrap32(acc), "conv s24 element");
            CHECK(yd[yi] == accd, "conv f64 element");
        }
        free(x); free(w); free(x32); free(w32); free(xf); free(wf); free(y1); free(y2); free(yd);
    }
}

static void attention(void) {
    const int64_t ls[][2] = {{1, 1}, {5, 3}, {17, 8}, {33, 16}, {0, 4}, {4, 0}};
    for (size_t s = 0; s < sizeof ls / sizeof ls[0]; ++s) {
        const int64_t L = ls[s][0], d = ls[s][1], n = L * d;
        int32_t* q = xmalloc(4 * n);
        int32_t* k = xmalloc(4 * n);
        int32_t* v = xmalloc(4 * n);
        int32_t* o1 = xmalloc(4 * n);
        int32_t* o2 = xmalloc(4 * n);
        float* qf = xmalloc(4 * n);
        float* kf = xmalloc(4 * n);
        float* vf = xmalloc(4 * n);
        float* of = xmalloc(4 * n);
        double* od1 = xmalloc(8 * n);
        double* od2 = xmalloc(8 * n);
        for (int64_t i = 0; i < n; ++i) {
            q[i] = (int32_t)next32();
            k[i] = (int32_t)next32();
            v[i] = (int32_t)next32();
            qf[i] = (float)rnd(-64, 64) / 32.0f;
            kf[i] = (float)rnd(-64, 64) / 32.0f;
            vf[i] = (float)rnd(-64, 64) / 32.0f;
        }
        oracle_attn_i32(q, k, v, o1, L, d);
        oracle_attn_i32_assoc(q, k, v, o2, L, d);
        CHECK(memcmp(o1, o2, 4 * n) == 0, "attention (QK^T)V vs Q(K^T V), L=%lld", (long long)L);
        oracle_attn_f64(qf, kf, vf, od1, L, d);
        oracle_attn_f64_assoc(qf, kf, vf, od2, L, d);
        for (int64_t i = 0; i < n; ++i) CHECK(od1[i] == od2[i], "attention f64 orders (exact on dyadic inputs)");
        oracle_attn_f32(qf, kf, vf, of, L, d);
        for (int64_t i = 0; i < n; ++i) CHECK(fabs(of[i] - od1[i]) <= 1e-3 * (1.0 + fabs(od1[i])), "attention f32");
        for (int causal = 0; causal < 2; ++causal) {
            oracle_sdpa_f64(qf, kf, vf, od1, 1, L, d, 0.5, causal);
            for (int64_t i = 0; i < n; ++i) CHECK(isfinite(od1[i]) && fabs(od1[i]) <= 2.0 + 1e-12, "sdpa range");
        }
        free(q); free(k); free(v); free(o1); free(o2); free(qf); free(kf); free(vf); free(of); free(od1); free(od2);
    }
}

static void reductions(void) {
    for (int64_t n = 1; n < 300; n += 37) {
        int32_t* x = xmalloc(4 * n);
        int16_t* h = xmalloc(2 * n);
        int32_t mm[2], lo = INT32_MAX, hi = INT32_MIN;
        int16_t mh[2];
        int lo16 = 32767, hi16 = -32768;
        for (int64_t i = 0; i < n; ++i) {
            x[i] = (int32_t)next32();
            h[i] = (int16_t)next32();
            lo = x[i] < lo ? x[i] : lo;
            hi = x[i] > hi ? x[i] : hi;
            lo16 = h[i] < lo16 ? h[i] : lo16;
            hi16 = h[i] > hi16 ? h[i] : hi16;
        }
        oracle_minmax_i32(x, n, mm);
        oracle_minmax_i16(h, n, mh);
        CHECK(mm[0] == lo && mm[1] == hi && mh[0] == lo16 && mh[1] == hi16, "minmax n=%lld", (long long)n);
        free(x); free(h);
    }
    const int64_t N = 2, C = 3, H = 7, W = 5, Ho = H / 2, Wo = W / 2;
    int32_t x[2 * 3 * 7 * 5], y[2 * 3 * 3 * 2];
    float xf[2 * 3 * 7 * 5], yf[2 * 3 * 3 * 2];
    for (int i = 0; i < 2 * 3 * 7 * 5; ++i) {
        x[i] = (int32_t)next32();
        xf[i] = (float)rnd(-1000, 1000);
    }
    oracle_avgpool2_i32(x, y, N, C, H, W);
    oracle_maxpool2_f32(xf, yf, N, C, H, W);
    for (int64_t p = 0; p < N * C; ++p)
        for (int64_t i = 0; i < Ho; ++i)
            for (int64_t j = 0; j < Wo; ++j) {
                const int32_t* b = x + (p * H + 2 * i) * W + 2 * j;
                const int64_t sum = (int64_t)b[0] + b[1] + b[W] + b[W + 1];
                const int64_t fl = sum >= 0 ? sum / 4 : -((-sum + 3) / 4);
                CHECK(y[(p * Ho + i) * Wo + j] == fl, "avgpool");
                const float* bf = xf + (p * H + 2 * i) * W + 2 * j;
                float m = bf[0];
                if (bf[1] > m) m = bf[1];
                if (bf[W] > m) m = bf[W];
                if (bf[W + 1] > m) m = bf[W + 1];
                CHECK(yf[(p * Ho + i) * Wo + j] == m, "maxpool");
            }
}

int main(void) {
    gemms();
    convs();
    attention();
    reductions();
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("ok\n");
    return 0;
}
