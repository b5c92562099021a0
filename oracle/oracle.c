/*
 * oracle.c -- plain, slow, obviously correct CPU definitions of what the
 * integer GEMM substrate computes.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header, table or constant
 * with the HIP library.
 *
 * Every function is the plain definition written out as nested loops, with
 * OpenMP over independent output rows and no blocking, fusion or reordering
 * of the contraction.  Integer results are defined modulo 2^32 (two's
 * complement), the reading of "INT32 accumulation" (Methodology; Table 1)
 * that also covers the smul24 contract, whose hardware product keeps the low
 * 32 bits.  Sums are carried in uint64_t, whose wrap-around is well defined
 * in C, so the low 32 bits are exact for every K.
 *
 * Paper sections cited: Methodology (operators, smul24 contract, GEMM-backed
 * convolution through lowering, attention core O = (Q K^T) V), Table 1
 * (INT32 and packed INT16-input / INT32-accumulation GEMM), Table 2 (Conv2D
 * and attention-core rows).
 *
 * Pins: every function here is checked against brute force in Python
 * integers, closed forms and invariants by tests/test_oracle_pins.py.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Two's-complement reinterpretation of the low 32 bits. */
static int32_t low32(uint64_t v) {
    uint32_t u = (uint32_t)v;
    int32_t r;
    memcpy(&r, &u, sizeof r);
    return r;
}

/* The smul24 operand reading (Methodology, smul24 contract): the low 24
 * bits of the word, read as a signed 24-bit integer. */
static int64_t sext24(int32_t x) {
    uint32_t u = (uint32_t)x & 0xFFFFFFu;
    return (u & 0x800000u) ? (int64_t)u - (int64_t)0x1000000 : (int64_t)u;
}

/* Packed INT16-input / INT32-accumulation GEMM (Table 1, right half):
 *   C[b,i,j] = sum_k A[b,i,k] * B[b,k,j]   (mod 2^32)
 * A [batch][M][K], B [batch][K][N], C [batch][M][N], all row-major. */
void oracle_gemm_i16i32(const int16_t* A, const int16_t* B, int32_t* C,
                        int64_t M, int64_t N, int64_t K, int64_t batch) {
    #pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t b = 0; b < batch; ++b) {
        for (int64_t i = 0; i < M; ++i) {
            const int16_t* a = A + (b * M + i) * K;
            const int16_t* bb = B + b * K * N;
            uint64_t* acc = (uint64_t*)calloc((size_t)(N > 0 ? N : 1), sizeof(uint64_t));
            for (int64_t k = 0; k < K; ++k) {
                int64_t av = a[k];
                const int16_t* brow = bb + k * N;
                for (int64_t j = 0; j < N; ++j)
                    acc[j] += (uint64_t)(av * (int64_t)brow[j]);
            }
            int32_t* c = C + (b * M + i) * N;
            for (int64_t j = 0; j < N; ++j) c[j] = low32(acc[j]);
            free(acc);
        }
    }
}

/* INT32 GEMM under the smul24 contract (Methodology; Table 1, left half):
 *   C[b,i,j] = sum_k sext24(A[b,i,k]) * sext24(B[b,k,j])   (mod 2^32)
 * Summing low-32-bit products with wrap-around gives the same value, since
 * reduction mod 2^32 is a ring homomorphism. */
void oracle_gemm_i32_s24(const int32_t* A, const int32_t* B, int32_t* C,
                         int64_t M, int64_t N, int64_t K, int64_t batch) {
    #pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t b = 0; b < batch; ++b) {
        for (int64_t i = 0; i < M; ++i) {
            const int32_t* a = A + (b * M + i) * K;
            const int32_t* bb = B + b * K * N;
            uint64_t* acc = (uint64_t*)calloc((size_t)(N > 0 ? N : 1), sizeof(uint64_t));
            for (int64_t k = 0; k < K; ++k) {
                int64_t av = sext24(a[k]);
                const int32_t* brow = bb + k * N;
                for (int64_t j = 0; j < N; ++j)
                    acc[j] += (uint64_t)(av * sext24(brow[j]));
            }
            int32_t* c = C + (b * M + i) * N;
            for (int64_t j = 0; j < N; ++j) c[j] = low32(acc[j]);
            free(acc);
        }
    }
}

static int64_t conv_out_dim(int64_t in, int64_t k, int64_t stride, int64_t pad) {
    return (in + 2 * pad - k) / stride + 1;
}

/* Conv2D, direct form (Methodology: GEMM-backed convolution; Table 2,
 * INT16-IN/INT32-ACC row).  Cross-correlation with zero padding, no bias,
 * dilation or groups; x NCHW int16, w OIHW int16, y NCHW (mod 2^32). */
void oracle_conv2d_direct(const int16_t* x, const int16_t* w, int32_t* y,
                          int64_t N, int64_t Ci, int64_t H, int64_t W, int64_t Co,
                          int64_t KH, int64_t KW, int64_t stride, int64_t pad) {
    int64_t Ho = conv_out_dim(H, KH, stride, pad);
    int64_t Wo = conv_out_dim(W, KW, stride, pad);
    #pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t co = 0; co < Co; ++co) {
            for (int64_t oh = 0; oh < Ho; ++oh) {
                for (int64_t ow = 0; ow < Wo; ++ow) {
                    uint64_t acc = 0;
                    for (int64_t ci = 0; ci < Ci; ++ci) {
                        for (int64_t kh = 0; kh < KH; ++kh) {
                            int64_t ih = oh * stride - pad + kh;
                            if (ih < 0 || ih >= H) continue;
                            for (int64_t kw = 0; kw < KW; ++kw) {
                                int64_t iw = ow * stride - pad + kw;
                                if (iw < 0 || iw >= W) continue;
                                int64_t xv = x[((n * Ci + ci) * H + ih) * W + iw];
                                int64_t wv = w[((co * Ci + ci) * KH + kh) * KW + kw];
                                acc += (uint64_t)(xv * wv);
                            }
                        }
                    }
                    y[((n * Co + co) * Ho + oh) * Wo + ow] = low32(acc);
                }
            }
        }
    }
}

/* Conv2D through lowering (Methodology): im2col then the GEMM above.
 *   col[(ci*KH + kh)*KW + kw][(n*Ho + oh)*Wo + ow] = x[n, ci, oh*s-p+kh, ow*s-p+kw]
 * (zero outside the image), Y = Wmat[Co][Ci*KH*KW] . col, scattered to NCHW. */
void oracle_conv2d_im2col(const int16_t* x, const int16_t* w, int32_t* y,
                          int64_t N, int64_t Ci, int64_t H, int64_t W, int64_t Co,
                          int64_t KH, int64_t KW, int64_t stride, int64_t pad) {
    int64_t Ho = conv_out_dim(H, KH, stride, pad);
    int64_t Wo = conv_out_dim(W, KW, stride, pad);
    int64_t Kd = Ci * KH * KW, P = N * Ho * Wo;
    int16_t* col = (int16_t*)calloc((size_t)(Kd * P > 0 ? Kd * P : 1), sizeof(int16_t));
    int32_t* g = (int32_t*)calloc((size_t)(Co * P > 0 ? Co * P : 1), sizeof(int32_t));
    for (int64_t ci = 0; ci < Ci; ++ci)
        for (int64_t kh = 0; kh < KH; ++kh)
            for (int64_t kw = 0; kw < KW; ++kw) {
                int64_t r = (ci * KH + kh) * KW + kw;
                for (int64_t n = 0; n < N; ++n)
                    for (int64_t oh = 0; oh < Ho; ++oh)
                        for (int64_t ow = 0; ow < Wo; ++ow) {
                            int64_t ih = oh * stride - pad + kh, iw = ow * stride - pad + kw;
                            int16_t v = 0;
                            if (ih >= 0 && ih < H && iw >= 0 && iw < W)
                                v = x[((n * Ci + ci) * H + ih) * W + iw];
                            col[r * P + (n * Ho + oh) * Wo + ow] = v;
                        }
            }
    oracle_gemm_i16i32(w, col, g, Co, P, Kd, 1);
    for (int64_t n = 0; n < N; ++n)
        for (int64_t co = 0; co < Co; ++co)
            for (int64_t p = 0; p < Ho * Wo; ++p)
                y[(n * Co + co) * Ho * Wo + p] = g[co * P + n * Ho * Wo + p];
    free(col);
    free(g);
}

/* Conv2D on INT32 operands (Table 2, Conv2D INT32 row) under the smul24
 * contract (Methodology): each operand word is read as sext24 of its low 24
 * bits, products keep their low 32 bits, sums wrap mod 2^32.  Same geometry
 * and layout as oracle_conv2d_direct. */
void oracle_conv2d_s24_direct(const int32_t* x, const int32_t* w, int32_t* y,
                              int64_t N, int64_t Ci, int64_t H, int64_t W, int64_t Co,
                              int64_t KH, int64_t KW, int64_t stride, int64_t pad) {
    int64_t Ho = conv_out_dim(H, KH, stride, pad);
    int64_t Wo = conv_out_dim(W, KW, stride, pad);
    #pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t co = 0; co < Co; ++co) {
            for (int64_t oh = 0; oh < Ho; ++oh) {
                for (int64_t ow = 0; ow < Wo; ++ow) {
                    uint64_t acc = 0;
                    for (int64_t ci = 0; ci < Ci; ++ci) {
                        for (int64_t kh = 0; kh < KH; ++kh) {
                            int64_t ih = oh * stride - pad + kh;
                            if (ih < 0 || ih >= H) continue;
                            for (int64_t kw = 0; kw < KW; ++kw) {
                                int64_t iw = ow * stride - pad + kw;
                                if (iw < 0 || iw >= W) continue;
                                int64_t xv = sext24(x[((n * Ci + ci) * H + ih) * W + iw]);
                                int64_t wv = sext24(w[((co * Ci + ci) * KH + kh) * KW + kw]);
                                acc += (uint64_t)(xv * wv);
                            }
                        }
                    }
                    y[((n * Co + co) * Ho + oh) * Wo + ow] = low32(acc);
                }
            }
        }
    }
}

/* Conv2D on FP32 operands (Table 2, Conv2D FP32 row), the reference the GPU
 * result is held to: every product and sum in float64 from the float32
 * inputs, in the plain (ci, kh, kw) order.  Same geometry and layout as
 * oracle_conv2d_direct; y is float64. */
void oracle_conv2d_f64_direct(const float* x, const float* w, double* y,
                              int64_t N, int64_t Ci, int64_t H, int64_t W, int64_t Co,
                              int64_t KH, int64_t KW, int64_t stride, int64_t pad) {
    int64_t Ho = conv_out_dim(H, KH, stride, pad);
    int64_t Wo = conv_out_dim(W, KW, stride, pad);
    #pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t co = 0; co < Co; ++co) {
            for (int64_t oh = 0; oh < Ho; ++oh) {
                for (int64_t ow = 0; ow < Wo; ++ow) {
                    double acc = 0.0;
                    for (int64_t ci = 0; ci < Ci; ++ci) {
                        for (int64_t kh = 0; kh < KH; ++kh) {
                            int64_t ih = oh * stride - pad + kh;
                            if (ih < 0 || ih >= H) continue;
                            for (int64_t kw = 0; kw < KW; ++kw) {
                                int64_t iw = ow * stride - pad + kw;
                                if (iw < 0 || iw >= W) continue;
                                double xv = x[((n * Ci + ci) * H + ih) * W + iw];
                                double wv = w[((co * Ci + ci) * KH + kh) * KW + kw];
                                acc += xv * wv;
                            }
                        }
                    }
                    y[((n * Co + co) * Ho + oh) * Wo + ow] = acc;
                }
            }
        }
    }
}

/* Min/max reduction (Table 2, Min/max rows): out[0] = min, out[1] = max of
 * the n values; n >= 1. */
void oracle_minmax_i32(const int32_t* x, int64_t n, int32_t* out) {
    int32_t lo = x[0], hi = x[0];
    for (int64_t i = 1; i < n; ++i) {
        if (x[i] < lo) lo = x[i];
        if (x[i] > hi) hi = x[i];
    }
    out[0] = lo;
    out[1] = hi;
}

void oracle_minmax_i16(const int16_t* x, int64_t n, int16_t* out) {
    int16_t lo = x[0], hi = x[0];
    for (int64_t i = 1; i < n; ++i) {
        if (x[i] < lo) lo = x[i];
        if (x[i] > hi) hi = x[i];
    }
    out[0] = lo;
    out[1] = hi;
}

/* 2x2 pooling with stride 2, no padding (Table 2, AvgPool INT32 and MaxPool
 * FP32 rows): x NCHW [N][C][H][W] -> y [N][C][H/2][W/2] (floor; a trailing
 * odd row or column is dropped).  The INT32 average is the floor of the
 * exact sum of the four values divided by 4. */
void oracle_avgpool2_i32(const int32_t* x, int32_t* y, int64_t N, int64_t C, int64_t H, int64_t W) {
    const int64_t Ho = H / 2, Wo = W / 2;
    for (int64_t nc = 0; nc < N * C; ++nc)
        for (int64_t oh = 0; oh < Ho; ++oh)
            for (int64_t ow = 0; ow < Wo; ++ow) {
                const int32_t* p = x + (nc * H + 2 * oh) * W + 2 * ow;
                int64_t s = (int64_t)p[0] + p[1] + p[W] + p[W + 1];
                int64_t q = s / 4;
                if (s % 4 != 0 && s < 0) q -= 1;   /* floor, not truncation */
                y[(nc * Ho + oh) * Wo + ow] = (int32_t)q;
            }
}

void oracle_maxpool2_f32(const float* x, float* y, int64_t N, int64_t C, int64_t H, int64_t W) {
    const int64_t Ho = H / 2, Wo = W / 2;
    for (int64_t nc = 0; nc < N * C; ++nc)
        for (int64_t oh = 0; oh < Ho; ++oh)
            for (int64_t ow = 0; ow < Wo; ++ow) {
                const float* p = x + (nc * H + 2 * oh) * W + 2 * ow;
                float m = p[0];
                if (p[1] > m) m = p[1];
                if (p[W] > m) m = p[W];
                if (p[W + 1] > m) m = p[W + 1];
                y[(nc * Ho + oh) * Wo + ow] = m;
            }
}

/* Scaled dot-product attention with softmax (Table 2 footnote: the FP32
 * attention baseline is SDPA with softmax; the attention core extended by
 * the softmax, Discussion), the float64 reference: for each of the BH heads
 * and each query i,
 *   s_j = scale * sum_t Q[i][t] K[j][t]   over keys j (j <= i if causal),
 *   O[i] = sum_j exp(s_j - max_j s_j) V[j] / sum_j exp(s_j - max_j s_j).
 * Q, K, V float32 [BH][L][d]; O float64 [BH][L][d]. */
void oracle_sdpa_f64(const float* Q, const float* K, const float* V, double* O,
                     int64_t BH, int64_t L, int64_t d, double scale, int32_t causal) {
    #pragma omp parallel for collapse(2) schedule(dynamic, 4)
    for (int64_t h = 0; h < BH; ++h) {
        for (int64_t i = 0; i < L; ++i) {
            const float* q = Q + (h * L + i) * d;
            const int64_t nk = causal ? i + 1 : L;
            double* s = (double*)malloc((size_t)(nk > 0 ? nk : 1) * sizeof(double));
            double mx = -INFINITY;
            for (int64_t j = 0; j < nk; ++j) {
                const float* k = K + (h * L + j) * d;
                double acc = 0.0;
                for (int64_t t = 0; t < d; ++t) acc += (double)q[t] * (double)k[t];
                s[j] = scale * acc;
                if (s[j] > mx) mx = s[j];
            }
            double den = 0.0;
            for (int64_t j = 0; j < nk; ++j) {
                s[j] = exp(s[j] - mx);
                den += s[j];
            }
            double* o = O + (h * L + i) * d;
            for (int64_t t = 0; t < d; ++t) o[t] = 0.0;
            for (int64_t j = 0; j < nk; ++j) {
                const float* v = V + (h * L + j) * d;
                for (int64_t t = 0; t < d; ++t) o[t] += s[j] * (double)v[t];
            }
            for (int64_t t = 0; t < d; ++t) o[t] /= den;
            free(s);
        }
    }
}

/* Attention core, INT32 (Methodology: O = (Q K^T) V; Table 2, INT32 row).
 * No scale, softmax or mask; one head; Q, K, V, O are [L][d] row-major.
 * S = Q K^T is formed exactly, then O = S V (mod 2^32). */
void oracle_attn_i32(const int32_t* Q, const int32_t* K, const int32_t* V, int32_t* O,
                     int64_t L, int64_t d) {
    #pragma omp parallel for schedule(dynamic, 4)
    for (int64_t i = 0; i < L; ++i) {
        uint64_t* acc = (uint64_t*)calloc((size_t)(d > 0 ? d : 1), sizeof(uint64_t));
        for (int64_t j = 0; j < L; ++j) {
            uint64_t s = 0;
            for (int64_t t = 0; t < d; ++t)
                s += (uint64_t)((int64_t)Q[i * d + t] * (int64_t)K[j * d + t]);
            for (int64_t t = 0; t < d; ++t)
                acc[t] += s * (uint64_t)(int64_t)V[j * d + t];
        }
        for (int64_t t = 0; t < d; ++t) O[i * d + t] = low32(acc[t]);
        free(acc);
    }
}

/* The other association, Q (K^T V) (mod 2^32).  Associativity holds exactly
 * in the ring Z/2^32, so this must equal oracle_attn_i32 bit for bit; it is
 * an invariant for the tests, never a route for the GPU (it does O(L d^2)
 * work instead of O(L^2 d)). */
void oracle_attn_i32_assoc(const int32_t* Q, const int32_t* K, const int32_t* V, int32_t* O,
                           int64_t L, int64_t d) {
    uint64_t* T = (uint64_t*)calloc((size_t)(d * d > 0 ? d * d : 1), sizeof(uint64_t));
    for (int64_t j = 0; j < L; ++j)
        for (int64_t a = 0; a < d; ++a)
            for (int64_t c = 0; c < d; ++c)
                T[a * d + c] += (uint64_t)((int64_t)K[j * d + a] * (int64_t)V[j * d + c]);
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < L; ++i)
        for (int64_t c = 0; c < d; ++c) {
            uint64_t s = 0;
            for (int64_t a = 0; a < d; ++a)
                s += (uint64_t)(int64_t)Q[i * d + a] * T[a * d + c];
            O[i * d + c] = low32(s);
        }
    free(T);
}

/* Attention core, FP32 inputs (Table 2, FP32 row): the reference R = (Q K^T) V
 * evaluated in float64 from the float32 inputs.  Sums run in index order. */
void oracle_attn_f64(const float* Q, const float* K, const float* V, double* O,
                     int64_t L, int64_t d) {
    #pragma omp parallel for schedule(dynamic, 4)
    for (int64_t i = 0; i < L; ++i) {
        double* acc = (double*)calloc((size_t)(d > 0 ? d : 1), sizeof(double));
        for (int64_t j = 0; j < L; ++j) {
            double s = 0.0;
            for (int64_t t = 0; t < d; ++t) s += (double)Q[i * d + t] * (double)K[j * d + t];
            for (int64_t t = 0; t < d; ++t) acc[t] += s * (double)V[j * d + t];
        }
        for (int64_t t = 0; t < d; ++t) O[i * d + t] = acc[t];
        free(acc);
    }
}

/* Q (K^T V) in float64: an independent evaluation order of the same
 * mathematical value, used only as a cross-check of the float64 reference. */
void oracle_attn_f64_assoc(const float* Q, const float* K, const float* V, double* O,
                           int64_t L, int64_t d) {
    double* T = (double*)calloc((size_t)(d * d > 0 ? d * d : 1), sizeof(double));
    for (int64_t j = 0; j < L; ++j)
        for (int64_t a = 0; a < d; ++a)
            for (int64_t c = 0; c < d; ++c)
                T[a * d + c] += (double)K[j * d + a] * (double)V[j * d + c];
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < L; ++i)
        for (int64_t c = 0; c < d; ++c) {
            double s = 0.0;
            for (int64_t a = 0; a < d; ++a) s += (double)Q[i * d + a] * T[a * d + c];
            O[i * d + c] = s;
        }
    free(T);
}

/* The same definition in plain float32 with sequential summation: the
 * textbook single-precision evaluation, whose error against the float64
 * reference shows what FP32 arithmetic alone costs. */
void oracle_attn_f32(const float* Q, const float* K, const float* V, float* O,
                     int64_t L, int64_t d) {
    #pragma omp parallel for schedule(dynamic, 4)
    for (int64_t i = 0; i < L; ++i) {
        float* acc = (float*)calloc((size_t)(d > 0 ? d : 1), sizeof(float));
        for (int64_t j = 0; j < L; ++j) {
            float s = 0.0f;
            for (int64_t t = 0; t < d; ++t) s += Q[i * d + t] * K[j * d + t];
            for (int64_t t = 0; t < d; ++t) acc[t] += s * V[j * d + t];
        }
        for (int64_t t = 0; t < d; ++t) O[i * d + t] = acc[t];
        free(acc);
    }
}
