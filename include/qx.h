/*
 * qx.h -- C ABI of the MI355X (gfx950) tiled integer matrix-multiplication
 * substrate: packed INT16-input / INT32-accumulation GEMM, INT32 GEMM under
 * the smul24 operand contract, GEMM-backed Conv2D through im2col lowering,
 * the single-head attention core O = (Q K^T) V, and a persistent executor.
 *
 * The operations follow the paper's Methodology: one tiled integer GEMM
 * that every operator reuses, convolution lowered onto it, the attention
 * core O = (Q K^T) V, handles that plan and allocate a single time, and
 * caller-declared operand bounds from which the exact route is chosen.  The
 * paper measures them in Table 1 (INT32 and packed INT16 / INT32-accumulation
 * GEMM) and Table 2 (Conv2D and attention-core rows).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensors are caller-owned DEVICE pointers (HIP device memory of the
 *    current device), dense and row-major, never freed or kept by the
 *    library.  Pointers to operands with zero elements may be NULL.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Work is enqueued on it; a return of QX_OK means "enqueued", nothing is
 *    synchronised.
 *  - Integer results are exact modulo 2^32 (two's complement), the reading
 *    of "INT32 accumulation" used throughout.  When the declared contract
 *    guarantees |result| < 2^31 no wrap ever happens.
 *  - Arguments are validated on the host before any HIP call; a failure
 *    returns a status and leaves a message in qx_last_error().  HIP errors
 *    map to QX_ERR_DEVICE (QX_ERR_OUT_OF_MEMORY for allocation failures).
 *  - Operand-range contracts (`bound_*` = largest |x| the caller promises)
 *    pick the exact route.  Operands outside a declared bound give an
 *    unspecified but memory-safe result.  0 means "no promise": the full
 *    range of the type.
 *  - With the environment variable QX_VALIDATE=1 (read at every run), a run
 *    first scans every bounded operand on the device and waits for the
 *    scan: if any |x| exceeds its declared bound the run returns
 *    QX_ERR_RANGE without launching the operation (the output is left
 *    untouched).  Such runs synchronise the stream.  The smul24 GEMM and
 *    FP32 attention have no bounds to check (smul24 reads the low 24 bits
 *    of any int32 by definition).
 *  - One-shot calls keep an internal plan + workspace cache keyed by shape,
 *    contract, route, device and stream; calls that share a key must not
 *    overlap in time.  Executor handles are not thread-safe; different
 *    handles may run concurrently on different streams.
 *  - Only gfx950 devices are supported (QX_ERR_UNSUPPORTED otherwise).
 */
#ifndef QX_H
#define QX_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    QX_OK = 0,
    QX_ERR_INVALID_ARG = 1,   /* null pointer, negative size, size overflow, bad enum */
    QX_ERR_UNSUPPORTED = 2,   /* valid request the library cannot run (device, route, shape) */
    QX_ERR_RANGE = 3,         /* declared bound outside what the operation accepts,
                                 or (QX_VALIDATE=1) an operand outside its declared bound */
    QX_ERR_OUT_OF_MEMORY = 4, /* workspace allocation failed */
    QX_ERR_DEVICE = 5         /* a HIP call failed; details in qx_last_error() */
} qx_status;

typedef enum { QX_DT_F32 = 0, QX_DT_I32 = 1 } qx_attn_dtype;

/* Exact routes of the integer contraction (chosen from the contract).
 *  I8_DIRECT    operands in [-127, 127]: one int8 MFMA product per multiply-add.
 *  F16_EXACT    |a|, |b| <= 2048 and chunk*|a|max*|b|max <= 2^24: fp16 MFMA with
 *               fp32 partial sums over `chunk` K-steps (every partial is an exactly
 *               representable integer), flushed into int32.  Large problems whose
 *               bounds are both <= 256 encode the operands as bf16 instead (also
 *               exact there) and run the bf16 MFMA; operand_format reports it.
 *  I8_KARATSUBA operands in [-8127, 8127]: balanced base-128 limbs h, l and h+l,
 *               three int8 MFMA products.
 *  I8_OFFSET4   any int16: offset base-256 limbs, four int8 MFMA products plus a
 *               rank-1 correction from row and column sums.
 *  VALU_DOT2    any int16: v_dot2_i32_i16 on the vector ALU (comparison path).
 *  S24_VALU     smul24: v_mad_i32_i24-class vector multiply (contract-native).
 *  S24_I8LIMB   smul24: three offset int8 limbs, eight int8 MFMA products with
 *               i+j <= 3, plus a rank-1 correction. */
typedef enum {
    QX_ROUTE_AUTO = 0,
    QX_ROUTE_I8_DIRECT = 1,
    QX_ROUTE_F16_EXACT = 2,
    QX_ROUTE_I8_KARATSUBA = 3,
    QX_ROUTE_I8_OFFSET4 = 4,
    QX_ROUTE_VALU_DOT2 = 5,
    QX_ROUTE_S24_VALU = 6,
    QX_ROUTE_S24_I8LIMB = 7,
    QX_ROUTE_ATTN_F32_MFMA = 8,  /* attention: fp32 MFMA, S tile kept on chip */
    QX_ROUTE_ATTN_I32_MFMA = 9,  /* attention: int8 MFMA for QK^T, S split into int8 limbs */
    QX_ROUTE_ATTN_I32_VALU = 10, /* attention: vector-ALU int32, any operand range */
    QX_ROUTE_ATTN_F32_VALU = 11, /* attention: vector-ALU fp32 (d outside the MFMA shapes) */
    QX_ROUTE_F32_MFMA = 12,      /* FP32 conv: fp32 matrix cores (C_in a multiple of 32) */
    QX_ROUTE_F32_VALU = 13       /* FP32 conv: vector-ALU fp32, any shape */
} qx_route;

/* What the planner decided for one operation (for tests and reporting). */
typedef struct {
    int32_t route;            /* qx_route that will run */
    int32_t chunk;            /* F16_EXACT: K elements per fp32 partial sum; else 0 */
    int32_t products;         /* matrix products issued per multiply-add (1, 3, 4, 8 ...) */
    int32_t tile_m, tile_n, tile_k;  /* workgroup tile of the main kernel */
    int32_t kernels;          /* kernel launches per run */
    int32_t exact_no_wrap;    /* 1: contract proves |result| < 2^31; 0: defined mod 2^32 */
    int32_t operand_format;   /* F16_EXACT with encoded operands: 1 = bf16 (both bounds
                                 <= 256, exact in bf16), 0 = fp16 (or not applicable) */
    int32_t k_splits;         /* int8 limb routes: K slices of the main kernel, added into
                                 the output (cleared first) with wrapping int32 atomics,
                                 exact mod 2^32; 0: K is not sliced */
    int64_t workspace_bytes;  /* device workspace owned by the plan */
} qx_plan_info;

typedef struct qx_exec_s* qx_exec;   /* opaque persistent executor */

/* ---- one-shot operations ------------------------------------------------ */

/* Packed INT16-input / INT32-accumulation GEMM (Methodology; Table 1, right).
 *   C[b] = A[b] . B[b]   for b < batch
 * A [batch][M][K] int16, B [batch][K][N] int16, C [batch][M][N] int32.
 * bound_a / bound_b: max |x| promised for A / B, in [0, 32768] (0 = 32768).
 * M, N, K, batch >= 0; K == 0 writes zeros; M, N or batch == 0 is a no-op. */
qx_status qgemm_i16i32(const int16_t* A, const int16_t* B, int32_t* C,
                       int64_t M, int64_t N, int64_t K, int64_t batch,
                       int32_t bound_a, int32_t bound_b, void* stream);

/* INT32 GEMM under the smul24 contract (Methodology; Table 1, left).
 *   C[b,i,j] = sum_k sext24(A[b,i,k]) * sext24(B[b,k,j])   (mod 2^32)
 * Each int32 operand is read as its low 24 bits, sign-extended (bits 24..31
 * are ignored, always -- this is the contract, not an error).  Shapes and
 * size rules as qgemm_i16i32. */
qx_status qgemm_i32_s24(const int32_t* A, const int32_t* B, int32_t* C,
                        int64_t M, int64_t N, int64_t K, int64_t batch, void* stream);

/* GEMM-backed Conv2D through im2col lowering (Methodology; Table 2,
 * INT16-IN/INT32-ACC row).  Cross-correlation with zero padding, no bias,
 * dilation or groups:
 *   y[n,co,oh,ow] = sum_{ci,kh,kw} x[n,ci,oh*s-p+kh,ow*s-p+kw] * w[co,ci,kh,kw]
 * x NCHW int16 [N][C_in][H][W], w OIHW int16 [C_out][C_in][KH][KW],
 * y NCHW int32 [N][C_out][Ho][Wo], Ho = (H+2p-KH)/s + 1, Wo likewise.
 * stride >= 1, pad >= 0, KH, KW >= 1, Ho, Wo >= 1; bounds as qgemm_i16i32. */
qx_status conv2d_gemm(const int16_t* x, const int16_t* w, int32_t* y,
                      int64_t N, int64_t C_in, int64_t H, int64_t W, int64_t C_out,
                      int64_t KH, int64_t KW, int64_t stride, int64_t pad,
                      int32_t bound_x, int32_t bound_w, void* stream);

/* Conv2D on FP32 or INT32 operands through the same lowering (Table 2,
 * Conv2D FP32 and INT32 rows).  Geometry, layouts and size rules as
 * conv2d_gemm; x, w and y have the element type of dt.
 *  QX_DT_F32: float32 in and out.  The sum is formed in fp32 (on the fp32
 *             matrix cores when C_in is a multiple of 32, else on the vector
 *             ALU) in a fixed order, so repeated runs are bit-identical; it
 *             meets max|y - R| <= 1e-4 max|R| against the float64 sum R.
 *  QX_DT_I32: int32 under the smul24 contract (Methodology): each operand
 *             word is read as sext24 of its low 24 bits; y exact mod 2^32. */
qx_status conv2d_gemm_t(qx_attn_dtype dt, const void* x, const void* w, void* y,
                        int64_t N, int64_t C_in, int64_t H, int64_t W, int64_t C_out,
                        int64_t KH, int64_t KW, int64_t stride, int64_t pad, void* stream);

/* Min/max (Table 2, Min/max rows): out[0] = min, out[1] = max of the n >= 1
 * values of x; elem_bytes 4 = int32, 2 = int16.  out is a device pointer to
 * two elements of the input type (aligned to the element size); x must be
 * 16-byte aligned.  n == 0 is QX_ERR_INVALID_ARG (no minimum exists). */
qx_status minmax(const void* x, int64_t n, int32_t elem_bytes, void* out, void* stream);

/* 2x2 / stride 2 pooling without padding (Table 2, AvgPool INT32 and MaxPool
 * FP32 rows): x NCHW [N][C][H][W] -> y [N][C][H/2][W/2] (a trailing odd row
 * or column is dropped).
 *  QX_POOL_AVG_I32: int32; y = floor((x00 + x01 + x10 + x11) / 4) of the exact sum.
 *  QX_POOL_MAX_F32: float32; y = the window maximum (first value, replaced by
 *                   each later one in row-major order that compares greater).
 * x must be 16-byte aligned; with W % 8 == 0 so must y. */
typedef enum { QX_POOL_AVG_I32 = 0, QX_POOL_MAX_F32 = 1 } qx_pool_kind;
qx_status pool2x2(int32_t kind, const void* x, void* y, int64_t N, int64_t C, int64_t H, int64_t W,
                  void* stream);

/* Single-head attention core (Methodology: O = (Q K^T) V; Table 2, attention
 * rows): no scale, softmax or mask.  Q, K, V, O are [L][d] row-major.
 *  QX_DT_F32: float32 in and out.  The association (Q K^T) V is evaluated
 *             (never Q (K^T V)); the sum order is fixed, so repeated runs are
 *             bit-identical.
 *  QX_DT_I32: int32 in and out, exact mod 2^32.  bound = max |q|, |k|, |v|
 *             (0 = full int32); bound <= 127 runs on int8 MFMA, larger on VALU.
 * L >= 0, d in [0, 256] (the MFMA routes need d % 32 == 0 and d <= 128). */
qx_status attn_core(qx_attn_dtype dt, const void* Q, const void* K, const void* V, void* O,
                    int64_t L, int64_t d, int32_t bound, void* stream);

/* qgemm_i16i32 for callers that cannot allocate device memory: code under
 * HIP graph capture, serving loops and harnesses that forbid allocation.
 * Same arguments, layouts, result (bit for bit) and errors as qgemm_i16i32,
 * and it calls no allocation routine: its workspace is a fixed per-device
 * scratch array of QX_NOALLOC_SCRATCH_BYTES, reserved when the library is
 * loaded on that device and held until the process ends.  Problems whose
 * encoded operands do not fit the scratch run the register-staged kernels
 * (no operand copies); one that needs more scratch even then returns
 * QX_ERR_UNSUPPORTED before anything is enqueued.  Every launch rewrites the
 * scratch it reads, so earlier calls' contents never leak into a result.
 * All calls on one GPU share its scratch: calls that overlap in time on that
 * GPU (other streams, other threads) race and must be serialised by the
 * caller.  Batched problems run every launch on `stream` in order (no side
 * stream).  The host keeps a small plan per distinct request. */
#define QX_NOALLOC_SCRATCH_BYTES (64u << 20)
qx_status qgemm_i16i32_noalloc(const int16_t* A, const int16_t* B, int32_t* C,
                               int64_t M, int64_t N, int64_t K, int64_t batch,
                               int32_t bound_a, int32_t bound_b, void* stream);

/* Multi-head scaled dot-product attention with softmax, FP32 (the SDPA
 * attention baseline of Table 2, whose footnote gives scale 1.0; the
 * attention core with a softmax, Discussion).  For every head b < BH:
 *   O[b] = softmax_rows(scale * Q[b] K[b]^T [+ causal mask]) V[b]
 * Q, K, V, O float32 [BH][L][d] row-major (heads outermost; a [B][H][L][d]
 * tensor is BH = B*H heads).  causal = 1 lets query i see keys j <= i only;
 * causal = 0 sees all L keys.  scale: any finite value (1/sqrt(d) is the
 * usual one).  The softmax is taken online over 32-key blocks with a
 * running maximum; key splits (used when BH * ceil(L/128) < 512) are merged
 * in a fixed order, so repeated runs are bit-identical.
 * BH in [0, 65535], L in [0, 2^20], d in [0, 128]; BH*L*d <= 2^34; any 0
 * size is a no-op.  Q, K, V 16-byte aligned when d % 32 == 0, 4-byte
 * otherwise.  Returns QX_ERR_INVALID_ARG for a non-finite scale or
 * causal outside {0, 1}. */
qx_status sdpa_f32(const float* Q, const float* K, const float* V, float* O,
                   int64_t BH, int64_t L, int64_t d, float scale, int32_t causal,
                   void* stream);

/* ---- persistent executor (Methodology: assemble and allocate once, cache
 *      launch metadata, re-dispatch) ---------------------------------------- */

/* Plan tiles, choose the exact route from the declared contract, allocate
 * the workspace and build the cached launch records, on the current device.
 * *out receives the handle (NULL on failure).  Nothing is enqueued.  Size and
 * bound rules are those of the matching one-shot call; the handle owns its
 * workspace until qx_exec_destroy. */
qx_status qx_exec_create_gemm_i16i32(qx_exec* out, int64_t M, int64_t N, int64_t K, int64_t batch,
                                     int32_t bound_a, int32_t bound_b);
qx_status qx_exec_create_gemm_i32_s24(qx_exec* out, int64_t M, int64_t N, int64_t K, int64_t batch);
qx_status qx_exec_create_conv2d(qx_exec* out, int64_t N, int64_t C_in, int64_t H, int64_t W,
                                int64_t C_out, int64_t KH, int64_t KW, int64_t stride, int64_t pad,
                                int32_t bound_x, int32_t bound_w);
qx_status qx_exec_create_attn(qx_exec* out, qx_attn_dtype dt, int64_t L, int64_t d, int32_t bound);

/* The same four calls with a forced route (tests and comparisons of the
 * routes, e.g. the vector-ALU smul24 GEMM against the int8 limb one):
 * route = QX_ROUTE_AUTO behaves exactly as the call without the suffix; a
 * route that does not apply to the operation returns QX_ERR_INVALID_ARG,
 * one that cannot be exact for the declared bounds QX_ERR_RANGE. */
qx_status qx_exec_create_gemm_i16i32_route(qx_exec* out, int64_t M, int64_t N, int64_t K,
                                           int64_t batch, int32_t bound_a, int32_t bound_b,
                                           int32_t route);
qx_status qx_exec_create_gemm_i32_s24_route(qx_exec* out, int64_t M, int64_t N, int64_t K,
                                            int64_t batch, int32_t route);
qx_status qx_exec_create_conv2d_route(qx_exec* out, int64_t N, int64_t C_in, int64_t H, int64_t W,
                                      int64_t C_out, int64_t KH, int64_t KW, int64_t stride,
                                      int64_t pad, int32_t bound_x, int32_t bound_w, int32_t route);
qx_status qx_exec_create_attn_route(qx_exec* out, qx_attn_dtype dt, int64_t L, int64_t d,
                                    int32_t bound, int32_t route);

/* FP32 / INT32 convolution (as conv2d_gemm_t).  dt QX_DT_F32: route AUTO,
 * F32_MFMA or F32_VALU; QX_DT_I32: AUTO, S24_I8LIMB or S24_VALU. */
qx_status qx_exec_create_conv2d_t(qx_exec* out, qx_attn_dtype dt, int64_t N, int64_t C_in,
                                  int64_t H, int64_t W, int64_t C_out, int64_t KH, int64_t KW,
                                  int64_t stride, int64_t pad, int32_t route);
qx_status qx_exec_create_minmax(qx_exec* out, int64_t n, int32_t elem_bytes);
/* LeNet-5-shaped INT32 pipeline (Results: end-to-end CNN), every layer one
 * of this library's operators chained through the workspace on one stream:
 *   x [B][1][32][32] -> conv 6@5x5 -> ReLU -> 2x2 avg -> conv 16@5x5 -> ReLU
 *   -> 2x2 avg -> [B][400] -> FC 120 -> ReLU -> FC 84 -> ReLU -> FC 10.
 * Convolutions and FC layers are INT32 under the smul24 contract (operand
 * words read as sext24 of their low 24 bits, results mod 2^32); pools are
 * the INT32 floor average; ReLU is max(x, 0).  inputs = {x, w1 [6][1][5][5],
 * w2 [16][6][5][5], f1 [400][120], f2 [120][84], f3 [84][10]} (FC weights
 * [in][out]); output [B][10] int32.  0 <= batch <= 2^20. */
qx_status qx_exec_create_lenet_i32(qx_exec* out, int64_t batch);
qx_status qx_exec_create_pool2x2(qx_exec* out, int32_t kind, int64_t N, int64_t C, int64_t H, int64_t W);
/* Softmax attention (as sdpa_f32): inputs {Q, K, V}, output O. */
qx_status qx_exec_create_sdpa_f32(qx_exec* out, int64_t BH, int64_t L, int64_t d, float scale,
                                  int32_t causal);

/* Enqueue one evaluation: inputs = {A, B} (GEMMs), {x, w} (convolutions), {x}
 * (min/max, pooling), {Q, K, V} (attention) or {x, w1, w2, f1, f2, f3}
 * (LeNet pipeline), device pointers with the shapes given at create.
 * Allocates nothing.  Calls on one handle must not overlap in time.  A
 * handle that is not live (never created, or already destroyed) returns
 * QX_ERR_INVALID_ARG. */
qx_status qx_exec_run(qx_exec h, const void* const* inputs, void* output, void* stream);

/* The plan a handle carries. */
qx_status qx_exec_plan(qx_exec h, qx_plan_info* out);

/* Execute-only timing (Methodology: separating setup, cached steady state
 * and execute-only kernel time): enqueue `reps` runs on `stream` with a HIP
 * event pair around every launch, wait for them, and write the mean duration
 * in milliseconds of launch i of the plan to kernel_ms[i] for i < min(kernels,
 * max_kernels); names[i] (if names is not NULL) receives a static kernel name.
 * Synchronises `stream`.  Not for use under graph capture. */
qx_status qx_exec_profile(qx_exec h, const void* const* inputs, void* output, void* stream,
                          int32_t reps, float* kernel_ms, const char** names, int32_t max_kernels);

/* Free the workspace and the handle (waits for the device to finish any
 * work that may use the workspace).  NULL is accepted.  Destroying a handle
 * that is not live (a second destroy, or a pointer that no create returned)
 * returns QX_ERR_INVALID_ARG and touches nothing. */
qx_status qx_exec_destroy(qx_exec h);

/* ---- planner queries (pure host logic, no device needed) ---------------- */
qx_status qx_plan_gemm_i16i32(qx_plan_info* out, int64_t M, int64_t N, int64_t K,
                              int64_t batch, int32_t bound_a, int32_t bound_b, int32_t route);
qx_status qx_plan_gemm_i32_s24(qx_plan_info* out, int64_t M, int64_t N, int64_t K,
                               int64_t batch, int32_t route);
qx_status qx_plan_conv2d(qx_plan_info* out, int64_t N, int64_t C_in, int64_t H, int64_t W,
                         int64_t C_out, int64_t KH, int64_t KW, int64_t stride, int64_t pad,
                         int32_t bound_x, int32_t bound_w, int32_t route);
qx_status qx_plan_conv2d_t(qx_plan_info* out, qx_attn_dtype dt, int64_t N, int64_t C_in,
                           int64_t H, int64_t W, int64_t C_out, int64_t KH, int64_t KW,
                           int64_t stride, int64_t pad, int32_t route);
qx_status qx_plan_attn(qx_plan_info* out, qx_attn_dtype dt, int64_t L, int64_t d,
                       int32_t bound, int32_t route);
qx_status qx_plan_sdpa_f32(qx_plan_info* out, int64_t BH, int64_t L, int64_t d, float scale,
                           int32_t causal);
qx_status qx_plan_minmax(qx_plan_info* out, int64_t n, int32_t elem_bytes);
qx_status qx_plan_lenet_i32(qx_plan_info* out, int64_t batch);
qx_status qx_plan_pool2x2(qx_plan_info* out, int32_t kind, int64_t N, int64_t C, int64_t H, int64_t W);

/* Message of the last failing call on this thread ("" if none).  Valid
 * until the next qx call on the same thread. */
const char* qx_last_error(void);

/* Release the one-shot plan cache (frees its workspaces). */
void qx_release_cache(void);

#ifdef __cplusplus
}
#endif

#endif /* QX_H */
