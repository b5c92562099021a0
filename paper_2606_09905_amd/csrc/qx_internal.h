// qx_internal.h -- definitions shared by the HIP kernels and the host side of
// the library (planner, executor, C ABI).  Not installed; the public
// interface is include/qx.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

namespace qx {

// ---------------------------------------------------------------------------
// Kernel parameter blocks.  Every kernel takes exactly one of these by value,
// so a launch is fully described by (function, grid, block, parameter bytes)
// and the executor can cache it and patch the pointer fields per run.
// ---------------------------------------------------------------------------

// Epilogue store modes of the GEMM kernels.
enum OutMode : int32_t {
    OUT_ROWMAJOR = 0,  // C[m][n] at C + m*ldc + n
    OUT_CONV = 1,      // C[m][n] -> y[(n / hw) * M * hw + m * hw + n % hw]  (NCHW scatter)
};

// B operand layouts.
enum BMode : int32_t {
    B_KN = 0,          // B[k][n] at B + k*ldb + n   (row-major K x N)
    B_IM2COL = 1,      // B[k][n] gathered from an NCHW image (implicit lowering)
    B_NHWC = 2,        // B^T[n][k] gathered from a zero-bordered NHWC fp16 image
};

struct ConvGeom {      // geometry for B_IM2COL / OUT_CONV
    int32_t Ci, H, W, KH, KW, stride, pad, Ho, Wo;
};

// Integer GEMM  C[b] = A[b] . B[b]  for every route.
struct GemmParams {
    const void* A;          // [M][lda] int16 or int32 (route dependent)
    const void* B;          // see BMode
    void* C;                // int32 output, see OutMode
    const int32_t* rowsum;  // limb routes with an offset: per (batch,row) sums of A
    const int32_t* colsum;  // per (batch,col) sums of B
    int64_t sA, sB, sC;     // batch strides (elements)
    int32_t M, N, K;
    int32_t lda, ldb, ldc;
    int32_t chunk_tiles;    // F16_EXACT: flush fp32 partials every chunk_tiles K-tiles
    int32_t corr_c;         // offset constant c of the limb split (0: none)
    int32_t out_mode;       // OutMode
    int32_t b_mode;         // BMode (int8 NT route: B_KN planes, or B_NHWC: gathered from the
                            // bordered NHWC limb planes of ConvLimbPrepParams, colsum from s)
    int32_t hw;             // OUT_CONV: Ho*Wo
    int32_t tiles_n;        // number of N tiles (grid swizzle)
    int32_t cs_slices;      // colsum holds this many partial rows per batch
    int32_t bf16;           // F16_EXACT NT contraction: operands are bf16 (|x| <= 256), else fp16
    int32_t ksplit;         // int8 NT route: K slices (grid y) added into a cleared C with
                            // wrapping int32 atomics; <= 1: one slice, plain stores
    int32_t flat_batch;     // int8 NT route: batch folded into grid x (each XCD gets whole batches)
    int32_t relu;           // int8 NT route without K slices: store max(C, 0)
    int32_t pad1;
    int64_t plane_a;        // int8 NT route: bytes between limb planes of A and of B
    int64_t plane_b;
    ConvGeom g;
};

// Per-row / per-column sums used by the rank-1 correction of offset limb routes.
struct SumsParams {
    const void* A;
    const void* B;
    int32_t* rowsum;        // [batch][M]
    int32_t* colsum;        // [batch][N]
    int64_t sA, sB;
    int32_t M, N, K, lda, ldb;
    int32_t s24;            // 1: operands are int32 read through sext24; 0: int16
    int32_t batch;
};

// Explicit im2col: col[k][p], k = (ci*KH + kh)*KW + kw, p = (n*Ho + oh)*Wo + ow,
// elements of elem_bytes (2: int16, 4: int32 or float32) copied as they are.
struct Im2colParams {
    const void* x;
    void* col;
    int64_t P;              // N*Ho*Wo
    int32_t Kd;             // Ci*KH*KW
    int32_t elem_bytes;
    ConvGeom g;
};

// int16 -> fp16 operand encoders of the large-problem fp16-exact route.
struct EncParams {
    const void* src;        // int16 [batch][rows][ld_src]
    void* dst;              // fp16 [batch][Mp|Np][Kp], zero padded
    int64_t s_src, s_dst;   // batch strides (elements)
    int32_t M, N, K;        // logical extents (A: M x K, B: K x N)
    int32_t Mp, Np, Kp;     // padded extents
    int32_t ld_src;
    int32_t batch;
    int32_t vec;            // rows and batch strides allow 16-byte source loads
    int32_t* sums;          // int8 limb routes with an offset: row sums [batch][M] of A
                            // (A encoder) or per-64-k-slice column sums [batch][Kp/64][N]
                            // of B (B^T encoder), of the values the split represents
    int32_t conv;           // B^T encoder: 1 = B is the im2col matrix of the NCHW image
                            // src with geometry g (gathered, never materialised)
    int32_t bf16;           // fp16 encoders: write bf16 (exact for |x| <= 256) instead of fp16
    ConvGeom g;
};

// Both operand encoders of the int8 limb routes in one launch.
struct EncPairParams {
    EncParams a;            // A -> A8 [batch][P][Mp][Kp]
    EncParams b;            // B -> B8T [batch][P][Np][Kp]
    int32_t blocks_a;       // leading blocks that encode A
};

// Convolution lowering into the transposed fp16 column matrix colT [Pp][Kp].
struct Im2colTParams {
    const int16_t* x;
    _Float16* colT;
    int32_t P, Pp;          // N*Ho*Wo and its padded extent
    int32_t Kd, Kp;         // Ci*KH*KW and its padded extent
    ConvGeom g;
};

// Implicit lowering of a convolution (C_in a multiple of 64): the input as a
// zero-bordered NHWC fp16 copy xp [N][H+2pad][W+2pad][Ci] and the weights as
// w16 [Cop][Kd] fp16 with k = (kh*KW + kw)*Ci + ci, in one launch.
// elem_bytes 2: int16 in, fp16 out (C_in a multiple of 64); 4: float32
// copied unchanged (C_in a multiple of 32).
struct ConvPrepParams {
    const void* x;          // NCHW
    const void* w;          // OIHW
    void* xp;
    void* w16;
    int32_t nimg, Co, Cop, Kd;
    int32_t xblocks, wblocks;
    int32_t elem_bytes;
    ConvGeom g;
};

// Implicit lowering of an INT32 (smul24) convolution for the int8 limb route
// (C_in a multiple of 64), in one launch: the input as three int8 limb
// planes of a zero-bordered NHWC image xp8 [3][N][H+2pad][W+2pad][Ci] (the
// border holds the limbs of 0), the per-position sums of the represented
// values over each 64-channel chunk s [N][Ci/64][H+2pad][W+2pad] (the column
// sums of the offset correction, gathered per K tile like the columns), and
// the weights as limb planes a8 [3][Mp][Kd], k = (kh*KW + kw)*Ci + ci, with
// their row sums.
struct ConvLimbPrepParams {
    const int32_t* x;       // NCHW
    const int32_t* w;       // OIHW
    int8_t* xp8;
    int32_t* s;
    int8_t* a8;
    int32_t* rowsum;        // [Co]
    int64_t plane_x;        // bytes between the image planes
    int64_t plane_a;        // bytes between the weight planes (Mp * Kd)
    int32_t nimg, Co, Kd;
    int32_t xblocks, wblocks;
    ConvGeom g;
};

// Direct smul24 convolution on the vector ALU for few output channels
// (C_out <= 16, C_in*KH*KW <= 1024, KW <= 8): a thread makes every output
// channel of one output pixel; the weights sit in LDS.
struct ConvDirectParams {
    const int32_t* x;       // NCHW
    const int32_t* w;       // OIHW
    int32_t* y;             // NCHW
    int64_t P;              // N*Ho*Wo
    int32_t Co, Kd;
    int32_t imgs;           // > 0: whole images per workgroup, staged in LDS
    int32_t pool;           // 1: ReLU + 2x2 average fused, y is [N][C_out][Ho/2][Wo/2]
    ConvGeom g;
};

// Attention core O = (Q K^T) V.
struct AttnParams {
    const void* Q;
    const void* K;
    const void* V;
    void* O;
    void* part;             // F32: split partials [splits][L][d] float
    int32_t L, d;
    int32_t splits;         // key splits
    int32_t keys_per_split;
    int32_t limbs;          // I32: int8 limbs of S
    // I32 with resident key splits: int8 copies made by the prep launch
    void* k8;               // [Lp][d] int8 rows of K
    void* v8;               // [d][Lp] int8 rows of V^T, keys of every 32-key block reordered
                            // so a lane half's 16 keys of one S V product are contiguous
    int32_t Lp;             // splits * keys_per_split (>= L), zero-padded keys
    int32_t clear_o;        // prep also clears O (split partials are added with atomics)
    int64_t prep_k, prep_v; // prep work items: 16-byte K8 chunks, 16-byte V8 chunks
    int32_t v_blocks;       // prep: 1 = write V8 block-major, [Lp/32][d][32] (each 32-key block of
                            // every column contiguous, keys reordered as above), for the
                            // streaming kernel; 0 = [d][Lp]
    int32_t qt;             // streaming kernel: query tiles of 32 per workgroup (1, 2 or 4)
    void* q8;               // prep_q > 0: int8 rows of Q, [L][d]
    int64_t prep_q;         // prep work items: 16-byte Q8 chunks (0: none)
};

// Softmax attention over BH heads (FP32): O = softmax(scale Q K^T [mask]) V.
struct SdpaParams {
    const float* Q;         // [BH][L][d]
    const float* K;
    const float* V;
    float* O;               // [BH][L][d]
    float* part;            // splits > 1: unnormalised outputs [splits][BH][L][d]
    float* stat;            // splits > 1: (max, sum) per row [splits][BH][L][2]
    int32_t L, d, BH;
    int32_t splits;         // key splits
    int32_t keys_per_split;
    int32_t causal;         // key j is seen by query i only when j <= i
    float c;                // scale * log2(e): scores in the base-2 exponent domain
};

struct SdpaCombineParams {
    const float* part;
    const float* stat;
    float* O;
    int64_t rows;           // BH * L
    int32_t d;
    int32_t splits;
};

struct ReduceParams {
    const float* part;      // [splits][n]
    float* out;             // [n]
    int64_t n;
    int32_t splits;
};

// Operand range scan (QX_VALIDATE): sets *flag when some |x| > bound.
struct RangeParams {
    const void* x;
    uint32_t* flag;
    int64_t n;              // elements
    int32_t bound;
    int32_t elem_bytes;     // 2 (int16) or 4 (int32)
    uint32_t bit;           // value or-ed into *flag
};

// Min/max: pass 1 writes one (min, max) pair per workgroup into part.
struct MinMaxParams {
    const void* x;
    int32_t* part;          // [blocks][2]
    void* out;              // two elements of the input type
    int64_t n, per;         // elements; elements per workgroup (multiple of 64)
    int32_t blocks;
    int32_t elem_bytes;     // 4 (int32) or 2 (int16)
};

// 2x2 / stride 2 pooling of NCHW 32-bit elements.
enum PoolKind : int32_t { POOL_AVG_I32 = 0, POOL_MAX_F32 = 1 };
struct PoolParams {
    const void* x;
    void* y;
    int64_t NC;
    int32_t H, W, Ho, Wo;
    int32_t vec;            // W % 8 == 0: 16-byte loads and stores
    int32_t relu;           // average of max(x, 0) (a ReLU fused ahead of the pool)
};

// In-place ReLU of int32 values: p[i] = max(p[i], 0).
struct ReluParams {
    int32_t* p;
    int64_t n;
};

// Largest grid of the fill kernel (a grid-stride loop beyond it).
constexpr int64_t kFillMaxBlocks = 16384;
struct FillParams {
    void* ptr;
    int64_t n32;            // number of 32-bit words
    int32_t value;
};

// Generic vector-ALU GEMM (fallbacks and attention on VALU).
enum ValuKind : int32_t {
    VK_I16_DOT2 = 0,        // int16 in, v_dot2_i32_i16, wrapping int32
    VK_S24 = 1,             // int32 in, sext24 products (v_mad_i32_i24 class), wrapping
    VK_I32 = 2,             // int32 in, low 32 bits of products, wrapping
    VK_F32 = 3,             // float in and out, fixed summation order
};

struct ValuGemmParams {
    const void* A;          // [M][lda]
    const void* B;          // b_trans ? [N][ldb] : [K][ldb]
    void* C;                // [M][ldc]
    int64_t sA, sB, sC;
    int32_t M, N, K, lda, ldb, ldc;
    int32_t b_trans;
    int32_t out_mode;
    int32_t hw;
    int32_t relu;           // skinny smul24 kernel only: max(c, 0) on store
    int32_t ksplit;         // k_valu_gemm, integer kinds: K slices on grid z (batch * ksplit),
                            // added with wrapping atomics into C cleared beforehand; 0 or 1: none
};

// ---------------------------------------------------------------------------
// Cached launch records.
// ---------------------------------------------------------------------------
enum Bind : uint8_t {
    BIND_IN0 = 0, BIND_IN1 = 1, BIND_IN2 = 2, BIND_IN3 = 3, BIND_IN4 = 4, BIND_IN5 = 5,
    BIND_OUT = 6, BIND_WS = 7
};
constexpr int kMaxInputs = 6;

struct Slot {
    uint16_t off;           // byte offset of a pointer field in the parameter blob
    uint8_t bind;           // what it points at
    uint64_t add;           // byte offset added to the bound pointer
};

// One kernel launch of a plan: kernel, geometry and parameter block, with
// the pointer fields bound at run time through slots.  Every launch of a
// plan goes to the caller's stream, in plan order.
struct LaunchRec {
    const void* fn = nullptr;
    dim3 grid{1, 1, 1};
    dim3 block{1, 1, 1};
    uint32_t shmem = 0;
    alignas(16) unsigned char blob[320];
    uint32_t blob_size = 0;
    Slot slots[8];
    int nslots = 0;
    const char* name = "";

    template <class P>
    void set_params(const P& p) {
        static_assert(sizeof(P) <= sizeof(blob), "parameter block too large");
        memcpy(blob, &p, sizeof(P));
        blob_size = sizeof(P);
    }
    void bind(size_t off, Bind b, uint64_t add = 0) {
        slots[nslots].off = (uint16_t)off;
        slots[nslots].bind = b;
        slots[nslots].add = add;
        ++nslots;
    }
};

// ---------------------------------------------------------------------------
// Kernel-family builders (defined in the .hip files).  Each fills a launch
// record for a fully planned problem; pointers are bound through slots.
// ---------------------------------------------------------------------------
enum Route : int32_t {
    R_AUTO = 0, R_I8_DIRECT = 1, R_F16_EXACT = 2, R_I8_KARATSUBA = 3, R_I8_OFFSET4 = 4,
    R_VALU_DOT2 = 5, R_S24_VALU = 6, R_S24_I8LIMB = 7,
    R_ATTN_F32_MFMA = 8, R_ATTN_I32_MFMA = 9, R_ATTN_I32_VALU = 10,
    R_ATTN_F32_VALU = 11,   // fp32 attention on the vector ALU (shapes the MFMA kernel does not take)
    R_F32_MFMA = 12, R_F32_VALU = 13,   // FP32 convolution: fp32 matrix cores / vector ALU
};

// Fixed device scratch of the allocation-free GEMM entry point: its size,
// and its device address on device `dev` (looked up once per device, with
// that device current).
constexpr uint64_t kScratchBytes = (uint64_t)64 << 20;
hipError_t scratch_device_ptr(int dev, void** out);

// Integer GEMM main kernel for an MFMA route; returns false if unsupported.
bool build_gemm_mfma(int32_t route, const GemmParams& p, int batch, LaunchRec* rec,
                     int* tile_m, int* tile_n, int* tile_k);
// Row sums [batch][M] and per-slice column sums [batch][slices][N] in one launch.
void build_sums(const SumsParams& p, LaunchRec* rec);
int sums_slices(int K);
void build_im2col(const Im2colParams& p, LaunchRec* rec);
void build_valu_gemm(int32_t kind, const ValuGemmParams& p, int batch, LaunchRec* rec);
void build_valu_skinny_s24(const ValuGemmParams& p, int batch, LaunchRec* rec);   // N of a few tens
bool build_attn_f32(const AttnParams& p, LaunchRec* rec);
bool build_attn_i32(const AttnParams& p, LaunchRec* rec);
// INT32 attention with resident key splits: applicable for d in {32, 64, 128}
// and splits of kps keys with kps * d a multiple of 4096 and 2 * kps * d <= 48 KiB
bool resident_attn_i32(int64_t d, int64_t kps);
bool build_attn_i32_prep(const AttnParams& p, LaunchRec* rec);
bool build_attn_i32r(const AttnParams& p, LaunchRec* rec);
// INT32 attention streaming its keys from the int8 copies into registers:
// d in {32, 64}, keys_per_split a multiple of 128, V8 block-major
bool build_attn_i32s(const AttnParams& p, LaunchRec* rec);
void build_reduce(const ReduceParams& p, LaunchRec* rec);
bool build_sdpa_f32(const SdpaParams& p, LaunchRec* rec);
void build_sdpa_combine(const SdpaCombineParams& p, LaunchRec* rec);
void build_fill(const FillParams& p, LaunchRec* rec);
void build_range(const RangeParams& p, LaunchRec* rec);
// Min/max reduction (two launches) and 2x2 pooling.
void minmax_blocks(int64_t n, int32_t* blocks, int64_t* per);
void build_minmax(const MinMaxParams& p, LaunchRec* partial, LaunchRec* final_rec);
void build_pool2(int32_t kind, const PoolParams& p, LaunchRec* rec);
void build_relu(const ReluParams& p, LaunchRec* rec);
int32_t conv_pool_images(const ConvDirectParams& p);
void build_conv_direct_s24(const ConvDirectParams& p, LaunchRec* rec);
// fp16-exact route for large problems: encoders + direct-to-LDS NT GEMM.
void nt_tile_shape(int64_t M, int64_t N, int64_t batch, int* bm, int* bn);
void build_gemm_nt(const GemmParams& p, int batch, LaunchRec* rec);
void build_enc_a(const EncParams& p, LaunchRec* rec);
void build_enc_bt(const EncParams& p, LaunchRec* rec);
void build_im2col_t(const Im2colTParams& p, LaunchRec* rec);
void build_conv_prep(const ConvPrepParams& p, LaunchRec* rec);
// FP32 NT GEMM on the fp32 matrix cores (conv FP32 row); same tile shapes.
void build_gemm_nt_f32(const GemmParams& p, int batch, LaunchRec* rec);
// int8 limb routes for large problems: limb-plane encoders + direct-to-LDS NT GEMM.
void i8nt_tile_shape(int32_t route, int64_t M, int64_t N, int64_t batch, int* bm, int* bn);
void build_enc_limb(int32_t route, bool s24, const EncPairParams& p, LaunchRec* rec);
void build_conv_prep_limb(const ConvLimbPrepParams& p, LaunchRec* rec);
bool build_gemm_i8nt(int32_t route, const GemmParams& p, int batch, LaunchRec* rec);

}  // namespace qx
