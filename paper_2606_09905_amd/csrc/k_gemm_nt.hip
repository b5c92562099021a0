// k_gemm_nt.hip -- the fp16-exact route for large contractions.
//
// Two stages:
//  1. Encode (HBM-bound): int16 operands become fp16 copies in the
//     workspace, A as [Mp][Kp] and B transposed as B^T [Np][Kp], both
//     K-contiguous and zero-padded to whole tiles (zero adds nothing to any
//     product).  Every int16 with |x| <= 2048 is exact in fp16.  For
//     convolution the lowering writes the transposed fp16 column matrix
//     directly (im2col, Methodology: convolution through lowering).
//  2. Contract: a tiled GEMM on v_mfma_f32_32x32x16_f16.  Tiles are staged
//     global -> LDS with global_load_lds_dwordx4 (no register staging) in a
//     three-deep ring; each wave accumulates a 64x64 block in fp32 for
//     `chunk` K elements, then converts and adds the partial into int32.
//     With chunk * max|a| * max|b| <= 2^24 every partial sum is an integer
//     fp32 holds exactly, whatever order the matrix core sums in; the int32
//     sum is exact mod 2^32 (Table 1: INT16 input, INT32 accumulation).
//
// LDS layout: a stage holds rows of 64 fp16 as eight 16-byte chunks; chunk c
// of row r sits at position c ^ ((r >> 1) & 7), so the 16 rows read by one
// ds_read_b128 pass fall in distinct banks.  The swizzle is applied on the
// global side (each lane fetches the chunk that belongs at its LDS slot).
#include <algorithm>

#include <type_traits>

#include "qx_internal.h"

namespace qx {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f16x __attribute__((ext_vector_type(16)));
typedef unsigned u16x __attribute__((ext_vector_type(16)));
typedef short s8v __attribute__((ext_vector_type(8)));
typedef float f4v __attribute__((ext_vector_type(4)));

// ===========================================================================
// Stage 1: encoders
// ===========================================================================
typedef __bf16 b8v __attribute__((ext_vector_type(8)));

// 8 int16 -> 8 fp16 (exact for |x| <= 2048), or with BF 8 bf16 (exact for
// |x| <= 256: eight significant bits) carried in the same 16-bit lanes.
template <bool BF>
__device__ __forceinline__ h8 to_h8(s8v v) {
    if constexpr (BF) {
        b8v o;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (__bf16)(float)v[e];
        return __builtin_bit_cast(h8, o);
    } else {
        h8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (_Float16)v[e];
        return o;
    }
}
template <bool BF>
__device__ __forceinline__ _Float16 to_h1(int v) {
    if constexpr (BF) return __builtin_bit_cast(_Float16, (__bf16)(float)v);
    else return (_Float16)v;
}

// A [batch][M][lda] int16 -> A16 [batch][Mp][Kp] fp16 (bf16 with BF); one
// thread = 8 k, four vectors per thread.  Both encoders read their int16
// source once, with non-temporal loads (whole lines per wave-wide load):
// the source then displaces less of the encoded operands the contraction
// reads next (2% on 8192^3 and 64 x 2048^3).
template <bool BF>
__global__ __launch_bounds__(256) void k_enc_a(const EncParams p) {
    const int kv = p.Kp / 8;
    const int64_t per_b = (int64_t)p.Mp * kv;
    const int64_t total = per_b * p.batch;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int64_t v = ((int64_t)blockIdx.x * 4 + q) * 256 + threadIdx.x;
        if (v >= total) return;
        const int b = (int)(v / per_b);
        const int64_t r = v - (int64_t)b * per_b;
        const int m = (int)(r / kv), k0 = (int)(r - (int64_t)m * kv) * 8;
        const int16_t* src = (const int16_t*)p.src + b * p.s_src + (int64_t)m * p.ld_src + k0;
        h8 out;
        if (p.vec && m < p.M && k0 + 8 <= p.K) {
            out = to_h8<BF>(__builtin_nontemporal_load((const s8v*)src));
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) out[e] = to_h1<BF>((m < p.M && k0 + e < p.K) ? src[e] : 0);
        }
        *(h8*)((_Float16*)p.dst + b * p.s_dst + (int64_t)m * p.Kp + k0) = out;
    }
}

// B [batch][K][ldb] int16 -> BT16 [batch][Np][Kp] fp16 (bf16 with BF),
// transposed through LDS with 256-byte segments on both sides (128-byte
// ones, transposing in registers only, took 57 us against 48 us for an
// 8192 x 8192 operand): a workgroup takes 128 (k) x 128 (n); wave w reads rows k = 32w .. 32w+31, lane (kb, nb)
// = (lane / 16, lane % 16) eight 16-byte rows k = 32w + 8kb + r (n = 8nb ..
// 8nb+7, sixteen lanes per 256-byte row segment), transposes its 8 x 8 block
// in registers and puts its eight 16-byte rows n = 8nb + e into the LDS
// tile [n][k]; the tile then leaves as 128 rows of 256 bytes.  Chunk c of
// tile row n sits at c ^ ((n / 8) & 15), so both sides are conflict-free.
template <bool BF>
__global__ __launch_bounds__(256) void k_enc_bt(const EncParams p) {
    __shared__ h8 t[128][16];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int kb = lane >> 4, nb = lane & 15;
    const int n0 = blockIdx.x * 128, k0 = blockIdx.y * 128, b = blockIdx.z;
    const int16_t* src = (const int16_t*)p.src + b * p.s_src;
    s8v in[8];
    const int n = n0 + nb * 8;
    const int kr = k0 + wave * 32 + kb * 8;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
        const int k = kr + r;
        const int16_t* sp = src + (int64_t)k * p.ld_src + n;
        if (p.vec && k < p.K && n + 8 <= p.N) {
            in[r] = __builtin_nontemporal_load((const s8v*)sp);
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) in[r][e] = (k < p.K && n + e < p.N) ? sp[e] : (short)0;
        }
    }
    const int c = wave * 4 + kb;              // this lane's k chunk of the tile
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        s8v col;
#pragma unroll
        for (int r = 0; r < 8; ++r) col[r] = in[r][e];
        const int row = nb * 8 + e;
        t[row][c ^ ((row >> 3) & 15)] = to_h8<BF>(col);
    }
    __syncthreads();
    _Float16* dst = (_Float16*)p.dst + b * p.s_dst;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int q = tid + 256 * i, row = q >> 4, cc = q & 15;
        const int gn = n0 + row, gk = k0 + cc * 8;
        if (gn < p.Np && gk < p.Kp) *(h8*)(dst + (int64_t)gn * p.Kp + gk) = t[row][cc ^ ((row >> 3) & 15)];
    }
}

// Convolution lowering straight into the transposed fp16 column matrix:
// colT[p][k] = x[n, ci, oh*s-p+kh, ow*s-p+kw] (0 outside the image and in the
// padding), p = (n*Ho + oh)*Wo + ow, k = (ci*KH + kh)*KW + kw.  One thread
// writes 8 consecutive k of one pixel.
__global__ __launch_bounds__(256) void k_im2col_t(const Im2colTParams p) {
    const int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int kv = p.Kp / 8;
    if (v >= (int64_t)p.Pp * kv) return;
    const int pix = (int)(v / kv), k0 = (int)(v - (int64_t)pix * kv) * 8;
    const ConvGeom& g = p.g;
    const int hw = g.Ho * g.Wo;
    h8 out;
    if (pix < p.P) {
        const int n = pix / hw, rem = pix - n * hw;
        const int oh = rem / g.Wo, ow = rem - oh * g.Wo;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int k = k0 + e;
            _Float16 val = (_Float16)0.0f;
            if (k < p.Kd) {
                const int kw = k % g.KW, kh = (k / g.KW) % g.KH, ci = k / (g.KW * g.KH);
                const int ih = oh * g.stride - g.pad + kh, iw = ow * g.stride - g.pad + kw;
                if (ih >= 0 && ih < g.H && iw >= 0 && iw < g.W)
                    val = (_Float16)p.x[(((int64_t)n * g.Ci + ci) * g.H + ih) * g.W + iw];
            }
            out[e] = val;
        }
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) out[e] = (_Float16)0.0f;
    }
    *(h8*)(p.colT + (int64_t)pix * p.Kp + k0) = out;
}

// The same lowering when C_in is a multiple of 8: a block owns one output
// row (n, oh) and 8 input channels; it stages the KH input rows those need
// (zero outside the image) in LDS, coalesced along W, then writes for every
// ow the 8*KH*KW consecutive k of its channel group as 16-byte stores.
__global__ __launch_bounds__(256) void k_im2col_t8(const Im2colTParams p) {
    extern __shared__ _Float16 xs[];   // [8][KH][Wp], Wp = (Wo-1)*stride + KW
    const ConvGeom& g = p.g;
    const int oh = blockIdx.x, cg = blockIdx.y, n = blockIdx.z;
    const int ci0 = cg * 8;
    const int Wp = (g.Wo - 1) * g.stride + g.KW;
    const int tid = threadIdx.x;
    const int total = 8 * g.KH * Wp;
    for (int idx = tid; idx < total; idx += 256) {
        const int c = idx / (g.KH * Wp), rem = idx - c * g.KH * Wp;
        const int kh = rem / Wp, iwp = rem - kh * Wp;
        const int ih = oh * g.stride - g.pad + kh, iw = iwp - g.pad;
        _Float16 v = (_Float16)0.0f;
        if (ih >= 0 && ih < g.H && iw >= 0 && iw < g.W)
            v = (_Float16)p.x[(((int64_t)n * g.Ci + ci0 + c) * g.H + ih) * g.W + iw];
        xs[idx] = v;
    }
    __syncthreads();
    const int kk = g.KH * g.KW;              // chunks of 8 k per pixel and group
    const int chunks = g.Wo * kk;
    const int64_t row0 = ((int64_t)n * g.Ho + oh) * g.Wo;
    for (int idx = tid; idx < chunks; idx += 256) {
        const int ow = idx / kk, q = idx - ow * kk;
        h8 out;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int kl = 8 * q + e;            // k within the group: c*KH*KW + kh*KW + kw
            const int c = kl / kk, r = kl - c * kk;
            const int kh = r / g.KW, kw = r - kh * g.KW;
            out[e] = xs[(c * g.KH + kh) * Wp + ow * g.stride + kw];
        }
        *(h8*)(p.colT + (row0 + ow) * p.Kp + ci0 * kk + 8 * q) = out;
    }
}

// Implicit lowering, C_in a multiple of 64.  The im2col column of pixel
// (n, oh, ow) for K tile t is 64 consecutive channels of one kernel tap
// (kh, kw): xp[n][oh*s + kh][ow*s + kw][ci0 .. ci0+64) of the zero-bordered
// NHWC copy, so the contraction gathers its B tiles straight from xp.  The
// weights take the matching order k = (kh*KW + kw)*Ci + ci; any order of the
// K sum gives the same exact integer result.
// blockIdx.y == 0: x NCHW int16 -> xp; a block covers 64 padded columns of
// one padded row of one image, 64 channels per pass through LDS.
// blockIdx.y == 1: w OIHW int16 -> w16 [Cop][Kd], one thread per 8 channels.
__global__ __launch_bounds__(256) void k_conv_prep(const ConvPrepParams p) {
    const ConvGeom& g = p.g;
    const int tid = threadIdx.x;
    if (blockIdx.y == 0) {
        if ((int)blockIdx.x >= p.xblocks) return;
        __shared__ short t[64][66];
        const int Hp = g.H + 2 * g.pad, Wp = g.W + 2 * g.pad;
        const int wch = (Wp + 63) / 64;
        const int n = blockIdx.x / (Hp * wch), rem = blockIdx.x - n * Hp * wch;
        const int hp = rem / wch, wp0 = (rem - hp * wch) * 64;
        const int h = hp - g.pad;
        const bool row_in = h >= 0 && h < g.H;
        const int wl = tid & 63, cq = tid >> 6;
        const int w = wp0 + wl - g.pad;
        const bool in = row_in && w >= 0 && w < g.W;
        _Float16* dst = (_Float16*)p.xp + ((int64_t)n * Hp + hp) * Wp * g.Ci;
        for (int c0 = 0; c0 < g.Ci; c0 += 64) {
            const int16_t* src = (const int16_t*)p.x + (((int64_t)n * g.Ci + c0) * g.H + h) * g.W + w;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int c = cq + 4 * r;
                t[c][wl] = in ? src[(int64_t)c * g.H * g.W] : (short)0;
            }
            __syncthreads();
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int q = tid + 256 * i, px = q >> 3, ch = q & 7;
                if (wp0 + px < Wp) {
                    h8 o;
#pragma unroll
                    for (int e = 0; e < 8; ++e) o[e] = (_Float16)t[ch * 8 + e][px];
                    *(h8*)(dst + (int64_t)(wp0 + px) * g.Ci + c0 + ch * 8) = o;
                }
            }
            __syncthreads();
        }
        return;
    }
    if ((int)blockIdx.x >= p.wblocks) return;
    const int kc = p.Kd / 8;
    const int64_t v = (int64_t)blockIdx.x * 256 + tid;
    if (v >= (int64_t)p.Cop * kc) return;
    const int co = (int)(v / kc), k0 = (int)(v - (int64_t)co * kc) * 8;
    const int tap = k0 / g.Ci, ci0 = k0 - tap * g.Ci;
    const int kh = tap / g.KW, kw = tap - kh * g.KW;
    h8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e)
        o[e] = co < p.Co ? (_Float16)((const int16_t*)p.w)[(((int64_t)co * g.Ci + ci0 + e) * g.KH + kh) * g.KW + kw]
                         : (_Float16)0.0f;
    *(h8*)((_Float16*)p.w16 + (int64_t)co * p.Kd + k0) = o;
}

// FP32 counterpart of k_conv_prep (C_in a multiple of 32): x NCHW float ->
// zero-bordered NHWC float xp; w OIHW float -> w32 [Cop][Kd] with
// k = (kh*KW + kw)*Ci + ci.  Values are copied unchanged.
__global__ __launch_bounds__(256) void k_conv_prep_f32(const ConvPrepParams p) {
    const ConvGeom& g = p.g;
    const int tid = threadIdx.x;
    if (blockIdx.y == 0) {
        if ((int)blockIdx.x >= p.xblocks) return;
        __shared__ float t[32][65];
        const int Hp = g.H + 2 * g.pad, Wp = g.W + 2 * g.pad;
        const int wch = (Wp + 63) / 64;
        const int n = blockIdx.x / (Hp * wch), rem = blockIdx.x - n * Hp * wch;
        const int hp = rem / wch, wp0 = (rem - hp * wch) * 64;
        const int h = hp - g.pad;
        const bool row_in = h >= 0 && h < g.H;
        const int wl = tid & 63, cq = tid >> 6;
        const int w = wp0 + wl - g.pad;
        const bool in = row_in && w >= 0 && w < g.W;
        float* dst = (float*)p.xp + ((int64_t)n * Hp + hp) * Wp * g.Ci;
        for (int c0 = 0; c0 < g.Ci; c0 += 32) {
            const float* src = (const float*)p.x + (((int64_t)n * g.Ci + c0) * g.H + h) * g.W + w;
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const int c = cq + 4 * r;
                t[c][wl] = in ? src[(int64_t)c * g.H * g.W] : 0.0f;
            }
            __syncthreads();
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int q = tid + 256 * i, px = q >> 3, ch = q & 7;
                if (wp0 + px < Wp) {
                    f4v o;
#pragma unroll
                    for (int e = 0; e < 4; ++e) o[e] = t[ch * 4 + e][px];
                    *(f4v*)(dst + (int64_t)(wp0 + px) * g.Ci + c0 + ch * 4) = o;
                }
            }
            __syncthreads();
        }
        return;
    }
    if ((int)blockIdx.x >= p.wblocks) return;
    const int kc = p.Kd / 4;
    const int64_t v = (int64_t)blockIdx.x * 256 + tid;
    if (v >= (int64_t)p.Cop * kc) return;
    const int co = (int)(v / kc), k0 = (int)(v - (int64_t)co * kc) * 4;
    const int tap = k0 / g.Ci, ci0 = k0 - tap * g.Ci;
    const int kh = tap / g.KW, kw = tap - kh * g.KW;
    f4v o;
#pragma unroll
    for (int e = 0; e < 4; ++e)
        o[e] = co < p.Co ? ((const float*)p.w)[(((int64_t)co * g.Ci + ci0 + e) * g.KH + kh) * g.KW + kw] : 0.0f;
    *(f4v*)((float*)p.w16 + (int64_t)co * p.Kd + k0) = o;
}

// ===========================================================================
// Stage 2: contraction
// ===========================================================================
__device__ __forceinline__ int chunk_swz(int r) { return (r >> 1) & 7; }

// FP32 contraction (conv FP32 row) on v_mfma_f32_32x32x2f32 with the same
// staging: a K tile is 32 fp32 = 128-byte rows of eight 16-byte chunks, same
// swizzle and direct-to-LDS ring.  In k-step ks (8 k) lane half h reads chunk
// 2*ks + h of its row / column, and MFMA e of the step takes element e of it:
// K-slot (h, e) is k = 8*ks + 4*h + e for both operands.  The sum is formed
// in fp32 in the matrix cores' order.  IMPL gathers B from the bordered NHWC
// fp32 image, 32 channels of one kernel tap per K tile.
template <int BM, int BN, int NW, bool IMPL, int WN = 64>
__global__ __launch_bounds__(NW * 64) void k_gemm_nt_f32(const GemmParams p) {
    constexpr int BK = 32, KCH = 8, WM = 64;
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int WAVES_N = BN / WN;
    static_assert((BM / WM) * (BN / WN) == NW, "wave grid");
    constexpr int NTH = NW * 64;
    constexpr int AL = BM * KCH / NTH, BL = BN * KCH / NTH, LPT = AL + BL;
    static_assert(AL * NTH == BM * KCH && BL * NTH == BN * KCH, "whole loads");
    constexpr int STAGES = 3;
    constexpr unsigned STAGE_A = BM * KCH * 16, STAGE_B = BN * KCH * 16;
    __shared__ f4v As[STAGES][BM][KCH];
    __shared__ f4v Bs[STAGES][BN][KCH];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, hh = lane >> 5;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int tiles_m = (p.M + BM - 1) / BM, tiles_n = p.tiles_n;
    int pid = blockIdx.x;
    const int total = gridDim.x;
    if ((total & 7) == 0) pid = (pid & 7) * (total >> 3) + (pid >> 3);
    int tm, tn;
    {
        constexpr int G = 8;
        const int per_group = G * tiles_n;
        const int gid = pid / per_group;
        const int first_m = gid * G;
        const int gsz = min(tiles_m - first_m, G);
        const int in = pid - gid * per_group;
        tm = first_m + in % gsz;
        tn = in / gsz;
    }
    const int m0 = tm * BM, n0 = tn * BN;
    const int b = blockIdx.z;
    const float* A = (const float*)p.A + b * p.sA;   // [Mp][lda], lda = Kp
    const float* B = (const float*)p.B + b * p.sB;   // [Np][ldb] or the NHWC image
    float* C = (float*)p.C + b * p.sC;

    unsigned oa[AL], ob[BL];
#pragma unroll
    for (int i = 0; i < AL; ++i) {
        const int q = tid + NTH * i, row = q / KCH, pc = q % KCH;
        oa[i] = (unsigned)(((int64_t)row * p.lda + (pc ^ chunk_swz(row)) * 4) * 4);
    }
    const ConvGeom& g = p.g;
    const int Hp = g.H + 2 * g.pad, Wp = g.W + 2 * g.pad;
#pragma unroll
    for (int i = 0; i < BL; ++i) {
        const int q = tid + NTH * i, row = q / KCH, pc = q % KCH;
        if (IMPL) {
            int pix = n0 + row;
            if (pix >= p.N) pix = 0;     // never stored
            const int img = pix / p.hw, rem = pix - img * p.hw;
            const int oh = rem / g.Wo, ow = rem - oh * g.Wo;
            const int64_t base = (((int64_t)img * Hp + oh * g.stride) * Wp + ow * g.stride) * g.Ci;
            ob[i] = (unsigned)((base + (pc ^ chunk_swz(row)) * 4) * 4);
        } else {
            ob[i] = (unsigned)(((int64_t)row * p.ldb + (pc ^ chunk_swz(row)) * 4) * 4);
        }
    }
    const char* a_panel = (const char*)(A + (int64_t)m0 * p.lda);
    const char* b_panel = IMPL ? (const char*)B : (const char*)(B + (int64_t)n0 * p.ldb);
    int tap_h = 0, tap_w = 0, tap_c = 0;
    const unsigned wave_u = __builtin_amdgcn_readfirstlane(wave);
    const unsigned lds_a0 = (unsigned)(uintptr_t)&As[0][0][0] + wave_u * 1024;
    const unsigned lds_b0 = (unsigned)(uintptr_t)&Bs[0][0][0] + wave_u * 1024;
    auto issue = [&](int t) {
        const int s = t % STAGES;
        const char* ab = a_panel + t * BK * 4;
        const char* bb;
        if (IMPL) {
            bb = b_panel + (int64_t)((tap_h * Wp + tap_w) * g.Ci + tap_c) * 4;
            tap_c += BK;
            if (tap_c == g.Ci) {
                tap_c = 0;
                if (++tap_w == g.KW) {
                    tap_w = 0;
                    ++tap_h;
                }
            }
        } else {
            bb = b_panel + t * BK * 4;
        }
        const unsigned la = lds_a0 + s * STAGE_A, lb = lds_b0 + s * STAGE_B;
#pragma unroll
        for (int i = 0; i < AL; ++i)
            asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                         :: "v"(oa[i]), "s"(ab), "s"(la + NTH * 16 * i) : "memory", "m0");
#pragma unroll
        for (int i = 0; i < BL; ++i)
            asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                         :: "v"(ob[i]), "s"(bb), "s"(lb + NTH * 16 * i) : "memory", "m0");
    };

    f16x acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f16x{};
    auto ldf = [&](int s, int ks, f4v (&a)[TM], f4v (&bv)[TN]) {
        const int c = ks * 2 + hh;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int row = wm * WM + i * 32 + l32;
            a[i] = As[s][row][c ^ chunk_swz(row)];
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = wn * WN + j * 32 + l32;
            bv[j] = Bs[s][col][c ^ chunk_swz(col)];
        }
    };
    const int ktiles = p.K / BK;   // K is padded to whole tiles
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
        if (s < ktiles) issue(s);
    for (int t = 0; t < ktiles; ++t) {
        if (t + 1 < ktiles) __builtin_amdgcn_s_waitcnt((LPT & 15) | ((LPT >> 4) << 14) | 0x0F70);
        else __builtin_amdgcn_s_waitcnt(0x0F70);
        __syncthreads();
        if (t + STAGES - 1 < ktiles) issue(t + STAGES - 1);
        const int s = t % STAGES;
        constexpr int KS = BK / 8;
        f4v fa[KS][TM], fb[KS][TN];
        ldf(s, 0, fa[0], fb[0]);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (ks + 1 < KS) ldf(s, ks + 1, fa[ks + 1], fb[ks + 1]);
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[ks][i][e], fb[ks][j][e], acc[i][j],
                                                                         0, 0, 0);
        }
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int gn = n0 + wn * WN + j * 32 + l32;
        if (gn >= p.N) continue;
        int64_t col_off, row_stride;
        if (p.out_mode == OUT_ROWMAJOR) {
            col_off = gn;
            row_stride = p.ldc;
        } else {
            const int img = gn / p.hw, pix = gn - img * p.hw;
            col_off = (int64_t)img * p.M * p.hw + pix;
            row_stride = p.hw;
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int gm = m0 + wm * WM + i * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
                // non-temporal, as in the integer contraction (FP32 conv
                // 8x64x56x56 -> 128: about 1 us of 43)
                if (gm < p.M) __builtin_nontemporal_store(acc[i][j][r], &C[(int64_t)gm * row_stride + col_off]);
            }
    }
}

// One 32x32x16 MFMA step of the fp16-exact route: fp16 operands, or bf16
// ones (the same 16-bit lanes) with BF; fp32 accumulation either way.
template <bool BF>
__device__ __forceinline__ f16x mfma_h(h8 a, h8 b, f16x c) {
    if constexpr (BF)
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(b8v, a), __builtin_bit_cast(b8v, b), c,
                                                       0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

template <int BM, int BN, int NW, bool IMPL, bool BF, int WN = 64>
__global__ __launch_bounds__(NW * 64) void k_gemm_nt(const GemmParams p) {
    constexpr int BK = 64, KCH = 8, WM = 64;
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int WAVES_N = BN / WN;
    static_assert((BM / WM) * (BN / WN) == NW, "wave grid");
    constexpr int NTH = NW * 64;
    constexpr int AL = BM * KCH / NTH, BL = BN * KCH / NTH, LPT = AL + BL;
    static_assert(AL * NTH == BM * KCH && BL * NTH == BN * KCH, "whole loads");
    constexpr int STAGES = 3;
    constexpr unsigned STAGE_A = BM * KCH * 16, STAGE_B = BN * KCH * 16;
    __shared__ h8 As[STAGES][BM][KCH];
    __shared__ h8 Bs[STAGES][BN][KCH];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, hh = lane >> 5;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    // Workgroup -> tile: consecutive ids go to different XCDs, so first
    // gather each XCD's ids into one contiguous range, then walk tiles in
    // groups of 8 tile-rows (neighbouring workgroups share B panels).
    const int tiles_m = (p.M + BM - 1) / BM, tiles_n = p.tiles_n;
    int pid = blockIdx.x;
    const int total = gridDim.x;
    if ((total & 7) == 0) pid = (pid & 7) * (total >> 3) + (pid >> 3);
    int tm, tn;
    {
        constexpr int G = 8;
        const int per_group = G * tiles_n;
        const int gid = pid / per_group;
        const int first_m = gid * G;
        const int gsz = min(tiles_m - first_m, G);
        const int in = pid - gid * per_group;
        tm = first_m + in % gsz;
        tn = in / gsz;
    }
    const int m0 = tm * BM, n0 = tn * BN;
    const int b = blockIdx.z;
    const _Float16* A = (const _Float16*)p.A + b * p.sA;   // [Mp][lda], lda = Kp
    const _Float16* B = (const _Float16*)p.B + b * p.sB;   // [Np][ldb], ldb = Kp
    int32_t* C = (int32_t*)p.C + b * p.sC;

    // Per-thread byte offsets of the chunks it fetches, relative to the panel.
    unsigned oa[AL], ob[BL];
#pragma unroll
    for (int i = 0; i < AL; ++i) {
        const int q = tid + NTH * i, row = q / KCH, pc = q % KCH;
        oa[i] = (unsigned)((row * p.lda + (pc ^ chunk_swz(row)) * 8) * 2);
    }
    const ConvGeom& g = p.g;
    const int Hp = g.H + 2 * g.pad, Wp = g.W + 2 * g.pad;
#pragma unroll
    for (int i = 0; i < BL; ++i) {
        const int q = tid + NTH * i, row = q / KCH, pc = q % KCH;
        if (IMPL) {
            // pixel base in xp; rows past the last pixel re-read pixel 0
            // (their results are never stored)
            int pix = n0 + row;
            if (pix >= p.N) pix = 0;
            const int img = pix / p.hw, rem = pix - img * p.hw;
            const int oh = rem / g.Wo, ow = rem - oh * g.Wo;
            const int64_t base = (((int64_t)img * Hp + oh * g.stride) * Wp + ow * g.stride) * g.Ci;
            ob[i] = (unsigned)((base + (pc ^ chunk_swz(row)) * 8) * 2);
        } else {
            ob[i] = (unsigned)((row * p.ldb + (pc ^ chunk_swz(row)) * 8) * 2);
        }
    }
    const char* a_panel = (const char*)(A + (int64_t)m0 * p.lda);
    const char* b_panel = IMPL ? (const char*)B : (const char*)(B + (int64_t)n0 * p.ldb);
    // IMPL: kernel tap and channel offset of the next K tile to be issued
    int tap_h = 0, tap_w = 0, tap_c = 0;
    const unsigned wave_u = __builtin_amdgcn_readfirstlane(wave);
    const unsigned lds_a0 = (unsigned)(uintptr_t)&As[0][0][0] + wave_u * 1024;
    const unsigned lds_b0 = (unsigned)(uintptr_t)&Bs[0][0][0] + wave_u * 1024;
    // One wave-wide global_load_lds_dwordx4 writes 64 lanes x 16 bytes
    // contiguously at M0; the lane -> global chunk mapping realises the swizzle.
    auto issue = [&](int t) {
        const int s = t % STAGES;
        const char* ab = a_panel + t * BK * 2;
        const char* bb;
        if (IMPL) {
            // tiles are issued in order 0, 1, 2, ...
            bb = b_panel + (int64_t)((tap_h * Wp + tap_w) * g.Ci + tap_c) * 2;
            tap_c += BK;
            if (tap_c == g.Ci) {
                tap_c = 0;
                if (++tap_w == g.KW) {
                    tap_w = 0;
                    ++tap_h;
                }
            }
        } else {
            bb = b_panel + t * BK * 2;
        }
        const unsigned la = lds_a0 + s * STAGE_A, lb = lds_b0 + s * STAGE_B;
#pragma unroll
        for (int i = 0; i < AL; ++i)
            asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                         :: "v"(oa[i]), "s"(ab), "s"(la + NTH * 16 * i) : "memory", "m0");
#pragma unroll
        for (int i = 0; i < BL; ++i)
            asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                         :: "v"(ob[i]), "s"(bb), "s"(lb + NTH * 16 * i) : "memory", "m0");
    };

    f16x acc[TM][TN];
    u16x iacc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) iacc[i][j] = u16x{};

    // K-slot (lane half h, element e) of the MFMA is k = 16*ks + 8*h + e for
    // both operands.  The fragments of k-step ks+1 are read while the MFMAs of
    // k-step ks run, and MFMA clusters raise the wave's issue priority so the
    // other wave on the SIMD issues its LDS reads and DMA in between.
    auto ldf = [&](int s, int ks, h8 (&a)[TM], h8 (&bv)[TN]) {
        const int c = ks * 2 + hh;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int row = wm * WM + i * 32 + l32;
            a[i] = As[s][row][c ^ chunk_swz(row)];
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = wn * WN + j * 32 + l32;
            bv[j] = Bs[s][col][c ^ chunk_swz(col)];
        }
    };
    auto compute = [&](int s, bool first) {
        constexpr int KS = BK / 16;
        h8 fa[KS][TM], fb[KS][TN];
        ldf(s, 0, fa[0], fb[0]);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (ks + 1 < KS) ldf(s, ks + 1, fa[ks + 1], fb[ks + 1]);
            __builtin_amdgcn_s_setprio(1);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = mfma_h<BF>(fa[ks][i], fb[ks][j], (first && ks == 0) ? f16x{} : acc[i][j]);
            __builtin_amdgcn_s_setprio(0);
        }
    };

    const int ktiles = p.K / BK;   // K is padded to whole tiles
    const int CT = p.chunk_tiles;
    if constexpr (NW == 8) {
        // Ping-pong: the waves form two groups, one wave of each per SIMD.
        // Phases alternate between barriers; in every phase one group reads
        // a whole tile's fragments from LDS and issues its share of the DMA
        // while the other runs the MFMAs of the tile it read in the phase
        // before, so the matrix cores and the LDS work side by side instead
        // of in turns.  Group 1 runs one phase behind group 0:
        //   phase 2t:   group 0 reads tile t      group 1 computes tile t-1
        //   phase 2t+1: group 0 computes tile t   group 1 reads tile t
        // Tile u is issued by each wave in its read phase of tile u-2 (tiles
        // 0 and 1 before the loop) into the stage of tile u-3, which both
        // groups finished reading by then; it must have landed before phase
        // 2u, so every wave ends phase 2t+1 with tile t+1 complete.
        constexpr int KS = BK / 16;
        // s_waitcnt immediates: vmcnt(n) with lgkmcnt(0)
        constexpr unsigned WAIT_VM_LPT = (LPT & 15) | ((LPT >> 4) << 14) | 0x0070;
        constexpr unsigned WAIT_VM_0 = 0x0070;
        const int grp = wave >> 2;
        // a phase boundary: no instruction moves across it
        auto phase_end = [] {
            __builtin_amdgcn_sched_barrier(0);
            __syncthreads();
            __builtin_amdgcn_sched_barrier(0);
        };
        h8 fa[KS][TM], fb[KS][TN];
        issue(0);
        if (1 < ktiles) {
            issue(1);
            __builtin_amdgcn_s_waitcnt(WAIT_VM_LPT);
        } else {
            __builtin_amdgcn_s_waitcnt(WAIT_VM_0);
        }
        phase_end();
        if (grp == 1) phase_end();
        // One tile: its read phase, then its compute phase.  ZERO (the first
        // tile of a flush chunk) starts the fp32 accumulators from zero; the
        // last tile of a chunk adds them into the int32 accumulators.
        auto ptile = [&](int tc, auto zero, bool flush) {
            constexpr bool ZERO = decltype(zero)::value;
            const int s = tc % STAGES;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) ldf(s, ks, fa[ks], fb[ks]);
            if (tc + 2 < ktiles) issue(tc + 2);
            if (grp == 1) {
                if (tc + 2 < ktiles) __builtin_amdgcn_s_waitcnt(WAIT_VM_LPT);
                else __builtin_amdgcn_s_waitcnt(WAIT_VM_0);
            } else {
                __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
            }
            phase_end();
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = mfma_h<BF>(fa[ks][i], fb[ks][j], (ZERO && ks == 0) ? f16x{} : acc[i][j]);
            if (flush) {
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
#pragma unroll
                        for (int r = 0; r < 16; ++r) iacc[i][j][r] += (uint32_t)(int32_t)acc[i][j][r];
            }
            if (grp == 0) {
                if (tc + 2 < ktiles) __builtin_amdgcn_s_waitcnt(WAIT_VM_LPT);
                else __builtin_amdgcn_s_waitcnt(WAIT_VM_0);
            }
            phase_end();
        };
        if (CT >= 4 && TM * TN == 4) {
            // Staggered flushes: the four 32x32 blocks of a wave close their
            // chunks on different tiles -- block b on every tile t with
            // t % 4 == b (t >= 1) -- so each compute phase converts and adds
            // one block (32 vector ops) while the same wave's 16 MFMAs run,
            // instead of all four blocks (128 vector ops, as long as the
            // MFMAs themselves) after every fourth tile.  Every chunk spans
            // at most four tiles (256 K), within the exactness bound since
            // CT >= 4.  FB = the block closed and restarted on this tile; 4 =
            // the first tile, where every block starts from zero.
            // Fragment reads at a stage offset the optimiser cannot see
            // through, so the per-lane addresses of the three stages are not
            // all precomputed and kept live (that alone would cost 48
            // registers).
            auto ldf_at = [&](unsigned soff_a, unsigned soff_b, int ks, h8 (&a)[TM], h8 (&bv)[TN]) {
                const int c = ks * 2 + hh;
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    const int row = wm * WM + i * 32 + l32;
                    a[i] = *(const h8*)((const char*)&As[0][row][c ^ chunk_swz(row)] + soff_a);
                }
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const int col = wn * WN + j * 32 + l32;
                    bv[j] = *(const h8*)((const char*)&Bs[0][col][c ^ chunk_swz(col)] + soff_b);
                }
            };
            auto stile = [&](int tc, auto fb_c) {
                constexpr int FB = decltype(fb_c)::value;
                unsigned soff = (unsigned)(tc % STAGES);
                asm volatile("" : "+s"(soff));
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) ldf_at(soff * STAGE_A, soff * STAGE_B, ks, fa[ks], fb[ks]);
                if (tc + 2 < ktiles) issue(tc + 2);
                if (grp == 1) {
                    if (tc + 2 < ktiles) __builtin_amdgcn_s_waitcnt(WAIT_VM_LPT);
                    else __builtin_amdgcn_s_waitcnt(WAIT_VM_0);
                } else {
                    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
                }
                phase_end();
                if constexpr (FB < 4) {
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        iacc[FB / 2][FB % 2][r] += (uint32_t)(int32_t)acc[FB / 2][FB % 2][r];
                    // pin the conversion to this phase: left to itself the
                    // optimiser sinks it past later tiles, which keeps the
                    // old fp32 block alive beside the restarted one
                    asm volatile("" : "+v"(iacc[FB / 2][FB % 2]));
                }
                // the restarted block comes last in the first k-step, so its
                // conversion has the other blocks' MFMAs to run beside
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
#pragma unroll
                    for (int q = 1; q <= 4; ++q) {
                        const int b = FB < 4 ? (FB + q) & 3 : q - 1;
                        const int i = b >> 1, j = b & 1;
                        const bool zero = ks == 0 && (FB == 4 || b == FB);
                        acc[i][j] = mfma_h<BF>(fa[ks][i], fb[ks][j], zero ? f16x{} : acc[i][j]);
                    }
                if (grp == 0) {
                    if (tc + 2 < ktiles) __builtin_amdgcn_s_waitcnt(WAIT_VM_LPT);
                    else __builtin_amdgcn_s_waitcnt(WAIT_VM_0);
                }
                phase_end();
            };
            using I0 = std::integral_constant<int, 0>;
            using I1 = std::integral_constant<int, 1>;
            using I2 = std::integral_constant<int, 2>;
            using I3 = std::integral_constant<int, 3>;
            stile(0, std::integral_constant<int, 4>{});
            int tc = 1;
            for (; tc + 3 < ktiles; tc += 4) {
                stile(tc, I1{});
                stile(tc + 1, I2{});
                stile(tc + 2, I3{});
                stile(tc + 3, I0{});
            }
            if (tc < ktiles) stile(tc, I1{});
            if (tc + 1 < ktiles) stile(tc + 1, I2{});
            if (tc + 2 < ktiles) stile(tc + 2, I3{});
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) iacc[i][j][r] += (uint32_t)(int32_t)acc[i][j][r];
        } else {
            for (int tc = 0; tc < ktiles;) {
                const int cend = min(tc + CT, ktiles);
                ptile(tc, std::true_type{}, tc + 1 == cend);
                for (++tc; tc < cend; ++tc) ptile(tc, std::false_type{}, tc + 1 == cend);
            }
        }
        if (grp == 0) phase_end();
    } else {
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
        if (s < ktiles) issue(s);
    int t = 0;
    while (t < ktiles) {
        const int cend = min(t + CT, ktiles);
        for (int tc = t; tc < cend; ++tc) {
            // Tile tc must have landed; the next one may still be in flight.
            if (tc + 1 < ktiles) __builtin_amdgcn_s_waitcnt((LPT & 15) | ((LPT >> 4) << 14) | 0x0F70);
            else __builtin_amdgcn_s_waitcnt(0x0F70);
            __syncthreads();
            if (tc + STAGES - 1 < ktiles) issue(tc + STAGES - 1);
            compute(tc % STAGES, tc == t);
        }
        t = cend;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) iacc[i][j][r] += (uint32_t)(int32_t)acc[i][j][r];
    }
    }

    // 32x32 accumulator layout: lane holds column (lane & 31), rows
    // 8*(r/4) + 4*(lane/32) + r%4.
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int gn = n0 + wn * WN + j * 32 + l32;
        if (gn >= p.N) continue;
        int64_t col_off;
        int64_t row_stride;
        if (p.out_mode == OUT_ROWMAJOR) {
            col_off = gn;
            row_stride = p.ldc;
        } else {
            const int img = gn / p.hw, pix = gn - img * p.hw;
            col_off = (int64_t)img * p.M * p.hw + pix;
            row_stride = p.hw;
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int gm = m0 + wm * WM + i * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
                // non-temporal: the output is not re-read here, and kept out
                // of L2 it does not evict the operand tiles other
                // workgroups are still streaming
                if (gm < p.M) __builtin_nontemporal_store((int32_t)iacc[i][j][r], &C[(int64_t)gm * row_stride + col_off]);
            }
    }
}

// ===========================================================================
// Builders
// ===========================================================================
void nt_tile_shape(int64_t M, int64_t N, int64_t batch, int* bm, int* bn) {
    // 128x256 (8 waves) when there are enough tiles to fill the chip,
    // otherwise 128x128 (4 waves).
    const int64_t big = ((M + 127) / 128) * ((N + 255) / 256) * batch;
    const int64_t mid = ((M + 127) / 128) * ((N + 127) / 128) * batch;
    if (big >= 512) {
        *bm = 128;
        *bn = 256;
    } else if (mid >= 256) {
        *bm = 128;
        *bn = 128;
    } else {
        *bm = 64;     // two 64x64 waves per workgroup: more workgroups for small M
        *bn = 128;
    }
}

void build_gemm_nt(const GemmParams& p0, int batch, LaunchRec* rec) {
    int bm, bn;
    nt_tile_shape(p0.M, p0.N, batch, &bm, &bn);
    GemmParams p = p0;
    const int tiles_m = (p.M + bm - 1) / bm;
    p.tiles_n = (p.N + bn - 1) / bn;
    rec->grid = dim3((unsigned)(tiles_m * p.tiles_n), 1, (unsigned)batch);
    const bool impl = p.b_mode == B_NHWC;
    const bool bf = p.bf16 != 0 && !impl;   // the conv image copy is fp16
    if (bn == 256) {
        rec->fn = impl ? (const void*)k_gemm_nt<128, 256, 8, true, false>
                       : bf ? (const void*)k_gemm_nt<128, 256, 8, false, true> : (const void*)k_gemm_nt<128, 256, 8, false, false>;
        rec->block = dim3(512, 1, 1);
        rec->name = impl ? "gemm_nt_conv_128x256" : bf ? "gemm_nt_bf16_128x256" : "gemm_nt_128x256";
    } else if (bm == 64) {
        // the conv gather runs four 64x32 waves (more loads in flight per
        // CU than two 64x64 ones: 14.0 -> 12.2 us on 8x64x56x56 -> 128)
        rec->fn = impl ? (const void*)k_gemm_nt<64, 128, 4, true, false, 32>
                       : bf ? (const void*)k_gemm_nt<64, 128, 2, false, true> : (const void*)k_gemm_nt<64, 128, 2, false, false>;
        rec->block = dim3(impl ? 256 : 128, 1, 1);
        rec->name = impl ? "gemm_nt_conv_64x128" : bf ? "gemm_nt_bf16_64x128" : "gemm_nt_64x128";
    } else {
        rec->fn = impl ? (const void*)k_gemm_nt<128, 128, 4, true, false>
                       : bf ? (const void*)k_gemm_nt<128, 128, 4, false, true> : (const void*)k_gemm_nt<128, 128, 4, false, false>;
        rec->block = dim3(256, 1, 1);
        rec->name = impl ? "gemm_nt_conv_128x128" : bf ? "gemm_nt_bf16_128x128" : "gemm_nt_128x128";
    }
    rec->set_params(p);
}

void build_gemm_nt_f32(const GemmParams& p0, int batch, LaunchRec* rec) {
    int bm, bn;
    nt_tile_shape(p0.M, p0.N, batch, &bm, &bn);
    GemmParams p = p0;
    const int tiles_m = (p.M + bm - 1) / bm;
    p.tiles_n = (p.N + bn - 1) / bn;
    rec->grid = dim3((unsigned)(tiles_m * p.tiles_n), 1, (unsigned)batch);
    const bool impl = p.b_mode == B_NHWC;
    if (bn == 256) {
        rec->fn = impl ? (const void*)k_gemm_nt_f32<128, 256, 8, true> : (const void*)k_gemm_nt_f32<128, 256, 8, false>;
        rec->block = dim3(512, 1, 1);
        rec->name = impl ? "gemm_nt_f32_conv_128x256" : "gemm_nt_f32_128x256";
    } else if (bm == 64) {
        // the conv gather runs four 64x32 waves, as the fp16 one does
        rec->fn = impl ? (const void*)k_gemm_nt_f32<64, 128, 4, true, 32> : (const void*)k_gemm_nt_f32<64, 128, 2, false>;
        rec->block = dim3(impl ? 256 : 128, 1, 1);
        rec->name = impl ? "gemm_nt_f32_conv_64x128" : "gemm_nt_f32_64x128";
    } else {
        rec->fn = impl ? (const void*)k_gemm_nt_f32<128, 128, 4, true> : (const void*)k_gemm_nt_f32<128, 128, 4, false>;
        rec->block = dim3(256, 1, 1);
        rec->name = impl ? "gemm_nt_f32_conv_128x128" : "gemm_nt_f32_128x128";
    }
    rec->set_params(p);
}

void build_conv_prep(const ConvPrepParams& p0, LaunchRec* rec) {
    ConvPrepParams p = p0;
    const ConvGeom& g = p.g;
    const int Hp = g.H + 2 * g.pad, Wp = g.W + 2 * g.pad;
    p.xblocks = p.nimg * Hp * ((Wp + 63) / 64);
    const bool f32 = p.elem_bytes == 4;
    p.wblocks = (int32_t)(((int64_t)p.Cop * (p.Kd / (f32 ? 4 : 8)) + 255) / 256);
    rec->fn = f32 ? (const void*)k_conv_prep_f32 : (const void*)k_conv_prep;
    rec->grid = dim3((unsigned)std::max(p.xblocks, p.wblocks), 2, 1);
    rec->block = dim3(256, 1, 1);
    rec->name = f32 ? "conv_prep_nhwc_f32" : "conv_prep_nhwc_f16";
    rec->set_params(p);
}

void build_enc_a(const EncParams& p, LaunchRec* rec) {
    const int64_t n = (int64_t)p.batch * p.Mp * (p.Kp / 8);
    rec->fn = p.bf16 ? (const void*)k_enc_a<true> : (const void*)k_enc_a<false>;
    rec->grid = dim3((unsigned)((n + 1023) / 1024), 1, 1);
    rec->block = dim3(256, 1, 1);
    rec->name = p.bf16 ? "enc_a_bf16" : "enc_a_f16";
    rec->set_params(p);
}

void build_enc_bt(const EncParams& p, LaunchRec* rec) {
    rec->fn = p.bf16 ? (const void*)k_enc_bt<true> : (const void*)k_enc_bt<false>;
    rec->grid = dim3((unsigned)((p.Np + 127) / 128), (unsigned)((p.Kp + 127) / 128), (unsigned)p.batch);
    rec->block = dim3(256, 1, 1);
    rec->name = p.bf16 ? "enc_bt_bf16" : "enc_bt_f16";
    rec->set_params(p);
}

void build_im2col_t(const Im2colTParams& p, LaunchRec* rec) {
    const ConvGeom& g = p.g;
    const int Wp = (g.Wo - 1) * g.stride + g.KW;
    const size_t lds = (size_t)8 * g.KH * Wp * 2;
    if (g.Ci % 8 == 0 && lds <= 32768 && g.Ho <= 65535 && g.Ci / 8 <= 65535) {
        rec->fn = (const void*)k_im2col_t8;
        rec->grid = dim3((unsigned)g.Ho, (unsigned)(g.Ci / 8), (unsigned)(p.P / (g.Ho * g.Wo)));
        rec->block = dim3(256, 1, 1);
        rec->shmem = (uint32_t)lds;
        rec->name = "im2col_t8_f16";
        rec->set_params(p);
        return;
    }
    const int64_t n = (int64_t)p.Pp * (p.Kp / 8);
    rec->fn = (const void*)k_im2col_t;
    rec->grid = dim3((unsigned)((n + 255) / 256), 1, 1);
    rec->block = dim3(256, 1, 1);
    rec->name = "im2col_t_f16";
    rec->set_params(p);
}

}  // namespace qx
