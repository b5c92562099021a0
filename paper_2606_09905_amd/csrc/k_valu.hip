// k_valu.hip -- vector-ALU GEMM paths.
//
// Comparison and fallback routes of the substrate that never touch the
// matrix cores: packed INT16 pairs through v_dot2_i32_i16, the smul24
// contract natively through the 24-bit multiplier (v_mul_i32_i24 /
// v_mad_i32_i24 class), plain wrapping int32, and float32 with a fixed
// summation order.  The smul24 path is the instruction the paper's integer
// kernels are built around (Methodology: smul24 operand contract).
//
// Tiling: a 64x64 output tile per 256-thread workgroup, 4x4 outputs per
// thread, K staged through LDS 16 elements at a time (k-major in LDS so
// that a thread's four rows / columns are one 16-byte read).
#include "qx_internal.h"

namespace qx {

constexpr int VT = 256;
constexpr int VBM = 64, VBN = 64, VBK = 16;

typedef short s2 __attribute__((ext_vector_type(2)));

template <int VK>
struct ValuT;
template <> struct ValuT<VK_I16_DOT2> { typedef int16_t In; typedef uint32_t Acc; };
template <> struct ValuT<VK_S24> { typedef int32_t In; typedef uint32_t Acc; };
template <> struct ValuT<VK_I32> { typedef int32_t In; typedef uint32_t Acc; };
template <> struct ValuT<VK_F32> { typedef float In; typedef float Acc; };

template <int VK>
__global__ __launch_bounds__(VT) void k_valu_gemm(const ValuGemmParams p) {
    typedef typename ValuT<VK>::In In;
    typedef typename ValuT<VK>::Acc Acc;
    __shared__ In As[VBK][VBM + 4];
    __shared__ In Bs[VBK][VBN + 4];

    const int tid = threadIdx.x;
    const int tx = tid % 16, ty = tid / 16;        // 16 x 16 threads, 4 x 4 outputs each
    const int m0 = blockIdx.y * VBM, n0 = blockIdx.x * VBN;
    const int b = blockIdx.z;
    const In* A = (const In*)p.A + b * p.sA;
    const In* B = (const In*)p.B + b * p.sB;

    Acc acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = (Acc)0;

    for (int k0 = 0; k0 < p.K; k0 += VBK) {
        // A tile: 64 rows x 16 k, 4 elements per thread.
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int idx = tid + VT * e, r = idx / VBK, kk = idx % VBK;
            const int gm = m0 + r, gk = k0 + kk;
            As[kk][r] = (gm < p.M && gk < p.K) ? A[(int64_t)gm * p.lda + gk] : (In)0;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int idx = tid + VT * e;
            int kk, c;
            if (p.b_trans) { c = idx / VBK; kk = idx % VBK; }
            else { kk = idx / VBN; c = idx % VBN; }
            const int gk = k0 + kk, gn = n0 + c;
            In v = (In)0;
            if (gk < p.K && gn < p.N)
                v = p.b_trans ? B[(int64_t)gn * p.ldb + gk] : B[(int64_t)gk * p.ldb + gn];
            Bs[kk][c] = v;
        }
        __syncthreads();
        if (VK == VK_I16_DOT2) {
#pragma unroll
            for (int kk = 0; kk < VBK; kk += 2) {
                s2 a[4], bb[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    a[i] = s2{(short)As[kk][ty * 4 + i], (short)As[kk + 1][ty * 4 + i]};
                    bb[i] = s2{(short)Bs[kk][tx * 4 + i], (short)Bs[kk + 1][tx * 4 + i]};
                }
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc[i][j] = (Acc)__builtin_amdgcn_sdot2(a[i], bb[j], (int)acc[i][j], false);
            }
        } else {
#pragma unroll
            for (int kk = 0; kk < VBK; ++kk) {
                In a[4], bb[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    a[i] = As[kk][ty * 4 + i];
                    bb[i] = Bs[kk][tx * 4 + i];
                }
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        if (VK == VK_S24)
                            acc[i][j] += (uint32_t)__mul24((int)a[i], (int)bb[j]);
                        else if (VK == VK_I32)
                            acc[i][j] += (uint32_t)a[i] * (uint32_t)bb[j];
                        else
                            acc[i][j] = fmaf((float)a[i], (float)bb[j], (float)acc[i][j]);
                    }
            }
        }
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int gm = m0 + ty * 4 + i, gn = n0 + tx * 4 + j;
            if (gm >= p.M || gn >= p.N) continue;
            int64_t off;
            if (p.out_mode == OUT_ROWMAJOR) {
                off = (int64_t)gm * p.ldc + gn;
            } else {
                const int img = gn / p.hw, pix = gn - img * p.hw;
                off = ((int64_t)img * p.M + gm) * p.hw + pix;
            }
            if (VK == VK_F32) ((float*)p.C + b * p.sC)[off] = (float)acc[i][j];
            else ((int32_t*)p.C + b * p.sC)[off] = (int32_t)acc[i][j];
        }
}

void build_valu_gemm(int32_t kind, const ValuGemmParams& p, int batch, LaunchRec* rec) {
    switch (kind) {
    case VK_I16_DOT2: rec->fn = (const void*)k_valu_gemm<VK_I16_DOT2>; rec->name = "valu_dot2"; break;
    case VK_S24: rec->fn = (const void*)k_valu_gemm<VK_S24>; rec->name = "valu_s24"; break;
    case VK_I32: rec->fn = (const void*)k_valu_gemm<VK_I32>; rec->name = "valu_i32"; break;
    default: rec->fn = (const void*)k_valu_gemm<VK_F32>; rec->name = "valu_f32"; break;
    }
    rec->grid = dim3((unsigned)((p.N + VBN - 1) / VBN), (unsigned)((p.M + VBM - 1) / VBM), (unsigned)batch);
    rec->block = dim3(VT, 1, 1);
    rec->set_params(p);
}

}  // namespace qx
