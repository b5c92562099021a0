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
typedef int i4v __attribute__((ext_vector_type(4)));

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
    // K slices (integer kinds): slice kz covers [kb, ke), whole 16-k steps
    const int ks = (VK != VK_F32 && p.ksplit > 1) ? p.ksplit : 1;
    const int b = (int)blockIdx.z / ks, kz = (int)blockIdx.z - b * ks;
    int kb = 0, ke = p.K;
    if (ks > 1) {
        const int per = ((p.K + ks - 1) / ks + VBK - 1) / VBK * VBK;
        kb = min(p.K, kz * per);
        ke = min(p.K, kb + per);
    }
    const In* A = (const In*)p.A + b * p.sA;
    const In* B = (const In*)p.B + b * p.sB;

    Acc acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = (Acc)0;

    // A tile: 64 rows x 16 k, B tile 16 k x 64 columns, 4 elements of each
    // per thread; the next step's elements are loaded into registers while
    // the current step's multiply-adds run
    In ra[4], rb[4];
    auto load_step = [&](int k0) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int idx = tid + VT * e, r = idx / VBK, kk = idx % VBK;
            const int gm = m0 + r, gk = k0 + kk;
            ra[e] = (gm < p.M && gk < ke) ? A[(int64_t)gm * p.lda + gk] : (In)0;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int idx = tid + VT * e;
            int kk, c;
            if (p.b_trans) { c = idx / VBK; kk = idx % VBK; }
            else { kk = idx / VBN; c = idx % VBN; }
            const int gk = k0 + kk, gn = n0 + c;
            In v = (In)0;
            if (gk < ke && gn < p.N)
                v = p.b_trans ? B[(int64_t)gn * p.ldb + gk] : B[(int64_t)gk * p.ldb + gn];
            rb[e] = v;
        }
    };
    if (kb < ke) load_step(kb);
    for (int k0 = kb; k0 < ke; k0 += VBK) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int idx = tid + VT * e;
            As[idx % VBK][idx / VBK] = ra[e];
            if (p.b_trans) Bs[idx % VBK][idx / VBK] = rb[e];
            else Bs[idx / VBN][idx % VBN] = rb[e];
        }
        __syncthreads();
        if (k0 + VBK < ke) load_step(k0 + VBK);
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
            if constexpr (VK == VK_F32) {
                ((float*)p.C + b * p.sC)[off] = (float)acc[i][j];
            } else {
                uint32_t* c = (uint32_t*)p.C + b * p.sC + off;
                if (ks > 1) atomicAdd(c, (uint32_t)acc[i][j]);   // wrapping: exact in any order
                else *c = (uint32_t)acc[i][j];
            }
        }
}

// smul24 GEMM with few output columns (the fully connected layers of a
// LeNet-shaped network: N of 10 to 120) on the vector ALU, instead of the
// (M/64) x (N/64) mostly empty 64x64 tiles of k_valu_gemm.  A workgroup
// owns 64 rows (one per lane) and NG columns; its four waves take a quarter
// of K each and their partial sums are added at the end (wrapping int32
// sums: the split changes nothing), so that a SIMD holds several waves,
// whose scalar, LDS and vector instructions interleave.
//  - B: every lane of a wave multiplies by the same B[k][n0 .. n0+NG), so B
//    is read with scalar loads (through the constant address space: B is
//    never written while the kernel runs) and each multiply-add takes its B
//    operand from a scalar register.
//  - A: a lane's own row, read straight from memory, would touch a
//    different cache line per lane and instruction; each wave stages its
//    64 rows through its own LDS slice instead, KC k at a time, with loads
//    whose lanes run along k (eight rows of 128 bytes per instruction), and
//    each lane then reads its row 16 bytes at a time (rows padded by 4
//    words: the eight lanes of one LDS cycle hit distinct banks).  Only the
//    wave touches its slice, so a wave-level fence orders the accesses; the
//    next chunk is fetched into registers while the current one is used.
template <int NG>
__global__ __launch_bounds__(VT) void k_valu_skinny_s24(const ValuGemmParams p) {
    constexpr int KC = 32, AP = KC + 4, WR = 64, NWV = VT / 64;
    typedef const __attribute__((address_space(4))) int32_t* cptr;
    __shared__ __align__(16) int32_t As[NWV][WR][AP];
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // Workgroups (row block, column group), column groups fastest.  The
    // dispatcher deals consecutive workgroups to the eight XCDs in turn;
    // when their count is a multiple of 8, XCD x is given the x-th eighth of
    // them instead, whole row blocks with all their column groups, so that
    // a block of A is fetched into that XCD's L2 once, not once per group.
    const int groups = (p.N + NG - 1) / NG, nwg = gridDim.x;
    int lin = blockIdx.x;
    if ((nwg & 7) == 0) lin = (lin & 7) * (nwg >> 3) + (lin >> 3);
    const int m0 = (lin / groups) * WR, m = m0 + lane;
    const int n0g = (lin % groups) * NG;
    // The last column group moves left to end at column N - 1 (it overlaps
    // the previous group and stores only its own columns), so every scalar
    // load of B reads NG contiguous words inside the matrix (N >= NG).
    const int n0 = min(n0g, p.N - NG);
    const int b = blockIdx.z;
    const int32_t* A = (const int32_t*)p.A + b * p.sA;
    const cptr B = (cptr)(uintptr_t)((const int32_t*)p.B + b * p.sB + n0);
    const bool vec = (p.K & 3) == 0 && (p.lda & 3) == 0 && (((uintptr_t)A) & 15) == 0;
    // this wave's share of K: quarters rounded up to whole 16-byte words
    const int kper = ((p.K + 4 * NWV - 1) / (4 * NWV)) * 4;
    const int kb = min(p.K, w * kper), ke = min(p.K, kb + kper);
    int32_t (*as)[AP] = As[w];
    // staging: lane loads rows lane / 8 + 8 i (i < 8), words 4 (lane % 8) .. +3 of the chunk
    const int sr = lane / (KC / 4), sq = (lane % (KC / 4)) * 4;
    auto load_a = [&](int k0, i4v* r) {
#pragma unroll
        for (int i = 0; i < WR / 8; ++i) {
            const int row = m0 + sr + 8 * i, k = k0 + sq;
            const int32_t* src = A + (int64_t)row * p.lda + k;
            if (vec) {
                r[i] = (row < p.M && k < p.K) ? *(const i4v*)src : i4v{0, 0, 0, 0};
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) r[i][e] = (row < p.M && k + e < p.K) ? src[e] : 0;
            }
        }
    };
    auto store_a = [&](const i4v* r) {
        // the previous chunk's reads of the slice are done before it is overwritten
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int i = 0; i < WR / 8; ++i) *(i4v*)&as[sr + 8 * i][sq] = r[i];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };
    // B rows are addressed by a 32-bit byte offset from B (the planner sends
    // K <= 4096 rows of ldb = N <= 128 words: under 2 MiB), stepped by one
    // row per load, which keeps the scalar address arithmetic to one add per
    // row
    typedef const __attribute__((address_space(4))) char* cbptr;
    const cbptr Bb = (cbptr)B;
    const uint32_t row_bytes = 4u * (uint32_t)p.ldb;
    auto load_b_at = [&](uint32_t off, int32_t* r) {
        const cptr row = (cptr)(Bb + off);
#pragma unroll
        for (int j = 0; j < NG; ++j) r[j] = row[j];
    };
    auto load_b = [&](int k, int32_t* r) { load_b_at((uint32_t)k * row_bytes, r); };
    uint32_t acc[NG];
#pragma unroll
    for (int j = 0; j < NG; ++j) acc[j] = 0u;
    // the next chunk of A is fetched into registers while the current one
    // is multiplied
    i4v a_reg[WR / 8];
    if (kb < ke) load_a(kb, a_reg);
    for (int k0 = kb; k0 < ke; k0 += KC) {
        store_a(a_reg);
        if (k0 + KC < ke) load_a(k0 + KC, a_reg);
        if (k0 + KC <= ke) {
            // whole chunk, four k at a time: one wait covers the scalar
            // loads of four B rows (scalar loads return out of order, so
            // any wait for one of them waits for all)
            uint32_t boff = (uint32_t)k0 * row_bytes;
#pragma unroll
            for (int q = 0; q < KC / 4; ++q) {
                int32_t bq[4][NG];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    load_b_at(boff, bq[e]);
                    boff += row_bytes;
                }
                const i4v a4 = *(const i4v*)&as[lane][4 * q];
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int j = 0; j < NG; ++j) acc[j] += (uint32_t)__mul24(a4[e], bq[e][j]);
            }
        } else {
            for (int kk = 0; kk < ke - k0; ++kk) {
                const int a = as[lane][kk];
                int32_t bk[NG];
                load_b(k0 + kk, bk);
#pragma unroll
                for (int j = 0; j < NG; ++j) acc[j] += (uint32_t)__mul24(a, bk[j]);
            }
        }
    }
    // join the four K quarters: wave w adds up and stores columns w, w + 4, ...
    __syncthreads();
    uint32_t* red = (uint32_t*)&As[0][0][0];   // [NG][NWV][64]
#pragma unroll
    for (int j = 0; j < NG; ++j) red[(j * NWV + w) * 64 + lane] = acc[j];
    __syncthreads();
    if (m >= p.M) return;
    int32_t* C = (int32_t*)p.C + b * p.sC;
    for (int j = w; j < NG; j += NWV) {
        const int gn = n0 + j;
        if (gn < n0g) continue;
        uint32_t v = 0u;
#pragma unroll
        for (int q = 0; q < NWV; ++q) v += red[(j * NWV + q) * 64 + lane];
        int64_t off;
        if (p.out_mode == OUT_ROWMAJOR) {
            off = (int64_t)m * p.ldc + gn;
        } else {
            const int img = gn / p.hw, pix = gn - img * p.hw;
            off = ((int64_t)img * p.M + m) * p.hw + pix;
        }
        C[off] = p.relu ? max((int32_t)v, 0) : (int32_t)v;
    }
}

void build_valu_skinny_s24(const ValuGemmParams& p, int batch, LaunchRec* rec) {
    // columns per workgroup: the largest of 8, 4, 2, 1 not above N
    const int ng = p.N >= 8 ? 8 : p.N >= 4 ? 4 : p.N >= 2 ? 2 : 1;
    rec->fn = ng == 8 ? (const void*)k_valu_skinny_s24<8> : ng == 4 ? (const void*)k_valu_skinny_s24<4>
            : ng == 2 ? (const void*)k_valu_skinny_s24<2> : (const void*)k_valu_skinny_s24<1>;
    rec->name = "valu_s24_skinny";
    rec->grid = dim3((unsigned)(((p.M + 63) / 64) * ((p.N + ng - 1) / ng)), 1u, (unsigned)batch);
    rec->block = dim3(VT, 1, 1);
    rec->set_params(p);
}

void build_valu_gemm(int32_t kind, const ValuGemmParams& p, int batch, LaunchRec* rec) {
    switch (kind) {
    case VK_I16_DOT2: rec->fn = (const void*)k_valu_gemm<VK_I16_DOT2>; rec->name = "valu_dot2"; break;
    case VK_S24: rec->fn = (const void*)k_valu_gemm<VK_S24>; rec->name = "valu_s24"; break;
    case VK_I32: rec->fn = (const void*)k_valu_gemm<VK_I32>; rec->name = "valu_i32"; break;
    default: rec->fn = (const void*)k_valu_gemm<VK_F32>; rec->name = "valu_f32"; break;
    }
    const int ks = (kind != VK_F32 && p.ksplit > 1) ? p.ksplit : 1;
    rec->grid = dim3((unsigned)((p.N + VBN - 1) / VBN), (unsigned)((p.M + VBM - 1) / VBM), (unsigned)(batch * ks));
    rec->block = dim3(VT, 1, 1);
    rec->set_params(p);
}

}  // namespace qx
