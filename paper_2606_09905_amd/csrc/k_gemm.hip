// k_gemm.hip -- the tiled integer GEMM substrate on gfx950 matrix cores.
//
// Two exact routes share one tile skeleton (global -> registers -> encode ->
// LDS, double-buffered; LDS -> registers -> MFMA; int32 epilogue):
//
//  * F16_EXACT: int16 operands with |a|,|b| <= 2048 are exact in fp16 and
//    their products exact in fp32.  v_mfma_f32_32x32x16_f16 accumulates in
//    fp32 for `chunk` K elements with chunk*max|a|*max|b| <= 2^24, so every
//    partial sum is an integer fp32 represents exactly whatever the internal
//    summation order; the partials are then converted and added into int32
//    (mod 2^32) accumulators.
//  * I8 limbs: operands are split into int8 limb planes while being staged,
//    each limb product runs on v_mfma_i32_32x32x32_i8 (int32 accumulation),
//    and the epilogue recombines the planes mod 2^32 (direct, Karatsuba
//    base 128, offset base 256 with a rank-1 correction, and the smul24
//    three-limb split with eight products).
//
// These realise the packed INT16-input / INT32-accumulation GEMM and the
// smul24 INT32 GEMM of the paper (Methodology; Table 1), with the operand
// range contract deciding the route (Methodology: contracts determine
// feasible tiling, packing and accumulation).
#include <algorithm>

#include <type_traits>

#include "qx_internal.h"

namespace qx {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef float f16x __attribute__((ext_vector_type(16)));
typedef int i16x __attribute__((ext_vector_type(16)));
typedef unsigned u16x __attribute__((ext_vector_type(16)));
typedef int i4 __attribute__((ext_vector_type(4)));
typedef short s8 __attribute__((ext_vector_type(8)));
typedef short s4 __attribute__((ext_vector_type(4)));

constexpr int NT = 256;  // threads per workgroup (4 waves)

// Workgroup -> output tile.  Tiles are walked in groups of 8 tile-rows so
// that consecutive workgroups share B panels.
__device__ __forceinline__ void tile_coords(int tiles_m, int tiles_n, int& tm, int& tn) {
    const int pid = blockIdx.x;
    constexpr int G = 8;
    const int per_group = G * tiles_n;
    const int gid = pid / per_group;
    const int first_m = gid * G;
    const int gsz = min(tiles_m - first_m, G);
    const int in = pid - gid * per_group;
    tm = first_m + in % gsz;
    tn = in / gsz;
}

// Store one int32 result with the epilogue's layout.
__device__ __forceinline__ int64_t c_index(const GemmParams& p, int gm, int gn) {
    if (p.out_mode == OUT_ROWMAJOR) return (int64_t)gm * p.ldc + gn;
    const int img = gn / p.hw, pix = gn - img * p.hw;
    return ((int64_t)img * p.M + gm) * p.hw + pix;
}

__device__ __forceinline__ void store_c(const GemmParams& p, int32_t* C, int gm, int gn, uint32_t v) {
    if (gm >= p.M || gn >= p.N) return;
    C[c_index(p, gm, gn)] = (int32_t)v;
}

// ===========================================================================
// F16_EXACT
// ===========================================================================
// LDS rows hold BK fp16 as 16-byte chunks; chunk index is XOR-swizzled with
// the row so that the eight consecutive rows read by one ds_read_b128 pass
// land in distinct banks.
__device__ __forceinline__ int swz_a(int row, int c) { return c ^ (row & 7); }
__device__ __forceinline__ int swz_b(int col, int c) { return c ^ ((col ^ (col >> 3)) & 7); }

template <int BM, int BN, int BK, int WM, int WN, bool ALIGNED, bool FLUSH_STEP>
__global__ __launch_bounds__(NT) void k_gemm_f16x(const GemmParams p) {
    static_assert(BK == 64, "chunk swizzle assumes 8 chunks per row");
    constexpr int KCH = BK / 8;
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int WAVES_N = BN / WN;
    static_assert((BM / WM) * (BN / WN) == 4, "four waves");
    constexpr int A_VECS = BM * KCH / NT;         // 16-byte A vectors per thread
    constexpr int B_NBLK = BN / 8;                // B staged as 4(k) x 8(n) blocks
    constexpr int B_THREADS = (BK / 4) * B_NBLK;  // threads that stage one B block each
    static_assert(B_THREADS <= NT && NT % B_THREADS == 0, "B blocks");

    __shared__ h8 As[2][BM][KCH];
    __shared__ h8 Bs[2][BN][KCH];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int tiles_m = (p.M + BM - 1) / BM;
    int tm, tn;
    tile_coords(tiles_m, p.tiles_n, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const int b = blockIdx.z;
    const int16_t* A = (const int16_t*)p.A + b * p.sA;
    const int16_t* B = (const int16_t*)p.B + b * p.sB;
    int32_t* C = (int32_t*)p.C + b * p.sC;

    s8 ra[A_VECS];
    s8 rb[4];
    const int bkb = tid / B_NBLK, bnb = tid % B_NBLK;

    auto load = [&](int k0) {
#pragma unroll
        for (int i = 0; i < A_VECS; ++i) {
            const int v = tid + NT * i, row = v / KCH, c = v % KCH;
            const int gm = m0 + row, gk = k0 + c * 8;
            if (ALIGNED) {
                ra[i] = (gm < p.M && gk < p.K) ? *(const s8*)(A + (int64_t)gm * p.lda + gk) : s8{};
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    ra[i][e] = (gm < p.M && gk + e < p.K) ? A[(int64_t)gm * p.lda + gk + e] : (short)0;
            }
        }
        if (B_THREADS < NT && tid >= B_THREADS) return;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int gk = k0 + bkb * 4 + r, gn = n0 + bnb * 8;
            if (ALIGNED) {
                rb[r] = (gk < p.K && gn < p.N) ? *(const s8*)(B + (int64_t)gk * p.ldb + gn) : s8{};
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    rb[r][e] = (gk < p.K && gn + e < p.N) ? B[(int64_t)gk * p.ldb + gn + e] : (short)0;
            }
        }
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int i = 0; i < A_VECS; ++i) {
            const int v = tid + NT * i, row = v / KCH, c = v % KCH;
            h8 h;
#pragma unroll
            for (int e = 0; e < 8; ++e) h[e] = (_Float16)ra[i][e];
            As[buf][row][swz_a(row, c)] = h;
        }
        if (B_THREADS < NT && tid >= B_THREADS) return;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const int col = bnb * 8 + c;
            h4 h;
#pragma unroll
            for (int r = 0; r < 4; ++r) h[r] = (_Float16)rb[r][c];
            h4* dst = (h4*)&Bs[buf][col][swz_b(col, bkb >> 1)];
            dst[bkb & 1] = h;
        }
    };

    f16x acc[TM][TN];
    u16x iacc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            acc[i][j] = f16x{};
            iacc[i][j] = u16x{};
        }
    auto flush = [&]() {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
#pragma unroll
                for (int r = 0; r < 16; ++r) iacc[i][j][r] += (uint32_t)(int32_t)acc[i][j][r];
                acc[i][j] = f16x{};
            }
    };

    const int ktiles = (p.K + BK - 1) / BK;
    // The MFMA steps of one staged K tile.  With FLUSH_STEP each step's
    // product block is a whole chunk (16 k): it starts from zero and is
    // converted and added on its own.
    auto compute = [&](int buf) {
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            h8 a[TM], bv[TN];
            const int c = ks * 2 + (lane >> 5);
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int row = wm * WM + i * 32 + (lane & 31);
                a[i] = As[buf][row][swz_a(row, c)];
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int col = wn * WN + j * 32 + (lane & 31);
                bv[j] = Bs[buf][col][swz_b(col, c)];
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    if (FLUSH_STEP) {
                        const f16x r = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[i], bv[j], f16x{}, 0, 0, 0);
#pragma unroll
                        for (int e = 0; e < 16; ++e) iacc[i][j][e] += (uint32_t)(int32_t)r[e];
                    } else {
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[i], bv[j], acc[i][j], 0, 0, 0);
                    }
                }
        }
    };
    int since_flush = 0;
    load(0);
    stash(0);
    __syncthreads();
    for (int t = 0; t < ktiles; ++t) {
        const int buf = t & 1;
        if (t + 1 < ktiles) load((t + 1) * BK);
        compute(buf);
        if (!FLUSH_STEP && ++since_flush == p.chunk_tiles) {
            flush();
            since_flush = 0;
        }
        if (t + 1 < ktiles) stash(buf ^ 1);
        __syncthreads();
    }
    if (!FLUSH_STEP) flush();

    // 32x32 accumulator layout: lane holds column (lane & 31) and rows
    // 8*(r/4) + 4*(lane/32) + r%4.
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int gm = m0 + wm * WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                const int gn = n0 + wn * WN + j * 32 + (lane & 31);
                store_c(p, C, gm, gn, iacc[i][j][r]);
            }
}

// Small fp16-exact GEMMs (K <= 256): a workgroup owns a 32 x 32 output tile
// and its four waves take one 64-k tile each, so a workgroup waits on memory
// once and each wave runs a quarter of the K steps; the waves' int32
// partials are then added through LDS.  A fragments come straight from
// global memory (8 consecutive k of a row are one 16-byte load); B goes
// through LDS to be transposed (k-contiguous per column).
template <bool ALIGNED, bool FLUSH_STEP>
__global__ __launch_bounds__(NT) void k_gemm_f16_ks(const GemmParams p) {
    constexpr int BK = 64;
    __shared__ h8 Bs[4][32][BK / 8];          // per wave: [col][k chunk], chunks swizzled
    __shared__ u16x red[3][64];               // partials of waves 1..3
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hh = lane >> 5;
    const int tiles_m = (p.M + 31) / 32;
    const int tm = (int)blockIdx.x % tiles_m, tn = (int)blockIdx.x / tiles_m;
    const int m0 = tm * 32, n0 = tn * 32;
    const int b = blockIdx.z;
    const int16_t* A = (const int16_t*)p.A + b * p.sA;
    const int16_t* B = (const int16_t*)p.B + b * p.sB;
    int32_t* C = (int32_t*)p.C + b * p.sC;
    const int k0 = wave * BK;                 // this wave's K tile (none past K)

    // A: lane (row l32, half hh) holds k = k0 + 16 ks + 8 hh .. +7
    s8 ra[4];
    const int gm = m0 + l32;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
        const int gk = k0 + 16 * ks + 8 * hh;
        if (ALIGNED) {
            ra[ks] = (gm < p.M && gk < p.K) ? *(const s8*)(A + (int64_t)gm * p.lda + gk) : s8{};
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                ra[ks][e] = (gm < p.M && gk + e < p.K) ? A[(int64_t)gm * p.lda + gk + e] : (short)0;
        }
    }
    // B: lane (kr, nc) loads k = k0 + 4 kr .. +3 of columns n0 + 8 nc .. +7
    const int kr = lane >> 2, nc = lane & 3;
    s8 rb[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int gk = k0 + 4 * kr + r, gn = n0 + 8 * nc;
        if (ALIGNED) {
            rb[r] = (gk < p.K && gn < p.N) ? *(const s8*)(B + (int64_t)gk * p.ldb + gn) : s8{};
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                rb[r][e] = (gk < p.K && gn + e < p.N) ? B[(int64_t)gk * p.ldb + gn + e] : (short)0;
        }
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const int col = 8 * nc + c;
        h4 h;
#pragma unroll
        for (int r = 0; r < 4; ++r) h[r] = (_Float16)rb[r][c];
        h4* dst = (h4*)&Bs[wave][col][swz_b(col, kr >> 1)];
        dst[kr & 1] = h;
    }
    __syncthreads();

    u16x iacc = u16x{};
    f16x acc = f16x{};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
        h8 a;
#pragma unroll
        for (int e = 0; e < 8; ++e) a[e] = (_Float16)ra[ks][e];
        const h8 bv = Bs[wave][l32][swz_b(l32, ks * 2 + hh)];
        if (FLUSH_STEP) {
            // each 16-k step is a whole chunk: converted and added on its own
            const f16x r = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bv, f16x{}, 0, 0, 0);
#pragma unroll
            for (int e = 0; e < 16; ++e) iacc[e] += (uint32_t)(int32_t)r[e];
        } else {
            acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bv, acc, 0, 0, 0);
        }
    }
    if (!FLUSH_STEP) {
#pragma unroll
        for (int e = 0; e < 16; ++e) iacc[e] = (uint32_t)(int32_t)acc[e];
    }
    if (wave > 0) red[wave - 1][lane] = iacc;
    __syncthreads();
    if (wave > 0) return;
#pragma unroll
    for (int w = 0; w < 3; ++w) {
        const u16x o = red[w][lane];
#pragma unroll
        for (int e = 0; e < 16; ++e) iacc[e] += o[e];
    }
    // 32x32 accumulator layout: lane holds column l32 and rows
    // 8*(r/4) + 4*hh + r%4.
#pragma unroll
    for (int r = 0; r < 16; ++r)
        store_c(p, C, m0 + 8 * (r >> 2) + 4 * hh + (r & 3), n0 + l32, iacc[r]);
}

// ===========================================================================
// int8 limb routes
// ===========================================================================
// A scheme splits each operand into PLANES int8 limbs, issues PRODUCTS limb
// products into GROUPS accumulators, and recombines them mod 2^32.
// PAD is the operand value whose limbs are all zero: padding a ragged K tail
// with it adds nothing to any limb product.
// value(x) is the integer the split represents (sext24 for smul24); offset
// schemes (PAD != 0) need its row and column sums for the rank-1 correction.
struct SchemeDirect {   // |x| <= 127
    static constexpr int PLANES = 1, GROUPS = 1, PRODUCTS = 1, PAD = 0;
    template <class T> __device__ static int32_t value(T x) { return (int32_t)x; }
    static constexpr int pa[1] = {0}, pb[1] = {0}, pg[1] = {0};
    template <class T> __device__ static void split(T x, uint32_t* l) { l[0] = (uint32_t)x & 0xFFu; }
    __device__ static uint32_t combine(const uint32_t* g) { return g[0]; }
};
struct SchemeKaratsuba {  // x in [-8256, 8127]: balanced base 128, h, l, h+l
    static constexpr int PLANES = 3, GROUPS = 3, PRODUCTS = 3, PAD = 0;
    template <class T> __device__ static int32_t value(T x) { return (int32_t)x; }
    static constexpr int pa[3] = {0, 1, 2}, pb[3] = {0, 1, 2}, pg[3] = {0, 1, 2};
    template <class T> __device__ static void split(T xv, uint32_t* l) {
        const int x = (int)xv;
        const int lo = ((x + 64) & 127) - 64;
        const int hi = (x - lo) >> 7;
        l[0] = (uint32_t)hi & 0xFFu;
        l[1] = (uint32_t)lo & 0xFFu;
        l[2] = (uint32_t)(hi + lo) & 0xFFu;
    }
    // a*b = 2^14 hh + 2^7 (mm - hh - ll) + ll
    __device__ static uint32_t combine(const uint32_t* g) {
        return (g[0] << 14) + ((g[2] - g[0] - g[1]) << 7) + g[1];
    }
};
struct SchemeOffset4 {  // any int16: x = 256*s1 + s0 + 128, s1 = x>>8, s0 = (x & 255) - 128
    static constexpr int PLANES = 2, GROUPS = 3, PRODUCTS = 4, PAD = 128;
    template <class T> __device__ static int32_t value(T x) { return (int32_t)x; }
    // product order keeps consecutive MFMAs on different accumulators
    static constexpr int pa[4] = {0, 0, 1, 1}, pb[4] = {0, 1, 1, 0}, pg[4] = {0, 1, 2, 1};
    template <class T> __device__ static void split(T xv, uint32_t* l) {
        const uint32_t x = (uint32_t)(int)xv;
        l[0] = (x >> 8) & 0xFFu;          // s1 (arithmetic high byte of an int16)
        l[1] = (x & 0xFFu) ^ 0x80u;       // s0 = low byte - 128
    }
    __device__ static uint32_t combine(const uint32_t* g) { return (g[0] << 16) + (g[1] << 8) + g[2]; }
};
struct SchemeS24 {  // smul24: u = sext24(x) + 2^23, s_i = byte_i(u) - 128, x = sum 2^(8i) s_i + 32896
    static constexpr int PLANES = 3, GROUPS = 4, PRODUCTS = 8, PAD = 0x8080;
    template <class T> __device__ static int32_t value(T x) { return (int32_t)((uint32_t)(int32_t)x << 8) >> 8; }
    // limb pairs (i, j) with i + j <= 3 into group i + j, ordered so that
    // consecutive MFMAs never accumulate into the same group
    static constexpr int pa[8] = {0, 0, 0, 1, 1, 1, 2, 2};
    static constexpr int pb[8] = {0, 1, 2, 2, 0, 1, 1, 0};
    static constexpr int pg[8] = {0, 1, 2, 3, 1, 2, 3, 2};
    template <class T> __device__ static void split(T xv, uint32_t* l) {
        const uint32_t u = ((uint32_t)(int)xv & 0xFFFFFFu) ^ 0x808080u ^ 0x800000u;
        l[0] = u & 0xFFu;
        l[1] = (u >> 8) & 0xFFu;
        l[2] = (u >> 16) & 0xFFu;
    }
    __device__ static uint32_t combine(const uint32_t* g) {
        return g[0] + (g[1] << 8) + (g[2] << 16) + (g[3] << 24);
    }
};

// Aligned vector load of N elements (whole 16-byte transactions).
template <class T, int N>
struct alignas(N * sizeof(T) >= 16 ? 16 : N * sizeof(T)) VecN {
    T v[N];
};
template <class T, int N>
__device__ __forceinline__ void load_vec(const T* src, T (&dst)[N]) {
    const VecN<T, N> x = *(const VecN<T, N>*)src;
#pragma unroll
    for (int e = 0; e < N; ++e) dst[e] = x.v[e];
}

// 64-byte LDS rows (BK = 64 int8) as four 16-byte chunks; the swizzle keeps
// the eight rows of one ds_read_b128 pass in distinct banks.
__device__ __forceinline__ int swz8(int row, int c) { return c ^ ((row >> 1) & 3); }

template <class S, class T, int BM, int BN, int WM, int WN, bool ALIGNED>
__global__ __launch_bounds__(NT) void k_gemm_i8limb(const GemmParams p) {
    constexpr int BK = 64, KCH = 4;
    constexpr int P = S::PLANES, G = S::GROUPS;
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int WAVES_N = BN / WN;
    static_assert((BM / WM) * (BN / WN) == 4, "four waves");
    constexpr int A_VECS = BM * BK / 8 / NT;      // 8-element A vectors per thread
    constexpr int BWN = BN / 16;                  // B staged as 4(k) x BWN(n) blocks
    static_assert((BK / 4) * (BN / BWN) == NT, "one B block per thread");

    __shared__ i4 As[2][P][BM][KCH];
    __shared__ i4 Bs[2][P][BN][KCH];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int tiles_m = (p.M + BM - 1) / BM;
    int tm, tn;
    tile_coords(tiles_m, p.tiles_n, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const int b = blockIdx.z;
    const T* A = (const T*)p.A + b * p.sA;
    const T* B = (const T*)p.B + b * p.sB;
    int32_t* C = (int32_t*)p.C + b * p.sC;

    T ra[A_VECS][8];
    T rb[4][BWN];
    const int bkb = tid / (BN / BWN), bnb = tid % (BN / BWN);

    auto load = [&](int k0) {
#pragma unroll
        for (int i = 0; i < A_VECS; ++i) {
            const int v = tid + NT * i, row = v / 8, e8 = v % 8;
            const int gm = m0 + row, gk = k0 + e8 * 8;
            const T* src = A + (int64_t)gm * p.lda + gk;
            if (ALIGNED && gm < p.M && gk < p.K) {
                load_vec<T, 8>(src, ra[i]);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) ra[i][e] = (gm < p.M && gk + e < p.K) ? src[e] : (T)S::PAD;
            }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int gk = k0 + bkb * 4 + r, gn = n0 + bnb * BWN;
            const T* src = B + (int64_t)gk * p.ldb + gn;
            if (ALIGNED && gk < p.K && gn < p.N) {
                load_vec<T, BWN>(src, rb[r]);
            } else {
#pragma unroll
                for (int e = 0; e < BWN; ++e) rb[r][e] = (gk < p.K && gn + e < p.N) ? src[e] : (T)S::PAD;
            }
        }
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int i = 0; i < A_VECS; ++i) {
            const int v = tid + NT * i, row = v / 8, e8 = v % 8;
            uint32_t w[P][2] = {};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                uint32_t l[P];
                S::split(ra[i][e], l);
#pragma unroll
                for (int q = 0; q < P; ++q) w[q][e >> 2] |= l[q] << (8 * (e & 3));
            }
#pragma unroll
            for (int q = 0; q < P; ++q) {
                uint32_t* dst = (uint32_t*)&As[buf][q][row][swz8(row, e8 >> 1)];
                dst[(e8 & 1) * 2 + 0] = w[q][0];
                dst[(e8 & 1) * 2 + 1] = w[q][1];
            }
        }
#pragma unroll
        for (int c = 0; c < BWN; ++c) {
            const int col = bnb * BWN + c;
            uint32_t w[P] = {};
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                uint32_t l[P];
                S::split(rb[r][c], l);
#pragma unroll
                for (int q = 0; q < P; ++q) w[q] |= l[q] << (8 * r);
            }
#pragma unroll
            for (int q = 0; q < P; ++q) {
                uint32_t* dst = (uint32_t*)&Bs[buf][q][col][swz8(col, bkb >> 2)];
                dst[bkb & 3] = w[q];
            }
        }
    };

    i16x acc[G][TM][TN];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[g][i][j] = i16x{};

    const int ktiles = (p.K + BK - 1) / BK;
    load(0);
    stash(0);
    __syncthreads();
    for (int t = 0; t < ktiles; ++t) {
        const int buf = t & 1;
        if (t + 1 < ktiles) load((t + 1) * BK);
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            const int c = ks * 2 + (lane >> 5);
            i4 a[P][TM], bv[P][TN];
#pragma unroll
            for (int q = 0; q < P; ++q) {
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    const int row = wm * WM + i * 32 + (lane & 31);
                    a[q][i] = As[buf][q][row][swz8(row, c)];
                }
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const int col = wn * WN + j * 32 + (lane & 31);
                    bv[q][j] = Bs[buf][q][col][swz8(col, c)];
                }
            }
#pragma unroll
            for (int pr = 0; pr < S::PRODUCTS; ++pr)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[S::pg[pr]][i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(
                            a[S::pa[pr]][i], bv[S::pb[pr]][j], acc[S::pg[pr]][i][j], 0, 0, 0);
        }
        if (t + 1 < ktiles) stash(buf ^ 1);
        __syncthreads();
    }

    const uint32_t cc = (uint32_t)p.corr_c;
    const uint32_t kcc = (uint32_t)p.K * cc * cc;
    const int32_t* rs = p.rowsum ? p.rowsum + (int64_t)b * p.M : nullptr;
    // column sums arrive as cs_slices partial rows [slice][N]
    const int32_t* cs = p.colsum ? p.colsum + (int64_t)b * p.cs_slices * p.N : nullptr;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int gn = n0 + wn * WN + j * 32 + (lane & 31);
        if (gn >= p.N) continue;
        uint32_t csum = 0;
        if (cc)
            for (int s = 0; s < p.cs_slices; ++s) csum += (uint32_t)cs[(int64_t)s * p.N + gn];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int gm = m0 + wm * WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                if (gm >= p.M) continue;
                uint32_t g[G];
#pragma unroll
                for (int q = 0; q < G; ++q) g[q] = (uint32_t)acc[q][i][j][r];
                uint32_t v = S::combine(g);
                if (cc) v += cc * ((uint32_t)rs[gm] + csum) - kcc;
                store_c(p, C, gm, gn, v);
            }
    }
}

// ===========================================================================
// int8 limb routes for large problems: encode to limb planes, then an NT
// int8 GEMM staged global -> LDS with global_load_lds_dwordx4.
// ===========================================================================
// smul24 limbs of four operands packed per plane with byte permutes: the
// dword of plane q holds limb q of u0..u3 in bytes 0..3.  Limb q is byte q
// of (x mod 2^24) ^ 0x008080 (bytes 0 and 1 flipped by 0x80), so the padding
// value 0x8080 packs to zero bytes.
__device__ __forceinline__ void pack_s24(uint32_t u0, uint32_t u1, uint32_t u2, uint32_t u3, uint32_t* d) {
    const uint32_t lo = __builtin_amdgcn_perm(u1, u0, 0x05010400u);   // (u0.b0, u1.b0, u0.b1, u1.b1)
    const uint32_t hi = __builtin_amdgcn_perm(u3, u2, 0x05010400u);   // (u2.b0, u3.b0, u2.b1, u3.b1)
    d[0] = __builtin_amdgcn_perm(hi, lo, 0x05040100u) ^ 0x80808080u;
    d[1] = __builtin_amdgcn_perm(hi, lo, 0x07060302u) ^ 0x80808080u;
    const uint32_t lo2 = __builtin_amdgcn_perm(u1, u0, 0x0C0C0602u);  // (u0.b2, u1.b2, 0, 0)
    const uint32_t hi2 = __builtin_amdgcn_perm(u3, u2, 0x0C0C0602u);
    d[2] = __builtin_amdgcn_perm(hi2, lo2, 0x05040100u);
}

// Limb dwords of four k-consecutive elements x[0..3] (ok[r] false: padding,
// all-zero limbs) for every plane, and their represented values' sum.
template <class S, class T>
__device__ __forceinline__ uint32_t pack4(const T* x, const bool* ok, uint32_t* w) {
    uint32_t sum = 0;
    if constexpr (std::is_same<S, SchemeS24>::value && sizeof(T) == 4) {
        uint32_t u[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            u[r] = ok[r] ? (uint32_t)x[r] : (uint32_t)S::PAD;
            sum += ok[r] ? (uint32_t)S::value(x[r]) : 0u;
        }
        pack_s24(u[0], u[1], u[2], u[3], w);
    } else {
#pragma unroll
        for (int q = 0; q < S::PLANES; ++q) w[q] = 0;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            uint32_t l[S::PLANES];
            S::split(x[r], l);
#pragma unroll
            for (int q = 0; q < S::PLANES; ++q) w[q] |= (ok[r] ? l[q] : 0u) << (8 * r);
            sum += ok[r] ? (uint32_t)S::value(x[r]) : 0u;
        }
    }
    return sum;
}

// A [batch][M][lda] (T) -> A8 [batch][P][Mp][Kp] int8 limb planes.  One wave
// per row (half a wave when Kp <= 512); a lane splits 16 consecutive k per
// step.  Elements outside M x K
// become all-zero limbs (the split of S::PAD), which add nothing to any limb
// product.  Offset schemes also get the row sums of the represented values
// (wrapping), reduced across the (half) wave.
template <class S, class T>
__device__ __forceinline__ void enc_limb_a(const EncParams& p, int blk) {
    constexpr int P = S::PLANES;
    constexpr bool SUMS = S::PAD != 0;
    // a wave per row, or half a wave for rows of at most 512 k (so that
    // every lane has 16 elements: smul24 16 x 512^3 encoder 15.2 -> 13.9 us)
    const bool half = p.Kp <= 512;
    const int LW = half ? 32 : 64;
    const int lane = threadIdx.x & (LW - 1);
    const int64_t rowg = half ? (int64_t)blk * (NT / 32) + (threadIdx.x >> 5)
                              : (int64_t)blk * (NT / 64) + (threadIdx.x >> 6);
    if (rowg >= (int64_t)p.batch * p.Mp) return;                     // whole (half) wave
    const int b = (int)(rowg / p.Mp), m = (int)(rowg - (int64_t)b * p.Mp);
    const T* src = (const T*)p.src + b * p.s_src + (int64_t)m * p.ld_src;
    int8_t* dst = (int8_t*)p.dst + b * p.s_dst + (int64_t)m * p.Kp;
    uint32_t sum = 0;
    for (int k0 = lane * 16; k0 < p.Kp; k0 += LW * 16) {
        T x[16];
        bool ok[16];
        if (p.vec && m < p.M && k0 + 16 <= p.K) {
            load_vec<T, 16>(src + k0, x);
#pragma unroll
            for (int e = 0; e < 16; ++e) ok[e] = true;
        } else {
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                ok[e] = m < p.M && k0 + e < p.K;
                x[e] = ok[e] ? src[k0 + e] : (T)0;
            }
        }
        uint32_t w[4][P];
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) sum += pack4<S, T>(x + 4 * g4, ok + 4 * g4, w[g4]);
#pragma unroll
        for (int q = 0; q < P; ++q)
            *(i4*)(dst + (int64_t)q * p.Mp * p.Kp + k0) = i4{(int)w[0][q], (int)w[1][q], (int)w[2][q], (int)w[3][q]};
    }
    if (SUMS) {
        for (int off = LW / 2; off > 0; off >>= 1) sum += __shfl_xor(sum, off, 64);
        if (lane == 0 && m < p.M) p.sums[(int64_t)b * p.M + m] = (int32_t)sum;
    }
}

// B [batch][K][ldb] (T) -> B8T [batch][P][Np][Kp]: a workgroup transposes a
// 64(k) x 64(n) block.  A thread takes four k rows of four columns, packs
// the four k bytes of each column and plane into one dword and stages it in
// LDS; the rows then leave as 16-byte runs along k.  Plain B: a thread's
// columns are consecutive (one 16-byte load per row).  Conv (B gathered
// from the NCHW input, k = (ci*KH + kh)*KW + kw, n = (img*Ho + oh)*Wo + ow):
// a thread's columns are 16 apart so that 16 lanes gather 16 consecutive
// pixels, and the workgroup first tabulates its 64 rows' tap offsets and its
// 64 columns' window origins in LDS, which leaves two adds, a bounds test
// and a load per element.
template <class S, class T>
__device__ __forceinline__ void enc_limb_bt(const EncParams& p, int blk) {
    constexpr int P = S::PLANES, RW = 17;     // LDS row: 16 dwords of k + 1 to spread banks
    constexpr bool SUMS = S::PAD != 0;
    __shared__ uint32_t t[P][64][RW];
    __shared__ uint32_t cpart[SUMS ? 16 : 1][64];
    __shared__ int64_t tab_base[64], tab_off[64];
    __shared__ int32_t tab_ih[64], tab_iw[64], tab_kh[64], tab_kw[64];
    const int nb64 = p.Np / 64, kb64 = p.Kp / 64;
    const int bx = blk % nb64, by = (blk / nb64) % kb64, b = blk / (nb64 * kb64);
    const int n0 = bx * 64, k0 = by * 64;
    const T* src = (const T*)p.src + b * p.s_src;
    const int tid = threadIdx.x, kg = tid >> 4, ng = tid & 15;
    const int kb = k0 + kg * 4;
    T x[4][4];
    bool ok[4][4];
    int col[4];
    if (p.conv) {
        const ConvGeom& g = p.g;
        if (tid < 64) {
            // column n0 + tid: window origin (clamped into N; columns past N are padding)
            const int hw = g.Ho * g.Wo;
            const int n = min(n0 + tid, p.N - 1);
            const int img = n / hw, rem = n - img * hw, oh = rem / g.Wo, ow = rem - oh * g.Wo;
            const int ih0 = oh * g.stride - g.pad, iw0 = ow * g.stride - g.pad;
            tab_base[tid] = ((int64_t)img * g.Ci * g.H + ih0) * g.W + iw0;
            tab_ih[tid] = ih0;
            tab_iw[tid] = iw0;
        } else if (tid < 128) {
            // row k0 + i: tap (ci, kh, kw) (clamped into K; rows past K are padding)
            const int i = tid - 64, k = min(k0 + i, p.K - 1);
            const int kw = k % g.KW, t2 = k / g.KW, kh = t2 % g.KH, ci = t2 / g.KH;
            tab_off[i] = ((int64_t)ci * g.H + kh) * g.W + kw;
            tab_kh[i] = kh;
            tab_kw[i] = kw;
        }
        __syncthreads();
        int64_t cb[4];
        int cih[4], ciw[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            col[c] = ng + 16 * c;
            cb[c] = tab_base[col[c]];
            cih[c] = tab_ih[col[c]];
            ciw[c] = tab_iw[col[c]];
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int i = kg * 4 + r;
            const int64_t off = tab_off[i];
            const int kh = tab_kh[i], kw = tab_kw[i];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                ok[r][c] = kb + r < p.K && n0 + col[c] < p.N;
                const int ih = cih[c] + kh, iw = ciw[c] + kw;
                const bool in = ok[r][c] && (unsigned)ih < (unsigned)g.H && (unsigned)iw < (unsigned)g.W;
                x[r][c] = in ? src[cb[c] + off] : (T)0;   // outside the image: a real zero operand
            }
        }
    } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) col[c] = ng * 4 + c;
        const int nb = n0 + ng * 4;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int k = kb + r;
            const T* row = src + (int64_t)k * p.ld_src + nb;
            if (p.vec && k < p.K && nb + 4 <= p.N) {
                load_vec<T, 4>(row, x[r]);
#pragma unroll
                for (int c = 0; c < 4; ++c) ok[r][c] = true;
            } else {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    ok[r][c] = k < p.K && nb + c < p.N;
                    x[r][c] = ok[r][c] ? row[c] : (T)0;
                }
            }
        }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const T xc[4] = {x[0][c], x[1][c], x[2][c], x[3][c]};
        const bool oc[4] = {ok[0][c], ok[1][c], ok[2][c], ok[3][c]};
        uint32_t w[P];
        const uint32_t cs = pack4<S, T>(xc, oc, w);
#pragma unroll
        for (int q = 0; q < P; ++q) t[q][col[c]][kg] = w[q];
        if (SUMS) cpart[kg][col[c]] = cs;
    }
    __syncthreads();
    // column sums of this 64-k slice: [batch][Kp/64][N]
    if (SUMS && tid < 64 && n0 + tid < p.N) {
        uint32_t cs = 0;
#pragma unroll
        for (int i = 0; i < 16; ++i) cs += cpart[i][tid];
        p.sums[((int64_t)b * kb64 + by) * p.N + n0 + tid] = (int32_t)cs;
    }
    const int nn = tid >> 2, kc = (tid & 3) * 4;
    int8_t* dst = (int8_t*)p.dst + b * p.s_dst + (int64_t)(n0 + nn) * p.Kp + k0 + kc * 4;
#pragma unroll
    for (int q = 0; q < P; ++q) {
        const uint32_t* s4 = &t[q][nn][kc];
        *(i4*)(dst + (int64_t)q * p.Np * p.Kp) = i4{(int)s4[0], (int)s4[1], (int)s4[2], (int)s4[3]};
    }
}

// Both limb encoders in one launch: blocks [0, blocks_a) encode A (four rows
// each), the rest encode 64 x 64 blocks of B^T.
template <class S, class T>
__global__ __launch_bounds__(NT) void k_enc_limb(const EncPairParams p) {
    if ((int)blockIdx.x < p.blocks_a) enc_limb_a<S, T>(p.a, blockIdx.x);
    else enc_limb_bt<S, T>(p.b, blockIdx.x - p.blocks_a);
}

// Implicit lowering of an INT32 convolution onto the int8 limb route
// (smul24 split, C_in a multiple of 64).  blockIdx.y == 0: a block takes
// one bordered image row (n, hp) and 64 of its positions, and for every
// 64-channel chunk stages the chunk's NCHW values in LDS (coalesced along
// W), then writes each position's 64 channels as three 64-byte limb rows
// (8 channels per thread) and the chunk's sum of the represented values at
// that position (positions outside the image hold the value 0).
// blockIdx.y == 1: one wave per output channel writes its weight row in
// (kh, kw, ci) order as limb planes and its row sum.
__global__ __launch_bounds__(NT) void k_conv_prep_limb(const ConvLimbPrepParams p) {
    const ConvGeom& g = p.g;
    const int tid = threadIdx.x;
    if (blockIdx.y == 0) {
        if ((int)blockIdx.x >= p.xblocks) return;
        __shared__ int32_t t[64][65];
        const int Hp = g.H + 2 * g.pad, Wp = g.W + 2 * g.pad;
        const int wch = (Wp + 63) / 64, CC = g.Ci / 64;
        const int n = blockIdx.x / (Hp * wch), rem = blockIdx.x - n * Hp * wch;
        const int hp = rem / wch, wp0 = (rem - hp * wch) * 64;
        const int h = hp - g.pad;
        const bool row_in = h >= 0 && h < g.H;
        const int wl = tid & 63, cq = tid >> 6;
        const int w = wp0 + wl - g.pad;
        const bool in = row_in && w >= 0 && w < g.W;
        const int64_t pos0 = ((int64_t)n * Hp + hp) * Wp;           // position of (n, hp, 0)
        for (int c0 = 0; c0 < g.Ci; c0 += 64) {
            const int32_t* src = p.x + (((int64_t)n * g.Ci + c0) * g.H + h) * g.W + w;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int c = cq + 4 * r;
                t[c][wl] = in ? src[(int64_t)c * g.H * g.W] : 0;
            }
            __syncthreads();
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int q = tid + NT * i, px = q >> 3, cg = q & 7;
                uint32_t u[8];
                uint32_t sum = 0;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    u[e] = (uint32_t)t[cg * 8 + e][px];
                    sum += (uint32_t)SchemeS24::value((int32_t)u[e]);
                }
                uint32_t lo[3], hi[3];
                pack_s24(u[0], u[1], u[2], u[3], lo);
                pack_s24(u[4], u[5], u[6], u[7], hi);
                // the eight threads of one position are eight consecutive lanes
                sum += __shfl_xor(sum, 1, 64);
                sum += __shfl_xor(sum, 2, 64);
                sum += __shfl_xor(sum, 4, 64);
                if (wp0 + px < Wp) {
                    const int64_t pos = pos0 + wp0 + px;
#pragma unroll
                    for (int pl = 0; pl < 3; ++pl) {
                        typedef uint32_t u2v __attribute__((ext_vector_type(2)));
                        *(u2v*)(p.xp8 + pl * p.plane_x + pos * g.Ci + c0 + cg * 8) = u2v{lo[pl], hi[pl]};
                    }
                    if (cg == 0)
                        p.s[(((int64_t)n * CC + c0 / 64) * Hp + hp) * Wp + wp0 + px] = (int32_t)sum;
                }
            }
            __syncthreads();
        }
        return;
    }
    // weights: wave -> output channel; lane -> 16 consecutive k (one tap, 16 channels)
    const int co = (int)blockIdx.x * (NT / 64) + (tid >> 6), lane = tid & 63;
    if ((int)blockIdx.x >= p.wblocks || co >= p.Co) return;   // whole wave
    const int taps = g.KH * g.KW;
    uint32_t sum = 0;
    for (int k0 = lane * 16; k0 < p.Kd; k0 += 64 * 16) {
        const int tap = k0 / g.Ci, ci0 = k0 - tap * g.Ci;
        const int32_t* src = p.w + ((int64_t)co * g.Ci + ci0) * taps + tap;
        uint32_t u[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            u[e] = (uint32_t)src[(int64_t)e * taps];
            sum += (uint32_t)SchemeS24::value((int32_t)u[e]);
        }
        uint32_t d[4][3];
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) pack_s24(u[4 * g4], u[4 * g4 + 1], u[4 * g4 + 2], u[4 * g4 + 3], d[g4]);
#pragma unroll
        for (int pl = 0; pl < 3; ++pl)
            *(i4*)(p.a8 + pl * p.plane_a + (int64_t)co * p.Kd + k0) =
                i4{(int)d[0][pl], (int)d[1][pl], (int)d[2][pl], (int)d[3][pl]};
    }
    for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off, 64);
    if (lane == 0) p.rowsum[co] = (int32_t)sum;
}

// 64-byte LDS rows (64 int8) as four 16-byte chunks; the 16 rows of one
// ds_read_b128 lane group land in distinct banks.
__device__ __forceinline__ int swz_i8(int row) { return (row >> 2) & 3; }

// Wait until at most n K tiles of LPT direct-to-LDS loads each are still in
// flight (s_waitcnt takes an immediate; a count past the 6-bit field waits
// for more, which is still correct).
template <int LPT>
__device__ __forceinline__ void wait_tiles(int n) {
#define QX_WAIT(k)                                                           \
    {                                                                        \
        constexpr int c = (k) * LPT > 63 ? 63 : (k) * LPT;                   \
        __builtin_amdgcn_s_waitcnt((c & 15) | ((c >> 4) << 14) | 0x0F70);   \
    }
    switch (n) {
    case 0: QX_WAIT(0) break;
    case 1: QX_WAIT(1) break;
    case 2: QX_WAIT(2) break;
    case 3: QX_WAIT(3) break;
    default: QX_WAIT(4) break;
    }
#undef QX_WAIT
}

// WAVES / KG = 4: a 2 x 2 grid of waves; 8: 2 (M) x 4 (N), two waves per
// SIMD, which halves a 128 x 128 tile's per-wave accumulators.  KG = 2: two
// such grids take alternate K tiles of the same output tile (two waves per
// SIMD for 64 x 64 tiles), each with its own STAGES-deep ring and its own
// barrier (a counter in LDS), so the two groups run out of step: one
// group's loads and barrier waits overlap the other's matrix products.
// The groups are added through LDS at the end.
template <class S, int BM, int BN, int STAGES, int WAVES, int KG = 1>
__global__ __launch_bounds__(64 * WAVES) void k_gemm_i8nt(const GemmParams p) {
    constexpr int NTH = 64 * WAVES, GW = WAVES / KG, GTH = 64 * GW, WGN = GW / 2;
    constexpr int BK = 64, KCH = 4, P = S::PLANES, G = S::GROUPS;
    constexpr int WM = BM / 2, WN = BN / WGN, TM = WM / 32, TN = WN / 32;
    static_assert(GW == 4 || GW == 8, "wave grid");
    static_assert(KG == 1 || KG == 2, "K groups");
    static_assert(TM >= 1 && TN >= 1, "whole 32 x 32 blocks per wave");
    static_assert(STAGES >= 3 && STAGES <= 6, "ring depth");
    // offset routes: besides its share of the two operand tiles, every wave
    // loads one dword per lane of the K tile's column-sum row (the encoder
    // writes one row of column sums per 64 K), so the column sums add up
    // alongside the K loop for any K; only the first BN/64 waves' values
    // are used
    constexpr bool OFFS = S::PAD != 0;
    // a stage holds the A planes' tile then the B planes' tile, 16-byte
    // chunks; every wave of a group issues LAB of its wave-wide (1 KB) loads
    constexpr int CH_A = P * BM * KCH, CH_B = P * BN * KCH, CH = CH_A + CH_B;
    constexpr int LAB = CH / GTH, LPT = LAB + (OFFS ? 1 : 0);
    static_assert(LAB * GTH == CH && CH_A % 64 == 0, "whole, wave-uniform loads");
    static_assert(BN <= GTH, "one column-sum dword per thread of a group");
    __shared__ i4 Stg[KG][STAGES][CH];
    __shared__ uint32_t cs_ring[OFFS ? KG : 1][OFFS ? STAGES : 1][GTH];
    __shared__ uint32_t rs_l[BM], csum_l[KG][BN];
    __shared__ uint32_t gbar[KG];

    const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hh = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: loop bounds and bases stay scalar
    const int kg = wave / GW, wl = wave % GW, tg = tid % GTH;
    const int wm = wl / WGN, wn = wl % WGN;
    const int tiles_m = (p.M + BM - 1) / BM;
    int pid = blockIdx.x;
    const int total = gridDim.x;
    // consecutive workgroup IDs go to the eight XCDs in turn: give each XCD
    // a contiguous run of tiles (with a folded batch, whole batches), whose
    // operand panels then share that XCD's L2
    if ((total & 7) == 0) pid = (pid & 7) * (total >> 3) + (pid >> 3);
    int b = blockIdx.z;
    if (p.flat_batch) {
        const int tpb = tiles_m * p.tiles_n;
        b = pid / tpb;
        pid -= b * tpb;
    }
    int tm, tn;
    {
        constexpr int GR = 8;
        const int per_group = GR * p.tiles_n;
        const int gid = pid / per_group;
        const int first_m = gid * GR;
        const int gsz = min(tiles_m - first_m, GR);
        const int in = pid - gid * per_group;
        tm = first_m + in % gsz;
        tn = in / gsz;
    }
    const int m0 = tm * BM, n0 = tn * BN;
    // K slices: slice y covers K tiles [y*per, y*per + ktiles); every slice
    // adds its partial products and the column-sum part of the offset
    // correction over its own K tiles into C (cleared beforehand) with
    // wrapping int32 atomics, which is exact mod 2^32 in any order; slice 0
    // also adds the row-sum part and subtracts K c^2
    const int ktiles_all = (p.K + BK - 1) / BK;   // planes are zero-limb padded to whole tiles
    const bool split = p.ksplit > 1;
    int kt0 = 0, ktiles = ktiles_all;
    if (split) {
        const int per = (ktiles_all + p.ksplit - 1) / p.ksplit;
        kt0 = (int)blockIdx.y * per;
        ktiles = min(per, ktiles_all - kt0);
        if (ktiles <= 0) return;   // whole workgroup, before any barrier; never slice 0
    }
    const bool lead = blockIdx.y == 0;
    // planes: A8 [batch][P][Mp][Kp] (sA = P*Mp*Kp, lda = Kp, plane_a = Mp*Kp), B8T likewise
    const char* a_panel = (const char*)p.A + b * p.sA + (int64_t)m0 * p.lda + kt0 * BK;
    // B_NHWC (implicit convolution, one image batch, no K slices): B^T column
    // n is output pixel n, and its K tile t is the 64 channels of chunk t % CC
    // of kernel tap t / CC at that pixel's window in the bordered NHWC limb
    // planes; the pixel's window origin goes into the lane offsets, the tap
    // and chunk into the tile's base
    const bool nhwc = p.b_mode == B_NHWC;
    const ConvGeom& cg = p.g;
    const int Hp = cg.H + 2 * cg.pad, Wp = cg.W + 2 * cg.pad, CC = cg.Ci / 64;
    auto win_origin = [&](int n) {   // (img, oh*stride, ow*stride) of output pixel n, as a bordered position
        const int pix = n < p.N ? n : 0;   // columns past N are never stored
        const int img = pix / p.hw, rem = pix - img * p.hw;
        const int oh = rem / cg.Wo, ow = rem - oh * cg.Wo;
        return ((int64_t)img * CC * Hp + oh * cg.stride) * Wp + ow * cg.stride;   // S index, chunk 0
    };
    auto tile_tap = [&](int t, int64_t& x_off, int64_t& s_off) {   // K tile t's offsets in xp8 (bytes) and s
        const int chunk = t % CC, tap = t / CC, kh = tap / cg.KW, kw = tap - kh * cg.KW;
        x_off = ((int64_t)kh * Wp + kw) * cg.Ci + chunk * 64;
        s_off = ((int64_t)chunk * Hp + kh) * Wp + kw;
    };
    const char* b_panel = nhwc ? (const char*)p.B : (const char*)p.B + b * p.sB + (int64_t)n0 * p.ldb + kt0 * BK;
    const unsigned wave_u = (unsigned)wave, wl_u = (unsigned)wl, kg_u = (unsigned)kg;
    // load k of this wave covers stage chunks (wl + GW*k)*64 + lane
    unsigned ol[LAB];
#pragma unroll
    for (int k = 0; k < LAB; ++k) {
        const int q = (wl + GW * k) * 64 + lane;
        if (q < CH_A) {
            const int plane = q / (BM * KCH), rem = q % (BM * KCH), row = rem / KCH, pc = rem % KCH;
            ol[k] = (unsigned)((int64_t)plane * p.plane_a + row * p.lda + (pc ^ swz_i8(row)) * 16);
        } else {
            const int qb = q - CH_A;
            const int plane = qb / (BN * KCH), rem = qb % (BN * KCH), row = rem / KCH, pc = rem % KCH;
            if (nhwc) {
                // window origin of pixel n0 + row in the NHWC planes: its S
                // index with the image's chunk stride taken out
                const int pix = n0 + row < p.N ? n0 + row : 0;
                const int img = pix / p.hw, prem = pix - img * p.hw;
                const int oh = prem / cg.Wo, ow = prem - oh * cg.Wo;
                const int64_t pos = ((int64_t)img * Hp + oh * cg.stride) * Wp + ow * cg.stride;
                ol[k] = (unsigned)((int64_t)plane * p.plane_b + pos * cg.Ci + (pc ^ swz_i8(row)) * 16);
            } else {
                ol[k] = (unsigned)((int64_t)plane * p.plane_b + row * p.ldb + (pc ^ swz_i8(row)) * 16);
            }
        }
    }
    const unsigned lds_s0 = (unsigned)(uintptr_t)&Stg[0][0][0] + kg_u * (unsigned)(STAGES * CH * 16);
    // column sums [batch][K/64][N]: this thread's column, clamped into N
    // (columns past N are never stored)
    const int32_t* csg = !OFFS ? nullptr : nhwc ? p.colsum : p.colsum + ((int64_t)b * p.cs_slices + kt0) * p.N;
    const unsigned cs_off = (unsigned)(nhwc ? win_origin(n0 + tg) : (int64_t)min(n0 + tg, p.N - 1)) * 4u;
    const unsigned lds_cs0 = (unsigned)(uintptr_t)&cs_ring[0][0][0] + (OFFS ? kg_u * (STAGES * GTH * 4) : 0u) + wl_u * 256;
    // this group's local tile u is K tile KG*u + kg, in slot u % STAGES
    auto issue = [&](int u) {
        const int s = u % STAGES, t = KG * u + (int)kg_u;
        const char* ab = a_panel + t * BK;
        int64_t x_off = 0, s_off = 0;
        if (nhwc) tile_tap(t, x_off, s_off);
        const char* bb = nhwc ? b_panel + x_off : b_panel + t * BK;
        const unsigned ls = lds_s0 + (unsigned)(s * CH * 16);
#pragma unroll
        for (int k = 0; k < LAB; ++k) {
            const unsigned blk = wl_u + GW * k;
            const char* base = (int)blk * 64 < CH_A ? ab : bb;
            asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                         :: "v"(ol[k]), "s"(base), "s"(ls + blk * 1024) : "memory", "m0");
        }
        if constexpr (OFFS)
            asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1"
                         :: "v"(cs_off), "s"(nhwc ? csg + s_off : csg + (int64_t)t * p.N), "s"(lds_cs0 + s * GTH * 4)
                         : "memory", "m0");
    };
    // barrier of this group's waves: all of them have waited for their part
    // of the current tile and have finished reading the slot about to be
    // refilled.  KG = 2: a counter in LDS (the group's waves are resident
    // together, so the wait ends); the data a wave's loads put in LDS has
    // landed before its vmcnt wait ends, hence before its increment
    uint32_t gen = 0;
    auto group_barrier = [&]() {
        if constexpr (KG == 1) {
            __syncthreads();
        } else {
            gen += GW;
            __builtin_amdgcn_s_waitcnt(0xC07F);          // lgkmcnt(0): this wave's LDS reads are done
            if (lane == 0) __hip_atomic_fetch_add(&gbar[kg], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            while (__hip_atomic_load(&gbar[kg], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) < gen)
                __builtin_amdgcn_s_sleep(1);
            asm volatile("" ::: "memory");
        }
    };

    i16x acc[G][TM][TN];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[g][i][j] = i16x{};

    if (OFFS && lead) {
        // the tile's row sums, one 4-byte direct-to-LDS load per lane ahead
        // of the first K tile; rows past M re-read the last valid one (they
        // are never stored)
        const int32_t* rsg = p.rowsum + (int64_t)b * p.M;
        for (int I = (int)wave_u; I < BM / 64; I += NTH / 64) {
            const unsigned off = (unsigned)min(m0 + I * 64 + lane, p.M - 1) * 4u;
            const unsigned lds = (unsigned)(uintptr_t)&rs_l[I * 64];
            asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1"
                         :: "v"(off), "s"(rsg), "s"(lds) : "memory", "m0");
        }
    }
    if (KG > 1 && tid < KG) gbar[tid] = 0;
    if constexpr (KG > 1) __syncthreads();
    uint32_t csum_acc = 0;   // this thread's column sum over its group's K tiles
    const int nloc = (ktiles - kg + KG - 1) / KG;   // this group's K tiles
#pragma unroll
    for (int u = 0; u < STAGES - 1; ++u)
        if (u < nloc) issue(u);
    for (int u = 0; u < nloc; ++u) {
        // local tile u must have landed; the ones after it may still be in
        // flight (and the sums, issued before tile 0, have landed with it)
        wait_tiles<LPT>(min(STAGES - 2, nloc - 1 - u));
        group_barrier();
        const int s = u % STAGES;
        if (OFFS && tg < BN) csum_acc += cs_ring[OFFS ? kg : 0][s][tg];   // before the slot is refilled
        // the slot of local tile u-1 is free: every wave of the group is
        // past the barrier, so done with it
        if (u + STAGES - 1 < nloc) issue(u + STAGES - 1);
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            const int c = ks * 2 + hh;
            i4 a[P][TM], bv[P][TN];
#pragma unroll
            for (int q = 0; q < P; ++q) {
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    const int row = wm * WM + i * 32 + l32;
                    a[q][i] = Stg[kg][s][(q * BM + row) * KCH + (c ^ swz_i8(row))];
                }
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const int col = wn * WN + j * 32 + l32;
                    bv[q][j] = Stg[kg][s][CH_A + (q * BN + col) * KCH + (c ^ swz_i8(col))];
                }
            }
#pragma unroll
            for (int pr = 0; pr < S::PRODUCTS; ++pr)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[S::pg[pr]][i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(
                            a[S::pa[pr]][i], bv[S::pb[pr]][j], acc[S::pg[pr]][i][j], 0, 0, 0);
        }
    }

    // limb groups recombined per output (wrapping int32: the sum of the K
    // groups' combinations is the combination of their sums)
    uint32_t vs[TM][TN][16];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                uint32_t gv[G];
#pragma unroll
                for (int q = 0; q < G; ++q) gv[q] = (uint32_t)acc[q][i][j][r];
                vs[i][j][r] = S::combine(gv);
            }
    if (OFFS && tg < BN) csum_l[kg][tg] = csum_acc;
    if constexpr (KG == 2) {
        // group 1 hands its sums to group 0 through the (drained) stage ring
        static_assert(GW * TM * TN * 16 * 64 * 4 <= (int)sizeof(Stg), "exchange fits the ring");
        uint32_t* xch = (uint32_t*)&Stg[0][0][0] + wl * (TM * TN * 16 * 64);
        __syncthreads();
        if (kg == 1) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) xch[((i * TN + j) * 16 + r) * 64 + lane] = vs[i][j][r];
        }
        __syncthreads();
        if (kg == 1) return;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) vs[i][j][r] += xch[((i * TN + j) * 16 + r) * 64 + lane];
    } else if (OFFS) {
        __syncthreads();
    }
    int32_t* C = (int32_t*)p.C + b * p.sC;
    const uint32_t cc = (uint32_t)p.corr_c;
    const uint32_t kcc = (uint32_t)p.K * cc * cc;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int gn = n0 + wn * WN + j * 32 + l32;
        if (gn >= p.N) continue;
        const uint32_t ccol = OFFS ? cc * (KG == 2 ? csum_l[0][wn * WN + j * 32 + l32] + csum_l[KG - 1][wn * WN + j * 32 + l32]
                                               : csum_l[0][wn * WN + j * 32 + l32]) : 0u;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int lr = wm * WM + i * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
                const int gm = m0 + lr;
                if (gm >= p.M) continue;
                uint32_t v = vs[i][j][r];
                if (OFFS) {
                    v += ccol;
                    if (lead) v += cc * rs_l[lr] - kcc;
                }
                // non-temporal: the output is not re-read by this launch and
                // kept out of L2 it does not evict other workgroups' operand
                // tiles (16 x 512^3: 27.0 -> 24.8 us, INT32 conv 30.2 -> 28.6)
                if (split) atomicAdd((uint32_t*)C + c_index(p, gm, gn), v);
                else __builtin_nontemporal_store(p.relu ? max((int32_t)v, 0) : (int32_t)v, &C[c_index(p, gm, gn)]);
            }
    }
}

// ===========================================================================
// Row / column sums for the rank-1 correction of offset limb routes.
// ===========================================================================
// Row sums of A (blockIdx.y == 0: one wave per row, lanes stride along the
// contiguous K) and per-slice column sums of B (blockIdx.y == 1: a block
// covers 64 columns x SUM_SLICE rows, 4 row groups of 64 threads coalesced
// along the row, reduced in LDS).  Column partials go to colsum[b][slice][N];
// consumers add the slices, so no atomics and no clearing are needed.
constexpr int SUM_SLICE = 64;

__global__ __launch_bounds__(NT) void k_sums(const SumsParams p) {
    __shared__ uint32_t part[4][64];
    const int b = blockIdx.z;
    if (blockIdx.y == 1) {
        if (p.N <= 0) return;
        const int ncb = (p.N + 63) / 64;
        const int cb = blockIdx.x % ncb, slice = blockIdx.x / ncb;
        const int k0 = slice * SUM_SLICE;
        if (k0 >= p.K) return;                      // whole block: uniform exit
        const int c = threadIdx.x & 63, g = threadIdx.x >> 6;
        const int col = cb * 64 + c;
        const int k1 = min(k0 + SUM_SLICE, p.K);
        uint32_t s = 0;
        if (col < p.N) {
            if (p.s24) {
                const int32_t* bb = (const int32_t*)p.B + b * p.sB + col;
                for (int k = k0 + g; k < k1; k += 4)
                    s += (uint32_t)((int32_t)((uint32_t)bb[(int64_t)k * p.ldb] << 8) >> 8);
            } else {
                const int16_t* bb = (const int16_t*)p.B + b * p.sB + col;
                for (int k = k0 + g; k < k1; k += 4) s += (uint32_t)(int32_t)bb[(int64_t)k * p.ldb];
            }
        }
        part[g][c] = s;
        __syncthreads();
        if (g == 0 && col < p.N) {
            const int slices = (p.K + SUM_SLICE - 1) / SUM_SLICE;
            p.colsum[((int64_t)b * slices + slice) * p.N + col] =
                (int32_t)(part[0][c] + part[1][c] + part[2][c] + part[3][c]);
        }
        return;
    }
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (row >= p.M) return;
    uint32_t s = 0;
    if (p.s24) {
        const int32_t* a = (const int32_t*)p.A + b * p.sA + (int64_t)row * p.lda;
        for (int k = lane; k < p.K; k += 64) s += (uint32_t)((int32_t)((uint32_t)a[k] << 8) >> 8);
    } else {
        const int16_t* a = (const int16_t*)p.A + b * p.sA + (int64_t)row * p.lda;
        for (int k = lane; k < p.K; k += 64) s += (uint32_t)(int32_t)a[k];
    }
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0) p.rowsum[(int64_t)b * p.M + row] = (int32_t)s;
}

// ===========================================================================
// Explicit im2col (Methodology: convolution through lowering).
// ===========================================================================
template <class T>
__global__ __launch_bounds__(NT) void k_im2col(const Im2colParams p) {
    const int64_t pix = (int64_t)blockIdx.x * NT + threadIdx.x;
    const int k = blockIdx.y;
    if (pix >= p.P) return;
    const ConvGeom& g = p.g;
    const int kw = k % g.KW, kh = (k / g.KW) % g.KH, ci = k / (g.KW * g.KH);
    const int hw = g.Ho * g.Wo;
    const int n = (int)(pix / hw), rem = (int)(pix - (int64_t)n * hw);
    const int oh = rem / g.Wo, ow = rem - oh * g.Wo;
    const int ih = oh * g.stride - g.pad + kh, iw = ow * g.stride - g.pad + kw;
    T v = (T)0;
    if (ih >= 0 && ih < g.H && iw >= 0 && iw < g.W)
        v = ((const T*)p.x)[(((int64_t)n * g.Ci + ci) * g.H + ih) * g.W + iw];
    ((T*)p.col)[(int64_t)k * p.P + pix] = v;
}

// Fill of 32-bit words: a grid-stride loop, so any count fits the capped grid.
__global__ __launch_bounds__(NT) void k_fill(const FillParams p) {
    const int64_t stride = (int64_t)gridDim.x * NT;
    for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < p.n32; i += stride)
        ((int32_t*)p.ptr)[i] = p.value;
}

// Range scan: a grid-stride pass; a wave with any lane out of range sets the
// flag once (vector atomic).
__global__ __launch_bounds__(NT) void k_range(const RangeParams p) {
    const int64_t stride = (int64_t)gridDim.x * NT;
    bool bad = false;
    for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < p.n; i += stride) {
        const int64_t v = p.elem_bytes == 2 ? (int64_t)((const int16_t*)p.x)[i] : (int64_t)((const int32_t*)p.x)[i];
        bad |= v > p.bound || v < -(int64_t)p.bound;
    }
    if (__any(bad) && (threadIdx.x & 63) == __builtin_ctzll(__ballot(bad))) atomicOr(p.flag, p.bit);
}

// ===========================================================================
// Builders
// ===========================================================================
template <class K>
static void fill_gemm_rec(LaunchRec* rec, K* fn, const GemmParams& p0, int BM, int BN, int batch,
                          const char* name) {
    GemmParams p = p0;
    const int tiles_m = (p.M + BM - 1) / BM;
    p.tiles_n = (p.N + BN - 1) / BN;
    rec->fn = (const void*)fn;
    rec->grid = dim3((unsigned)(tiles_m * p.tiles_n), 1, (unsigned)batch);
    rec->block = dim3(NT, 1, 1);
    rec->shmem = 0;
    rec->name = name;
    rec->set_params(p);
}

// Vector loads need 16-byte aligned rows and batch strides, and whole
// vectors inside K (A vectors of 8) and N (B vectors of bvec); pointers are
// bound per run and the executor checks their alignment there.
static bool aligned_for(const GemmParams& p, int elem, int bvec) {
    const int v = 16 / elem;
    return p.lda % v == 0 && p.ldb % v == 0 && p.sA % v == 0 && p.sB % v == 0 &&
           p.K % 8 == 0 && p.N % bvec == 0 && p.b_mode == B_KN;
}

bool build_gemm_mfma(int32_t route, const GemmParams& p, int batch, LaunchRec* rec,
                     int* tile_m, int* tile_n, int* tile_k) {
    *tile_k = 64;
    switch (route) {
    case R_F16_EXACT: {
        const bool al = aligned_for(p, 2, 8);
        const bool step = p.chunk_tiles == 0;  // chunk of 16: flush after every MFMA step
        // fewer than 64 tiles of 128 x 128: 64 x 64 tiles give 4x the workgroups
        const int64_t tiles128 = (int64_t)((p.M + 127) / 128) * ((p.N + 127) / 128) * batch;
        if (tiles128 < 64) {
            *tile_m = 64;
            *tile_n = 64;
            // K within four tiles: 32 x 32 tiles, K split over the four waves
            if (p.K <= 4 * 64) {
                *tile_m = 32;
                *tile_n = 32;
                if (al && !step) fill_gemm_rec(rec, k_gemm_f16_ks<true, false>, p, 32, 32, batch, "gemm_f16_ksplit");
                else if (al) fill_gemm_rec(rec, k_gemm_f16_ks<true, true>, p, 32, 32, batch, "gemm_f16_ksplit_step");
                else if (!step) fill_gemm_rec(rec, k_gemm_f16_ks<false, false>, p, 32, 32, batch, "gemm_f16_ksplit_u");
                else fill_gemm_rec(rec, k_gemm_f16_ks<false, true>, p, 32, 32, batch, "gemm_f16_ksplit_step_u");
                return true;
            }
            if (al && !step) fill_gemm_rec(rec, k_gemm_f16x<64, 64, 64, 32, 32, true, false>, p, 64, 64, batch, "gemm_f16x_64");
            else if (al) fill_gemm_rec(rec, k_gemm_f16x<64, 64, 64, 32, 32, true, true>, p, 64, 64, batch, "gemm_f16x_step_64");
            else if (!step) fill_gemm_rec(rec, k_gemm_f16x<64, 64, 64, 32, 32, false, false>, p, 64, 64, batch, "gemm_f16x_u_64");
            else fill_gemm_rec(rec, k_gemm_f16x<64, 64, 64, 32, 32, false, true>, p, 64, 64, batch, "gemm_f16x_step_u_64");
            return true;
        }
        *tile_m = 128;
        *tile_n = 128;
        if (al && !step) fill_gemm_rec(rec, k_gemm_f16x<128, 128, 64, 64, 64, true, false>, p, 128, 128, batch, "gemm_f16x");
        else if (al) fill_gemm_rec(rec, k_gemm_f16x<128, 128, 64, 64, 64, true, true>, p, 128, 128, batch, "gemm_f16x_step");
        else if (!step) fill_gemm_rec(rec, k_gemm_f16x<128, 128, 64, 64, 64, false, false>, p, 128, 128, batch, "gemm_f16x_u");
        else fill_gemm_rec(rec, k_gemm_f16x<128, 128, 64, 64, 64, false, true>, p, 128, 128, batch, "gemm_f16x_step_u");
        return true;
    }
    case R_I8_DIRECT:
    case R_I8_KARATSUBA:
    case R_I8_OFFSET4: {
        *tile_m = 128;
        *tile_n = 128;
        const bool al = aligned_for(p, 2, 8);
#define QX_I8(S, NAME)                                                                                       \
    if (al) fill_gemm_rec(rec, k_gemm_i8limb<S, int16_t, 128, 128, 64, 64, true>, p, 128, 128, batch, NAME);  \
    else fill_gemm_rec(rec, k_gemm_i8limb<S, int16_t, 128, 128, 64, 64, false>, p, 128, 128, batch, NAME "_u");
        if (route == R_I8_DIRECT) { QX_I8(SchemeDirect, "gemm_i8_direct") }
        else if (route == R_I8_KARATSUBA) { QX_I8(SchemeKaratsuba, "gemm_i8_karatsuba") }
        else { QX_I8(SchemeOffset4, "gemm_i8_offset4") }
#undef QX_I8
        return true;
    }
    case R_S24_I8LIMB: {
        *tile_m = 128;
        *tile_n = 64;
        const bool al = aligned_for(p, 4, 4);
        if (al) fill_gemm_rec(rec, k_gemm_i8limb<SchemeS24, int32_t, 128, 64, 64, 32, true>, p, 128, 64, batch, "gemm_s24_i8limb");
        else fill_gemm_rec(rec, k_gemm_i8limb<SchemeS24, int32_t, 128, 64, 64, 32, false>, p, 128, 64, batch, "gemm_s24_i8limb_u");
        return true;
    }
    default:
        return false;
    }
}

// int8 NT route: 128x128 workgroup tiles (four 64x64 waves) when they fill
// the chip, else 64x64 (four 32x32 waves).
void i8nt_tile_shape(int32_t route, int64_t M, int64_t N, int64_t batch, int* bm, int* bn) {
    // 128x128 tiles (eight waves, two per SIMD, 64x32 each) move half the
    // operand bytes per product of 64x64 tiles; they take over once there
    // are 128 of them
    (void)route;
    const int64_t big = ((M + 127) / 128) * ((N + 127) / 128) * batch;
    *bm = *bn = big >= 128 ? 128 : 64;
}

template <class S>
static void enc_limb_rec(bool s24, const EncPairParams& p0, LaunchRec* rec, const char* name) {
    EncPairParams p = p0;
    const int rows_per_block = p.a.Kp <= 512 ? NT / 32 : NT / 64;   // half a wave or a wave per row
    p.blocks_a = (int32_t)(((int64_t)p.a.batch * p.a.Mp + rows_per_block - 1) / rows_per_block);
    const int64_t blocks_b = (int64_t)(p.b.Np / 64) * (p.b.Kp / 64) * p.b.batch;
    rec->fn = s24 ? (const void*)k_enc_limb<S, int32_t> : (const void*)k_enc_limb<S, int16_t>;
    rec->grid = dim3((unsigned)(p.blocks_a + blocks_b), 1, 1);
    rec->block = dim3(NT, 1, 1);
    rec->shmem = 0;
    rec->name = name;
    rec->set_params(p);
}

void build_enc_limb(int32_t route, bool s24, const EncPairParams& p, LaunchRec* rec) {
    switch (route) {
    case R_I8_DIRECT: enc_limb_rec<SchemeDirect>(s24, p, rec, "enc_limb_direct"); break;
    case R_I8_KARATSUBA: enc_limb_rec<SchemeKaratsuba>(s24, p, rec, "enc_limb_karatsuba"); break;
    case R_I8_OFFSET4: enc_limb_rec<SchemeOffset4>(s24, p, rec, "enc_limb_offset4"); break;
    default: enc_limb_rec<SchemeS24>(s24, p, rec, "enc_limb_s24"); break;
    }
}

void build_conv_prep_limb(const ConvLimbPrepParams& p0, LaunchRec* rec) {
    ConvLimbPrepParams p = p0;
    const ConvGeom& g = p.g;
    const int Hp = g.H + 2 * g.pad, Wp = g.W + 2 * g.pad;
    p.xblocks = p.nimg * Hp * ((Wp + 63) / 64);
    p.wblocks = (p.Co + NT / 64 - 1) / (NT / 64);
    rec->fn = (const void*)k_conv_prep_limb;
    rec->grid = dim3((unsigned)std::max(p.xblocks, p.wblocks), 2, 1);
    rec->block = dim3(NT, 1, 1);
    rec->name = "conv_prep_limb_s24";
    rec->set_params(p);
}

bool build_gemm_i8nt(int32_t route, const GemmParams& p0, int batch, LaunchRec* rec) {
    int bm, bn;
    i8nt_tile_shape(route, p0.M, p0.N, batch, &bm, &bn);
    const bool big = bm == 128;
    // 64x64 tiles: a 6-deep ring (one workgroup per CU) while the grid,
    // K slices included, fits the chip in one round, else 3 deep (two per CU)
    const bool deep = (int64_t)((p0.M + 63) / 64) * ((p0.N + 63) / 64) * batch * std::max(p0.ksplit, 1) <= 256;
#define QX_NT(S, NAME)                                                                               \
    if (big) fill_gemm_rec(rec, k_gemm_i8nt<S, 128, 128, 3, 8>, p0, 128, 128, batch, "gemm_i8nt_" NAME "_128x128"); \
    else if (deep) fill_gemm_rec(rec, k_gemm_i8nt<S, 64, 64, 3, 8, 2>, p0, 64, 64, batch, "gemm_i8nt_" NAME "_64x64"); \
    else fill_gemm_rec(rec, k_gemm_i8nt<S, 64, 64, 3, 4>, p0, 64, 64, batch, "gemm_i8nt_" NAME "_64x64_3");
    switch (route) {
    case R_I8_DIRECT: QX_NT(SchemeDirect, "direct") break;
    case R_I8_KARATSUBA: QX_NT(SchemeKaratsuba, "karatsuba") break;
    case R_I8_OFFSET4: QX_NT(SchemeOffset4, "offset4") break;
    case R_S24_I8LIMB: QX_NT(SchemeS24, "s24") break;
    default: return false;
    }
#undef QX_NT
    if (big || deep) rec->block = dim3(512, 1, 1);
    if (p0.ksplit > 1) rec->grid.y = (unsigned)p0.ksplit;
    if (batch > 1 && (int64_t)rec->grid.x * batch < ((int64_t)1 << 31)) {
        GemmParams p = *(const GemmParams*)rec->blob;
        p.flat_batch = 1;
        rec->set_params(p);
        rec->grid.x *= (unsigned)batch;
        rec->grid.z = 1;
    }
    return true;
}

int sums_slices(int K) { return std::max((K + SUM_SLICE - 1) / SUM_SLICE, 1); }

void build_sums(const SumsParams& p, LaunchRec* rec) {
    const int row_blocks = (p.M + 3) / 4;
    const int col_blocks = ((p.N + 63) / 64) * sums_slices(p.K);
    rec->fn = (const void*)k_sums;
    rec->grid = dim3((unsigned)std::max(std::max(row_blocks, col_blocks), 1), 2, (unsigned)p.batch);
    rec->block = dim3(NT, 1, 1);
    rec->name = "rowcol_sums";
    rec->set_params(p);
}

void build_im2col(const Im2colParams& p, LaunchRec* rec) {
    rec->fn = p.elem_bytes == 4 ? (const void*)k_im2col<uint32_t> : (const void*)k_im2col<uint16_t>;
    rec->grid = dim3((unsigned)((p.P + NT - 1) / NT), (unsigned)p.Kd, 1);
    rec->block = dim3(NT, 1, 1);
    rec->name = "im2col";
    rec->set_params(p);
}

void build_range(const RangeParams& p, LaunchRec* rec) {
    const int64_t blocks = std::min<int64_t>((p.n + NT - 1) / NT, 2048);
    rec->fn = (const void*)k_range;
    rec->grid = dim3((unsigned)std::max<int64_t>(blocks, 1), 1, 1);
    rec->block = dim3(NT, 1, 1);
    rec->shmem = 0;
    rec->name = "range_check";
    rec->set_params(p);
}

void build_fill(const FillParams& p, LaunchRec* rec) {
    rec->fn = (const void*)k_fill;
    rec->grid = dim3((unsigned)std::min<int64_t>(std::max<int64_t>((p.n32 + NT - 1) / NT, 1), kFillMaxBlocks), 1, 1);
    rec->block = dim3(NT, 1, 1);
    rec->name = "fill";
    rec->set_params(p);
}

}  // namespace qx
