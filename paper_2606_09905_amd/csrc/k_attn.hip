// k_attn.hip -- the single-head attention core O = (Q K^T) V on matrix cores
// (Methodology: attention operator of the form O = (Q K^T) V; Table 2,
// attention rows).  No scale, softmax or mask.
//
// Both kernels keep S on chip.  A wave owns 32 queries; per block of 32 keys
// it forms S^T = K_blk Q^T with one MFMA chain, whose 32x32 accumulator
// (lane = query, 16 registers = 16 keys) is exactly the A operand layout of
// the second product O += S V once the V operand is gathered with the same
// key permutation (the order of a contraction's terms is free).  Keys are
// split across workgroups; partial results are combined in a fixed order.
//
//  * FP32: v_mfma_f32_32x32x2f32 for both products; per-split partials are
//    reduced in split order, so repeated runs are bit-identical.
//  * INT32 (|q|,|k|,|v| <= 127 and d*max^2 < 2^23): S^T on
//    v_mfma_i32_32x32x32_i8; every S is read as three offset int8 limbs,
//    S = s0 + 2^8 s1 + 2^16 s2 + 32896, where the limbs are the bytes of
//    S xor 0x8080; O gets three int8 products mod 2^32 plus 32896 * colsum(V).
//    Integer partials from different splits are added with atomics (exact
//    and order-independent mod 2^32).
#include "qx_internal.h"

namespace qx {

typedef float f16x __attribute__((ext_vector_type(16)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef int i16x __attribute__((ext_vector_type(16)));
typedef int i4 __attribute__((ext_vector_type(4)));

constexpr int AT = 256;      // 4 waves
constexpr int AQW = 32;      // queries per wave
constexpr int AQ = 4 * AQW;  // queries per workgroup
constexpr int AKB = 32;      // keys per block

// ---------------------------------------------------------------------------
// FP32
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(AT) void k_attn_f32(const AttnParams p) {
    constexpr int DP = D + 4;            // padded LDS row (floats)
    constexpr int HALF = D / 2;          // K-slot h of a 32x32x2 MFMA covers d-half h
    constexpr int NTO = D / 32;          // output column tiles
    constexpr int LD4 = AKB * D / 4 / AT;  // float4 loads per thread per operand
    __shared__ float Ks[AKB][DP];
    __shared__ float Vs[AKB][DP];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, l32 = lane & 31;
    const int q0 = blockIdx.x * AQ + wave * AQW;
    const int split = blockIdx.y;
    const int key_lo = split * p.keys_per_split;
    const int key_hi = min(p.L, key_lo + p.keys_per_split);
    const float* Q = (const float*)p.Q;
    const float* Kp = (const float*)p.K;
    const float* Vp = (const float*)p.V;

    float qf[HALF];
    {
        const int q = q0 + l32;
#pragma unroll
        for (int t = 0; t < HALF; t += 4) {
            f4 v = (q < p.L) ? *(const f4*)(Q + (int64_t)q * D + HALF * h + t) : f4{};
            qf[t] = v[0]; qf[t + 1] = v[1]; qf[t + 2] = v[2]; qf[t + 3] = v[3];
        }
    }
    f16x o[NTO];
#pragma unroll
    for (int n = 0; n < NTO; ++n) o[n] = f16x{};

    f4 rk[LD4], rv[LD4];
    auto load = [&](int kb) {
#pragma unroll
        for (int i = 0; i < LD4; ++i) {
            const int v = tid + AT * i, row = v / (D / 4), c4 = v % (D / 4);
            const int key = kb + row;
            const bool in = key < key_hi;
            rk[i] = in ? *(const f4*)(Kp + (int64_t)key * D + c4 * 4) : f4{};
            rv[i] = in ? *(const f4*)(Vp + (int64_t)key * D + c4 * 4) : f4{};
        }
    };
    auto stash = [&]() {
#pragma unroll
        for (int i = 0; i < LD4; ++i) {
            const int v = tid + AT * i, row = v / (D / 4), c4 = v % (D / 4);
            *(f4*)&Ks[row][c4 * 4] = rk[i];
            *(f4*)&Vs[row][c4 * 4] = rv[i];
        }
    };

    if (key_lo < key_hi) load(key_lo);
    for (int kb = key_lo; kb < key_hi; kb += AKB) {
        __syncthreads();              // previous block fully consumed
        stash();
        __syncthreads();
        if (kb + AKB < key_hi) load(kb + AKB);
        // S^T[key][query] = sum_t K[key][t] Q[query][t]
        f16x s = f16x{};
#pragma unroll
        for (int t = 0; t < HALF; t += 4) {
            const f4 kv = *(const f4*)&Ks[l32][HALF * h + t];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                s = __builtin_amdgcn_mfma_f32_32x32x2f32(kv[e], qf[t + e], s, 0, 0, 0);
        }
        // O[query][c] += sum_key S[query][key] V[key][c]; register r of lane
        // half h holds key 8*(r/4) + 4*h + r%4.
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int key = 8 * (r >> 2) + 4 * h + (r & 3);
#pragma unroll
            for (int n = 0; n < NTO; ++n)
                o[n] = __builtin_amdgcn_mfma_f32_32x32x2f32(s[r], Vs[key][n * 32 + l32], o[n], 0, 0, 0);
        }
    }

    float* dst = p.splits > 1 ? (float*)p.part + (int64_t)split * p.L * D : (float*)p.O;
#pragma unroll
    for (int n = 0; n < NTO; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int q = q0 + 8 * (r >> 2) + 4 * h + (r & 3);
            if (q < p.L) dst[(int64_t)q * D + n * 32 + l32] = o[n][r];
        }
}

__global__ __launch_bounds__(AT) void k_reduce_splits(const ReduceParams p) {
    const int64_t i = (int64_t)blockIdx.x * AT + threadIdx.x;
    if (i >= p.n) return;
    float s = p.part[i];
    for (int k = 1; k < p.splits; ++k) s += p.part[(int64_t)k * p.n + i];
    p.out[i] = s;
}

// ---------------------------------------------------------------------------
// INT32 through int8 matrix cores
// ---------------------------------------------------------------------------
// Byte j of four words, packed into one word (a, b, c, d -> bytes 0..3).
__device__ __forceinline__ uint32_t gather_byte(uint32_t a, uint32_t b, uint32_t c, uint32_t d, int j) {
    const uint32_t sel = (uint32_t)j | ((uint32_t)(4 + j) << 8) | (0x0C0Cu << 16);
    const uint32_t lo = __builtin_amdgcn_perm(b, a, sel);   // (a_j, b_j, 0, 0)
    const uint32_t hi = __builtin_amdgcn_perm(d, c, sel);   // (c_j, d_j, 0, 0)
    return __builtin_amdgcn_perm(hi, lo, 0x05040100u);      // (a_j, b_j, c_j, d_j)
}

template <int D>
__global__ __launch_bounds__(AT) void k_attn_i32(const AttnParams p) {
    constexpr int NTO = D / 32;
    constexpr int KCH = D / 16;                 // 16-byte chunks per key row (int8)
    constexpr int KW = AKB * D / 4 / AT;        // packed K words per thread
    __shared__ i4 Ks8[AKB][KCH];                // int8 K rows
    __shared__ uint32_t Vt8[D][AKB / 4 + 1];    // int8 V^T: [column][keys], padded

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, l32 = lane & 31;
    const int q0 = blockIdx.x * AQ + wave * AQW;
    const int split = blockIdx.y;
    const int key_lo = split * p.keys_per_split;
    const int key_hi = min(p.L, key_lo + p.keys_per_split);
    const int32_t* Q = (const int32_t*)p.Q;
    const int32_t* Kp = (const int32_t*)p.K;
    const int32_t* Vp = (const int32_t*)p.V;

    auto pack4 = [](i4 v) -> uint32_t {
        return ((uint32_t)v[0] & 0xFFu) | (((uint32_t)v[1] & 0xFFu) << 8) |
               (((uint32_t)v[2] & 0xFFu) << 16) | ((uint32_t)v[3] << 24);
    };
    // Q fragment: lane (query, half h), MFMA t: Q[query][32t + 16h + e], e < 16.
    i4 qf[NTO];
    {
        const int q = q0 + l32;
#pragma unroll
        for (int t = 0; t < NTO; ++t) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const i4 v = (q < p.L) ? *(const i4*)(Q + (int64_t)q * D + 32 * t + 16 * h + 4 * w) : i4{};
                qf[t][w] = (int)pack4(v);
            }
        }
    }
    i16x o[3][NTO];
#pragma unroll
    for (int j = 0; j < 3; ++j)
#pragma unroll
        for (int n = 0; n < NTO; ++n) o[j][n] = i16x{};

    // Column sums of V over this split's keys, for the offset correction.
    __shared__ uint32_t vsum[D];
    if (tid < D) vsum[tid] = 0u;
    __syncthreads();
    uint32_t vpart[KW];
#pragma unroll
    for (int i = 0; i < KW; ++i) vpart[i] = 0u;

    uint32_t rk[KW], rv[KW];
    auto load = [&](int kb) {
#pragma unroll
        for (int i = 0; i < KW; ++i) {
            const int v = tid + AT * i;
            // K: word v covers key v/(D/4), columns 4*(v%(D/4)) .. +3
            const int krow = v / (D / 4), kc = v % (D / 4);
            const int key = kb + krow;
            rk[i] = key < key_hi ? pack4(*(const i4*)(Kp + (int64_t)key * D + kc * 4)) : 0u;
            // V^T: word v covers column v % D, keys 4*(v / D) .. +3
            const int col = v % D, kq = v / D;
            uint32_t w = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int key2 = kb + kq * 4 + e;
                const uint32_t x = key2 < key_hi ? (uint32_t)Vp[(int64_t)key2 * D + col] : 0u;
                w |= (x & 0xFFu) << (8 * e);
                vpart[i] += x;
            }
            rv[i] = w;
        }
    };
    auto stash = [&]() {
#pragma unroll
        for (int i = 0; i < KW; ++i) {
            const int v = tid + AT * i;
            const int krow = v / (D / 4), kc = v % (D / 4);
            ((uint32_t*)&Ks8[krow][0])[kc] = rk[i];
            Vt8[v % D][v / D] = rv[i];
        }
    };

    if (key_lo < key_hi) load(key_lo);
    for (int kb = key_lo; kb < key_hi; kb += AKB) {
        __syncthreads();
        stash();
        __syncthreads();
        if (kb + AKB < key_hi) load(kb + AKB);
        i16x s = i16x{};
#pragma unroll
        for (int t = 0; t < NTO; ++t)
            s = __builtin_amdgcn_mfma_i32_32x32x32_i8(Ks8[l32][2 * t + h], qf[t], s, 0, 0, 0);
        // Offset limbs: bytes 0..2 of S ^ 0x8080.  K-slot (h, e) of the
        // second product is key 8*(e/4) + 4*h + e%4, as the S^T layout gives.
        uint32_t x[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) x[r] = (uint32_t)s[r] ^ 0x8080u;
        i4 limb[3];
#pragma unroll
        for (int j = 0; j < 3; ++j)
#pragma unroll
            for (int w = 0; w < 4; ++w)
                limb[j][w] = (int)gather_byte(x[4 * w], x[4 * w + 1], x[4 * w + 2], x[4 * w + 3], j);
#pragma unroll
        for (int n = 0; n < NTO; ++n) {
            i4 vb;
#pragma unroll
            for (int w = 0; w < 4; ++w) vb[w] = (int)Vt8[n * 32 + l32][2 * w + h];
#pragma unroll
            for (int j = 0; j < 3; ++j)
                o[j][n] = __builtin_amdgcn_mfma_i32_32x32x32_i8(limb[j], vb, o[j][n], 0, 0, 0);
        }
    }

#pragma unroll
    for (int i = 0; i < KW; ++i) atomicAdd(&vsum[(tid + AT * i) % D], vpart[i]);
    __syncthreads();

    int32_t* O = (int32_t*)p.O;
#pragma unroll
    for (int n = 0; n < NTO; ++n) {
        const int c = n * 32 + l32;
        // every split adds 32896 * sum over its own keys of V[key][c]
        const uint32_t corr = 32896u * vsum[c];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int q = q0 + 8 * (r >> 2) + 4 * h + (r & 3);
            if (q >= p.L) continue;
            const uint32_t v = (uint32_t)o[0][n][r] + ((uint32_t)o[1][n][r] << 8) +
                               ((uint32_t)o[2][n][r] << 16) + corr;
            if (p.splits > 1) atomicAdd(O + (int64_t)q * D + c, (int)v);
            else O[(int64_t)q * D + c] = (int32_t)v;
        }
    }
}

// ---------------------------------------------------------------------------
// INT32 with resident key splits.  A prep launch writes int8 copies of K
// (rows) and V^T (rows of keys, each 32-key block reordered as in the V
// operand gather below) into the workspace and clears O; then each workgroup
// loads its whole key split -- kps keys of K8 and of V8 -- into LDS with
// direct-to-LDS loads in one batch, and runs every key block from LDS with
// no further global loads or barriers.  The S^T tile and the limb split are
// those of k_attn_i32.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(AT) void k_attn_i32_prep(const AttnParams p) {
    const int64_t i = (int64_t)blockIdx.x * AT + threadIdx.x;
    const int32_t* Kp = (const int32_t*)p.K;
    const int32_t* Vp = (const int32_t*)p.V;
    auto pack4 = [](i4 v) -> uint32_t {
        return ((uint32_t)v[0] & 0xFFu) | (((uint32_t)v[1] & 0xFFu) << 8) |
               (((uint32_t)v[2] & 0xFFu) << 16) | ((uint32_t)v[3] << 24);
    };
    if (i < p.prep_k) {
        // 16 consecutive d of one key row
        const int key = (int)(i / (D / 16)), c0 = (int)(i % (D / 16)) * 16;
        i4 o = i4{};
        if (key < p.L) {
#pragma unroll
            for (int w = 0; w < 4; ++w) o[w] = (int)pack4(*(const i4*)(Kp + (int64_t)key * D + c0 + 4 * w));
        }
        *(i4*)((int8_t*)p.k8 + (int64_t)key * D + c0) = o;
        return;
    }
    const int64_t iv = i - p.prep_k;
    if (iv < p.prep_v) {
        // column c, half-block hb (16 keys): byte 4w + e holds key
        // 32*(hb/2) + 8w + 4*(hb%2) + e
        const int c = (int)(iv % D);
        const int hb = (int)(iv / D);
        const int kb = (hb >> 1) * 32 + 4 * (hb & 1);
        i4 o;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            uint32_t x = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int key = kb + 8 * w + e;
                const uint32_t v = key < p.L ? (uint32_t)Vp[(int64_t)key * D + c] : 0u;
                x |= (v & 0xFFu) << (8 * e);
            }
            o[w] = (int)x;
        }
        int8_t* dst = p.v_blocks ? (int8_t*)p.v8 + ((int64_t)(hb >> 1) * D + c) * 32 + 16 * (hb & 1)
                                 : (int8_t*)p.v8 + (int64_t)c * p.Lp + 16 * (int64_t)hb;
        *(i4*)dst = o;
        return;
    }
    const int64_t iq = iv - p.prep_v;
    if (iq < p.prep_q) {
        // 16 consecutive d of one query row
        const int q = (int)(iq / (D / 16)), c0 = (int)(iq % (D / 16)) * 16;
        const int32_t* Qp = (const int32_t*)p.Q;
        i4 o;
#pragma unroll
        for (int w = 0; w < 4; ++w) o[w] = (int)pack4(*(const i4*)(Qp + (int64_t)q * D + c0 + 4 * w));
        *(i4*)((int8_t*)p.q8 + (int64_t)q * D + c0) = o;
        return;
    }
    const int64_t io = iq - p.prep_q;
    if (p.clear_o && io < (int64_t)p.L * D / 4) ((i4*)p.O)[io] = i4{};
}

// chunk swizzles of the resident tiles: K rows of D bytes (16 lanes of one
// ds_read_b128 read 16 rows at one chunk: spread them over the 64 banks), and
// V rows of kps bytes (swizzle within the largest power-of-two group of
// chunks that divides the row, at most 16)
template <int D>
__device__ __forceinline__ int swz_k(int row) { return (row / (256 / D)) & (D / 16 - 1); }
__device__ __forceinline__ int swz_v(int row, int vmask) { return row & vmask; }

template <int D>
__global__ __launch_bounds__(AT) void k_attn_i32r(const AttnParams p) {
    constexpr int NTO = D / 32;
    constexpr int CK = D / 16;                   // 16-byte chunks per K row
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int kps = p.keys_per_split;
    char* Ks = smem;                             // [kps][D] int8
    char* Vs = smem + (int64_t)kps * D;          // [D][kps] int8
    __shared__ uint32_t vsum[D];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, l32 = lane & 31;
    const int q0 = blockIdx.x * AQ + wave * AQW;
    const int split = blockIdx.y;
    const int key_lo = split * kps;
    const int CV = kps / 16;                     // 16-byte chunks per V row
    const int vmask = min(CV & -CV, 16) - 1;
    const unsigned wave_u = __builtin_amdgcn_readfirstlane(wave);

    // the split's K8 rows and V8 columns, 1 KB per wave instruction
    {
        const char* k8 = (const char*)p.k8 + (int64_t)key_lo * D;
        const char* v8 = (const char*)p.v8 + key_lo;
        const unsigned lds_k = (unsigned)(uintptr_t)Ks, lds_v = (unsigned)(uintptr_t)Vs;
        const int nk = kps * D / 1024, nv = D * kps / 1024;
        for (int I = (int)wave_u; I < nk; I += 4) {
            const int q = I * 64 + lane, row = q / CK, pos = q % CK;
            const unsigned off = (unsigned)(row * D + ((pos ^ swz_k<D>(row)) * 16));
            asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                         :: "v"(off), "s"(k8), "s"(lds_k + I * 1024) : "memory", "m0");
        }
        for (int I = (int)wave_u; I < nv; I += 4) {
            const int q = I * 64 + lane, row = q / CV, pos = q % CV;
            const unsigned off = (unsigned)(row * p.Lp + ((pos ^ swz_v(row, vmask)) * 16));
            asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                         :: "v"(off), "s"(v8), "s"(lds_v + I * 1024) : "memory", "m0");
        }
    }
    const int32_t* Q = (const int32_t*)p.Q;
    auto pack4 = [](i4 v) -> uint32_t {
        return ((uint32_t)v[0] & 0xFFu) | (((uint32_t)v[1] & 0xFFu) << 8) |
               (((uint32_t)v[2] & 0xFFu) << 16) | ((uint32_t)v[3] << 24);
    };
    i4 qf[NTO];
    {
        const int q = q0 + l32;
#pragma unroll
        for (int t = 0; t < NTO; ++t) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const i4 v = (q < p.L) ? *(const i4*)(Q + (int64_t)q * D + 32 * t + 16 * h + 4 * w) : i4{};
                qf[t][w] = (int)pack4(v);
            }
        }
    }
    if (tid < D) vsum[tid] = 0u;
    __builtin_amdgcn_s_waitcnt(0x0070);          // vmcnt(0), lgkmcnt(0): the tiles have landed
    __syncthreads();
    // column sums of V over the split's keys (padding keys are zero)
    {
        constexpr int TPR = AT / D;              // threads per V row
        const int row = tid / TPR, part = tid % TPR;
        const uint32_t* vr = (const uint32_t*)(Vs + (int64_t)row * kps);
        // thread `part` sums words [part*per, (part+1)*per), visited in an
        // order rotated by the row so that lanes on different rows (whose
        // rows start in the same bank) read different banks
        const int per = kps / 4 / TPR;
        int acc = 0;
        for (int i = 0; i < per; ++i)
            acc = __builtin_amdgcn_sdot4((int)vr[part * per + (i + row) % per], 0x01010101, acc, false);
        atomicAdd(&vsum[row], (uint32_t)acc);
    }

    i16x o[3][NTO];
#pragma unroll
    for (int j = 0; j < 3; ++j)
#pragma unroll
        for (int n = 0; n < NTO; ++n) o[j][n] = i16x{};
    for (int blk = 0; blk < kps / 32; ++blk) {
        const int krow = blk * 32 + l32;
        i16x s = i16x{};
#pragma unroll
        for (int t = 0; t < NTO; ++t) {
            const i4 kf = *(const i4*)(Ks + (int64_t)krow * D + (((2 * t + h) ^ swz_k<D>(krow)) * 16));
            s = __builtin_amdgcn_mfma_i32_32x32x32_i8(kf, qf[t], s, 0, 0, 0);
        }
        uint32_t x[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) x[r] = (uint32_t)s[r] ^ 0x8080u;
        i4 limb[3];
#pragma unroll
        for (int jj = 0; jj < 3; ++jj)
#pragma unroll
            for (int w = 0; w < 4; ++w)
                limb[jj][w] = (int)gather_byte(x[4 * w], x[4 * w + 1], x[4 * w + 2], x[4 * w + 3], jj);
#pragma unroll
        for (int n = 0; n < NTO; ++n) {
            const int vrow = n * 32 + l32;
            const i4 vb = *(const i4*)(Vs + (int64_t)vrow * kps + (((2 * blk + h) ^ swz_v(vrow, vmask)) * 16));
#pragma unroll
            for (int jj = 0; jj < 3; ++jj)
                o[jj][n] = __builtin_amdgcn_mfma_i32_32x32x32_i8(limb[jj], vb, o[jj][n], 0, 0, 0);
        }
    }
    __syncthreads();                             // vsum complete

    int32_t* O = (int32_t*)p.O;
#pragma unroll
    for (int n = 0; n < NTO; ++n) {
        const int c = n * 32 + l32;
        const uint32_t corr = 32896u * vsum[c];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int q = q0 + 8 * (r >> 2) + 4 * h + (r & 3);
            if (q >= p.L) continue;
            const uint32_t v = (uint32_t)o[0][n][r] + ((uint32_t)o[1][n][r] << 8) +
                               ((uint32_t)o[2][n][r] << 16) + corr;
            if (p.splits > 1) atomicAdd(O + (int64_t)q * D + c, (int)v);
            else O[(int64_t)q * D + c] = (int32_t)v;
        }
    }
}

// ---------------------------------------------------------------------------
// INT32, streaming.  A workgroup of eight waves takes QT query tiles of 32
// queries and one key split, cut into KQ = 8 / QT key parts: wave w holds
// query tile w % QT over key part w / QT.  Per 32-key block: S^T on the int8
// matrix cores, the offset limb split of S, three limb products into O, and
// the block's V column sums (for the offset correction) from the same V
// registers.  The KQ partial outputs of a query tile are added through LDS,
// each wave adding a slice of the tile, and one wrapping int32 atomic per
// output joins the key splits (exact mod 2^32 in any order).
// ---------------------------------------------------------------------------
template <int D, int QT>
struct AttnStream {
    static constexpr int NTO = D / 32;
    static constexpr int KQ = 8 / QT;                    // key parts
    static constexpr int BLK = 2 * NTO * 1024;           // bytes of one block's K and V
    static constexpr int PER_PAIR = 4 * NTO;             // 1 KB loads per pair of blocks
    static constexpr int PW = PER_PAIR / QT;             // of them issued by each wave
    static constexpr int R0 = (128 * 1024) / (KQ * 2 * BLK);
    static constexpr int R = R0 > 8 ? 8 : R0;            // ring depth in pairs
    static_assert(PER_PAIR % QT == 0 && R >= 2 && (R & (R - 1)) == 0, "ring geometry");
    static_assert(PW * (R - 2) < 64, "loads in flight fit the vmcnt counter");
    static constexpr int KEYS = 64 * KQ;                 // keys_per_split is a multiple of this
};

// s_waitcnt vmcnt(N) (expcnt and lgkmcnt left alone), N in [0, 63]
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// wait until at most STEP * n of this wave's vector memory loads are in flight,
// n in [0, NMAX] (the immediate is a constant: dispatch on n)
template <int STEP, int NMAX>
__device__ __forceinline__ void wait_vmcnt_steps(int n) {
    if constexpr (NMAX <= 0) {
        wait_vmcnt<0>();
    } else {
        if (n >= NMAX) wait_vmcnt<STEP * NMAX>();
        else wait_vmcnt_steps<STEP, NMAX - 1>(n);
    }
}

template <int D, int QT>
__global__ __launch_bounds__(512) void k_attn_i32s(const AttnParams p) {
    using G = AttnStream<D, QT>;
    constexpr int NTO = G::NTO, KQ = G::KQ, BLK = G::BLK, PW = G::PW, R = G::R;
    // per key part a ring of R pairs of blocks; after the loop the ring
    // carries the partial outputs between the waves of a query tile
    __shared__ __attribute__((aligned(16))) char ring[KQ][R][2][BLK];
    __shared__ __attribute__((aligned(16))) char qs[8][NTO * 1024];

    const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: block addresses stay scalar
    const int qw = wave % QT, kp = wave / QT;
    const int q0 = blockIdx.x * (32 * QT) + qw * 32;
    const int kps = p.keys_per_split;            // a multiple of G::KEYS
    const int npair = kps / G::KEYS;             // pairs of 32-key blocks per key part
    const int blk0 = (int)(((int64_t)blockIdx.y * kps + (int64_t)kp * (kps / KQ)) / 32);
    const char* K8 = (const char*)p.k8;          // [Lp][D]
    const char* V8 = (const char*)p.v8;          // [Lp/32][D][32]

    // The QT waves of a key part stage its blocks in the part's ring with
    // direct-to-LDS loads, R-1 pairs ahead, each wave PW of the 1 KB loads
    // of every pair.  A lane's 16 bytes land where the MFMA operand layout
    // reads them (lane (key | column l32, half h): K row chunk 2t + h, V 16
    // keys of column n*32 + l32), which is the same for every query tile,
    // so the ring reads are contiguous.
    const unsigned koff = (unsigned)(l32 * D + h * 16), voff = (unsigned)(l32 * 32 + h * 16);
    auto issue = [&](int pr) {
        const unsigned lds = (unsigned)(uintptr_t)&ring[kp][pr & (R - 1)][0][0];
#pragma unroll
        for (int u = 0; u < PW; ++u) {
            const int l = qw * PW + u;                           // 0 .. PER_PAIR-1
            const int e = l / (2 * NTO), part = l % (2 * NTO);   // block of the pair, 1 KB part
            const int64_t bg = blk0 + 2 * pr + e;
            const unsigned dst = lds + (unsigned)(e * BLK + part * 1024);
            if (part < NTO) {
                const char* kb = K8 + bg * 32 * D;
                asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                             :: "v"(koff + part * 32), "s"(kb), "s"(dst) : "memory", "m0");
            } else {
                const char* vb = V8 + bg * D * 32;
                asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                             :: "v"(voff + (part - NTO) * 1024), "s"(vb), "s"(dst) : "memory", "m0");
            }
        }
    };
    // this wave's Q rows as int8 (written by the prep launch), staged the
    // same way ahead of the key blocks: lane (query l32, half h), MFMA t
    // reads Q[query][32t + 16h + e]; rows past L repeat the last row
    {
        const int qr = min(q0, p.L - 1);         // a tile past L (last workgroup) reads row L-1
        const char* qb = (const char*)p.q8 + (int64_t)qr * D;
        const unsigned qoff = (unsigned)((min(q0 + l32, p.L - 1) - qr) * D + 16 * h);
        const unsigned dst = (unsigned)(uintptr_t)&qs[wave][0];
#pragma unroll
        for (int t = 0; t < NTO; ++t)
            asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                         :: "v"(qoff + 32 * t), "s"(qb), "s"(dst + t * 1024) : "memory", "m0");
    }
    for (int pr = 0; pr < R - 1 && pr < npair; ++pr) issue(pr);

    i16x o[3][NTO];
#pragma unroll
    for (int j = 0; j < 3; ++j)
#pragma unroll
        for (int n = 0; n < NTO; ++n) o[j][n] = i16x{};
    int vs[NTO];                                 // V column n*32 + l32, keys of half h
#pragma unroll
    for (int n = 0; n < NTO; ++n) vs[n] = 0;
    i4 qf[NTO];

    // the offset limbs of S (bytes of S ^ 0x8080, read as int8): K-slot
    // (h, e) of the second product is key 8*(e/4) + 4*h + e%4, as the S^T
    // accumulator layout gives.  Per four elements a, b, c, d a byte
    // transpose: (a0 b0 a1 b1), (c0 d0 c1 d1), (a2 b2 - -), (c2 d2 - -), then
    // limb j = (a_j b_j c_j d_j); the XOR with 0x80 of bytes 0 and 1 is done
    // on the transposed words.
    auto limbs = [](const i16x& s, i4 (&limb)[3]) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const uint32_t a = (uint32_t)s[4 * w], b = (uint32_t)s[4 * w + 1];
            const uint32_t c = (uint32_t)s[4 * w + 2], d = (uint32_t)s[4 * w + 3];
            const uint32_t ab01 = __builtin_amdgcn_perm(b, a, 0x05010400u);
            const uint32_t cd01 = __builtin_amdgcn_perm(d, c, 0x05010400u);
            const uint32_t ab2 = __builtin_amdgcn_perm(b, a, 0x0C0C0602u);
            const uint32_t cd2 = __builtin_amdgcn_perm(d, c, 0x0C0C0602u);
            limb[0][w] = (int)(__builtin_amdgcn_perm(cd01, ab01, 0x05040100u) ^ 0x80808080u);
            limb[1][w] = (int)(__builtin_amdgcn_perm(cd01, ab01, 0x07060302u) ^ 0x80808080u);
            limb[2][w] = (int)__builtin_amdgcn_perm(cd2, ab2, 0x05040100u);
        }
    };
    // Software pipeline: the second block's limb products of pair pr run at
    // the start of pair pr+1, beside its S^T chains and first limb split
    // (zero limbs stand in before the first pair: they add nothing).
    i4 lp[3] = {i4{}, i4{}, i4{}};
    i4 vp[NTO];
#pragma unroll
    for (int n = 0; n < NTO; ++n) vp[n] = i4{};
    for (int pr = 0; pr < npair; ++pr) {
        // this wave's loads of pair pr (and, before them, its Q rows) have
        // landed once no more than those of the later pairs are in flight
        wait_vmcnt_steps<PW, R - 2>(npair - 1 - pr);
        __syncthreads();                         // every part landed; slot of pair pr-1 read by all
        if (pr + R - 1 < npair) issue(pr + R - 1);
        if (pr == 0) {
#pragma unroll
            for (int t = 0; t < NTO; ++t) qf[t] = *(const i4*)(&qs[wave][t * 1024 + lane * 16]);
        }
        const char* st0 = &ring[kp][pr & (R - 1)][0][0];
        const char* st1 = &ring[kp][pr & (R - 1)][1][0];
        i4 kf0[NTO], kf1[NTO], vf0[NTO], vf1[NTO];
#pragma unroll
        for (int t = 0; t < NTO; ++t) {
            kf0[t] = *(const i4*)(st0 + t * 1024 + lane * 16);
            kf1[t] = *(const i4*)(st1 + t * 1024 + lane * 16);
        }
#pragma unroll
        for (int n = 0; n < NTO; ++n) {
            vf0[n] = *(const i4*)(st0 + (NTO + n) * 1024 + lane * 16);
            vf1[n] = *(const i4*)(st1 + (NTO + n) * 1024 + lane * 16);
        }
        // both S^T chains first (pinned: left alone, the scheduler ran the
        // second chain after the first block's products, so every limb split
        // waited on its own chain)
        i16x s0 = i16x{}, s1 = i16x{};
#pragma unroll
        for (int t = 0; t < NTO; ++t) {
            s0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(kf0[t], qf[t], s0, 0, 0, 0);
            s1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(kf1[t], qf[t], s1, 0, 0, 0);
        }
        asm volatile("" : "+v"(s1));
        __builtin_amdgcn_sched_barrier(0);
        // the previous pair's second-block products beside this pair's first
        // limb split
        i4 l0[3], l1[3];
#pragma unroll
        for (int n = 0; n < NTO; ++n)
#pragma unroll
            for (int jj = 0; jj < 3; ++jj)
                o[jj][n] = __builtin_amdgcn_mfma_i32_32x32x32_i8(lp[jj], vp[n], o[jj][n], 0, 0, 0);
        limbs(s0, l0);
#pragma unroll
        for (int g = 0; g < 3 * NTO; ++g) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 36 / (3 * NTO), 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        // the first block's products beside the second block's limb split
#pragma unroll
        for (int n = 0; n < NTO; ++n)
#pragma unroll
            for (int jj = 0; jj < 3; ++jj)
                o[jj][n] = __builtin_amdgcn_mfma_i32_32x32x32_i8(l0[jj], vf0[n], o[jj][n], 0, 0, 0);
        limbs(s1, l1);
#pragma unroll
        for (int g = 0; g < 3 * NTO; ++g) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
            __builtin_amdgcn_sched_group_barrier(0x002, 36 / (3 * NTO), 1);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int n = 0; n < NTO; ++n)
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                vs[n] = __builtin_amdgcn_sdot4(vf0[n][w], 0x01010101, vs[n], false);
                vs[n] = __builtin_amdgcn_sdot4(vf1[n][w], 0x01010101, vs[n], false);
            }
#pragma unroll
        for (int jj = 0; jj < 3; ++jj) lp[jj] = l1[jj];
#pragma unroll
        for (int n = 0; n < NTO; ++n) vp[n] = vf1[n];
    }
#pragma unroll
    for (int n = 0; n < NTO; ++n)
#pragma unroll
        for (int jj = 0; jj < 3; ++jj)
            o[jj][n] = __builtin_amdgcn_mfma_i32_32x32x32_i8(lp[jj], vp[n], o[jj][n], 0, 0, 0);

    // recombine the limbs and add the offset correction of this wave's keys
    uint32_t v[NTO][16];
#pragma unroll
    for (int n = 0; n < NTO; ++n) {
        const uint32_t cs = (uint32_t)(vs[n] + __shfl_xor(vs[n], 32, 64));
        const uint32_t corr = 32896u * cs;
#pragma unroll
        for (int r = 0; r < 16; ++r)
            v[n][r] = (uint32_t)o[0][n][r] + ((uint32_t)o[1][n][r] << 8) + ((uint32_t)o[2][n][r] << 16) + corr;
    }
    // the partial outputs of the KQ key parts, [QT][KQ][32][D], through the
    // ring once every wave is done reading it
    uint32_t* red = (uint32_t*)&ring[0][0][0][0];
    static_assert(8 * 32 * D * 4 <= (int)sizeof(ring), "partial outputs fit the ring");
    __syncthreads();
    {
        uint32_t* mine = red + (qw * KQ + kp) * (32 * D);
#pragma unroll
        for (int n = 0; n < NTO; ++n)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                mine[(8 * (r >> 2) + 4 * h + (r & 3)) * D + n * 32 + l32] = v[n][r];
    }
    __syncthreads();
    // wave (qw, kp) adds slice kp of query tile qw: 64 consecutive outputs
    // (row-major, query by column) per step, one atomic per output
    constexpr int PERW = 32 * D / 64 / KQ;
    const uint32_t* tile = red + qw * KQ * (32 * D);
    int32_t* dst = (int32_t*)p.O;
#pragma unroll
    for (int i = 0; i < PERW; ++i) {
        const int e = (kp * PERW + i) * 64 + lane;
        uint32_t t = 0;
#pragma unroll
        for (int k = 0; k < KQ; ++k) t += tile[k * 32 * D + e];
        const int q = q0 + e / D, c = e % D;
        if (q >= p.L) continue;
        // splits add into the output cleared by the prep launch:
        // wrapping int32 atomics, exact mod 2^32 in any order
        if (p.splits > 1) atomicAdd(dst + (int64_t)q * D + c, (int)t);
        else dst[(int64_t)q * D + c] = (int32_t)t;
    }
}

// ---------------------------------------------------------------------------
// Softmax attention, FP32, BH heads (the SDPA-with-softmax form of the
// attention baseline, Table 2 footnote; the attention core with a softmax,
// Discussion).  Same S^T = K_blk Q^T layout as k_attn_f32: lane (query l32,
// half h) holds 16 of the 32 scores of its query in a key block.  Per block
// the running maximum m (base-2 exponent domain, t = scale*log2(e)*s) and the
// running sum are updated online; the exponentials are the A operand of
// O += P V, and O's rows (registers, not lanes) are rescaled by the factor of
// their query, fetched from the lane that owns it.  With key splits every
// split writes unnormalised O, its maximum and its sum; k_sdpa_combine merges
// them in split order, so repeated runs are bit-identical.
// RAG: d < D, columns d..D-1 read as zeros and are not written.
// ---------------------------------------------------------------------------
template <int D, bool RAG>
__global__ __launch_bounds__(AT) void k_sdpa_f32(const SdpaParams p) {
    constexpr int DP = D + 4;
    constexpr int HALF = D / 2;
    constexpr int NTO = D / 32;
    constexpr int LD4 = AKB * D / 4 / AT;
    // two LDS buffers: block j is staged into buffer j&1 while the other
    // holds block j-1, so one barrier per block suffices
    __shared__ float Ksb[2][AKB][DP];
    __shared__ float Vsb[2][AKB][DP];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, l32 = lane & 31;
    // Under the mask a query block's work grows with its index: the dispatch
    // order (x fastest, then z) hands out the longest blocks of every head
    // first, so that the short ones fill in behind them.
    int qblk = blockIdx.x;
    int64_t head = blockIdx.z;
    if (p.causal) {
        const int id = (int)blockIdx.x + (int)gridDim.x * (int)blockIdx.z;
        qblk = (int)gridDim.x - 1 - id / (int)gridDim.z;
        head = id % (int)gridDim.z;
    }
    const int qb = qblk * AQ;
    const int q0 = qb + wave * AQW;
    const int split = blockIdx.y;
    const int d = RAG ? p.d : D;
    const int key_lo = split * p.keys_per_split;
    int key_hi = min(p.L, key_lo + p.keys_per_split);
    if (p.causal) key_hi = min(key_hi, qb + AQ);
    const int64_t hoff = head * p.L * d;
    const float* Q = p.Q + hoff;
    const float* Kp = p.K + hoff;
    const float* Vp = p.V + hoff;

    auto ld4 = [&](const float* base, int row, int c4) -> f4 {
        if (!RAG) return *(const f4*)(base + (int64_t)row * D + c4 * 4);
        f4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int col = c4 * 4 + e;
            v[e] = col < d ? base[(int64_t)row * d + col] : 0.f;
        }
        return v;
    };

    const int q = q0 + l32;           // this lane's query in the S^T layout
    // Q is taken pre-multiplied by c = scale*log2(e), so the scores come out
    // of the MFMAs already in the base-2 exponent domain.
    const float c = p.c;
    float qf[HALF];
#pragma unroll
    for (int t = 0; t < HALF; t += 4) {
        const f4 v = q < p.L ? ld4(Q, q, (HALF * h + t) / 4) : f4{};
        qf[t] = v[0] * c; qf[t + 1] = v[1] * c; qf[t + 2] = v[2] * c; qf[t + 3] = v[3] * c;
    }
    f16x o[NTO];
#pragma unroll
    for (int n = 0; n < NTO; ++n) o[n] = f16x{};
    float m = -INFINITY;              // running maximum of t for query q
    float lsum = 0.f;                 // this half's share of the running sum

    f4 rk[LD4], rv[LD4];
    auto load = [&](int kb) {
#pragma unroll
        for (int i = 0; i < LD4; ++i) {
            const int v = tid + AT * i, row = v / (D / 4), c4 = v % (D / 4);
            const int key = kb + row;
            const bool in = key < key_hi;
            rk[i] = in ? ld4(Kp, key, c4) : f4{};
            rv[i] = in ? ld4(Vp, key, c4) : f4{};
        }
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int i = 0; i < LD4; ++i) {
            const int v = tid + AT * i, row = v / (D / 4), c4 = v % (D / 4);
            *(f4*)&Ksb[buf][row][c4 * 4] = rk[i];
            *(f4*)&Vsb[buf][row][c4 * 4] = rv[i];
        }
    };

    if (key_lo < key_hi) load(key_lo);
    int buf = 0;
    for (int kb = key_lo; kb < key_hi; kb += AKB, buf ^= 1) {
        // Buffer buf was last read two blocks ago: every wave finished that
        // block before the previous iteration's barrier.
        stash(buf);
        __syncthreads();
        if (kb + AKB < key_hi) load(kb + AKB);
        float (&Ks)[AKB][DP] = Ksb[buf];
        float (&Vs)[AKB][DP] = Vsb[buf];
        if (p.causal && kb > q0 + AQW - 1) continue;   // every key after every query of this wave
        f16x s = f16x{};
#pragma unroll
        for (int t = 0; t < HALF; t += 4) {
            const f4 kv = *(const f4*)&Ks[l32][HALF * h + t];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                s = __builtin_amdgcn_mfma_f32_32x32x2f32(kv[e], qf[t + e], s, 0, 0, 0);
        }
        // Register r holds key kb + 8*(r/4) + 4*h + r%4.  In a block that
        // reaches past key_hi or (causal) past a query of this wave, keys at
        // or past key_lim are set to -inf, whose exponential is 0.
        if (kb + AKB > key_hi || (p.causal && kb + AKB - 1 > q0)) {
            const int key_lim = p.causal ? min(key_hi, q + 1) : key_hi;
            const int kl = key_lim - kb - 4 * h;    // register r is kept iff 8*(r/4) + r%4 < kl
#pragma unroll
            for (int r = 0; r < 16; ++r)
                if (8 * (r >> 2) + (r & 3) >= kl) s[r] = -INFINITY;
        }
        float mx = fmaxf(fmaxf(s[0], s[1]), s[2]);
#pragma unroll
        for (int r = 3; r < 15; r += 2) mx = fmaxf(fmaxf(mx, s[r]), s[r + 1]);
        mx = fmaxf(mx, s[15]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m, mx);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        // v_exp_f32 directly: arguments are <= 0 here, results below 2^-126
        // flush to 0, which no sum of a row with its maximum term 1 can see
        const float alpha = __builtin_amdgcn_exp2f(m - m_use);
        m = m_new;
        float ps = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            s[r] = __builtin_amdgcn_exp2f(s[r] - m_use);
            ps += s[r];
        }
        lsum = lsum * alpha + ps;
        if (__ballot(alpha != 1.f) != 0) {
            // row r of O is query 8*(r/4) + 4*h + r%4, whose factor lane that index holds
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float a = __shfl(alpha, 8 * (r >> 2) + 4 * h + (r & 3));
#pragma unroll
                for (int n = 0; n < NTO; ++n) o[n][r] *= a;
            }
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int key = 8 * (r >> 2) + 4 * h + (r & 3);
#pragma unroll
            for (int n = 0; n < NTO; ++n)
                o[n] = __builtin_amdgcn_mfma_f32_32x32x2f32(s[r], Vs[key][n * 32 + l32], o[n], 0, 0, 0);
        }
    }

    const float l = lsum + __shfl_xor(lsum, 32);
    const int64_t rows = (int64_t)p.BH * p.L;
    if (p.splits > 1) {
        float* part = p.part + ((int64_t)split * rows + head * p.L) * d;
#pragma unroll
        for (int n = 0; n < NTO; ++n)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int qr = q0 + 8 * (r >> 2) + 4 * h + (r & 3), col = n * 32 + l32;
                if (qr < p.L && (!RAG || col < d)) part[(int64_t)qr * d + col] = o[n][r];
            }
        if (h == 0 && q < p.L) {
            float* st = p.stat + ((int64_t)split * rows + head * p.L + q) * 2;
            st[0] = m;
            st[1] = l;
        }
    } else {
        const float inv = l > 0.f ? 1.f / l : 0.f;
        float* O = p.O + hoff;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int qi = 8 * (r >> 2) + 4 * h + (r & 3);
            const float f = __shfl(inv, qi);
            const int qr = q0 + qi;
#pragma unroll
            for (int n = 0; n < NTO; ++n) {
                const int col = n * 32 + l32;
                if (qr < p.L && (!RAG || col < d)) O[(int64_t)qr * d + col] = o[n][r] * f;
            }
        }
    }
}

// Merge of the key splits, one thread per output element, splits in order:
// O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s with M = max_s m_s.
__global__ __launch_bounds__(AT) void k_sdpa_combine(const SdpaCombineParams p) {
    const int64_t i = (int64_t)blockIdx.x * AT + threadIdx.x;
    if (i >= p.rows * p.d) return;
    const int64_t row = i / p.d;
    float M = -INFINITY;
    for (int s = 0; s < p.splits; ++s) M = fmaxf(M, p.stat[((int64_t)s * p.rows + row) * 2]);
    float num = 0.f, den = 0.f;
    for (int s = 0; s < p.splits; ++s) {
        const float* st = p.stat + ((int64_t)s * p.rows + row) * 2;
        const float w = exp2f(st[0] - M);
        num += w * p.part[(int64_t)s * p.rows * p.d + i];
        den += w * st[1];
    }
    p.O[i] = num / den;
}

// ---------------------------------------------------------------------------
// Builders
// ---------------------------------------------------------------------------
bool build_attn_f32(const AttnParams& p, LaunchRec* rec) {
    switch (p.d) {
    case 32: rec->fn = (const void*)k_attn_f32<32>; break;
    case 64: rec->fn = (const void*)k_attn_f32<64>; break;
    case 96: rec->fn = (const void*)k_attn_f32<96>; break;
    case 128: rec->fn = (const void*)k_attn_f32<128>; break;
    default: return false;
    }
    rec->name = "attn_f32";
    rec->grid = dim3((unsigned)((p.L + AQ - 1) / AQ), (unsigned)p.splits, 1);
    rec->block = dim3(AT, 1, 1);
    rec->set_params(p);
    return true;
}

bool build_attn_i32(const AttnParams& p, LaunchRec* rec) {
    switch (p.d) {
    case 32: rec->fn = (const void*)k_attn_i32<32>; break;
    case 64: rec->fn = (const void*)k_attn_i32<64>; break;
    case 96: rec->fn = (const void*)k_attn_i32<96>; break;
    case 128: rec->fn = (const void*)k_attn_i32<128>; break;
    default: return false;
    }
    rec->name = "attn_i32";
    rec->grid = dim3((unsigned)((p.L + AQ - 1) / AQ), (unsigned)p.splits, 1);
    rec->block = dim3(AT, 1, 1);
    rec->set_params(p);
    return true;
}

bool resident_attn_i32(int64_t d, int64_t kps) {
    return (d == 32 || d == 64 || d == 128) && kps % 32 == 0 && (kps * d) % 4096 == 0 && 2 * kps * d <= 49152;
}

bool build_attn_i32_prep(const AttnParams& p, LaunchRec* rec) {
    switch (p.d) {
    case 32: rec->fn = (const void*)k_attn_i32_prep<32>; break;
    case 64: rec->fn = (const void*)k_attn_i32_prep<64>; break;
    case 128: rec->fn = (const void*)k_attn_i32_prep<128>; break;
    default: return false;
    }
    const int64_t items = p.prep_k + p.prep_v + p.prep_q + (p.clear_o ? (int64_t)p.L * p.d / 4 : 0);
    rec->name = "attn_i32_prep";
    rec->grid = dim3((unsigned)((items + AT - 1) / AT), 1, 1);
    rec->block = dim3(AT, 1, 1);
    rec->set_params(p);
    return true;
}

bool build_attn_i32r(const AttnParams& p, LaunchRec* rec) {
    switch (p.d) {
    case 32: rec->fn = (const void*)k_attn_i32r<32>; break;
    case 64: rec->fn = (const void*)k_attn_i32r<64>; break;
    case 128: rec->fn = (const void*)k_attn_i32r<128>; break;
    default: return false;
    }
    rec->name = "attn_i32_resident";
    rec->grid = dim3((unsigned)((p.L + AQ - 1) / AQ), (unsigned)p.splits, 1);
    rec->block = dim3(AT, 1, 1);
    rec->shmem = (uint32_t)(2 * (int64_t)p.keys_per_split * p.d);
    rec->set_params(p);
    return true;
}

bool build_attn_i32s(const AttnParams& p, LaunchRec* rec) {
    int keys = 0;
#define QX_ATTN_S(DD, QQ) \
    if (p.d == DD && p.qt == QQ) { rec->fn = (const void*)k_attn_i32s<DD, QQ>; keys = AttnStream<DD, QQ>::KEYS; }
    QX_ATTN_S(32, 2) QX_ATTN_S(64, 2)
#undef QX_ATTN_S
    if (keys == 0 || p.keys_per_split % keys != 0 || !p.v_blocks) return false;
    rec->name = "attn_i32_stream";
    rec->grid = dim3((unsigned)((p.L + 32 * p.qt - 1) / (32 * p.qt)), (unsigned)p.splits, 1);
    rec->block = dim3(512, 1, 1);
    rec->set_params(p);
    return true;
}

void build_reduce(const ReduceParams& p, LaunchRec* rec) {
    rec->fn = (const void*)k_reduce_splits;
    rec->grid = dim3((unsigned)((p.n + AT - 1) / AT), 1, 1);
    rec->block = dim3(AT, 1, 1);
    rec->name = "reduce_splits";
    rec->set_params(p);
}

bool build_sdpa_f32(const SdpaParams& p, LaunchRec* rec) {
    const int D = (p.d + 31) / 32 * 32;
    const bool rag = p.d != D;
#define QX_SDPA_CASE(DD) \
    case DD: rec->fn = rag ? (const void*)k_sdpa_f32<DD, true> : (const void*)k_sdpa_f32<DD, false>; break;
    switch (D) {
    QX_SDPA_CASE(32)
    QX_SDPA_CASE(64)
    QX_SDPA_CASE(96)
    QX_SDPA_CASE(128)
    default: return false;
    }
#undef QX_SDPA_CASE
    rec->name = "sdpa_f32";
    rec->grid = dim3((unsigned)((p.L + AQ - 1) / AQ), (unsigned)p.splits, (unsigned)p.BH);
    rec->block = dim3(AT, 1, 1);
    rec->set_params(p);
    return true;
}

void build_sdpa_combine(const SdpaCombineParams& p, LaunchRec* rec) {
    rec->fn = (const void*)k_sdpa_combine;
    rec->grid = dim3((unsigned)((p.rows * p.d + AT - 1) / AT), 1, 1);
    rec->block = dim3(AT, 1, 1);
    rec->name = "sdpa_combine";
    rec->set_params(p);
}

}  // namespace qx
