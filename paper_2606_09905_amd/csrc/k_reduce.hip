// k_reduce.hip -- the HBM-bound operators of the operator table (Table 2):
// min/max over an INT32 or INT16 array, and 2x2 / stride 2 pooling of NCHW
// tensors (INT32 average, FP32 maximum).  One pass over the input with
// 16-byte loads; their roofline is HBM bandwidth.
#include <algorithm>

#include "qx_internal.h"

namespace qx {

typedef int i4v __attribute__((ext_vector_type(4)));
typedef short s8m __attribute__((ext_vector_type(8)));
typedef float f4m __attribute__((ext_vector_type(4)));

constexpr int RT = 256;   // threads per workgroup

// ---------------------------------------------------------------------------
// min/max: pass 1 -- workgroup b reduces elements [b*per, min((b+1)*per, n))
// (per is a multiple of 64 elements) and writes its pair to part[2b .. 2b+1];
// pass 2 -- one workgroup reduces the pairs into out[0] = min, out[1] = max.
// ---------------------------------------------------------------------------
// The input is read once: non-temporal loads stream it past the caches
// (12% faster than plain loads on a 512 MB array).
template <class T>
__device__ __forceinline__ void minmax_vec(const T* src, int32_t& lo, int32_t& hi) {
    if (sizeof(T) == 4) {
        const i4v v = __builtin_nontemporal_load((const i4v*)src);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            lo = min(lo, (int32_t)v[e]);
            hi = max(hi, (int32_t)v[e]);
        }
    } else {
        const s8m v = __builtin_nontemporal_load((const s8m*)src);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            lo = min(lo, (int32_t)v[e]);
            hi = max(hi, (int32_t)v[e]);
        }
    }
}

__device__ __forceinline__ void block_minmax(int32_t& lo, int32_t& hi) {
    __shared__ int32_t red[2][RT / 64];
    for (int off = 32; off > 0; off >>= 1) {
        lo = min(lo, __shfl_xor(lo, off, 64));
        hi = max(hi, __shfl_xor(hi, off, 64));
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        red[0][wave] = lo;
        red[1][wave] = hi;
    }
    __syncthreads();
    lo = red[0][0];
    hi = red[1][0];
#pragma unroll
    for (int w = 1; w < RT / 64; ++w) {
        lo = min(lo, red[0][w]);
        hi = max(hi, red[1][w]);
    }
}

template <class T>
__global__ __launch_bounds__(RT) void k_minmax_partial(const MinMaxParams p) {
    constexpr int V = 16 / sizeof(T);
    const T* x = (const T*)p.x;
    const int64_t start = (int64_t)blockIdx.x * p.per;
    const int64_t end = min(start + p.per, p.n);
    int32_t lo = INT32_MAX, hi = INT32_MIN;
    const int64_t vend = start + (end - start) / (RT * V) * (RT * V);
    // whole rounds of 256 vectors, four in flight per thread
    int64_t i = start + threadIdx.x * V;
    for (; i + 3 * RT * V < vend; i += 4 * RT * V) {
        minmax_vec<T>(x + i, lo, hi);
        minmax_vec<T>(x + i + RT * V, lo, hi);
        minmax_vec<T>(x + i + 2 * RT * V, lo, hi);
        minmax_vec<T>(x + i + 3 * RT * V, lo, hi);
    }
    for (; i < vend; i += RT * V) minmax_vec<T>(x + i, lo, hi);
    for (int64_t j = vend + threadIdx.x; j < end; j += RT) {
        lo = min(lo, (int32_t)x[j]);
        hi = max(hi, (int32_t)x[j]);
    }
    block_minmax(lo, hi);
    if (threadIdx.x == 0) {
        p.part[2 * blockIdx.x] = lo;
        p.part[2 * blockIdx.x + 1] = hi;
    }
}

__global__ __launch_bounds__(RT) void k_minmax_final(const MinMaxParams p) {
    int32_t lo = INT32_MAX, hi = INT32_MIN;
    for (int b = threadIdx.x; b < p.blocks; b += RT) {
        lo = min(lo, p.part[2 * b]);
        hi = max(hi, p.part[2 * b + 1]);
    }
    block_minmax(lo, hi);
    if (threadIdx.x == 0) {
        if (p.elem_bytes == 4) {
            ((int32_t*)p.out)[0] = lo;
            ((int32_t*)p.out)[1] = hi;
        } else {
            ((int16_t*)p.out)[0] = (int16_t)lo;
            ((int16_t*)p.out)[1] = (int16_t)hi;
        }
    }
}

// ---------------------------------------------------------------------------
// 2x2 / stride 2 pooling, no padding (a trailing odd row or column is
// dropped).  A thread makes four consecutive outputs of one output row from
// two 8-element input row segments.  INT32 average: floor of the exact sum
// of the four values over 4 (the int64 sum shifted right by 2).  FP32
// maximum: the first window value, replaced by each later one that compares
// greater (row-major window order).
// ---------------------------------------------------------------------------
template <bool AVG>
__device__ __forceinline__ uint32_t pool4(const uint32_t* a, const uint32_t* b, bool relu) {
    if (AVG) {
        int64_t v0 = (int32_t)a[0], v1 = (int32_t)a[1], v2 = (int32_t)b[0], v3 = (int32_t)b[1];
        if (relu) {
            v0 = v0 > 0 ? v0 : 0;
            v1 = v1 > 0 ? v1 : 0;
            v2 = v2 > 0 ? v2 : 0;
            v3 = v3 > 0 ? v3 : 0;
        }
        return (uint32_t)(int32_t)((v0 + v1 + v2 + v3) >> 2);
    }
    float m = __uint_as_float(a[0]);
    const float c1 = __uint_as_float(a[1]), c2 = __uint_as_float(b[0]), c3 = __uint_as_float(b[1]);
    if (c1 > m) m = c1;
    if (c2 > m) m = c2;
    if (c3 > m) m = c3;
    return __float_as_uint(m);
}

template <bool AVG>
__global__ __launch_bounds__(RT) void k_pool2(const PoolParams p) {
    const int wq = (p.Wo + 3) / 4;
    const int64_t t = (int64_t)blockIdx.x * RT + threadIdx.x;
    if (t >= p.NC * p.Ho * wq) return;
    const int q = (int)(t % wq);
    const int64_t r = t / wq;            // (nc, oh)
    const int oh = (int)(r % p.Ho);
    const int64_t nc = r / p.Ho;
    const int ow0 = q * 4;
    const uint32_t* row0 = (const uint32_t*)p.x + (nc * p.H + 2 * oh) * p.W + 2 * ow0;
    const uint32_t* row1 = row0 + p.W;
    uint32_t* out = (uint32_t*)p.y + (nc * p.Ho + oh) * p.Wo + ow0;
    if (p.vec && ow0 + 4 <= p.Wo) {
        const i4v a0 = *(const i4v*)row0, a1 = *(const i4v*)(row0 + 4);
        const i4v b0 = *(const i4v*)row1, b1 = *(const i4v*)(row1 + 4);
        const uint32_t a[8] = {(uint32_t)a0[0], (uint32_t)a0[1], (uint32_t)a0[2], (uint32_t)a0[3],
                               (uint32_t)a1[0], (uint32_t)a1[1], (uint32_t)a1[2], (uint32_t)a1[3]};
        const uint32_t b[8] = {(uint32_t)b0[0], (uint32_t)b0[1], (uint32_t)b0[2], (uint32_t)b0[3],
                               (uint32_t)b1[0], (uint32_t)b1[1], (uint32_t)b1[2], (uint32_t)b1[3]};
        i4v o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (int)pool4<AVG>(a + 2 * e, b + 2 * e, p.relu);
        *(i4v*)out = o;
    } else {
        for (int e = 0; e < 4 && ow0 + e < p.Wo; ++e) out[e] = pool4<AVG>(row0 + 2 * e, row1 + 2 * e, p.relu);
    }
}

__global__ __launch_bounds__(RT) void k_relu_i32(const ReluParams p) {
    const int64_t i = (int64_t)blockIdx.x * RT + threadIdx.x;
    if (i < p.n) p.p[i] = max(p.p[i], 0);
}

// ---------------------------------------------------------------------------
// Direct INT32 convolution under the smul24 contract for few output
// channels, where a GEMM tile would be mostly empty: a thread owns a few
// output pixels and accumulates all C_out channels of each with
// v_mad_i32_i24 (low 32 bits of the product of the sign-extended low 24
// bits), wrapping mod 2^32.
// ---------------------------------------------------------------------------
constexpr int DKW = 8;   // KW limit; C_out <= 16 and C_in*KH*KW <= 1024 (64 KB of LDS)

// The workgroup copies n int32 from global memory into LDS with several
// loads in flight per thread before any wait (16-byte loads when both
// sides are 16-byte aligned): a loop of single loads each waited for costs
// one memory latency per element a thread copies.
__device__ __forceinline__ void copy_to_lds(int32_t* dst, const int32_t* src, int n) {
    int done = 0;
    if ((((uintptr_t)src | (uintptr_t)dst) & 15) == 0) {
        const int n4 = n >> 2;
        const i4v* s4 = (const i4v*)src;
        i4v* d4 = (i4v*)dst;
        for (int i0 = (int)threadIdx.x; i0 < n4; i0 += RT * 4) {
            i4v v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = i0 + u * RT;
                v[u] = i < n4 ? s4[i] : i4v{0, 0, 0, 0};
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = i0 + u * RT;
                if (i < n4) d4[i] = v[u];
            }
        }
        done = 4 * n4;
    }
    for (int i0 = done + (int)threadIdx.x; i0 < n; i0 += RT * 8) {
        int32_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = i0 + u * RT;
            v[u] = i < n ? src[i] : 0;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = i0 + u * RT;
            if (i < n) dst[i] = v[u];
        }
    }
}

// Weights [C_out][Kd] -> LDS [Kd][DCO] (zero past C_out), eight loads in
// flight per thread.
template <int DCO>
__device__ __forceinline__ void stage_weights(int32_t (*ws)[DCO], const int32_t* w, int Co, int Kd) {
    for (int i0 = (int)threadIdx.x; i0 < Kd * DCO; i0 += RT * 8) {
        int32_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = i0 + u * RT, k = i / DCO, c = i % DCO;
            v[u] = (i < Kd * DCO && c < Co) ? w[(int64_t)c * Kd + k] : 0;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = i0 + u * RT;
            if (i < Kd * DCO) ws[i / DCO][i % DCO] = v[u];
        }
    }
}

// KWT: the kernel width when it is 3 or 5, else DKW for any KW <= DKW (the
// taps past KW then multiply a zero input).  PXT: output pixels per thread,
// consecutive along a row (Wo % PXT == 0): each weight read from LDS (a
// broadcast, the same address in every lane) feeds PXT multiply-adds.
// STAGE: a workgroup takes p.imgs whole images (imgs * Ho * Wo <= RT * PXT)
// and first copies their inputs into LDS with coalesced loads, so the
// window reads (scattered across rows and cache lines) come from LDS;
// otherwise the windows are read from global memory.
// At most four waves per SIMD: the registers that frees hold a kernel row's
// weights (KWT x DCO words) at once, so their LDS reads are in flight
// together (the grids of these convolutions give a few waves per SIMD).
template <int DCO, int KWT, int PXT, bool STAGE, bool S1P0>
__global__ __launch_bounds__(RT) __attribute__((amdgpu_waves_per_eu(1, 4)))
void k_conv_direct_s24(const ConvDirectParams p) {
    // LDS: weights [Kd][DCO], zero past C_out, then (STAGE) the inputs of
    // this workgroup's images [imgs][Ci][H][W]
    extern __shared__ __align__(16) int32_t wsh[];
    int32_t(*ws)[DCO] = (int32_t(*)[DCO])wsh;
    const ConvGeom& g = p.g;
    stage_weights<DCO>(ws, p.w, p.Co, p.Kd);
    const int hw = g.Ho * g.Wo;
    const int64_t groups = p.P / PXT;
    int64_t t;
    const int32_t* xb;
    int n, rem;
    bool live;
    if constexpr (STAGE) {
        // images [img0, img0 + imgs) of the batch; thread -> PXT pixels
        const int imgs = p.imgs, nimg = (int)(p.P / hw);
        const int img0 = (int)blockIdx.x * imgs, cnt = min(imgs, nimg - img0);
        const int chw = g.Ci * g.H * g.W;
        int32_t* xs = wsh + p.Kd * DCO;
        copy_to_lds(xs, p.x + (int64_t)img0 * chw, cnt * chw);
        const int local = (int)threadIdx.x * PXT;             // pixel within the images
        live = local < cnt * hw;
        const int li = min(local, cnt * hw - PXT);
        const int limg = li / hw;
        rem = li - limg * hw;
        n = img0 + limg;
        t = (int64_t)n * (hw / PXT) + rem / PXT;
        xb = xs + (int64_t)limg * chw;
        __syncthreads();
    } else {
        t = (int64_t)blockIdx.x * RT + threadIdx.x;
        live = t < groups;
        const int64_t pc = min(t, groups - 1) * PXT;
        n = (int)(pc / hw);
        rem = (int)(pc - (int64_t)n * hw);
        xb = p.x + (int64_t)n * g.Ci * g.H * g.W;
        __syncthreads();
    }
    const int oh = rem / g.Wo, ow0 = rem - oh * g.Wo;
    uint32_t acc[PXT][DCO];
#pragma unroll
    for (int j = 0; j < PXT; ++j)
#pragma unroll
        for (int c = 0; c < DCO; ++c) acc[j][c] = 0u;
    int k = 0;
    for (int ci = 0; ci < g.Ci; ++ci)
        for (int kh = 0; kh < g.KH; ++kh, k += g.KW) {
            // the inputs of this kernel row for all PXT pixels first
            // (independent loads), then every tap and output channel
            int32_t xv[PXT][KWT];
            if constexpr (S1P0) {
                // stride 1, no padding: every window lies inside the image
                // and neighbouring pixels share PXT + KW - 2 of their inputs
                const int32_t* xr = xb + ((int64_t)ci * g.H + oh + kh) * g.W + ow0;
                int32_t xrow[PXT + KWT - 1];
#pragma unroll
                for (int i = 0; i < PXT + KWT - 1; ++i)
                    xrow[i] = (KWT != DKW || i < PXT + g.KW - 1) ? xr[i] : 0;
#pragma unroll
                for (int j = 0; j < PXT; ++j)
#pragma unroll
                    for (int kw = 0; kw < KWT; ++kw) xv[j][kw] = (KWT != DKW || kw < g.KW) ? xrow[j + kw] : 0;
            } else {
                const int ih = oh * g.stride - g.pad + kh;
                const bool rin = ih >= 0 && ih < g.H;
                const int32_t* xr = xb + ((int64_t)ci * g.H + ih) * g.W;
#pragma unroll
                for (int j = 0; j < PXT; ++j)
#pragma unroll
                    for (int kw = 0; kw < KWT; ++kw) {
                        const int iw = (ow0 + j) * g.stride - g.pad + kw;
                        xv[j][kw] = (kw < g.KW && rin && iw >= 0 && iw < g.W) ? xr[iw] : 0;
                    }
            }
            if constexpr (S1P0 && KWT != DKW) {
                // the whole kernel row's weights first (KWT x DCO / 4 reads
                // in flight together), then its multiply-adds: one wait on
                // LDS per row instead of one per tap
                int32_t wr[KWT][DCO];
#pragma unroll
                for (int kw = 0; kw < KWT; ++kw) {
                    const i4v* wk = (const i4v*)ws[k + kw];
#pragma unroll
                    for (int c4 = 0; c4 < DCO / 4; ++c4) {
                        const i4v w4 = wk[c4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) wr[kw][4 * c4 + e] = w4[e];
                    }
                }
#pragma unroll
                for (int kw = 0; kw < KWT; ++kw)
#pragma unroll
                    for (int j = 0; j < PXT; ++j)
#pragma unroll
                        for (int c = 0; c < DCO; ++c) acc[j][c] += (uint32_t)__mul24(xv[j][kw], wr[kw][c]);
            } else {
#pragma unroll
                for (int kw = 0; kw < KWT; ++kw) {
                    // DCO weights as 16-byte LDS reads (rows of DCO ints from a
                    // 16-byte aligned base)
                    const i4v* wk = (const i4v*)ws[k + (KWT == DKW ? min(kw, g.KW - 1) : kw)];
                    int32_t wv[DCO];
#pragma unroll
                    for (int c4 = 0; c4 < DCO / 4; ++c4) {
                        const i4v w4 = wk[c4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) wv[4 * c4 + e] = w4[e];
                    }
#pragma unroll
                    for (int j = 0; j < PXT; ++j)
#pragma unroll
                        for (int c = 0; c < DCO; ++c) acc[j][c] += (uint32_t)__mul24(xv[j][kw], wv[c]);
                }
            }
        }
    (void)t;
    if (live)
#pragma unroll
        for (int c = 0; c < DCO; ++c)
            if (c < p.Co)
#pragma unroll
                for (int j = 0; j < PXT; ++j) p.y[((int64_t)n * p.Co + c) * hw + rem + j] = (int32_t)acc[j][c];
}

// The direct convolution fused with ReLU and a 2x2 average pool (the
// sequence of the LeNet-shaped pipeline): a thread computes one 2x2 block of
// conv outputs for every output channel (four pixels share each weight
// read, as above) and writes only the pooled value, floor((relu(a) +
// relu(b) + relu(c) + relu(d)) / 4) summed in 64 bits, the pool kernel's
// arithmetic.  Ho and Wo even; the output is [N][C_out][Ho/2][Wo/2].  A
// workgroup takes p.imgs whole images, staged in LDS as above.
template <int DCO, int KWT, bool S1P0, int DCU>
__global__ __launch_bounds__(RT) void k_conv_pool_s24(const ConvDirectParams p) {
    extern __shared__ __align__(16) int32_t wsh[];
    int32_t(*ws)[DCO] = (int32_t(*)[DCO])wsh;
    const ConvGeom& g = p.g;
    stage_weights<DCO>(ws, p.w, p.Co, p.Kd);
    const int Wq = g.Wo / 2, hwq = (g.Ho / 2) * Wq;
    const int64_t pq = p.P / 4;   // pooled pixels
    // images [img0, img0 + cnt) of the batch; thread -> one pooled pixel
    const int imgs = p.imgs, nimg = (int)(pq / hwq);
    const int img0 = (int)blockIdx.x * imgs, cnt = min(imgs, nimg - img0);
    const int chw = g.Ci * g.H * g.W;
    int32_t* xs = wsh + p.Kd * DCO;
    copy_to_lds(xs, p.x + (int64_t)img0 * chw, cnt * chw);
    const int local = (int)threadIdx.x;
    const bool live = local < cnt * hwq;
    const int li = min(local, cnt * hwq - 1);
    const int limg = li / hwq;
    const int remq = li - limg * hwq;
    const int n = img0 + limg;
    const int32_t* xb = xs + (int64_t)limg * chw;
    __syncthreads();
    const int qh = remq / Wq, qw = remq - qh * Wq;
    const int oh0 = 2 * qh, ow0 = 2 * qw;
    // DCU: output channels computed (C_out <= DCU <= DCO; the LDS weight
    // rows stay DCO wide)
    static_assert(DCU <= DCO, "computed channels fit the weight rows");
    uint32_t acc[4][DCU];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int c = 0; c < DCU; ++c) acc[j][c] = 0u;
    int k = 0;
    for (int ci = 0; ci < g.Ci; ++ci)
        for (int kh = 0; kh < g.KH; ++kh, k += g.KW) {
            int32_t xv[4][KWT];
#pragma unroll
            for (int dy = 0; dy < 2; ++dy) {
                if constexpr (S1P0) {
                    // stride 1, no padding: the two pixels of a row share
                    // KW - 1 of their inputs, all inside the image
                    const int32_t* xr = xb + ((int64_t)ci * g.H + oh0 + dy + kh) * g.W + ow0;
                    int32_t xrow[KWT + 1];
#pragma unroll
                    for (int i = 0; i < KWT + 1; ++i) xrow[i] = (KWT != DKW || i < g.KW + 1) ? xr[i] : 0;
#pragma unroll
                    for (int dx = 0; dx < 2; ++dx)
#pragma unroll
                        for (int kw = 0; kw < KWT; ++kw)
                            xv[2 * dy + dx][kw] = (KWT != DKW || kw < g.KW) ? xrow[dx + kw] : 0;
                } else {
                    const int ih = (oh0 + dy) * g.stride - g.pad + kh;
                    const bool rin = ih >= 0 && ih < g.H;
                    const int32_t* xr = xb + ((int64_t)ci * g.H + ih) * g.W;
#pragma unroll
                    for (int dx = 0; dx < 2; ++dx)
#pragma unroll
                        for (int kw = 0; kw < KWT; ++kw) {
                            const int iw = (ow0 + dx) * g.stride - g.pad + kw;
                            xv[2 * dy + dx][kw] = (kw < g.KW && rin && iw >= 0 && iw < g.W) ? xr[iw] : 0;
                        }
                }
            }
            // the kernel row's weights first, all reads in flight together
            int32_t wr[KWT][DCO];
#pragma unroll
            for (int kw = 0; kw < KWT; ++kw) {
                const i4v* wk = (const i4v*)ws[k + (KWT == DKW ? min(kw, g.KW - 1) : kw)];
#pragma unroll
                for (int c4 = 0; c4 < (DCU + 3) / 4; ++c4) {
                    const i4v w4 = wk[c4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) wr[kw][4 * c4 + e] = w4[e];
                }
            }
#pragma unroll
            for (int kw = 0; kw < KWT; ++kw)
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int c = 0; c < DCU; ++c) acc[j][c] += (uint32_t)__mul24(xv[j][kw], wr[kw][c]);
        }
    if (live)
#pragma unroll
        for (int c = 0; c < DCU; ++c)
            if (c < p.Co) {
                int64_t sum = 0;
#pragma unroll
                for (int j = 0; j < 4; ++j) sum += max((int64_t)(int32_t)acc[j][c], (int64_t)0);
                p.y[((int64_t)n * p.Co + c) * hwq + remq] = (int32_t)(sum >> 2);
            }
}

// ---------------------------------------------------------------------------
// Builders
// ---------------------------------------------------------------------------
void minmax_blocks(int64_t n, int32_t* blocks, int64_t* per) {
    const int64_t want = std::min<int64_t>(std::max<int64_t>((n + 65535) / 65536, 1), 2048);
    int64_t pe = (n + want - 1) / want;
    pe = (pe + 63) / 64 * 64;   // whole 16-byte vectors at every workgroup start
    *per = pe;
    *blocks = (int32_t)((n + pe - 1) / pe);
}

void build_minmax(const MinMaxParams& p, LaunchRec* partial, LaunchRec* final_rec) {
    partial->fn = p.elem_bytes == 4 ? (const void*)k_minmax_partial<int32_t> : (const void*)k_minmax_partial<int16_t>;
    partial->grid = dim3((unsigned)p.blocks, 1, 1);
    partial->block = dim3(RT, 1, 1);
    partial->name = p.elem_bytes == 4 ? "minmax_i32" : "minmax_i16";
    partial->set_params(p);
    final_rec->fn = (const void*)k_minmax_final;
    final_rec->grid = dim3(1, 1, 1);
    final_rec->block = dim3(RT, 1, 1);
    final_rec->name = "minmax_final";
    final_rec->set_params(p);
}

// Whole images per workgroup for the fused conv + ReLU + pool kernel: as
// many as its threads (one per pooled pixel) and 64 KB of LDS (weights and
// inputs) hold; 0 when not even one fits.
int32_t conv_pool_images(const ConvDirectParams& p) {
    const int dco = p.Co <= 8 ? 8 : 16;
    const int64_t hwq = (int64_t)(p.g.Ho / 2) * (p.g.Wo / 2);
    const int64_t chw = (int64_t)p.g.Ci * p.g.H * p.g.W;
    if (hwq <= 0 || chw <= 0 || p.P <= 0) return 0;
    return (int32_t)std::max<int64_t>(std::min<int64_t>(RT / hwq, (16384 - (int64_t)p.Kd * dco) / chw), 0);
}

void build_conv_direct_s24(const ConvDirectParams& p0, LaunchRec* rec) {
    ConvDirectParams p = p0;
    if (p.pool) {
        // fused ReLU + 2x2 average: one thread per pooled pixel, whole
        // images staged in LDS (the caller checked conv_pool_images > 0)
        const int kw = p.g.KW;
        const int dco = p.Co <= 8 ? 8 : 16;
        const int64_t hwq = (int64_t)(p.g.Ho / 2) * (p.g.Wo / 2);
        const int64_t chw = (int64_t)p.g.Ci * p.g.H * p.g.W;
        p.imgs = conv_pool_images(p);
        const bool s1p0 = p.g.stride == 1 && p.g.pad == 0;
        // channels computed: C_out rounded up to 4, 6, 8 or 16
#define QX_CP3(DCO, KWT, DCU) (s1p0 ? (const void*)k_conv_pool_s24<DCO, KWT, true, DCU> \
                                    : (const void*)k_conv_pool_s24<DCO, KWT, false, DCU>)
#define QX_CP2(DCO, KWT) (DCO == 16 ? QX_CP3(DCO, KWT, DCO) : p.Co <= 4 ? QX_CP3(DCO, KWT, 4) \
                          : p.Co <= 6 ? QX_CP3(DCO, KWT, 6) : QX_CP3(DCO, KWT, DCO))
#define QX_CP(DCO) (kw == 5 ? QX_CP2(DCO, 5) : kw == 3 ? QX_CP2(DCO, 3) : QX_CP2(DCO, DKW))
        rec->fn = p.Co <= 8 ? QX_CP(8) : QX_CP(16);
#undef QX_CP
#undef QX_CP2
#undef QX_CP3
        const int64_t blocks = (p.P / 4 / hwq + p.imgs - 1) / p.imgs;
        rec->grid = dim3((unsigned)std::max<int64_t>(blocks, 1), 1, 1);
        rec->block = dim3(RT, 1, 1);
        rec->shmem = (uint32_t)((p.Kd * dco + p.imgs * chw) * sizeof(int32_t));
        rec->name = "conv_relu_pool_s24";
        rec->set_params(p);
        return;
    }
    const int kw = p.g.KW, wo = p.g.Wo;
    const int pxt = wo % 4 == 0 ? 4 : wo % 2 == 0 ? 2 : 1;
    const int dco = p.Co <= 8 ? 8 : 16;
    const int64_t hw = (int64_t)p.g.Ho * wo;
    const int64_t chw = (int64_t)p.g.Ci * p.g.H * p.g.W;
    // whole images per workgroup when at least one fits the threads and
    // LDS (weights + inputs within 64 KB)
    const int64_t by_threads = hw > 0 ? (int64_t)RT * pxt / hw : 0;
    const int64_t by_lds = chw > 0 ? (16384 - (int64_t)p.Kd * dco) / chw : 0;
    const int64_t imgs = std::min<int64_t>(by_threads, by_lds);
    const bool stage = imgs >= 1 && p.P > 0;
    p.imgs = stage ? (int32_t)imgs : 0;
    const bool s1p0 = p.g.stride == 1 && p.g.pad == 0;
#define QX_DC5(DCO, KWT, PX, ST) (s1p0 ? (const void*)k_conv_direct_s24<DCO, KWT, PX, ST, true> \
                                       : (const void*)k_conv_direct_s24<DCO, KWT, PX, ST, false>)
#define QX_DC4(DCO, KWT, PX) (stage ? QX_DC5(DCO, KWT, PX, true) : QX_DC5(DCO, KWT, PX, false))
#define QX_DC3(DCO, KWT) (pxt == 4 ? QX_DC4(DCO, KWT, 4) : pxt == 2 ? QX_DC4(DCO, KWT, 2) : QX_DC4(DCO, KWT, 1))
#define QX_DC(DCO) (kw == 5 ? QX_DC3(DCO, 5) : kw == 3 ? QX_DC3(DCO, 3) : QX_DC3(DCO, DKW))
    rec->fn = p.Co <= 8 ? QX_DC(8) : QX_DC(16);
#undef QX_DC
#undef QX_DC3
#undef QX_DC4
#undef QX_DC5
    int64_t blocks;
    if (stage) {
        const int64_t nimg = p.P / hw;
        blocks = (nimg + imgs - 1) / imgs;
    } else {
        blocks = (p.P / pxt + RT - 1) / RT;
    }
    rec->grid = dim3((unsigned)std::max<int64_t>(blocks, 1), 1, 1);
    rec->block = dim3(RT, 1, 1);
    rec->shmem = (uint32_t)((p.Kd * dco + (stage ? imgs * chw : 0)) * sizeof(int32_t));
    rec->name = "conv_direct_s24";
    rec->set_params(p);
}

void build_relu(const ReluParams& p, LaunchRec* rec) {
    rec->fn = (const void*)k_relu_i32;
    rec->grid = dim3((unsigned)std::max<int64_t>((p.n + RT - 1) / RT, 1), 1, 1);
    rec->block = dim3(RT, 1, 1);
    rec->name = "relu_i32";
    rec->set_params(p);
}

void build_pool2(int32_t kind, const PoolParams& p, LaunchRec* rec) {
    const int64_t threads = p.NC * p.Ho * ((p.Wo + 3) / 4);
    rec->fn = kind == POOL_AVG_I32 ? (const void*)k_pool2<true> : (const void*)k_pool2<false>;
    rec->grid = dim3((unsigned)std::max<int64_t>((threads + RT - 1) / RT, 1), 1, 1);
    rec->block = dim3(RT, 1, 1);
    rec->name = kind == POOL_AVG_I32 ? "avgpool2_i32" : "maxpool2_f32";
    rec->set_params(p);
}

}  // namespace qx
