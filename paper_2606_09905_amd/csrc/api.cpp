// api.cpp -- planner, persistent executor and the C ABI of libqx.
//
// Planner: from an operation, its shape and the caller's declared operand
// bounds it derives which exact route can run (the bounds prove how large
// every partial sum can get), the tile shapes, the launch records and the
// workspace size (Methodology: operand-range contracts).  Pure host logic,
// exported through the qx_plan_* queries so it can be checked without a
// device.
//
// Executor: a handle holding one planned operation.  Its workspace is
// allocated and its launch parameter blocks built when it is created; a run
// only writes the caller's pointers into copies of those blocks and enqueues
// the launches (Methodology: persistent executors).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <atomic>
#include <map>
#include <set>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/qx.h"
#include "../../include/qx_testing.h"
#include "qx_internal.h"

using namespace qx;

namespace {

thread_local std::string g_err;

qx_status fail(qx_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

qx_status hip_fail(hipError_t e, const char* what) {
    return fail(e == hipErrorOutOfMemory ? QX_ERR_OUT_OF_MEMORY : QX_ERR_DEVICE, "%s: %s (%d)", what,
                hipGetErrorString(e), (int)e);
}

constexpr int64_t kMaxDim = (int64_t)1 << 30;
constexpr int64_t kMaxBatch = 65535;
constexpr uint32_t kMagic = 0x71786578u;  // "qxex"

enum OpKind : int32_t {
    OP_GEMM_I16 = 1, OP_GEMM_S24 = 2, OP_CONV = 3, OP_ATTN_F32 = 4, OP_ATTN_I32 = 5, OP_CONV_F32 = 6, OP_CONV_I32 = 7,
    OP_MINMAX = 8, OP_POOL = 9, OP_LENET = 10, OP_SDPA = 11
};

// A fully planned operation: route facts plus launch records with unbound
// pointers.  Built on the host with no device call.
struct Plan {
    OpKind op{};
    qx_plan_info info{};
    std::vector<LaunchRec> launches;
    // operands with a declared bound, scanned on the device when QX_VALIDATE=1
    struct RangeCheck {
        int input;
        int elem_bytes;
        int64_t n;
        int32_t bound;
    };
    std::vector<RangeCheck> checks;
    int n_inputs = 0;
    uint64_t in_align = 16;  // required alignment of every input pointer
    uint64_t out_align = 4;  // required alignment of the output pointer
};

bool mul_ok(int64_t a, int64_t b, int64_t lim, int64_t* out) {
    if (a < 0 || b < 0) return false;
    if (a != 0 && b > lim / a) return false;
    *out = a * b;
    return true;
}

uint64_t round_up(uint64_t v, uint64_t a) { return (v + a - 1) / a * a; }

// The dtype argument as the caller passed it.  A C caller may pass any int;
// reading it through the enum type would be undefined for values outside
// the enumerators, so its bytes are copied and validated as an int32.
int32_t dt_raw(const qx_attn_dtype& dt) {
    int32_t v;
    static_assert(sizeof(qx_attn_dtype) == sizeof(int32_t), "enum passed as int");
    memcpy(&v, &dt, sizeof v);
    return v;
}

// ---------------------------------------------------------------------------
// Exactness rules of the integer routes.
// ---------------------------------------------------------------------------
// Largest multiple of 16 with chunk * ba * bb <= 2^24: every partial sum of
// that many products is an integer of magnitude <= 2^24, exactly
// representable in fp32.  0 if infeasible (operands beyond fp16's exact
// integer range, or fewer than 16 products per partial).
int64_t f16_chunk(int64_t ba, int64_t bb) {
    if (ba > 2048 || bb > 2048) return 0;
    const int64_t prod = std::max<int64_t>(ba * bb, 1);
    int64_t c = ((int64_t)1 << 24) / prod;
    c = c / 16 * 16;
    return c >= 16 ? c : 0;
}

bool route_applies_i16(int32_t r) {
    return r == R_I8_DIRECT || r == R_F16_EXACT || r == R_I8_KARATSUBA || r == R_I8_OFFSET4 ||
           r == R_VALU_DOT2;
}

// Route feasibility for an int16 contraction with bounds ba, bb (max |x|).
bool feasible_i16(int32_t r, int64_t ba, int64_t bb) {
    switch (r) {
    case R_I8_DIRECT: return ba <= 127 && bb <= 127;
    case R_F16_EXACT: return f16_chunk(ba, bb) > 0;
    case R_I8_KARATSUBA: return ba <= 8127 && bb <= 8127;
    case R_I8_OFFSET4:
    case R_VALU_DOT2: return true;
    default: return false;
    }
}

int32_t auto_i16(int64_t ba, int64_t bb) {
    if (feasible_i16(R_I8_DIRECT, ba, bb)) return R_I8_DIRECT;
    if (feasible_i16(R_F16_EXACT, ba, bb)) return R_F16_EXACT;
    if (feasible_i16(R_I8_KARATSUBA, ba, bb)) return R_I8_KARATSUBA;
    return R_I8_OFFSET4;
}

int32_t products_of(int32_t r) {
    switch (r) {
    case R_I8_KARATSUBA: return 3;
    case R_I8_OFFSET4: return 4;
    case R_S24_I8LIMB: return 8;
    case R_ATTN_I32_MFMA: return 3;
    default: return 1;
    }
}

qx_status check_bound16(int32_t b, const char* name, int64_t* out) {
    if (b < 0 || b > 32768) return fail(QX_ERR_INVALID_ARG, "%s = %d: must be in [0, 32768]", name, b);
    *out = b == 0 ? 32768 : b;
    return QX_OK;
}

// ---------------------------------------------------------------------------
// Integer GEMM planning shared by the GEMM and convolution operators.
// ---------------------------------------------------------------------------
struct GemmSpec {
    int64_t M, N, K, batch;
    int64_t ba, bb;      // bounds (i16 routes); unused for s24
    bool s24;
    int32_t route;       // requested
    // operand bindings
    Bind a_bind, b_bind;
    uint64_t b_ws_off;   // when b_bind == BIND_WS
    int64_t lda, ldb, ldc, sA, sB, sC;
    int32_t out_mode, hw;
    bool allow_nt;       // plain GEMM: large fp16-exact problems may take encode + NT GEMM
    bool b_conv;         // B is the im2col matrix of the image bound by b_bind (geometry
                         // geo), gathered by the limb-plane encoder (NT int8 path only)
    ConvGeom geo;
};

// The encode + direct-to-LDS route pays two HBM-bound encoding passes; it is
// used when the contraction is large enough for them to be small change and
// the chunk covers at least one 64-wide K tile.
// The NT kernel forms each lane's byte offset into an operand panel (at
// most 256 rows of Kp fp16 elements) in 32-bit int arithmetic, and the B^T
// encoder puts Kp/128 workgroups in grid y, so Kp is held below 2^22 (every
// offset below 2^31); longer K takes the register-staged kernel, which
// addresses in 64 bits.
constexpr int64_t kNtMaxKp = (int64_t)1 << 22;
bool use_nt(int32_t route, int64_t chunk, int64_t M, int64_t N, int64_t K, int64_t batch) {
    if (route != R_F16_EXACT || chunk < 64) return false;
    if ((K + 63) / 64 * 64 >= kNtMaxKp) return false;
    const double macs = (double)M * (double)N * (double)K * (double)batch;
    return macs >= (double)(1 << 24) && M >= 32 && N >= 32 && K >= 64;
}

int64_t pad_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

int32_t planes_of(int32_t r) {
    switch (r) {
    case R_I8_DIRECT: return 1;
    case R_I8_OFFSET4: return 2;
    default: return 3;
    }
}

// The int8 limb routes take the same encode + direct-to-LDS structure for
// large problems; the GEMM addresses every limb plane with 32-bit offsets.
bool use_i8nt(int32_t route, int64_t M, int64_t N, int64_t K, int64_t batch) {
    if (route != R_I8_DIRECT && route != R_I8_KARATSUBA && route != R_I8_OFFSET4 && route != R_S24_I8LIMB)
        return false;
    const double macs = (double)M * (double)N * (double)K * (double)batch;
    if (!(macs >= (double)(1 << 24) && M >= 32 && N >= 32 && K >= 64)) return false;
    int bm, bn;
    i8nt_tile_shape(route, M, N, batch, &bm, &bn);
    const int64_t P = planes_of(route), Kp = pad_up(K, 64);
    const int64_t lim = (int64_t)1 << 31;
    return P * pad_up(M, bm) * Kp < lim && P * pad_up(N, bn) * Kp < lim;
}

void add_fill_out(Plan* pl, int64_t n32);

// The skinny smul24 kernel (one row per thread, eight columns per
// workgroup) takes GEMMs of at most 128 columns with at least 1024 rows over
// the batch, enough workgroups to occupy the chip, and K up to 4096.
static bool skinny_s24(const GemmSpec& s) {
    // (its B row offsets are 32-bit: K x ldb words stay under 2 MiB)
    return s.s24 && s.N <= 128 && s.ldb <= 128 && s.M * s.batch >= 1024 && s.K <= 4096;
}

// Appends the launches of one integer GEMM; ws_used is the workspace end.
qx_status plan_int_gemm(const GemmSpec& s, Plan* pl, uint64_t* ws_used) {
    int32_t route = s.route;
    if (!s.s24) {
        if (route == R_AUTO) route = auto_i16(s.ba, s.bb);
        if (!route_applies_i16(route))
            return fail(QX_ERR_INVALID_ARG, "route %d does not apply to an int16 contraction", route);
        if (!feasible_i16(route, s.ba, s.bb))
            return fail(QX_ERR_RANGE, "route %d cannot be exact for bounds %lld x %lld", route,
                        (long long)s.ba, (long long)s.bb);
    } else {
        // Few output columns, many rows and at most 2^26 multiply-adds (the
        // last two fully connected layers of a LeNet-shaped network): the
        // skinny vector-ALU kernel, one launch without encoders or sums.
        // Through the limb planes / skinny kernel: 4096 x 10 x 84 18.1 /
        // 5.2 us, 4096 x 84 x 120 11.7 / 7.1, 4096 x 64 x 120 11.5 / 8.9;
        // larger ones favour the matrix cores: 4096 x 120 x 400 16.6 /
        // 16.7, 16384 x 128 x 512 35.6 / 73.9.
        if (route == R_AUTO) {
            const double macs = (double)s.M * (double)s.N * (double)s.K * (double)s.batch;
            route = (skinny_s24(s) && macs <= (double)(1 << 26) && !s.b_conv) ? R_S24_VALU : R_S24_I8LIMB;
        }
        if (route != R_S24_I8LIMB && route != R_S24_VALU)
            return fail(QX_ERR_INVALID_ARG, "route %d does not apply to the smul24 GEMM", route);
    }
    qx_plan_info& info = pl->info;
    info.route = route;
    info.products = products_of(route);
    info.chunk = 0;
    if (s.s24) {
        info.exact_no_wrap = 0;
    } else {
        const double maxabs = (double)s.K * (double)s.ba * (double)s.bb;
        info.exact_no_wrap = maxabs < 2147483648.0 ? 1 : 0;
    }

    if (route == R_VALU_DOT2 || route == R_S24_VALU) {
        if ((s.M + 63) / 64 > 65535) return fail(QX_ERR_UNSUPPORTED, "M too large for the VALU route");
        ValuGemmParams v{};
        v.sA = s.sA; v.sB = s.sB; v.sC = s.sC;
        v.M = (int32_t)s.M; v.N = (int32_t)s.N; v.K = (int32_t)s.K;
        v.lda = (int32_t)s.lda; v.ldb = (int32_t)s.ldb; v.ldc = (int32_t)s.ldc;
        v.b_trans = 0; v.out_mode = s.out_mode; v.hw = s.hw;
        LaunchRec rec;
        const bool skinny = route == R_S24_VALU && skinny_s24(s);
        // K slices when the 64x64 tiles give under four waves per SIMD
        // (1024 workgroups) and K is long: the slices add into the output,
        // cleared first, with wrapping int32 atomics (exact in any order).
        // smul24 1024^3: 256 tiles, 4 slices of 256.
        int32_t ksplit = 1;
        if (!skinny) {
            const int64_t tiles = ((s.M + 63) / 64) * ((s.N + 63) / 64) * s.batch;
            const bool dense_out = s.out_mode == OUT_CONV ||
                                   (s.ldc == s.N && (s.batch == 1 || s.sC == s.M * s.N));
            if (dense_out && tiles > 0 && tiles < 1024 && s.K >= 256) {
                const int64_t want = std::min<int64_t>({(1024 + tiles - 1) / tiles, s.K / 128, 8});
                if (want > 1 && s.batch * want <= 65535) ksplit = (int32_t)want;
            }
        }
        v.ksplit = ksplit;
        info.k_splits = ksplit > 1 ? ksplit : 0;
        if (ksplit > 1) add_fill_out(pl, s.M * s.N * s.batch);
        if (skinny) build_valu_skinny_s24(v, (int)s.batch, &rec);
        else build_valu_gemm(route == R_VALU_DOT2 ? VK_I16_DOT2 : VK_S24, v, (int)s.batch, &rec);
        rec.bind(offsetof(ValuGemmParams, A), s.a_bind);
        rec.bind(offsetof(ValuGemmParams, B), s.b_bind, s.b_ws_off);
        rec.bind(offsetof(ValuGemmParams, C), BIND_OUT);
        pl->launches.push_back(rec);
        if (skinny) { info.tile_m = 64; info.tile_n = 8; info.tile_k = 32; }
        else { info.tile_m = 64; info.tile_n = 64; info.tile_k = 16; }
        return QX_OK;
    }

    if (s.allow_nt && use_nt(route, f16_chunk(s.ba, s.bb), s.M, s.N, s.K, s.batch)) {
        const int64_t chunk = f16_chunk(s.ba, s.bb);
        // Operands within [-256, 256] are exact in bf16 as well (eight
        // significant bits); the bf16 matrix cores sustain a slightly higher
        // clock on such data, so the encoders write bf16 then.
        const int32_t bf = std::max(s.ba, s.bb) <= 256 ? 1 : 0;
        info.operand_format = bf;
        int bm, bn;
        nt_tile_shape(s.M, s.N, s.batch, &bm, &bn);
        // A and B^T are padded to whole 128-row / 256-column tiles so that
        // every tile shape a batch group or column panel picks divides them.
        const int64_t Mp = pad_up(s.M, 128), Np = pad_up(s.N, 256), Kp = pad_up(s.K, 64);
        const uint64_t a_off = round_up(*ws_used, 256);
        const uint64_t b_off = round_up(a_off + 2 * (uint64_t)s.batch * Mp * Kp, 256);
        *ws_used = b_off + 2 * (uint64_t)s.batch * Np * Kp;
        // Batch groups: the batches run in groups whose encoded operands
        // fill at most the 256 MiB last-level cache, each group encoded and
        // then contracted, so that the contraction reads operands the
        // encoders have just left in that cache.  64 x 2048^3 (1 GiB
        // encoded, 16 MiB per batch): 4 groups 1.42 ms per step, 8 groups
        // 1.48, 2 groups 1.50, one 1.50 (the contraction slows once a
        // group outgrows the cache; smaller groups pay more encoder tails).
        // Encoding the next group on a second stream while the current one
        // contracts measured 4% slower still (the encoders then take CUs
        // between the contraction's workgroups).
        constexpr uint64_t kGroupBytes = (uint64_t)256 << 20;
        const uint64_t batch_bytes = 2 * (uint64_t)(Mp + Np) * (uint64_t)Kp;
        const int64_t fit = std::max<int64_t>((int64_t)(kGroupBytes / batch_bytes), 1);
        const int64_t groups = (s.batch + fit - 1) / fit;
        const int64_t per_group = (s.batch + groups - 1) / groups;
        auto enc_a = [&](int64_t b0, int64_t cnt) {
            EncParams ea{};
            ea.s_src = s.sA; ea.s_dst = Mp * Kp;
            ea.M = (int32_t)s.M; ea.N = 0; ea.K = (int32_t)s.K;
            ea.Mp = (int32_t)Mp; ea.Np = 0; ea.Kp = (int32_t)Kp;
            ea.ld_src = (int32_t)s.lda; ea.batch = (int32_t)cnt;
            ea.vec = (s.lda % 8 == 0 && s.sA % 8 == 0) ? 1 : 0;
            ea.bf16 = bf;
            LaunchRec r;
            build_enc_a(ea, &r);
            r.bind(offsetof(EncParams, src), s.a_bind, 2 * (uint64_t)(b0 * s.sA));
            r.bind(offsetof(EncParams, dst), BIND_WS, a_off + 2 * (uint64_t)(b0 * Mp * Kp));
            return r;
        };
        // encode B^T columns [n0, n0 + nw) of batches [b0, b0 + cnt), then contract them
        auto enc_b_and_gemm = [&](int64_t b0, int64_t cnt, int64_t n0, int64_t nw) {
            const int64_t nwp = std::min(pad_up(nw, 256), Np - n0);
            EncParams eb{};
            eb.s_src = s.sB; eb.s_dst = Np * Kp;
            eb.M = 0; eb.N = (int32_t)nw; eb.K = (int32_t)s.K;
            eb.Mp = 0; eb.Np = (int32_t)nwp; eb.Kp = (int32_t)Kp;
            eb.ld_src = (int32_t)s.ldb; eb.batch = (int32_t)cnt;
            eb.vec = (s.ldb % 8 == 0 && s.sB % 8 == 0 && n0 % 8 == 0) ? 1 : 0;
            eb.bf16 = bf;
            LaunchRec r2;
            build_enc_bt(eb, &r2);
            const uint64_t bt_add = b_off + 2 * (uint64_t)(b0 * Np * Kp + n0 * Kp);
            r2.bind(offsetof(EncParams, src), s.b_bind, s.b_ws_off + 2 * (uint64_t)(b0 * s.sB + n0));
            r2.bind(offsetof(EncParams, dst), BIND_WS, bt_add);
            GemmParams g{};
            g.sA = Mp * Kp; g.sB = Np * Kp; g.sC = s.sC;
            g.M = (int32_t)s.M; g.N = (int32_t)nw; g.K = (int32_t)Kp;
            g.lda = (int32_t)Kp; g.ldb = (int32_t)Kp; g.ldc = (int32_t)s.ldc;
            g.out_mode = s.out_mode; g.hw = s.hw; g.b_mode = B_KN;
            g.chunk_tiles = (int32_t)(chunk / 64);
            g.bf16 = bf;
            LaunchRec r3;
            build_gemm_nt(g, (int)cnt, &r3);
            r3.bind(offsetof(GemmParams, A), BIND_WS, a_off + 2 * (uint64_t)(b0 * Mp * Kp));
            r3.bind(offsetof(GemmParams, B), BIND_WS, bt_add);
            r3.bind(offsetof(GemmParams, C), BIND_OUT, 4 * (uint64_t)(b0 * s.sC + n0));
            pl->launches.push_back(r2);
            pl->launches.push_back(r3);
        };
        for (int64_t b0 = 0; b0 < s.batch; b0 += per_group) {
            const int64_t cnt = std::min(per_group, s.batch - b0);
            pl->launches.push_back(enc_a(b0, cnt));
            enc_b_and_gemm(b0, cnt, 0, s.N);
        }
        info.chunk = (int32_t)(chunk / 64 * 64);
        info.tile_m = bm; info.tile_n = bn; info.tile_k = 64;
        return QX_OK;
    }

    GemmParams g{};
    g.sA = s.sA; g.sB = s.sB; g.sC = s.sC;
    g.M = (int32_t)s.M; g.N = (int32_t)s.N; g.K = (int32_t)s.K;
    g.lda = (int32_t)s.lda; g.ldb = (int32_t)s.ldb; g.ldc = (int32_t)s.ldc;
    g.out_mode = s.out_mode; g.hw = s.hw; g.b_mode = B_KN;
    const bool nt8 = s.allow_nt && use_i8nt(route, s.M, s.N, s.K, s.batch);
    if (s.b_conv && !nt8) return fail(QX_ERR_UNSUPPORTED, "gathered B needs the NT int8 route");
    const bool offset = route == R_I8_OFFSET4 || route == R_S24_I8LIMB;
    // Implicit INT32 convolution (C_in a multiple of 64): one launch writes
    // the image as bordered NHWC limb planes with per-chunk position sums and
    // the weights as limb planes in (kh, kw, ci) order with their row sums;
    // the contraction then gathers each 64-k tile of B^T (64 channels of one
    // tap per pixel) from the planes, as the fp16 conv does from its NHWC
    // copy, instead of reading a materialised column matrix (9x the image
    // for a 3x3 kernel).  Offsets into the planes are 32-bit.
    const ConvGeom& cgeo = s.geo;
    const int64_t conv_hp = cgeo.H + 2 * cgeo.pad, conv_wp = cgeo.W + 2 * cgeo.pad;
    const int64_t conv_imgs = s.hw > 0 ? s.N / s.hw : 0;
    const int64_t plane_x = conv_imgs * conv_hp * conv_wp * cgeo.Ci;
    const bool conv_nhwc = nt8 && s.b_conv && s.s24 && route == R_S24_I8LIMB && cgeo.Ci % 64 == 0 &&
                           s.batch == 1 && 3 * plane_x < ((int64_t)1 << 31);
    uint64_t rs_off = 0, cs_off = 0;
    if (offset) {
        g.corr_c = route == R_I8_OFFSET4 ? 128 : 32896;
        const int slices = sums_slices((int)s.K);
        g.cs_slices = slices;
        rs_off = round_up(*ws_used, 256);
        cs_off = round_up(rs_off + 4 * (uint64_t)s.batch * (uint64_t)s.M, 256);
        // column sums: [batch][K/64][N], or for the implicit convolution the
        // per-chunk position sums [N_img][C_in/64][H+2p][W+2p]
        const uint64_t cs_n = conv_nhwc ? (uint64_t)(conv_imgs * (cgeo.Ci / 64) * conv_hp * conv_wp)
                                        : (uint64_t)s.batch * (uint64_t)slices * (uint64_t)s.N;
        *ws_used = cs_off + 4 * cs_n;
        if (!nt8) {  // the limb-plane encoders produce the sums themselves
            SumsParams sp{};
            sp.sA = s.sA; sp.sB = s.sB;
            sp.M = (int32_t)s.M; sp.N = (int32_t)s.N; sp.K = (int32_t)s.K;
            sp.lda = (int32_t)s.lda; sp.ldb = (int32_t)s.ldb;
            sp.s24 = s.s24 ? 1 : 0; sp.batch = (int32_t)s.batch;
            LaunchRec rr;
            build_sums(sp, &rr);
            rr.bind(offsetof(SumsParams, A), s.a_bind);
            rr.bind(offsetof(SumsParams, B), s.b_bind, s.b_ws_off);
            rr.bind(offsetof(SumsParams, rowsum), BIND_WS, rs_off);
            rr.bind(offsetof(SumsParams, colsum), BIND_WS, cs_off);
            pl->launches.push_back(rr);
        }
    }
    if (nt8) {
        // limb planes: A8 [batch][P][Mp][Kp], B8T [batch][P][Np][Kp] (int8)
        int bm, bn;
        i8nt_tile_shape(route, s.M, s.N, s.batch, &bm, &bn);
        const int64_t P = planes_of(route);
        const int64_t Mp = pad_up(s.M, bm), Np = pad_up(s.N, bn), Kp = pad_up(s.K, 64);
        // K slices: a grid with fewer 64x64 tiles than the chip has CUs
        // leaves CUs idle while each tile walks all of K; slicing K (at least
        // four K tiles per slice, at most 16 slices) fills the CUs once.  Two
        // slices per CU do not pay: a CU's throughput on these tiles is the
        // same with one workgroup or two.  The slices add into the output,
        // cleared first, so it must be one dense block.
        int32_t ksplit = 1;
        {
            const int64_t tiles = (Mp / bm) * (Np / bn) * s.batch, kt = Kp / 64;
            const bool dense_out = s.out_mode == OUT_ROWMAJOR && s.ldc == s.N &&
                                   (s.batch == 1 || s.sC == s.M * s.N);
            if (bm == 64 && dense_out && tiles <= 128 && kt >= 8) {
                const int64_t want = std::min<int64_t>({256 / tiles, 16, kt / 4});
                const int64_t per = (kt + want - 1) / want;
                ksplit = (int32_t)((kt + per - 1) / per);   // no empty slice
            }
        }
        g.ksplit = ksplit;
        info.k_splits = ksplit > 1 ? ksplit : 0;
        if (ksplit > 1) add_fill_out(pl, s.M * s.N * s.batch);
        if (conv_nhwc) {
            const uint64_t a_off = round_up(*ws_used, 256);
            const uint64_t x_off = round_up(a_off + (uint64_t)P * Mp * Kp, 256);
            *ws_used = x_off + (uint64_t)P * plane_x;
            ConvLimbPrepParams cp{};
            cp.plane_x = plane_x;
            cp.plane_a = Mp * Kp;
            cp.nimg = (int32_t)conv_imgs; cp.Co = (int32_t)s.M; cp.Kd = (int32_t)s.K;
            cp.g = cgeo;
            LaunchRec r1;
            build_conv_prep_limb(cp, &r1);
            r1.bind(offsetof(ConvLimbPrepParams, x), s.b_bind, s.b_ws_off);
            r1.bind(offsetof(ConvLimbPrepParams, w), s.a_bind);
            r1.bind(offsetof(ConvLimbPrepParams, xp8), BIND_WS, x_off);
            r1.bind(offsetof(ConvLimbPrepParams, s), BIND_WS, cs_off);
            r1.bind(offsetof(ConvLimbPrepParams, a8), BIND_WS, a_off);
            r1.bind(offsetof(ConvLimbPrepParams, rowsum), BIND_WS, rs_off);
            g.b_mode = B_NHWC;
            g.g = cgeo;
            g.sA = P * Mp * Kp; g.sB = 0;
            g.lda = (int32_t)Kp; g.ldb = 0;
            g.plane_a = Mp * Kp; g.plane_b = plane_x;
            LaunchRec r3;
            if (!build_gemm_i8nt(route, g, 1, &r3)) return fail(QX_ERR_UNSUPPORTED, "no kernel for route %d", route);
            r3.bind(offsetof(GemmParams, A), BIND_WS, a_off);
            r3.bind(offsetof(GemmParams, B), BIND_WS, x_off);
            r3.bind(offsetof(GemmParams, C), BIND_OUT);
            r3.bind(offsetof(GemmParams, rowsum), BIND_WS, rs_off);
            r3.bind(offsetof(GemmParams, colsum), BIND_WS, cs_off);
            pl->launches.push_back(r1);
            pl->launches.push_back(r3);
            info.tile_m = bm; info.tile_n = bn; info.tile_k = 64;
            return QX_OK;
        }
        const uint64_t a_off = round_up(*ws_used, 256);
        const uint64_t b_off = round_up(a_off + (uint64_t)s.batch * P * Mp * Kp, 256);
        *ws_used = b_off + (uint64_t)s.batch * P * Np * Kp;
        const int64_t v16 = s.s24 ? 4 : 8;   // elements per 16 bytes
        EncPairParams ep{};
        EncParams& ea = ep.a;
        ea.s_src = s.sA; ea.s_dst = P * Mp * Kp;
        ea.M = (int32_t)s.M; ea.K = (int32_t)s.K;
        ea.Mp = (int32_t)Mp; ea.Kp = (int32_t)Kp;
        ea.ld_src = (int32_t)s.lda; ea.batch = (int32_t)s.batch;
        ea.vec = (s.lda % v16 == 0 && s.sA % v16 == 0) ? 1 : 0;
        EncParams& eb = ep.b;
        eb.s_src = s.sB; eb.s_dst = P * Np * Kp;
        eb.N = (int32_t)s.N; eb.K = (int32_t)s.K;
        eb.Np = (int32_t)Np; eb.Kp = (int32_t)Kp;
        eb.ld_src = (int32_t)s.ldb; eb.batch = (int32_t)s.batch;
        eb.vec = (s.ldb % 4 == 0 && s.sB % 4 == 0) ? 1 : 0;
        if (s.b_conv) {
            eb.conv = 1;
            eb.g = s.geo;
            eb.vec = 0;
        }
        LaunchRec r1;
        build_enc_limb(route, s.s24, ep, &r1);
        r1.bind(offsetof(EncPairParams, a) + offsetof(EncParams, src), s.a_bind);
        r1.bind(offsetof(EncPairParams, a) + offsetof(EncParams, dst), BIND_WS, a_off);
        r1.bind(offsetof(EncPairParams, b) + offsetof(EncParams, src), s.b_bind, s.b_ws_off);
        r1.bind(offsetof(EncPairParams, b) + offsetof(EncParams, dst), BIND_WS, b_off);
        if (offset) {
            r1.bind(offsetof(EncPairParams, a) + offsetof(EncParams, sums), BIND_WS, rs_off);
            r1.bind(offsetof(EncPairParams, b) + offsetof(EncParams, sums), BIND_WS, cs_off);
        }
        g.sA = P * Mp * Kp; g.sB = P * Np * Kp;
        g.lda = (int32_t)Kp; g.ldb = (int32_t)Kp;
        g.plane_a = Mp * Kp; g.plane_b = Np * Kp;
        LaunchRec r3;
        if (!build_gemm_i8nt(route, g, (int)s.batch, &r3))
            return fail(QX_ERR_UNSUPPORTED, "no kernel for route %d", route);
        r3.bind(offsetof(GemmParams, A), BIND_WS, a_off);
        r3.bind(offsetof(GemmParams, B), BIND_WS, b_off);
        r3.bind(offsetof(GemmParams, C), BIND_OUT);
        if (offset) {
            r3.bind(offsetof(GemmParams, rowsum), BIND_WS, rs_off);
            r3.bind(offsetof(GemmParams, colsum), BIND_WS, cs_off);
        }
        pl->launches.push_back(r1);
        pl->launches.push_back(r3);
        info.tile_m = bm; info.tile_n = bn; info.tile_k = 64;
        return QX_OK;
    }
    if (route == R_F16_EXACT) {
        const int64_t chunk = f16_chunk(s.ba, s.bb);
        g.chunk_tiles = chunk >= 64 ? (int32_t)(chunk / 64) : 0;
        info.chunk = chunk >= 64 ? (int32_t)(chunk / 64 * 64) : 16;
    }
    LaunchRec rec;
    int tm = 0, tn = 0, tk = 0;
    if (!build_gemm_mfma(route, g, (int)s.batch, &rec, &tm, &tn, &tk))
        return fail(QX_ERR_UNSUPPORTED, "no kernel for route %d", route);
    rec.bind(offsetof(GemmParams, A), s.a_bind);
    rec.bind(offsetof(GemmParams, B), s.b_bind, s.b_ws_off);
    rec.bind(offsetof(GemmParams, C), BIND_OUT);
    if (offset) {
        rec.bind(offsetof(GemmParams, rowsum), BIND_WS, rs_off);
        rec.bind(offsetof(GemmParams, colsum), BIND_WS, cs_off);
    }
    pl->launches.push_back(rec);
    info.tile_m = tm; info.tile_n = tn; info.tile_k = tk;
    return QX_OK;
}

void add_fill_out(Plan* pl, int64_t n32) {
    FillParams f{};
    f.n32 = n32;
    f.value = 0;
    LaunchRec rec;
    build_fill(f, &rec);
    rec.bind(offsetof(FillParams, ptr), BIND_OUT);
    pl->launches.push_back(rec);
}

qx_status check_dims(std::initializer_list<std::pair<const char*, int64_t>> dims) {
    for (auto& d : dims) {
        if (d.second < 0) return fail(QX_ERR_INVALID_ARG, "%s = %lld must be >= 0", d.first, (long long)d.second);
        if (d.second > kMaxDim)
            return fail(QX_ERR_UNSUPPORTED, "%s = %lld exceeds 2^30", d.first, (long long)d.second);
    }
    return QX_OK;
}

qx_status plan_gemm(Plan* pl, bool s24, int64_t M, int64_t N, int64_t K, int64_t batch, int32_t bound_a,
                    int32_t bound_b, int32_t route, bool allow_nt = true) {
    qx_status st = check_dims({{"M", M}, {"N", N}, {"K", K}, {"batch", batch}});
    if (st) return st;
    if (batch > kMaxBatch) return fail(QX_ERR_UNSUPPORTED, "batch = %lld exceeds 65535", (long long)batch);
    int64_t ba = 0, bb = 0;
    if (!s24) {
        if ((st = check_bound16(bound_a, "bound_a", &ba))) return st;
        if ((st = check_bound16(bound_b, "bound_b", &bb))) return st;
    }
    int64_t t;
    if (!mul_ok(M, K, (int64_t)1 << 40, &t) || !mul_ok(K, N, (int64_t)1 << 40, &t) ||
        !mul_ok(M, N, (int64_t)1 << 40, &t))
        return fail(QX_ERR_UNSUPPORTED, "matrix larger than 2^40 elements");
    int64_t total;
    if (!mul_ok(M * N, batch, (int64_t)1 << 42, &total) || !mul_ok(M * K, batch, (int64_t)1 << 42, &total) ||
        !mul_ok(K * N, batch, (int64_t)1 << 42, &total))
        return fail(QX_ERR_UNSUPPORTED, "batched operands larger than 2^42 elements");
    pl->op = s24 ? OP_GEMM_S24 : OP_GEMM_I16;
    pl->n_inputs = 2;
    pl->in_align = 16;
    if (route < 0 || route > R_ATTN_I32_VALU) return fail(QX_ERR_INVALID_ARG, "unknown route %d", route);
    // Route choice happens even for empty problems so that plan queries and
    // forced-route errors do not depend on the sizes.
    GemmSpec s{};
    s.M = M; s.N = N; s.K = K; s.batch = batch; s.ba = ba; s.bb = bb; s.s24 = s24; s.route = route;
    s.a_bind = BIND_IN0; s.b_bind = BIND_IN1; s.b_ws_off = 0;
    s.lda = K; s.ldb = N; s.ldc = N; s.sA = M * K; s.sB = K * N; s.sC = M * N;
    s.out_mode = OUT_ROWMAJOR; s.hw = 1;
    s.allow_nt = allow_nt;
    uint64_t ws = 0;
    Plan scratch;
    scratch.info = pl->info;
    if ((st = plan_int_gemm(s, &scratch, &ws))) return st;
    pl->info = scratch.info;
    if (M == 0 || N == 0 || batch == 0) {
        pl->launches.clear();
        pl->info.kernels = 0;
        pl->info.workspace_bytes = 0;
        return QX_OK;
    }
    if (K == 0) {
        add_fill_out(pl, M * N * batch);
        pl->info.kernels = 1;
        pl->info.workspace_bytes = 0;
        return QX_OK;
    }
    pl->launches = scratch.launches;
    if (!s24) {
        if (ba < 32768) pl->checks.push_back({0, 2, M * K * batch, (int32_t)ba});
        if (bb < 32768) pl->checks.push_back({1, 2, K * N * batch, (int32_t)bb});
    }
    pl->info.kernels = (int32_t)pl->launches.size();
    pl->info.workspace_bytes = (int64_t)ws;
    return QX_OK;
}

// Geometry shared by every convolution: validates the arguments and gives
// the output size and the GEMM view (Kd = C_in*KH*KW, P = N*Ho*Wo).
qx_status conv_shape(int64_t N, int64_t Ci, int64_t H, int64_t W, int64_t Co, int64_t KH, int64_t KW,
                     int64_t stride, int64_t pad, int64_t* Ho_, int64_t* Wo_, int64_t* Kd_, int64_t* P_) {
    qx_status st = check_dims({{"N", N}, {"C_in", Ci}, {"H", H}, {"W", W}, {"C_out", Co}, {"KH", KH},
                               {"KW", KW}, {"stride", stride}, {"pad", pad}});
    if (st) return st;
    if (stride < 1) return fail(QX_ERR_INVALID_ARG, "stride = %lld must be >= 1", (long long)stride);
    if (KH < 1 || KW < 1) return fail(QX_ERR_INVALID_ARG, "kernel size must be >= 1");
    const int64_t Ho = (H + 2 * pad - KH) >= 0 ? (H + 2 * pad - KH) / stride + 1 : 0;
    const int64_t Wo = (W + 2 * pad - KW) >= 0 ? (W + 2 * pad - KW) / stride + 1 : 0;
    if (Ho < 1 || Wo < 1)
        return fail(QX_ERR_INVALID_ARG, "kernel %lldx%lld larger than the padded %lldx%lld input", (long long)KH,
                    (long long)KW, (long long)(H + 2 * pad), (long long)(W + 2 * pad));
    int64_t Kd, P, t;
    if (!mul_ok(Ci, KH * KW, kMaxDim, &Kd) || !mul_ok(N, Ho * Wo, kMaxDim, &P) ||
        !mul_ok(Kd, P, (int64_t)1 << 40, &t) || !mul_ok(Co, P, (int64_t)1 << 40, &t))
        return fail(QX_ERR_UNSUPPORTED, "convolution too large");
    if (Kd > 65535) return fail(QX_ERR_UNSUPPORTED, "C_in*KH*KW = %lld exceeds 65535", (long long)Kd);
    *Ho_ = Ho; *Wo_ = Wo; *Kd_ = Kd; *P_ = P;
    return QX_OK;
}

qx_status plan_conv(Plan* pl, int64_t N, int64_t Ci, int64_t H, int64_t W, int64_t Co, int64_t KH, int64_t KW,
                    int64_t stride, int64_t pad, int32_t bound_x, int32_t bound_w, int32_t route) {
    int64_t Ho, Wo, Kd, P;
    qx_status st = conv_shape(N, Ci, H, W, Co, KH, KW, stride, pad, &Ho, &Wo, &Kd, &P);
    if (st) return st;
    int64_t ba, bb;
    if ((st = check_bound16(bound_w, "bound_w", &ba))) return st;
    if ((st = check_bound16(bound_x, "bound_x", &bb))) return st;
    if (route < 0 || route > R_ATTN_I32_VALU) return fail(QX_ERR_INVALID_ARG, "unknown route %d", route);
    pl->op = OP_CONV;
    pl->n_inputs = 2;
    pl->in_align = 16;
    // GEMM view: A = w [Co][Kd], B = col [Kd][P] in the workspace, C = y (NCHW scatter).
    GemmSpec s{};
    s.M = Co; s.N = P; s.K = Kd; s.batch = 1; s.ba = ba; s.bb = bb; s.s24 = false; s.route = route;
    s.a_bind = BIND_IN1; s.b_bind = BIND_WS; s.b_ws_off = 0;
    s.lda = Kd; s.ldb = P; s.ldc = P; s.sA = 0; s.sB = 0; s.sC = 0;
    s.out_mode = OUT_CONV; s.hw = (int32_t)(Ho * Wo);
    uint64_t ws = round_up(2 * (uint64_t)Kd * (uint64_t)P, 256);
    Plan g;
    g.info = pl->info;
    if ((st = plan_int_gemm(s, &g, &ws))) return st;
    pl->info = g.info;
    if (N == 0 || Co == 0) {
        pl->launches.clear();
        pl->info.kernels = 0;
        pl->info.workspace_bytes = 0;
        return QX_OK;
    }
    if (Ci == 0) {
        add_fill_out(pl, N * Co * Ho * Wo);
        pl->info.kernels = 1;
        pl->info.workspace_bytes = 0;
        return QX_OK;
    }
    if (bb < 32768) pl->checks.push_back({0, 2, N * Ci * H * W, (int32_t)bb});
    if (ba < 32768) pl->checks.push_back({1, 2, Co * Ci * KH * KW, (int32_t)ba});
    const int64_t Hp = H + 2 * pad, Wp = W + 2 * pad;
    const bool nt = use_nt(pl->info.route, f16_chunk(ba, bb), Co, P, Kd, 1);
    if (nt && Ci % 64 == 0 && 2 * N * Hp * Wp * Ci < ((int64_t)1 << 31)) {
        // fp16-exact, implicit lowering: one launch writes the zero-bordered
        // NHWC fp16 copy of x and the tap-major fp16 weights; the NT GEMM
        // gathers its B tiles from that copy and scatters y to NCHW.
        const int64_t chunk = f16_chunk(ba, bb);
        int bm, bn;
        nt_tile_shape(Co, P, 1, &bm, &bn);
        const int64_t Mp = pad_up(Co, bm);
        const uint64_t x_off = round_up(2 * (uint64_t)Mp * Kd, 256);
        const uint64_t wsz = x_off + 2 * (uint64_t)(N * Hp * Wp * Ci);
        const ConvGeom geo{(int32_t)Ci, (int32_t)H, (int32_t)W, (int32_t)KH, (int32_t)KW, (int32_t)stride,
                           (int32_t)pad, (int32_t)Ho, (int32_t)Wo};
        ConvPrepParams cp{};
        cp.nimg = (int32_t)N; cp.Co = (int32_t)Co; cp.Cop = (int32_t)Mp; cp.Kd = (int32_t)Kd;
        cp.elem_bytes = 2;
        cp.g = geo;
        LaunchRec r1;
        build_conv_prep(cp, &r1);
        r1.bind(offsetof(ConvPrepParams, x), BIND_IN0);
        r1.bind(offsetof(ConvPrepParams, w), BIND_IN1);
        r1.bind(offsetof(ConvPrepParams, xp), BIND_WS, x_off);
        r1.bind(offsetof(ConvPrepParams, w16), BIND_WS, 0);
        GemmParams gp{};
        gp.M = (int32_t)Co; gp.N = (int32_t)P; gp.K = (int32_t)Kd;
        gp.lda = (int32_t)Kd; gp.ldb = 0; gp.ldc = (int32_t)P;
        gp.out_mode = OUT_CONV; gp.hw = (int32_t)(Ho * Wo); gp.b_mode = B_NHWC;
        gp.chunk_tiles = (int32_t)(chunk / 64);
        gp.g = geo;
        LaunchRec r2;
        build_gemm_nt(gp, 1, &r2);
        r2.bind(offsetof(GemmParams, A), BIND_WS, 0);
        r2.bind(offsetof(GemmParams, B), BIND_WS, x_off);
        r2.bind(offsetof(GemmParams, C), BIND_OUT);
        pl->launches = {r1, r2};
        pl->info.chunk = (int32_t)(chunk / 64 * 64);
        pl->info.tile_m = bm; pl->info.tile_n = bn; pl->info.tile_k = 64;
        pl->info.kernels = 2;
        pl->info.workspace_bytes = (int64_t)wsz;
        return QX_OK;
    }
    if (nt) {
        // fp16-exact: weights encoded to fp16 [Mp][Kp], lowering written as
        // the transposed fp16 column matrix [Pp][Kp], then the NT GEMM with
        // an NCHW scatter epilogue.
        const int64_t chunk = f16_chunk(ba, bb);
        int bm, bn;
        nt_tile_shape(Co, P, 1, &bm, &bn);
        const int64_t Mp = pad_up(Co, bm), Pp = pad_up(P, bn), Kp = pad_up(Kd, 64);
        const uint64_t b_off = round_up(2 * (uint64_t)Mp * Kp, 256);
        const uint64_t wsz = b_off + 2 * (uint64_t)Pp * Kp;
        EncParams ea{};
        ea.s_src = 0; ea.s_dst = 0;
        ea.M = (int32_t)Co; ea.K = (int32_t)Kd; ea.Mp = (int32_t)Mp; ea.Kp = (int32_t)Kp;
        ea.ld_src = (int32_t)Kd; ea.batch = 1;
        ea.vec = Kd % 8 == 0 ? 1 : 0;
        LaunchRec r1;
        build_enc_a(ea, &r1);
        r1.bind(offsetof(EncParams, src), BIND_IN1);
        r1.bind(offsetof(EncParams, dst), BIND_WS, 0);
        Im2colTParams it{};
        it.P = (int32_t)P; it.Pp = (int32_t)Pp; it.Kd = (int32_t)Kd; it.Kp = (int32_t)Kp;
        it.g = ConvGeom{(int32_t)Ci, (int32_t)H, (int32_t)W, (int32_t)KH, (int32_t)KW, (int32_t)stride,
                        (int32_t)pad, (int32_t)Ho, (int32_t)Wo};
        LaunchRec r2;
        build_im2col_t(it, &r2);
        r2.bind(offsetof(Im2colTParams, x), BIND_IN0);
        r2.bind(offsetof(Im2colTParams, colT), BIND_WS, b_off);
        GemmParams gp{};
        gp.M = (int32_t)Co; gp.N = (int32_t)P; gp.K = (int32_t)Kp;
        gp.lda = (int32_t)Kp; gp.ldb = (int32_t)Kp; gp.ldc = (int32_t)P;
        gp.out_mode = OUT_CONV; gp.hw = (int32_t)(Ho * Wo); gp.b_mode = B_KN;
        gp.chunk_tiles = (int32_t)(chunk / 64);
        LaunchRec r3;
        build_gemm_nt(gp, 1, &r3);
        r3.bind(offsetof(GemmParams, A), BIND_WS, 0);
        r3.bind(offsetof(GemmParams, B), BIND_WS, b_off);
        r3.bind(offsetof(GemmParams, C), BIND_OUT);
        pl->launches = {r1, r2, r3};
        pl->info.chunk = (int32_t)(chunk / 64 * 64);
        pl->info.tile_m = bm; pl->info.tile_n = bn; pl->info.tile_k = 64;
        pl->info.kernels = 3;
        pl->info.workspace_bytes = (int64_t)wsz;
        return QX_OK;
    }
    Im2colParams ip{};
    ip.P = P;
    ip.Kd = (int32_t)Kd;
    ip.elem_bytes = 2;
    ip.g = ConvGeom{(int32_t)Ci, (int32_t)H, (int32_t)W, (int32_t)KH, (int32_t)KW, (int32_t)stride, (int32_t)pad,
                    (int32_t)Ho, (int32_t)Wo};
    LaunchRec rec;
    build_im2col(ip, &rec);
    rec.bind(offsetof(Im2colParams, x), BIND_IN0);
    rec.bind(offsetof(Im2colParams, col), BIND_WS, 0);
    pl->launches.push_back(rec);
    for (auto& r : g.launches) pl->launches.push_back(r);
    pl->info.kernels = (int32_t)pl->launches.size();
    pl->info.workspace_bytes = (int64_t)ws;
    return QX_OK;
}

// Conv2D on FP32 or INT32 (smul24 contract) operands (Table 2, Conv2D FP32
// and INT32 rows): the same lowering onto the FP32 and smul24 GEMMs.
qx_status plan_conv_t(Plan* pl, int32_t dt, int64_t N, int64_t Ci, int64_t H, int64_t W, int64_t Co,
                      int64_t KH, int64_t KW, int64_t stride, int64_t pad, int32_t route) {
    int64_t Ho, Wo, Kd, P;
    qx_status st = conv_shape(N, Ci, H, W, Co, KH, KW, stride, pad, &Ho, &Wo, &Kd, &P);
    if (st) return st;
    if (dt != QX_DT_F32 && dt != QX_DT_I32) return fail(QX_ERR_INVALID_ARG, "unknown dtype %d", (int)dt);
    pl->op = dt == QX_DT_F32 ? OP_CONV_F32 : OP_CONV_I32;
    pl->n_inputs = 2;
    pl->in_align = 16;
    qx_plan_info& info = pl->info;
    const int64_t Hp = H + 2 * pad, Wp = W + 2 * pad;
    const ConvGeom geo{(int32_t)Ci, (int32_t)H, (int32_t)W, (int32_t)KH, (int32_t)KW, (int32_t)stride,
                       (int32_t)pad, (int32_t)Ho, (int32_t)Wo};
    if (dt == QX_DT_F32) {
        const bool mfma_ok = Ci % 32 == 0 && 4 * N * Hp * Wp * Ci < ((int64_t)1 << 31);
        int32_t r = route == R_AUTO ? (mfma_ok ? R_F32_MFMA : R_F32_VALU) : route;
        if (r != R_F32_MFMA && r != R_F32_VALU)
            return fail(QX_ERR_INVALID_ARG, "route %d does not apply to an FP32 convolution", route);
        if (r == R_F32_MFMA && !mfma_ok)
            return fail(QX_ERR_UNSUPPORTED, "the fp32 MFMA convolution needs C_in a multiple of 32");
        info.route = r;
        info.products = 1;
        info.chunk = 0;
        info.exact_no_wrap = 0;
        if (N == 0 || Co == 0) {
            info.kernels = 0;
            info.workspace_bytes = 0;
            return QX_OK;
        }
        if (Ci == 0) {
            add_fill_out(pl, N * Co * Ho * Wo);
            info.kernels = 1;
            info.workspace_bytes = 0;
            return QX_OK;
        }
        if (r == R_F32_MFMA) {
            // bordered NHWC fp32 image + tap-major weights, then the gathering
            // fp32 NT GEMM with an NCHW scatter
            int bm, bn;
            nt_tile_shape(Co, P, 1, &bm, &bn);
            const int64_t Mp = pad_up(Co, bm);
            const uint64_t x_off = round_up(4 * (uint64_t)Mp * Kd, 256);
            ConvPrepParams cp{};
            cp.nimg = (int32_t)N; cp.Co = (int32_t)Co; cp.Cop = (int32_t)Mp; cp.Kd = (int32_t)Kd;
            cp.elem_bytes = 4;
            cp.g = geo;
            LaunchRec r1;
            build_conv_prep(cp, &r1);
            r1.bind(offsetof(ConvPrepParams, x), BIND_IN0);
            r1.bind(offsetof(ConvPrepParams, w), BIND_IN1);
            r1.bind(offsetof(ConvPrepParams, xp), BIND_WS, x_off);
            r1.bind(offsetof(ConvPrepParams, w16), BIND_WS, 0);
            GemmParams gp{};
            gp.M = (int32_t)Co; gp.N = (int32_t)P; gp.K = (int32_t)Kd;
            gp.lda = (int32_t)Kd; gp.ldb = 0; gp.ldc = (int32_t)P;
            gp.out_mode = OUT_CONV; gp.hw = (int32_t)(Ho * Wo); gp.b_mode = B_NHWC;
            gp.g = geo;
            LaunchRec r2;
            build_gemm_nt_f32(gp, 1, &r2);
            r2.bind(offsetof(GemmParams, A), BIND_WS, 0);
            r2.bind(offsetof(GemmParams, B), BIND_WS, x_off);
            r2.bind(offsetof(GemmParams, C), BIND_OUT);
            pl->launches = {r1, r2};
            info.tile_m = bm; info.tile_n = bn; info.tile_k = 32;
            info.kernels = 2;
            info.workspace_bytes = (int64_t)(x_off + 4 * (uint64_t)(N * Hp * Wp * Ci));
            return QX_OK;
        }
        // explicit lowering col [Kd][P] fp32, then the vector-ALU fp32 GEMM
        if ((Co + 63) / 64 > 65535) return fail(QX_ERR_UNSUPPORTED, "C_out too large for the VALU route");
        Im2colParams ip{};
        ip.P = P; ip.Kd = (int32_t)Kd; ip.elem_bytes = 4; ip.g = geo;
        LaunchRec r1;
        build_im2col(ip, &r1);
        r1.bind(offsetof(Im2colParams, x), BIND_IN0);
        r1.bind(offsetof(Im2colParams, col), BIND_WS, 0);
        ValuGemmParams v{};
        v.M = (int32_t)Co; v.N = (int32_t)P; v.K = (int32_t)Kd;
        v.lda = (int32_t)Kd; v.ldb = (int32_t)P; v.ldc = (int32_t)P; v.b_trans = 0;
        v.out_mode = OUT_CONV; v.hw = (int32_t)(Ho * Wo);
        LaunchRec r2;
        build_valu_gemm(VK_F32, v, 1, &r2);
        r2.bind(offsetof(ValuGemmParams, A), BIND_IN1);
        r2.bind(offsetof(ValuGemmParams, B), BIND_WS, 0);
        r2.bind(offsetof(ValuGemmParams, C), BIND_OUT);
        pl->launches = {r1, r2};
        info.tile_m = 64; info.tile_n = 64; info.tile_k = 16;
        info.kernels = 2;
        info.workspace_bytes = (int64_t)(4 * (uint64_t)Kd * (uint64_t)P);
        return QX_OK;
    }
    // INT32 under smul24.  Large problems: the limb-plane encoder gathers the
    // im2col columns straight from x, then the NT int8 contraction.  Small
    // ones: explicit lowering col [Kd][P] int32, then the smul24 GEMM.
    if (route < 0 || route > R_F32_VALU) return fail(QX_ERR_INVALID_ARG, "unknown route %d", route);
    const bool gather = (route == R_AUTO || route == R_S24_I8LIMB) && use_i8nt(R_S24_I8LIMB, Co, P, Kd, 1);
    // few output channels: a direct vector-ALU kernel (a GEMM tile would be
    // mostly empty)
    const bool direct = Co <= 16 && Kd <= 1024 && KW <= 8 && (route == R_S24_VALU || (route == R_AUTO && !gather));
    if (direct) {
        info.route = R_S24_VALU;
        info.products = 1;
        info.chunk = 0;
        info.exact_no_wrap = 0;
        info.workspace_bytes = 0;
        if (N == 0 || Co == 0) {
            info.kernels = 0;
            return QX_OK;
        }
        if (Ci == 0) {
            add_fill_out(pl, N * Co * Ho * Wo);
            info.kernels = 1;
            return QX_OK;
        }
        ConvDirectParams cd{};
        cd.P = P; cd.Co = (int32_t)Co; cd.Kd = (int32_t)Kd; cd.g = geo;
        LaunchRec r;
        build_conv_direct_s24(cd, &r);
        r.bind(offsetof(ConvDirectParams, x), BIND_IN0);
        r.bind(offsetof(ConvDirectParams, w), BIND_IN1);
        r.bind(offsetof(ConvDirectParams, y), BIND_OUT);
        pl->launches = {r};
        info.kernels = 1;
        info.tile_m = 1; info.tile_n = 256; info.tile_k = 1;
        return QX_OK;
    }
    GemmSpec s{};
    s.M = Co; s.N = P; s.K = Kd; s.batch = 1; s.s24 = true; s.route = route;
    s.a_bind = BIND_IN1; s.b_bind = gather ? BIND_IN0 : BIND_WS; s.b_ws_off = 0;
    s.lda = Kd; s.ldb = P; s.ldc = P; s.sA = 0; s.sB = 0; s.sC = 0;
    s.out_mode = OUT_CONV; s.hw = (int32_t)(Ho * Wo);
    s.allow_nt = true;
    s.b_conv = gather;
    s.geo = geo;
    uint64_t ws = gather ? 0 : round_up(4 * (uint64_t)Kd * (uint64_t)P, 256);
    Plan g;
    g.info = pl->info;
    if ((st = plan_int_gemm(s, &g, &ws))) return st;
    pl->info = g.info;
    if (N == 0 || Co == 0) {
        pl->launches.clear();
        pl->info.kernels = 0;
        pl->info.workspace_bytes = 0;
        return QX_OK;
    }
    if (Ci == 0) {
        add_fill_out(pl, N * Co * Ho * Wo);
        pl->info.kernels = 1;
        pl->info.workspace_bytes = 0;
        return QX_OK;
    }
    if (!gather) {
        Im2colParams ip{};
        ip.P = P; ip.Kd = (int32_t)Kd; ip.elem_bytes = 4; ip.g = geo;
        LaunchRec rec;
        build_im2col(ip, &rec);
        rec.bind(offsetof(Im2colParams, x), BIND_IN0);
        rec.bind(offsetof(Im2colParams, col), BIND_WS, 0);
        pl->launches.push_back(rec);
    }
    for (auto& r : g.launches) pl->launches.push_back(r);
    pl->info.kernels = (int32_t)pl->launches.size();
    pl->info.workspace_bytes = (int64_t)ws;
    return QX_OK;
}

// Min/max over n >= 1 int32 or int16 values (Table 2, Min/max rows).
qx_status plan_minmax(Plan* pl, int64_t n, int32_t elem_bytes) {
    if (elem_bytes != 2 && elem_bytes != 4) return fail(QX_ERR_INVALID_ARG, "elem_bytes = %d must be 2 or 4", elem_bytes);
    if (n < 1) return fail(QX_ERR_INVALID_ARG, "min/max needs n >= 1 (n = %lld)", (long long)n);
    if (n > ((int64_t)1 << 40)) return fail(QX_ERR_UNSUPPORTED, "n = %lld exceeds 2^40", (long long)n);
    pl->op = OP_MINMAX;
    pl->n_inputs = 1;
    pl->in_align = 16;
    pl->out_align = (uint64_t)elem_bytes;
    MinMaxParams m{};
    m.n = n;
    m.elem_bytes = elem_bytes;
    minmax_blocks(n, &m.blocks, &m.per);
    LaunchRec r1, r2;
    build_minmax(m, &r1, &r2);
    r1.bind(offsetof(MinMaxParams, x), BIND_IN0);
    r1.bind(offsetof(MinMaxParams, part), BIND_WS, 0);
    r2.bind(offsetof(MinMaxParams, part), BIND_WS, 0);
    r2.bind(offsetof(MinMaxParams, out), BIND_OUT);
    pl->launches = {r1, r2};
    qx_plan_info& info = pl->info;
    info.route = R_AUTO;
    info.kernels = 2;
    info.workspace_bytes = 8 * (int64_t)m.blocks;
    info.tile_m = 1; info.tile_n = (int32_t)std::min<int64_t>(m.per, INT32_MAX); info.tile_k = 1;
    return QX_OK;
}

// 2x2 / stride 2 pooling of NCHW tensors (Table 2, AvgPool INT32 and MaxPool
// FP32 rows): y [N][C][H/2][W/2].
qx_status plan_pool2(Plan* pl, int32_t kind, int64_t N, int64_t C, int64_t H, int64_t W) {
    if (kind != POOL_AVG_I32 && kind != POOL_MAX_F32) return fail(QX_ERR_INVALID_ARG, "unknown pool kind %d", kind);
    qx_status st = check_dims({{"N", N}, {"C", C}, {"H", H}, {"W", W}});
    if (st) return st;
    int64_t nc, t;
    if (!mul_ok(N, C, kMaxDim, &nc) || !mul_ok(nc * H, W, (int64_t)1 << 40, &t))
        return fail(QX_ERR_UNSUPPORTED, "tensor larger than 2^40 elements");
    pl->op = OP_POOL;
    pl->n_inputs = 1;
    pl->in_align = 16;
    const int64_t Ho = H / 2, Wo = W / 2;
    qx_plan_info& info = pl->info;
    info.route = R_AUTO;
    info.workspace_bytes = 0;
    if (nc == 0 || Ho == 0 || Wo == 0) {
        info.kernels = 0;
        return QX_OK;
    }
    PoolParams pp{};
    pp.NC = nc; pp.H = (int32_t)H; pp.W = (int32_t)W; pp.Ho = (int32_t)Ho; pp.Wo = (int32_t)Wo;
    pp.vec = W % 8 == 0 ? 1 : 0;
    pl->out_align = pp.vec ? 16 : 4;
    LaunchRec r;
    build_pool2(kind, pp, &r);
    r.bind(offsetof(PoolParams, x), BIND_IN0);
    r.bind(offsetof(PoolParams, y), BIND_OUT);
    pl->launches = {r};
    info.kernels = 1;
    info.tile_m = 2; info.tile_n = 8; info.tile_k = 1;
    return QX_OK;
}

// Where a sub-plan's input or output binding goes when plans are chained.
struct Target {
    Bind bind;
    uint64_t add;
};

// Appends the launches of sub-plan sp to pl: its workspace moves to
// [base, base + its size) of pl's workspace, its inputs and output are
// rebound to the given targets.
void append_plan(Plan* pl, const Plan& sp, uint64_t base, std::initializer_list<Target> ins, Target out) {
    const Target* in = ins.begin();
    for (const LaunchRec& r0 : sp.launches) {
        LaunchRec r = r0;
        for (int i = 0; i < r.nslots; ++i) {
            Slot& sl = r.slots[i];
            if (sl.bind == BIND_WS) {
                sl.add += base;
            } else if (sl.bind == BIND_OUT) {
                sl.bind = out.bind;
                sl.add += out.add;
            } else {
                sl.add += in[sl.bind].add;
                sl.bind = in[sl.bind].bind;
            }
        }
        pl->launches.push_back(r);
    }
}

// LeNet-5-shaped INT32 pipeline (Results: end-to-end CNN on the substrate),
// every layer an executor-planned operator of this library, chained on one
// stream through the workspace:
//   x [B][1][32][32] -> conv 6@5x5 -> ReLU -> 2x2 avg -> conv 16@5x5 -> ReLU
//   -> 2x2 avg -> [B][400] -> FC 120 -> ReLU -> FC 84 -> ReLU -> FC 10.
// Convolutions and FC layers are INT32 under the smul24 contract (each
// operand word read as sext24, results mod 2^32); the pools are the INT32
// floor average of the ReLU'd values.  Inputs: x, w1 [6][1][5][5],
// w2 [16][6][5][5], f1 [400][120], f2 [120][84], f3 [84][10]; output [B][10].
qx_status plan_lenet(Plan* pl, int64_t B) {
    qx_status st = check_dims({{"batch", B}});
    if (st) return st;
    if (B > (1 << 20)) return fail(QX_ERR_UNSUPPORTED, "batch = %lld exceeds 2^20", (long long)B);
    pl->op = OP_LENET;
    pl->n_inputs = 6;
    pl->in_align = 16;
    qx_plan_info& info = pl->info;
    info.route = R_S24_I8LIMB;
    info.products = products_of(R_S24_I8LIMB);
    info.exact_no_wrap = 0;
    if (B == 0) {
        info.kernels = 0;
        info.workspace_bytes = 0;
        return QX_OK;
    }
    uint64_t off = 0;
    auto take = [&](uint64_t bytes) {
        const uint64_t o = round_up(off, 256);
        off = o + bytes;
        return o;
    };
    const uint64_t o_p1 = take(4 * (uint64_t)B * 6 * 14 * 14), o_p2 = take(4 * (uint64_t)B * 400);
    const uint64_t o_h1 = take(4 * (uint64_t)B * 120), o_h2 = take(4 * (uint64_t)B * 84);
    auto sub = [&](Plan& sp, std::initializer_list<Target> ins, Target out) -> qx_status {
        append_plan(pl, sp, take((uint64_t)sp.info.workspace_bytes), ins, out);
        return QX_OK;
    };
    auto pool = [&](uint64_t from, uint64_t to, int64_t C, int32_t H) {
        PoolParams pp{};
        pp.NC = B * C; pp.H = H; pp.W = H; pp.Ho = H / 2; pp.Wo = H / 2;
        pp.vec = H % 8 == 0 ? 1 : 0;
        pp.relu = 1;
        LaunchRec r;
        build_pool2(POOL_AVG_I32, pp, &r);
        r.bind(offsetof(PoolParams, x), BIND_WS, from);
        r.bind(offsetof(PoolParams, y), BIND_WS, to);
        pl->launches.push_back(r);
    };
    // conv 5x5 (smul24, few output channels: the direct kernel), ReLU and the
    // 2x2 average pool into the workspace: one launch (one thread per pooled
    // pixel) when an image fits the kernel's LDS, else the conv and the pool
    // as two launches.  The second conv at batch 4096 fused: 48.8 us against
    // 49.6 + 11.5 (the grid is smaller, 1.6 waves per SIMD, but its busiest
    // CUs carry the same work and the conv map never reaches HBM).
    auto conv_pool = [&](Target x, Bind w, uint64_t to, int64_t Ci, int32_t H, int64_t Co) {
        const int32_t Ho = H - 4;
        ConvDirectParams cd{};
        cd.P = B * Ho * Ho; cd.Co = (int32_t)Co; cd.Kd = (int32_t)(Ci * 25);
        cd.g = ConvGeom{(int32_t)Ci, H, H, 5, 5, 1, 0, Ho, Ho};
        const bool fuse = conv_pool_images(cd) > 0;
        cd.pool = fuse ? 1 : 0;
        const uint64_t y = fuse ? to : take(4 * (uint64_t)B * Co * Ho * Ho);
        LaunchRec r;
        build_conv_direct_s24(cd, &r);
        r.bind(offsetof(ConvDirectParams, x), x.bind, x.add);
        r.bind(offsetof(ConvDirectParams, w), w);
        r.bind(offsetof(ConvDirectParams, y), BIND_WS, y);
        pl->launches.push_back(r);
        if (!fuse) pool(y, to, Co, Ho);
    };
    // ReLU after a fully connected layer: folded into the stores of the
    // layer's last launch when that is the int8 NT contraction (K not
    // sliced) or the skinny vector-ALU kernel, else a launch of its own
    auto relu = [&](uint64_t at, int64_t n) {
        LaunchRec& last = pl->launches.back();
        if (strcmp(last.name, "valu_s24_skinny") == 0) {
            ValuGemmParams vp;
            memcpy(&vp, last.blob, sizeof(vp));
            vp.relu = 1;
            memcpy(last.blob, &vp, sizeof(vp));
            return;
        }
        if (strncmp(last.name, "gemm_i8nt_", 10) == 0) {
            GemmParams gp;
            memcpy(&gp, last.blob, sizeof(gp));
            if (gp.ksplit <= 1) {
                gp.relu = 1;
                memcpy(last.blob, &gp, sizeof(gp));
                return;
            }
        }
        ReluParams rp{};
        rp.n = n;
        LaunchRec r;
        build_relu(rp, &r);
        r.bind(offsetof(ReluParams, p), BIND_WS, at);
        pl->launches.push_back(r);
    };
    Plan g1, g2, g3;
    conv_pool({BIND_IN0, 0}, BIND_IN1, o_p1, 1, 32, 6);
    conv_pool({BIND_WS, o_p1}, BIND_IN2, o_p2, 6, 14, 16);
    if ((st = plan_gemm(&g1, true, B, 120, 400, 1, 0, 0, R_AUTO))) return st;
    if ((st = sub(g1, {{BIND_WS, o_p2}, {BIND_IN3, 0}}, {BIND_WS, o_h1}))) return st;
    relu(o_h1, B * 120);
    if ((st = plan_gemm(&g2, true, B, 84, 120, 1, 0, 0, R_AUTO))) return st;
    if ((st = sub(g2, {{BIND_WS, o_h1}, {BIND_IN4, 0}}, {BIND_WS, o_h2}))) return st;
    relu(o_h2, B * 84);
    if ((st = plan_gemm(&g3, true, B, 10, 84, 1, 0, 0, R_AUTO))) return st;
    if ((st = sub(g3, {{BIND_WS, o_h2}, {BIND_IN5, 0}}, {BIND_OUT, 0}))) return st;
    info.kernels = (int32_t)pl->launches.size();
    info.workspace_bytes = (int64_t)round_up(off, 256);
    info.tile_m = info.tile_n = info.tile_k = 0;
    return QX_OK;
}

// Query tiles of 32 per workgroup of the streaming INT32 attention core
// (eight waves: qt query tiles x 8/qt key parts).  At L = 4096, d = 64 two
// tiles (64 queries x 4 splits of 1024 keys) measured best: four (8
// splits) doubled the wrapping atomics that join the splits, and one (2
// splits of 2048 keys) doubled each workgroup's key traffic and left its
// LDS ring one pair deep.
static int attn_stream_qt(int64_t L) {
    (void)L;
    return 2;
}

qx_status plan_attn(Plan* pl, int32_t dt, int64_t L, int64_t d, int32_t bound, int32_t route) {
    qx_status st = check_dims({{"L", L}, {"d", d}});
    if (st) return st;
    if (dt != QX_DT_F32 && dt != QX_DT_I32) return fail(QX_ERR_INVALID_ARG, "unknown attention dtype %d", (int)dt);
    if (d > 256) return fail(QX_ERR_UNSUPPORTED, "d = %lld exceeds 256", (long long)d);
    if (L > (1 << 20)) return fail(QX_ERR_UNSUPPORTED, "L = %lld exceeds 2^20", (long long)L);
    if (bound < 0) return fail(QX_ERR_INVALID_ARG, "bound = %d must be >= 0", bound);
    pl->op = dt == QX_DT_F32 ? OP_ATTN_F32 : OP_ATTN_I32;
    pl->n_inputs = 3;
    pl->in_align = 16;
    qx_plan_info& info = pl->info;
    const bool mfma_shape = d >= 32 && d <= 128 && d % 32 == 0;
    int32_t r = route;
    if (dt == QX_DT_F32) {
        if (r == R_AUTO) r = mfma_shape ? R_ATTN_F32_MFMA : R_ATTN_F32_VALU;
        if (r != R_ATTN_F32_MFMA && r != R_ATTN_F32_VALU)
            return fail(QX_ERR_INVALID_ARG, "route %d does not apply to FP32 attention", route);
        if (r == R_ATTN_F32_MFMA && !mfma_shape)
            return fail(QX_ERR_UNSUPPORTED, "fp32 MFMA attention needs d in {32, 64, 96, 128}");
        info.exact_no_wrap = 0;
    } else {
        const int64_t b = bound == 0 ? ((int64_t)1 << 31) : bound;
        const bool in8 = b <= 127 && (double)d * (double)b * (double)b < 8388608.0;
        if (r == R_AUTO) r = (mfma_shape && in8) ? R_ATTN_I32_MFMA : R_ATTN_I32_VALU;
        if (r != R_ATTN_I32_MFMA && r != R_ATTN_I32_VALU)
            return fail(QX_ERR_INVALID_ARG, "route %d does not apply to INT32 attention", route);
        if (r == R_ATTN_I32_MFMA && !in8)
            return fail(QX_ERR_RANGE, "int8 attention needs bound <= 127 and d*bound^2 < 2^23");
        if (r == R_ATTN_I32_MFMA && !mfma_shape)
            return fail(QX_ERR_UNSUPPORTED, "int8 MFMA attention needs d in {32, 64, 96, 128}");
        info.exact_no_wrap = ((double)L * (double)d * (double)b * (double)b * (double)b < 2147483648.0) ? 1 : 0;
    }
    info.route = r;
    info.products = r == R_ATTN_I32_MFMA ? 3 : 1;
    info.chunk = 0;
    if (L == 0 || d == 0) {
        info.kernels = 0;
        info.workspace_bytes = 0;
        return QX_OK;
    }
    if (dt == QX_DT_I32 && bound > 0)
        for (int i = 0; i < 3; ++i) pl->checks.push_back({i, 4, L * d, bound});
    uint64_t ws = 0;
    if (r == R_ATTN_F32_VALU || r == R_ATTN_I32_VALU) {
        // S = Q K^T into the workspace, then O = S V, both on the vector ALU.
        const int kind = r == R_ATTN_F32_VALU ? VK_F32 : VK_I32;
        int64_t ss;
        if (!mul_ok(L, L, (int64_t)1 << 34, &ss) || (L + 63) / 64 > 65535)
            return fail(QX_ERR_UNSUPPORTED, "L too large for the VALU route");
        ws = 4 * (uint64_t)ss;
        ValuGemmParams v{};
        v.M = (int32_t)L; v.N = (int32_t)L; v.K = (int32_t)d;
        v.lda = (int32_t)d; v.ldb = (int32_t)d; v.ldc = (int32_t)L; v.b_trans = 1; v.out_mode = OUT_ROWMAJOR;
        LaunchRec r1;
        build_valu_gemm(kind, v, 1, &r1);
        r1.bind(offsetof(ValuGemmParams, A), BIND_IN0);
        r1.bind(offsetof(ValuGemmParams, B), BIND_IN1);
        r1.bind(offsetof(ValuGemmParams, C), BIND_WS, 0);
        ValuGemmParams v2{};
        v2.M = (int32_t)L; v2.N = (int32_t)d; v2.K = (int32_t)L;
        v2.lda = (int32_t)L; v2.ldb = (int32_t)d; v2.ldc = (int32_t)d; v2.b_trans = 0; v2.out_mode = OUT_ROWMAJOR;
        LaunchRec r2;
        build_valu_gemm(kind, v2, 1, &r2);
        r2.bind(offsetof(ValuGemmParams, A), BIND_WS, 0);
        r2.bind(offsetof(ValuGemmParams, B), BIND_IN2);
        r2.bind(offsetof(ValuGemmParams, C), BIND_OUT);
        pl->launches.push_back(r1);
        pl->launches.push_back(r2);
        info.tile_m = 64; info.tile_n = 64; info.tile_k = 16;
    } else {
        // Key splits: enough workgroups for one per CU (>= 256), split
        // boundaries on 32-key blocks.  Twice that many (shorter splits)
        // measured 10% slower on L = 4096, d = 64 (more per-workgroup
        // set-up and more partial outputs to combine); half as many left
        // CUs idle (FP32 1.6x slower).
        const bool stream = r == R_ATTN_I32_MFMA && (d == 32 || d == 64);
        const int qt = stream ? attn_stream_qt(L) : 4;       // query tiles of 32 per workgroup
        const int64_t qgroups = (L + 32 * qt - 1) / (32 * qt);
        const int64_t kblocks = (L + 31) / 32;
        int64_t splits = std::min<int64_t>(std::max<int64_t>((256 + qgroups - 1) / qgroups, 1), kblocks);
        int64_t kps = ((kblocks + splits - 1) / splits) * 32;
        if (stream) {
            // streaming kernel: each split is 8 / qt key parts of an even
            // number of whole 32-key blocks
            const int64_t g = 64 * (8 / qt);
            kps = (kps + g - 1) / g * g;
        } else if (r == R_ATTN_I32_MFMA && d == 128) {
            // resident splits: kps * d a multiple of 4096 (whole 1 KB loads
            // per wave) and both int8 tiles within 48 KiB of LDS
            const int64_t g = std::max<int64_t>(32, 4096 / d), cap = 24576 / d / g * g;
            kps = std::min((kps + g - 1) / g * g, cap);
        }
        splits = (L + kps - 1) / kps;
        AttnParams a{};
        a.L = (int32_t)L; a.d = (int32_t)d; a.splits = (int32_t)splits; a.keys_per_split = (int32_t)kps;
        a.limbs = 3;
        a.qt = qt;
        LaunchRec rec;
        if (r == R_ATTN_F32_MFMA) {
            build_attn_f32(a, &rec);
            rec.bind(offsetof(AttnParams, Q), BIND_IN0);
            rec.bind(offsetof(AttnParams, K), BIND_IN1);
            rec.bind(offsetof(AttnParams, V), BIND_IN2);
            rec.bind(offsetof(AttnParams, O), BIND_OUT);
            if (splits > 1) {
                ws = 4 * (uint64_t)splits * (uint64_t)L * (uint64_t)d;
                rec.bind(offsetof(AttnParams, part), BIND_WS, 0);
                pl->launches.push_back(rec);
                ReduceParams rp{};
                rp.n = L * d;
                rp.splits = (int32_t)splits;
                LaunchRec rr;
                build_reduce(rp, &rr);
                rr.bind(offsetof(ReduceParams, part), BIND_WS, 0);
                rr.bind(offsetof(ReduceParams, out), BIND_OUT);
                pl->launches.push_back(rr);
            } else {
                pl->launches.push_back(rec);
            }
        } else if (stream) {
            // prep: int8 K rows and block-major int8 V in the workspace, O
            // cleared for split accumulation; then eight waves per
            // workgroup stream their keys from them (no LDS staging)
            a.Lp = (int32_t)(splits * kps);
            a.clear_o = splits > 1 ? 1 : 0;
            a.v_blocks = 1;
            a.prep_k = (int64_t)a.Lp * d / 16;
            a.prep_v = d * (int64_t)a.Lp / 16;
            a.prep_q = L * d / 16;
            const uint64_t v8_off = round_up((uint64_t)a.Lp * (uint64_t)d, 256);
            const uint64_t q8_off = round_up(v8_off + (uint64_t)a.Lp * (uint64_t)d, 256);
            ws = q8_off + (uint64_t)L * (uint64_t)d;
            LaunchRec r1;
            build_attn_i32_prep(a, &r1);
            r1.bind(offsetof(AttnParams, Q), BIND_IN0);
            r1.bind(offsetof(AttnParams, K), BIND_IN1);
            r1.bind(offsetof(AttnParams, V), BIND_IN2);
            r1.bind(offsetof(AttnParams, O), BIND_OUT);
            r1.bind(offsetof(AttnParams, k8), BIND_WS, 0);
            r1.bind(offsetof(AttnParams, v8), BIND_WS, v8_off);
            r1.bind(offsetof(AttnParams, q8), BIND_WS, q8_off);
            pl->launches.push_back(r1);
            if (!build_attn_i32s(a, &rec)) return fail(QX_ERR_UNSUPPORTED, "no streaming attention kernel");
            rec.bind(offsetof(AttnParams, O), BIND_OUT);
            rec.bind(offsetof(AttnParams, k8), BIND_WS, 0);
            rec.bind(offsetof(AttnParams, v8), BIND_WS, v8_off);
            rec.bind(offsetof(AttnParams, q8), BIND_WS, q8_off);
            pl->launches.push_back(rec);
        } else if (resident_attn_i32(d, kps)) {
            // prep: int8 K rows and reordered V^T rows in the workspace, O
            // cleared for split accumulation; then every workgroup loads its
            // whole key split into LDS once (and forms the V column sums of
            // the offset correction from it)
            a.Lp = (int32_t)(splits * kps);
            a.clear_o = splits > 1 ? 1 : 0;
            a.prep_k = (int64_t)a.Lp * d / 16;
            a.prep_v = d * (int64_t)a.Lp / 16;
            const uint64_t v8_off = round_up((uint64_t)a.Lp * (uint64_t)d, 256);
            ws = v8_off + (uint64_t)a.Lp * (uint64_t)d;
            LaunchRec r1;
            build_attn_i32_prep(a, &r1);
            r1.bind(offsetof(AttnParams, K), BIND_IN1);
            r1.bind(offsetof(AttnParams, V), BIND_IN2);
            r1.bind(offsetof(AttnParams, O), BIND_OUT);
            r1.bind(offsetof(AttnParams, k8), BIND_WS, 0);
            r1.bind(offsetof(AttnParams, v8), BIND_WS, v8_off);
            pl->launches.push_back(r1);
            build_attn_i32r(a, &rec);
            rec.bind(offsetof(AttnParams, Q), BIND_IN0);
            rec.bind(offsetof(AttnParams, O), BIND_OUT);
            rec.bind(offsetof(AttnParams, k8), BIND_WS, 0);
            rec.bind(offsetof(AttnParams, v8), BIND_WS, v8_off);
            pl->launches.push_back(rec);
        } else {
            // the output cleared for split accumulation, then the kernel
            // (which also forms the V column sums of the offset correction)
            if (splits > 1) add_fill_out(pl, L * d);
            build_attn_i32(a, &rec);
            rec.bind(offsetof(AttnParams, Q), BIND_IN0);
            rec.bind(offsetof(AttnParams, K), BIND_IN1);
            rec.bind(offsetof(AttnParams, V), BIND_IN2);
            rec.bind(offsetof(AttnParams, O), BIND_OUT);
            pl->launches.push_back(rec);
        }
        info.tile_m = 128; info.tile_n = (int32_t)d; info.tile_k = (int32_t)kps;
    }
    info.kernels = (int32_t)pl->launches.size();
    info.workspace_bytes = (int64_t)ws;
    return QX_OK;
}

qx_status plan_sdpa(Plan* pl, int64_t BH, int64_t L, int64_t d, float scale, int32_t causal) {
    qx_status st = check_dims({{"BH", BH}, {"L", L}, {"d", d}});
    if (st) return st;
    if (d > 128) return fail(QX_ERR_UNSUPPORTED, "d = %lld exceeds 128", (long long)d);
    if (L > (1 << 20)) return fail(QX_ERR_UNSUPPORTED, "L = %lld exceeds 2^20", (long long)L);
    if (BH > 65535) return fail(QX_ERR_UNSUPPORTED, "BH = %lld exceeds 65535", (long long)BH);
    if (!std::isfinite(scale)) return fail(QX_ERR_INVALID_ARG, "scale must be finite");
    if (causal != 0 && causal != 1) return fail(QX_ERR_INVALID_ARG, "causal = %d must be 0 or 1", causal);
    int64_t n;
    if (!mul_ok(BH, L, (int64_t)1 << 40, &n) || !mul_ok(n, d, (int64_t)1 << 34, &n))
        return fail(QX_ERR_UNSUPPORTED, "BH*L*d exceeds 2^34");
    pl->op = OP_SDPA;
    pl->n_inputs = 3;
    pl->in_align = d % 32 == 0 ? 16 : 4;
    qx_plan_info& info = pl->info;
    info.route = R_ATTN_F32_MFMA;
    info.products = 1;
    info.chunk = 0;
    info.exact_no_wrap = 0;
    if (BH == 0 || L == 0 || d == 0) {
        info.kernels = 0;
        info.workspace_bytes = 0;
        return QX_OK;
    }
    // Key splits only while the query blocks of all heads leave the chip
    // short of 512 workgroups; split boundaries on 32-key blocks.
    const int64_t wgs = (L + 127) / 128 * BH;
    const int64_t kblocks = (L + 31) / 32;
    int64_t splits = std::min<int64_t>(std::max<int64_t>((512 + wgs - 1) / wgs, 1), kblocks);
    const int64_t kps = ((kblocks + splits - 1) / splits) * 32;
    splits = (L + kps - 1) / kps;
    SdpaParams a{};
    a.L = (int32_t)L; a.d = (int32_t)d; a.BH = (int32_t)BH;
    a.splits = (int32_t)splits; a.keys_per_split = (int32_t)kps;
    a.causal = causal;
    a.c = (float)((double)scale * 1.4426950408889634);   // log2(e)
    LaunchRec rec;
    if (!build_sdpa_f32(a, &rec)) return fail(QX_ERR_UNSUPPORTED, "no attention kernel for d = %lld", (long long)d);
    rec.bind(offsetof(SdpaParams, Q), BIND_IN0);
    rec.bind(offsetof(SdpaParams, K), BIND_IN1);
    rec.bind(offsetof(SdpaParams, V), BIND_IN2);
    rec.bind(offsetof(SdpaParams, O), BIND_OUT);
    uint64_t ws = 0;
    if (splits > 1) {
        const uint64_t part_bytes = round_up(4 * (uint64_t)splits * (uint64_t)n, 256);
        ws = part_bytes + 8 * (uint64_t)splits * (uint64_t)BH * (uint64_t)L;
        rec.bind(offsetof(SdpaParams, part), BIND_WS, 0);
        rec.bind(offsetof(SdpaParams, stat), BIND_WS, part_bytes);
        pl->launches.push_back(rec);
        SdpaCombineParams cp{};
        cp.rows = BH * L;
        cp.d = (int32_t)d;
        cp.splits = (int32_t)splits;
        LaunchRec rc;
        build_sdpa_combine(cp, &rc);
        rc.bind(offsetof(SdpaCombineParams, part), BIND_WS, 0);
        rc.bind(offsetof(SdpaCombineParams, stat), BIND_WS, part_bytes);
        rc.bind(offsetof(SdpaCombineParams, O), BIND_OUT);
        pl->launches.push_back(rc);
    } else {
        pl->launches.push_back(rec);
    }
    info.tile_m = 128; info.tile_n = (int32_t)d; info.tile_k = (int32_t)kps;
    info.kernels = (int32_t)pl->launches.size();
    info.workspace_bytes = (int64_t)ws;
    return QX_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// Device runtime calls of the executor
//
// Every HIP call the executor makes (device query, workspace, timing
// events, launches, the validation read-back) goes through one table.  The
// default table is the HIP runtime.  A host-only test double (switched on by
// qx_testing_host_double, for tests of the executor's bookkeeping on machines
// without a GPU) records instead: it reports one gfx950 device, hands out
// host memory for workspaces, checks every launch's geometry and enqueues
// nothing, so no operation result is ever computed while it is on.  Each
// handle keeps the table it was created with.
// ---------------------------------------------------------------------------
namespace {

struct RtTable {
    const char* name;
    hipError_t (*get_device)(int*);
    hipError_t (*set_device)(int);
    hipError_t (*arch_name)(int, char*, size_t);
    hipError_t (*malloc)(void**, size_t);
    hipError_t (*free)(void*);
    hipError_t (*clear_sync)(void*, size_t);    // zero, then wait for the device
    hipError_t (*device_sync)();
    hipError_t (*stream_sync)(hipStream_t);
    hipError_t (*event_create)(hipEvent_t*, bool timing);
    hipError_t (*event_destroy)(hipEvent_t);
    hipError_t (*event_record)(hipEvent_t, hipStream_t);
    hipError_t (*event_elapsed)(float*, hipEvent_t, hipEvent_t);
    hipError_t (*launch)(const LaunchRec&, void**, hipStream_t);
    hipError_t (*read_async)(void*, const void*, size_t, hipStream_t);
};

hipError_t hip_arch_name(int dev, char* buf, size_t n) {
    hipDeviceProp_t prop;
    hipError_t e = hipGetDeviceProperties(&prop, dev);
    if (e == hipSuccess) snprintf(buf, n, "%s", prop.gcnArchName);
    return e;
}

const RtTable kHip = {
    "hip",
    [](int* d) { return hipGetDevice(d); },
    [](int d) { return hipSetDevice(d); },
    hip_arch_name,
    [](void** p, size_t n) { return hipMalloc(p, n); },
    [](void* p) { return hipFree(p); },
    [](void* p, size_t n) {
        hipError_t e = hipMemset(p, 0, n);
        return e == hipSuccess ? hipDeviceSynchronize() : e;
    },
    []() { return hipDeviceSynchronize(); },
    [](hipStream_t s) { return hipStreamSynchronize(s); },
    [](hipEvent_t* ev, bool timing) {
        return timing ? hipEventCreate(ev) : hipEventCreateWithFlags(ev, hipEventDisableTiming);
    },
    [](hipEvent_t ev) { return hipEventDestroy(ev); },
    [](hipEvent_t ev, hipStream_t s) { return hipEventRecord(ev, s); },
    [](float* ms, hipEvent_t a, hipEvent_t b) { return hipEventElapsedTime(ms, a, b); },
    [](const LaunchRec& r, void** args, hipStream_t s) {
        return hipLaunchKernel(r.fn, r.grid, r.block, args, r.shmem, s);
    },
    [](void* dst, const void* src, size_t n, hipStream_t s) {
        return hipMemcpyAsync(dst, src, n, hipMemcpyDeviceToHost, s);
    },
};

// Host double: streams and events are distinct dummy objects so that leaks
// show up in the counters; a launch is checked against the hardware's grid
// and workgroup limits and every pointer slot of its parameter block must be
// bound.
struct Dummy { uint32_t tag; };
hipError_t dbl_new(void** p) { *p = new Dummy{0x64626c}; return hipSuccess; }
hipError_t dbl_delete(void* p) {
    if (!p || ((Dummy*)p)->tag != 0x64626c) return hipErrorInvalidValue;
    ((Dummy*)p)->tag = 0;
    delete (Dummy*)p;
    return hipSuccess;
}
hipError_t dbl_launch(const LaunchRec& r, void** args, hipStream_t) {
    if (!r.fn || !args) return hipErrorInvalidValue;
    if (r.grid.x < 1 || r.grid.y < 1 || r.grid.z < 1 || r.grid.y > 65535 || r.grid.z > 65535 ||
        (uint64_t)r.grid.x * r.block.x > 0xFFFFFFFFull)
        return hipErrorInvalidConfiguration;
    if (r.block.x * r.block.y * r.block.z < 1 || r.block.x * r.block.y * r.block.z > 1024)
        return hipErrorInvalidConfiguration;
    if (r.shmem > 160 * 1024) return hipErrorInvalidConfiguration;
    for (int i = 0; i < r.nslots; ++i) {
        void* ptr = nullptr;
        memcpy(&ptr, (const unsigned char*)args[0] + r.slots[i].off, sizeof ptr);
        if (!ptr) return hipErrorInvalidValue;
    }
    return hipSuccess;
}

const RtTable kHostDouble = {
    "host double",
    [](int* d) { *d = 0; return hipSuccess; },
    [](int d) { return d == 0 ? hipSuccess : hipErrorInvalidDevice; },
    [](int, char* buf, size_t n) { snprintf(buf, n, "gfx950:sramecc+:xnack-"); return hipSuccess; },
    [](void** p, size_t n) {
        *p = aligned_alloc(256, round_up(n, 256));
        return *p ? hipSuccess : hipErrorOutOfMemory;
    },
    [](void* p) { std::free(p); return hipSuccess; },
    [](void* p, size_t n) { memset(p, 0, n); return hipSuccess; },
    []() { return hipSuccess; },
    [](hipStream_t) { return hipSuccess; },
    [](hipEvent_t* ev, bool) { return dbl_new((void**)ev); },
    [](hipEvent_t ev) { return dbl_delete((void*)ev); },
    [](hipEvent_t ev, hipStream_t) { return ev ? hipSuccess : hipErrorInvalidHandle; },
    [](float* ms, hipEvent_t, hipEvent_t) { *ms = 0.0f; return hipSuccess; },
    dbl_launch,
    [](void* dst, const void* src, size_t n, hipStream_t) { memcpy(dst, src, n); return hipSuccess; },
};

std::atomic<const RtTable*> g_rt{&kHip};

// Counters of every device resource the executor acquires and releases
// (both tables), for the tests of "run allocates nothing" and of cleanup
// after a failed create.
enum Counter { C_ALLOCS, C_FREES, C_EVENTS, C_EVENTS_FREED, C_LAUNCHES, C_LIVE_HANDLES, C_N };
std::atomic<int64_t> g_count[C_N];

}  // namespace

struct qx_exec_s {
    uint32_t magic;
    int device;
    const RtTable* rt;      // runtime the handle was created with
    Plan plan;
    void* ws;
    uint64_t ws_bytes;
    uint64_t flag_off;      // QX_VALIDATE flag word in the workspace
};

namespace {

// Live handles: a handle is usable only between its create and its destroy,
// so a second destroy or a stray pointer is refused without being read.
std::mutex g_live_mu;
std::set<qx_exec>* g_live = new std::set<qx_exec>();

bool is_live(qx_exec h) {
    if (!h) return false;
    std::lock_guard<std::mutex> lk(g_live_mu);
    return g_live->count(h) != 0;
}

qx_status check_device(const RtTable& rt, int* dev) {
    hipError_t e = rt.get_device(dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    char arch[256] = {0};
    e = rt.arch_name(*dev, arch, sizeof arch);
    if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
    if (strncmp(arch, "gfx950", 6) != 0)
        return fail(QX_ERR_UNSUPPORTED, "device %d is %s; this library is built for gfx950 only", *dev, arch);
    return QX_OK;
}

// Releases everything a handle holds (any part may be missing); returns the
// first error, after trying every release.
hipError_t release_exec(qx_exec h) {
    const RtTable& rt = *h->rt;
    hipError_t first = hipSuccess;
    auto note = [&](hipError_t e) { if (first == hipSuccess && e != hipSuccess) first = e; };
    if (h->ws) {
        note(rt.device_sync());
        note(rt.free(h->ws));
        g_count[C_FREES]++;
        h->ws = nullptr;
    }
    return first;
}

// QX_TEST_FAIL_ALLOC=k: the k-th device resource a create acquires (counted
// from 1; a create acquires at most one, its workspace) fails as if the
// device were out of memory, so that the cleanup path of a failed create
// can be exercised.
int fail_alloc_at() {
    const char* v = getenv("QX_TEST_FAIL_ALLOC");
    return v ? atoi(v) : 0;
}

qx_status make_exec(Plan&& pl, qx_exec* out) {
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    const RtTable& rt = *g_rt.load();
    int dev = 0;
    qx_status st = check_device(rt, &dev);
    if (st) return st;
    const int fail_at = fail_alloc_at();
    int acquired = 0;
    auto injected = [&]() { return ++acquired == fail_at; };
    qx_exec h = new qx_exec_s();
    h->magic = kMagic;
    h->device = dev;
    h->rt = &rt;
    h->ws = nullptr;
    h->ws_bytes = (uint64_t)pl.info.workspace_bytes;
    h->plan = std::move(pl);
    // QX_VALIDATE flag word behind the plan's workspace
    h->flag_off = round_up(h->ws_bytes, 256);
    if (!h->plan.checks.empty()) h->ws_bytes = h->flag_off + 256;
    hipError_t e = hipSuccess;
    const char* what = "";
    if (h->ws_bytes) {
        what = "workspace allocation";
        e = injected() ? hipErrorOutOfMemory : rt.malloc(&h->ws, h->ws_bytes);
        if (e == hipSuccess) {
            g_count[C_ALLOCS]++;
            // Zero once: padding that no run writes (tile tails of the encoded
            // operands) must hold finite zeros.
            what = "workspace clear";
            e = rt.clear_sync(h->ws, h->ws_bytes);
        } else {
            h->ws = nullptr;
        }
    }
    if (e != hipSuccess) {
        if (h->rt == &kHip) (void)hipGetLastError();
        (void)release_exec(h);
        h->magic = 0;
        delete h;
        return hip_fail(e, what);
    }
    {
        std::lock_guard<std::mutex> lk(g_live_mu);
        g_live->insert(h);
    }
    g_count[C_LIVE_HANDLES]++;
    *out = h;
    return QX_OK;
}

// What a run needs: the plan, the runtime and the workspace (with the
// validation flag word at flag_off).  Every launch goes to the caller's
// stream in plan order.
struct RunCtx {
    const Plan* plan;
    const RtTable* rt;
    void* ws;
    uint64_t flag_off;
    int device;
};

qx_status launch_direct(const RtTable& rt, LaunchRec& r, hipStream_t s) {
    void* args[1] = {r.blob};
    g_count[C_LAUNCHES]++;
    hipError_t e = rt.launch(r, args, s);
    return e == hipSuccess ? QX_OK : hip_fail(e, r.name);
}

// QX_VALIDATE: scan every bounded operand, wait, and refuse the run if one
// is outside its declared bound.
qx_status validate_ranges(const RunCtx& c, const void* const* inputs, hipStream_t s) {
    const Plan& pl = *c.plan;
    const RtTable& rt = *c.rt;
    uint32_t* flag = (uint32_t*)((char*)c.ws + c.flag_off);
    FillParams f{};
    f.ptr = flag;
    f.n32 = 1;
    f.value = 0;
    LaunchRec rf;
    build_fill(f, &rf);
    qx_status st = launch_direct(rt, rf, s);
    for (size_t i = 0; st == QX_OK && i < pl.checks.size(); ++i) {
        const Plan::RangeCheck& c = pl.checks[i];
        if (c.n == 0) continue;
        RangeParams rp{};
        rp.x = inputs[c.input];
        rp.flag = flag;
        rp.n = c.n;
        rp.bound = c.bound;
        rp.elem_bytes = c.elem_bytes;
        rp.bit = 1u << i;
        LaunchRec rr;
        build_range(rp, &rr);
        st = launch_direct(rt, rr, s);
    }
    if (st) return st;
    uint32_t bad = 0;
    hipError_t e = rt.read_async(&bad, flag, sizeof bad, s);
    if (e == hipSuccess) e = rt.stream_sync(s);
    if (e != hipSuccess) return hip_fail(e, "range scan");
    for (size_t i = 0; i < pl.checks.size(); ++i)
        if (bad & (1u << i))
            return fail(QX_ERR_RANGE, "input %d has an element with |x| > %d (declared bound)", pl.checks[i].input,
                        pl.checks[i].bound);
    return QX_OK;
}

qx_status run_plan(const RunCtx& c, const void* const* inputs, void* output, void* stream,
                   std::vector<hipEvent_t>* evs) {
    const Plan& pl = *c.plan;
    const RtTable& rt = *c.rt;
    if (pl.launches.empty()) return QX_OK;
    // Only inputs some launch reads are required (a K == 0 GEMM just clears
    // its output and may get NULL operands).
    unsigned used = 0;
    for (const LaunchRec& r : pl.launches)
        for (int i = 0; i < r.nslots; ++i)
            if (r.slots[i].bind < BIND_OUT) used |= 1u << r.slots[i].bind;
    if (used && !inputs) return fail(QX_ERR_INVALID_ARG, "inputs is NULL");
    for (int i = 0; i < pl.n_inputs; ++i) {
        if (!(used & (1u << i))) continue;
        if (!inputs[i]) return fail(QX_ERR_INVALID_ARG, "input %d is NULL", i);
        if ((uintptr_t)inputs[i] % pl.in_align)
            return fail(QX_ERR_INVALID_ARG, "input %d is not %llu-byte aligned", i, (unsigned long long)pl.in_align);
    }
    if (!output) return fail(QX_ERR_INVALID_ARG, "output is NULL");
    if ((uintptr_t)output % pl.out_align)
        return fail(QX_ERR_INVALID_ARG, "output is not %llu-byte aligned", (unsigned long long)pl.out_align);
    int dev = -1;
    hipError_t e = rt.get_device(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != c.device)
        return fail(QX_ERR_INVALID_ARG, "plan was made for device %d, current device is %d", c.device, dev);
    hipStream_t s = (hipStream_t)stream;
    const char* val = getenv("QX_VALIDATE");
    if (val && val[0] == '1' && !pl.checks.empty()) {
        const qx_status st = validate_ranges(c, inputs, s);
        if (st) return st;
    }
    for (const LaunchRec& r0 : pl.launches) {
        LaunchRec r = r0;
        for (int i = 0; i < r.nslots; ++i) {
            const Slot& sl = r.slots[i];
            const char* ptr = nullptr;
            if (sl.bind < BIND_OUT) ptr = (const char*)inputs[sl.bind];
            else if (sl.bind == BIND_OUT) ptr = (const char*)output;
            else ptr = (const char*)c.ws;
            ptr += sl.add;
            memcpy(r.blob + sl.off, &ptr, sizeof(void*));
        }
        void* args[1] = {r.blob};
        const size_t li = (size_t)(&r0 - pl.launches.data());
        if (evs && (e = rt.event_record((*evs)[2 * li], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
        g_count[C_LAUNCHES]++;
        e = rt.launch(r, args, s);
        if (e != hipSuccess) return hip_fail(e, r.name);
        if (evs && (e = rt.event_record((*evs)[2 * li + 1], s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    }
    return QX_OK;
}

qx_status run_exec(qx_exec h, const void* const* inputs, void* output, void* stream,
                   std::vector<hipEvent_t>* evs = nullptr) {
    if (!is_live(h) || h->magic != kMagic) return fail(QX_ERR_INVALID_ARG, "invalid executor handle");
    const RunCtx c{&h->plan, h->rt, h->ws, h->flag_off, h->device};
    return run_plan(c, inputs, output, stream, evs);
}

qx_status profile_exec(qx_exec h, const void* const* inputs, void* output, void* stream, int32_t reps,
                       float* kernel_ms, const char** names, int32_t max_kernels) {
    if (!is_live(h) || h->magic != kMagic) return fail(QX_ERR_INVALID_ARG, "invalid executor handle");
    if (reps < 1 || max_kernels < 0 || (max_kernels > 0 && !kernel_ms))
        return fail(QX_ERR_INVALID_ARG, "reps must be >= 1 and kernel_ms non-NULL");
    const RtTable& rt = *h->rt;
    const size_t nl = h->plan.launches.size();
    const int nout = (int)std::min<size_t>(nl, (size_t)max_kernels);
    for (int i = 0; i < nout; ++i) {
        kernel_ms[i] = 0.0f;
        if (names) names[i] = h->plan.launches[i].name;
    }
    if (nl == 0) return QX_OK;
    std::vector<hipEvent_t> evs(2 * nl * (size_t)reps, nullptr);
    qx_status st = QX_OK;
    hipError_t e = hipSuccess;
    for (auto& ev : evs) {
        if ((e = rt.event_create(&ev, true)) != hipSuccess) {
            ev = nullptr;
            break;
        }
        g_count[C_EVENTS]++;
    }
    if (e != hipSuccess) {
        st = hip_fail(e, "hipEventCreate");
    } else {
        for (int r = 0; r < reps && st == QX_OK; ++r) {
            std::vector<hipEvent_t> sub(evs.begin() + 2 * nl * r, evs.begin() + 2 * nl * (r + 1));
            st = run_exec(h, inputs, output, stream, &sub);
        }
        if (st == QX_OK && (e = rt.stream_sync((hipStream_t)stream)) != hipSuccess)
            st = hip_fail(e, "hipStreamSynchronize");
        for (int r = 0; r < reps && st == QX_OK; ++r)
            for (int i = 0; i < nout; ++i) {
                float ms = 0.0f;
                if ((e = rt.event_elapsed(&ms, evs[2 * nl * r + 2 * i], evs[2 * nl * r + 2 * i + 1])) !=
                    hipSuccess) {
                    st = hip_fail(e, "hipEventElapsedTime");
                    break;
                }
                kernel_ms[i] += ms / (float)reps;
            }
    }
    for (auto& ev : evs)
        if (ev) {
            (void)rt.event_destroy(ev);
            g_count[C_EVENTS_FREED]++;
        }
    return st;
}

// One-shot calls: a cache of executors keyed by the full request.  The lock
// is held while a missing entry is created, so concurrent first calls with
// one key create it once.
typedef std::tuple<int, int, int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, int64_t,
                   int64_t, int64_t, int64_t, uintptr_t>
    Key;
std::mutex g_cache_mu;
std::map<Key, qx_exec>* g_cache = new std::map<Key, qx_exec>();

template <class MakePlan>
qx_status oneshot(const Key& key0, MakePlan make_plan, const void* const* inputs, void* output, void* stream) {
    int dev = -1;
    hipError_t e = g_rt.load()->get_device(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    Key key = key0;
    std::get<1>(key) = dev;
    qx_exec h = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_cache_mu);
        auto it = g_cache->find(key);
        if (it != g_cache->end()) {
            h = it->second;
        } else {
            Plan pl;
            qx_status st = make_plan(&pl);
            if (st) return st;
            if ((st = make_exec(std::move(pl), &h))) return st;
            g_cache->emplace(key, h);
        }
    }
    return run_exec(h, inputs, output, stream);
}

}  // namespace

// Allocation-free GEMM: plans are cached on the host per request; the
// workspace is the per-device scratch array, whose device address is looked
// up (and the device checked) on the first call on each device.
namespace {
typedef std::tuple<int64_t, int64_t, int64_t, int64_t, int32_t, int32_t> NoAllocKey;
std::mutex g_noalloc_mu;
std::map<NoAllocKey, Plan>* g_noalloc_plans = new std::map<NoAllocKey, Plan>();
std::atomic<bool> g_noalloc_dev_ok[64];

static_assert(QX_NOALLOC_SCRATCH_BYTES == kScratchBytes, "scratch size in the header and the library");

uint64_t scratch_need(const Plan& pl) {
    const uint64_t ws = (uint64_t)pl.info.workspace_bytes;
    return pl.checks.empty() ? ws : round_up(ws, 256) + 256;
}
}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" {

const char* qx_last_error(void) { return g_err.c_str(); }

qx_status qx_plan_gemm_i16i32(qx_plan_info* out, int64_t M, int64_t N, int64_t K, int64_t batch, int32_t bound_a,
                              int32_t bound_b, int32_t route) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    Plan pl;
    qx_status st = plan_gemm(&pl, false, M, N, K, batch, bound_a, bound_b, route);
    if (!st) *out = pl.info;
    return st;
}

qx_status qx_plan_gemm_i32_s24(qx_plan_info* out, int64_t M, int64_t N, int64_t K, int64_t batch, int32_t route) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    Plan pl;
    qx_status st = plan_gemm(&pl, true, M, N, K, batch, 0, 0, route);
    if (!st) *out = pl.info;
    return st;
}

qx_status qx_plan_conv2d(qx_plan_info* out, int64_t N, int64_t C_in, int64_t H, int64_t W, int64_t C_out,
                         int64_t KH, int64_t KW, int64_t stride, int64_t pad, int32_t bound_x, int32_t bound_w,
                         int32_t route) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    Plan pl;
    qx_status st = plan_conv(&pl, N, C_in, H, W, C_out, KH, KW, stride, pad, bound_x, bound_w, route);
    if (!st) *out = pl.info;
    return st;
}

qx_status qx_plan_conv2d_t(qx_plan_info* out, qx_attn_dtype dt, int64_t N, int64_t C_in, int64_t H, int64_t W,
                           int64_t C_out, int64_t KH, int64_t KW, int64_t stride, int64_t pad, int32_t route) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    Plan pl;
    qx_status st = plan_conv_t(&pl, dt_raw(dt), N, C_in, H, W, C_out, KH, KW, stride, pad, route);
    if (!st) *out = pl.info;
    return st;
}

qx_status qx_plan_minmax(qx_plan_info* out, int64_t n, int32_t elem_bytes) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    Plan pl;
    qx_status st = plan_minmax(&pl, n, elem_bytes);
    if (!st) *out = pl.info;
    return st;
}

qx_status qx_plan_pool2x2(qx_plan_info* out, int32_t kind, int64_t N, int64_t C, int64_t H, int64_t W) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    Plan pl;
    qx_status st = plan_pool2(&pl, kind, N, C, H, W);
    if (!st) *out = pl.info;
    return st;
}

qx_status qx_plan_lenet_i32(qx_plan_info* out, int64_t batch) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    Plan pl;
    qx_status st = plan_lenet(&pl, batch);
    if (!st) *out = pl.info;
    return st;
}

qx_status qx_plan_attn(qx_plan_info* out, qx_attn_dtype dt, int64_t L, int64_t d, int32_t bound, int32_t route) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    Plan pl;
    qx_status st = plan_attn(&pl, dt_raw(dt), L, d, bound, route);
    if (!st) *out = pl.info;
    return st;
}

qx_status qx_plan_sdpa_f32(qx_plan_info* out, int64_t BH, int64_t L, int64_t d, float scale, int32_t causal) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    Plan pl;
    qx_status st = plan_sdpa(&pl, BH, L, d, scale, causal);
    if (!st) *out = pl.info;
    return st;
}

qx_status qx_exec_create_sdpa_f32(qx_exec* out, int64_t BH, int64_t L, int64_t d, float scale, int32_t causal) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    Plan pl;
    qx_status st = plan_sdpa(&pl, BH, L, d, scale, causal);
    if (st) return st;
    return make_exec(std::move(pl), out);
}

qx_status qx_exec_create_gemm_i16i32_route(qx_exec* out, int64_t M, int64_t N, int64_t K, int64_t batch,
                                           int32_t bound_a, int32_t bound_b, int32_t route) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    Plan pl;
    qx_status st = plan_gemm(&pl, false, M, N, K, batch, bound_a, bound_b, route);
    if (st) return st;
    return make_exec(std::move(pl), out);
}

qx_status qx_exec_create_gemm_i32_s24_route(qx_exec* out, int64_t M, int64_t N, int64_t K, int64_t batch,
                                            int32_t route) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    Plan pl;
    qx_status st = plan_gemm(&pl, true, M, N, K, batch, 0, 0, route);
    if (st) return st;
    return make_exec(std::move(pl), out);
}

qx_status qx_exec_create_conv2d_route(qx_exec* out, int64_t N, int64_t C_in, int64_t H, int64_t W, int64_t C_out,
                                      int64_t KH, int64_t KW, int64_t stride, int64_t pad, int32_t bound_x,
                                      int32_t bound_w, int32_t route) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    Plan pl;
    qx_status st = plan_conv(&pl, N, C_in, H, W, C_out, KH, KW, stride, pad, bound_x, bound_w, route);
    if (st) return st;
    return make_exec(std::move(pl), out);
}

qx_status qx_exec_create_conv2d_t(qx_exec* out, qx_attn_dtype dt, int64_t N, int64_t C_in, int64_t H, int64_t W,
                                  int64_t C_out, int64_t KH, int64_t KW, int64_t stride, int64_t pad, int32_t route) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    Plan pl;
    qx_status st = plan_conv_t(&pl, dt_raw(dt), N, C_in, H, W, C_out, KH, KW, stride, pad, route);
    if (st) return st;
    return make_exec(std::move(pl), out);
}

qx_status qx_exec_create_minmax(qx_exec* out, int64_t n, int32_t elem_bytes) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    Plan pl;
    qx_status st = plan_minmax(&pl, n, elem_bytes);
    if (st) return st;
    return make_exec(std::move(pl), out);
}

qx_status qx_exec_create_pool2x2(qx_exec* out, int32_t kind, int64_t N, int64_t C, int64_t H, int64_t W) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    Plan pl;
    qx_status st = plan_pool2(&pl, kind, N, C, H, W);
    if (st) return st;
    return make_exec(std::move(pl), out);
}

qx_status qx_exec_create_lenet_i32(qx_exec* out, int64_t batch) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    Plan pl;
    qx_status st = plan_lenet(&pl, batch);
    if (st) return st;
    return make_exec(std::move(pl), out);
}

qx_status qx_exec_create_attn_route(qx_exec* out, qx_attn_dtype dt, int64_t L, int64_t d, int32_t bound,
                                    int32_t route) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    Plan pl;
    qx_status st = plan_attn(&pl, dt_raw(dt), L, d, bound, route);
    if (st) return st;
    return make_exec(std::move(pl), out);
}

// The executor-create calls of the operations' specified interface take no
// route: the planner chooses it from the contract.
qx_status qx_exec_create_gemm_i16i32(qx_exec* out, int64_t M, int64_t N, int64_t K, int64_t batch, int32_t bound_a,
                                     int32_t bound_b) {
    return qx_exec_create_gemm_i16i32_route(out, M, N, K, batch, bound_a, bound_b, R_AUTO);
}

qx_status qx_exec_create_gemm_i32_s24(qx_exec* out, int64_t M, int64_t N, int64_t K, int64_t batch) {
    return qx_exec_create_gemm_i32_s24_route(out, M, N, K, batch, R_AUTO);
}

qx_status qx_exec_create_conv2d(qx_exec* out, int64_t N, int64_t C_in, int64_t H, int64_t W, int64_t C_out,
                                int64_t KH, int64_t KW, int64_t stride, int64_t pad, int32_t bound_x,
                                int32_t bound_w) {
    return qx_exec_create_conv2d_route(out, N, C_in, H, W, C_out, KH, KW, stride, pad, bound_x, bound_w, R_AUTO);
}

qx_status qx_exec_create_attn(qx_exec* out, qx_attn_dtype dt, int64_t L, int64_t d, int32_t bound) {
    g_err.clear();
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    Plan pl;
    qx_status st = plan_attn(&pl, dt_raw(dt), L, d, bound, R_AUTO);
    if (st) return st;
    return make_exec(std::move(pl), out);
}

qx_status qx_exec_run(qx_exec h, const void* const* inputs, void* output, void* stream) {
    g_err.clear();
    return run_exec(h, inputs, output, stream);
}

qx_status qx_exec_profile(qx_exec h, const void* const* inputs, void* output, void* stream, int32_t reps,
                          float* kernel_ms, const char** names, int32_t max_kernels) {
    g_err.clear();
    return profile_exec(h, inputs, output, stream, reps, kernel_ms, names, max_kernels);
}

qx_status qx_exec_plan(qx_exec h, qx_plan_info* out) {
    g_err.clear();
    if (!is_live(h) || h->magic != kMagic) return fail(QX_ERR_INVALID_ARG, "invalid executor handle");
    if (!out) return fail(QX_ERR_INVALID_ARG, "out is NULL");
    *out = h->plan.info;
    return QX_OK;
}

qx_status qx_exec_destroy(qx_exec h) {
    g_err.clear();
    if (!h) return QX_OK;
    {
        std::lock_guard<std::mutex> lk(g_live_mu);
        if (!g_live->erase(h)) return fail(QX_ERR_INVALID_ARG, "invalid executor handle (not live)");
    }
    g_count[C_LIVE_HANDLES]--;
    h->magic = 0;
    const RtTable& rt = *h->rt;
    int cur = -1;
    (void)rt.get_device(&cur);
    if (cur != h->device) (void)rt.set_device(h->device);
    const hipError_t e = release_exec(h);
    if (cur != h->device && cur >= 0) (void)rt.set_device(cur);
    delete h;
    return e == hipSuccess ? QX_OK : hip_fail(e, "executor release");
}

void qx_release_cache(void) {
    std::map<Key, qx_exec> old;
    {
        std::lock_guard<std::mutex> lk(g_cache_mu);
        old.swap(*g_cache);
    }
    for (auto& kv : old) qx_exec_destroy(kv.second);
}

// ---- test seams (include/qx_testing.h) ----------------------------------

qx_status qx_testing_host_double(int32_t on) {
    g_err.clear();
    if (on != 0 && on != 1) return fail(QX_ERR_INVALID_ARG, "on must be 0 or 1");
    const RtTable* want = on ? &kHostDouble : &kHip;
    if (g_rt.load() == want) return QX_OK;
    qx_release_cache();
    {
        std::lock_guard<std::mutex> lk(g_live_mu);
        if (!g_live->empty())
            return fail(QX_ERR_INVALID_ARG, "%zu executor handles are still live", g_live->size());
    }
    g_rt.store(want);
    return QX_OK;
}

void qx_testing_counters(int64_t* out, int32_t n) {
    for (int i = 0; out && i < n && i < C_N; ++i) out[i] = g_count[i].load();
}

static bool empty_ok(const void* p, int64_t n) { return p != nullptr || n == 0; }

qx_status qgemm_i16i32(const int16_t* A, const int16_t* B, int32_t* C, int64_t M, int64_t N, int64_t K,
                       int64_t batch, int32_t bound_a, int32_t bound_b, void* stream) {
    g_err.clear();
    Plan probe;
    qx_status st = plan_gemm(&probe, false, M, N, K, batch, bound_a, bound_b, R_AUTO);
    if (st) return st;
    if (!empty_ok(A, M * K * batch) || !empty_ok(B, K * N * batch) || !empty_ok(C, M * N * batch))
        return fail(QX_ERR_INVALID_ARG, "NULL pointer for a non-empty operand");
    if (probe.launches.empty()) return QX_OK;
    const void* in[2] = {A, B};
    Key key{OP_GEMM_I16, 0, M, N, K, batch, bound_a, bound_b, 0, 0, 0, 0, 0, 0, (uintptr_t)stream};
    return oneshot(key, [&](Plan* pl) { return plan_gemm(pl, false, M, N, K, batch, bound_a, bound_b, R_AUTO); },
                   in, C, stream);
}

qx_status qgemm_i32_s24(const int32_t* A, const int32_t* B, int32_t* C, int64_t M, int64_t N, int64_t K,
                        int64_t batch, void* stream) {
    g_err.clear();
    Plan probe;
    qx_status st = plan_gemm(&probe, true, M, N, K, batch, 0, 0, R_AUTO);
    if (st) return st;
    if (!empty_ok(A, M * K * batch) || !empty_ok(B, K * N * batch) || !empty_ok(C, M * N * batch))
        return fail(QX_ERR_INVALID_ARG, "NULL pointer for a non-empty operand");
    if (probe.launches.empty()) return QX_OK;
    const void* in[2] = {A, B};
    Key key{OP_GEMM_S24, 0, M, N, K, batch, 0, 0, 0, 0, 0, 0, 0, 0, (uintptr_t)stream};
    return oneshot(key, [&](Plan* pl) { return plan_gemm(pl, true, M, N, K, batch, 0, 0, R_AUTO); }, in, C,
                   stream);
}

qx_status conv2d_gemm(const int16_t* x, const int16_t* w, int32_t* y, int64_t N, int64_t C_in, int64_t H, int64_t W,
                      int64_t C_out, int64_t KH, int64_t KW, int64_t stride, int64_t pad, int32_t bound_x,
                      int32_t bound_w, void* stream) {
    g_err.clear();
    Plan probe;
    qx_status st = plan_conv(&probe, N, C_in, H, W, C_out, KH, KW, stride, pad, bound_x, bound_w, R_AUTO);
    if (st) return st;
    if (probe.launches.empty()) return QX_OK;
    if (!empty_ok(x, N * C_in * H * W) || !empty_ok(w, C_out * C_in * KH * KW) || !y)
        return fail(QX_ERR_INVALID_ARG, "NULL pointer for a non-empty operand");
    const void* in[2] = {x, w};
    Key key{OP_CONV, 0, N, C_in, H, W, C_out, KH, KW, stride, pad, bound_x, bound_w, 0, (uintptr_t)stream};
    return oneshot(key,
                   [&](Plan* pl) {
                       return plan_conv(pl, N, C_in, H, W, C_out, KH, KW, stride, pad, bound_x, bound_w, R_AUTO);
                   },
                   in, y, stream);
}

qx_status conv2d_gemm_t(qx_attn_dtype dt, const void* x, const void* w, void* y, int64_t N, int64_t C_in,
                        int64_t H, int64_t W, int64_t C_out, int64_t KH, int64_t KW, int64_t stride, int64_t pad,
                        void* stream) {
    g_err.clear();
    Plan probe;
    qx_status st = plan_conv_t(&probe, dt_raw(dt), N, C_in, H, W, C_out, KH, KW, stride, pad, R_AUTO);
    if (st) return st;
    if (probe.launches.empty()) return QX_OK;
    if (!empty_ok(x, N * C_in * H * W) || !empty_ok(w, C_out * C_in * KH * KW) || !y)
        return fail(QX_ERR_INVALID_ARG, "NULL pointer for a non-empty operand");
    const void* in[2] = {x, w};
    Key key{dt_raw(dt) == QX_DT_F32 ? OP_CONV_F32 : OP_CONV_I32, 0, N, C_in, H, W, C_out, KH, KW, stride, pad, 0, 0, 0,
            (uintptr_t)stream};
    return oneshot(key,
                   [&](Plan* pl) { return plan_conv_t(pl, dt_raw(dt), N, C_in, H, W, C_out, KH, KW, stride, pad, R_AUTO); },
                   in, y, stream);
}

qx_status minmax(const void* x, int64_t n, int32_t elem_bytes, void* out, void* stream) {
    g_err.clear();
    Plan probe;
    qx_status st = plan_minmax(&probe, n, elem_bytes);
    if (st) return st;
    if (!x || !out) return fail(QX_ERR_INVALID_ARG, "NULL pointer");
    const void* in[1] = {x};
    Key key{OP_MINMAX, 0, n, elem_bytes, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, (uintptr_t)stream};
    return oneshot(key, [&](Plan* pl) { return plan_minmax(pl, n, elem_bytes); }, in, out, stream);
}

qx_status pool2x2(int32_t kind, const void* x, void* y, int64_t N, int64_t C, int64_t H, int64_t W, void* stream) {
    g_err.clear();
    Plan probe;
    qx_status st = plan_pool2(&probe, kind, N, C, H, W);
    if (st) return st;
    if (probe.launches.empty()) return QX_OK;
    if (!x || !y) return fail(QX_ERR_INVALID_ARG, "NULL pointer for a non-empty operand");
    const void* in[1] = {x};
    Key key{OP_POOL, 0, kind, N, C, H, W, 0, 0, 0, 0, 0, 0, 0, (uintptr_t)stream};
    return oneshot(key, [&](Plan* pl) { return plan_pool2(pl, kind, N, C, H, W); }, in, y, stream);
}

qx_status attn_core(qx_attn_dtype dt, const void* Q, const void* K, const void* V, void* O, int64_t L, int64_t d,
                    int32_t bound, void* stream) {
    g_err.clear();
    Plan probe;
    qx_status st = plan_attn(&probe, dt_raw(dt), L, d, bound, R_AUTO);
    if (st) return st;
    if (probe.launches.empty()) return QX_OK;
    if (!Q || !K || !V || !O) return fail(QX_ERR_INVALID_ARG, "NULL pointer for a non-empty operand");
    const void* in[3] = {Q, K, V};
    Key key{dt_raw(dt) == QX_DT_F32 ? OP_ATTN_F32 : OP_ATTN_I32, 0, L, d, bound, 0, 0, 0, 0, 0, 0, 0, 0, 0,
            (uintptr_t)stream};
    return oneshot(key, [&](Plan* pl) { return plan_attn(pl, dt_raw(dt), L, d, bound, R_AUTO); }, in, O, stream);
}

qx_status qgemm_i16i32_noalloc(const int16_t* A, const int16_t* B, int32_t* C, int64_t M, int64_t N, int64_t K,
                               int64_t batch, int32_t bound_a, int32_t bound_b, void* stream) {
    g_err.clear();
    const Plan* pl = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_noalloc_mu);
        const NoAllocKey key{M, N, K, batch, bound_a, bound_b};
        auto it = g_noalloc_plans->find(key);
        if (it == g_noalloc_plans->end()) {
            Plan p;
            qx_status st = plan_gemm(&p, false, M, N, K, batch, bound_a, bound_b, R_AUTO);
            if (st) return st;
            if (scratch_need(p) > kScratchBytes) {
                // the encoded operands do not fit: the register-staged
                // kernels convert while staging and need only the row and
                // column sums of the offset routes
                Plan q;
                if ((st = plan_gemm(&q, false, M, N, K, batch, bound_a, bound_b, R_AUTO, false))) return st;
                p = std::move(q);
            }
            if (scratch_need(p) > kScratchBytes)
                return fail(QX_ERR_UNSUPPORTED,
                            "this GEMM needs %llu bytes of workspace; the allocation-free entry point has %llu",
                            (unsigned long long)scratch_need(p), (unsigned long long)kScratchBytes);
            it = g_noalloc_plans->emplace(key, std::move(p)).first;
        }
        pl = &it->second;
    }
    if (!empty_ok(A, M * K * batch) || !empty_ok(B, K * N * batch) || !empty_ok(C, M * N * batch))
        return fail(QX_ERR_INVALID_ARG, "NULL pointer for a non-empty operand");
    if (pl->launches.empty()) return QX_OK;
    int dev = -1;
    hipError_t e = kHip.get_device(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= 64) return fail(QX_ERR_UNSUPPORTED, "device %d: at most 64 devices", dev);
    if (!g_noalloc_dev_ok[dev].load()) {
        int d2 = dev;
        qx_status st = check_device(kHip, &d2);
        if (st) return st;
        g_noalloc_dev_ok[dev].store(true);
    }
    void* ws = nullptr;
    if ((e = scratch_device_ptr(dev, &ws)) != hipSuccess) return hip_fail(e, "scratch lookup");
    const void* in[2] = {A, B};
    const RunCtx c{pl, &kHip, ws, round_up((uint64_t)pl->info.workspace_bytes, 256), dev};
    return run_plan(c, in, C, stream, nullptr);
}

qx_status sdpa_f32(const float* Q, const float* K, const float* V, float* O, int64_t BH, int64_t L, int64_t d,
                   float scale, int32_t causal, void* stream) {
    g_err.clear();
    Plan probe;
    qx_status st = plan_sdpa(&probe, BH, L, d, scale, causal);
    if (st) return st;
    if (probe.launches.empty()) return QX_OK;
    if (!Q || !K || !V || !O) return fail(QX_ERR_INVALID_ARG, "NULL pointer for a non-empty operand");
    const void* in[3] = {Q, K, V};
    uint32_t sbits;
    std::memcpy(&sbits, &scale, 4);
    Key key{OP_SDPA, 0, BH, L, d, (int64_t)sbits, causal, 0, 0, 0, 0, 0, 0, 0, (uintptr_t)stream};
    return oneshot(key, [&](Plan* pl) { return plan_sdpa(pl, BH, L, d, scale, causal); }, in, O, stream);
}

}  // extern "C"
