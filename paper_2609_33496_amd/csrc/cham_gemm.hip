// Mixed-format linear layer: Y = DQ(X codes) . DQ(W codes)^T with a per-output-channel
// weight format (Sec. 4.5) and one activation format per call (Sec. 4.3).
//
// Design (gfx950): per-channel formats do not map onto one native MFMA operand type
// (Sec. 6), so weights are dequantized on the fly, per 128x32 tile, into a common
// half-precision operand in LDS ("weights dequantized in registers").  Every weight code
// becomes a value that half precision holds exactly -- integers, E2M1 values, MX integer or
// E2M1 mantissas times 2^(E_block - E_ref) -- except the NF4 levels, which are carried to
// 11 significant bits (relative error <= 2^-11).  The per-channel factor (the INT/FP4 scale,
// or 2^E_ref for block-scaled channels) and the per-tensor activation scale are applied in
// the binary32 epilogue.  Activation codes become exact half-precision values: INT8-asym
// q - z, E4M3/E5M2 values, MX values relative to the row's largest block exponent.  The
// contraction runs on v_mfma_f32_16x16x32_f16 with binary32 accumulation.
#include "cham_device.h"

namespace cham {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float4v __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 128, BK = 32, LDK = BK + 8;  // LDS row stride (halves)
constexpr int kThreads = 256;

struct GemmArgs {
    const uint8_t* xc;   // [M][K]
    const uint8_t* xe8;  // [M][K/32] (MX act)
    const float* xs;     // [1]
    const float* xz;     // [1]
    int afmt;
    const uint8_t* wfmt;  // [N]
    const uint8_t* wc;    // codes
    const float* wscale;  // [N]
    const int32_t* wzero; // [N]
    const float* wnf4;    // [N][K/64]
    const uint8_t* we8;   // [N][K/32]
    float* Y;
    int M, N, K;
    uint32_t mask;  // palette: a channel whose format is outside it decodes as zero
};

// Per-channel decode parameters, computed once per tile.
struct ColInfo {
    int fmt;
    int eref;      // exponent removed from block-scaled values (0 for INT/FP4)
    float zero;    // INT-asym zero point
    float colscale;
};

CHAM_DEV float wdecode(int fmt, uint32_t c, float zero, int kblk_e, float nf4a, int eref) {
    switch (fmt) {
    case CHAM_W_INT8_SYM: return (float)(int8_t)c;
    case CHAM_W_INT8_ASYM:
    case CHAM_W_INT4_ASYM: return (float)c - zero;
    case CHAM_W_MXINT8: return ldexpf((float)(int8_t)c, kblk_e - 6 - eref);
    case CHAM_W_INT4_SYM: return (float)((int)(c << 28) >> 28);
    case CHAM_W_NF4: return ldexpf(nf4_level(c) * nf4a, -eref);
    case CHAM_W_FP4: return e2m1_decode(c);
    case CHAM_W_MXINT4: return ldexpf((float)((int)(c << 28) >> 28), kblk_e - 2 - eref);
    default: return ldexpf(e2m1_decode(c), kblk_e - eref);  // MXFP4
    }
}

CHAM_DEV float adecode(int afmt, uint32_t c, float z, int kblk_e, int eref) {
    switch (afmt) {
    case CHAM_A_INT8_ASYM: return (float)c - z;
    case CHAM_A_FP8_E4M3: return e4m3_decode(c);
    case CHAM_A_FP8_E5M2: return e5m2_decode(c);
    case CHAM_A_MXFP8_E4M3: return ldexpf(e4m3_decode(c), kblk_e - eref);
    default: return ldexpf((float)(int8_t)c, kblk_e - 6 - eref);  // MXINT8
    }
}

template <int CODE_BITS>
__global__ __launch_bounds__(kThreads) void gemm_f16_kernel(GemmArgs a) {
    __shared__ _Float16 As[BM][LDK];
    __shared__ _Float16 Bs[BN][LDK];
    __shared__ ColInfo cinfo[BN];
    __shared__ int rowE[BM];

    const int t = threadIdx.x;
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const int K = a.K;
    const bool amx = a.afmt == CHAM_A_MXFP8_E4M3 || a.afmt == CHAM_A_MXINT8;
    const float az = *a.xz;

    // ---- per-channel / per-row prologue
    if (t < BN) {
        const int n = n0 + t;
        ColInfo ci{CHAM_W_INT8_SYM, 0, 0.0f, 0.0f};
        if (n < a.N && a.wfmt[n] < CHAM_W_NFMT && ((a.mask >> a.wfmt[n]) & 1u)) {
            const int f = a.wfmt[n];
            ci.fmt = f;
            ci.zero = (float)a.wzero[n];
            if (f == CHAM_W_NF4) {
                float mx = 0.0f;
                for (int b = 0; b < K / 64; ++b) mx = fmaxf(mx, a.wnf4[(int64_t)n * (K / 64) + b]);
                ci.eref = floor_log2(floor_scale(mx));
                ci.colscale = ldexpf(1.0f, ci.eref);
            } else if (f == CHAM_W_MXINT8 || f == CHAM_W_MXINT4 || f == CHAM_W_MXFP4) {
                int mx = 0;
                for (int b = 0; b < K / 32; ++b) mx = max(mx, (int)a.we8[(int64_t)n * (K / 32) + b]);
                const int F = f == CHAM_W_MXINT8 ? 6 : (f == CHAM_W_MXINT4 ? 2 : 0);
                ci.eref = mx - 127 - F;
                ci.colscale = ldexpf(1.0f, ci.eref);
            } else {
                ci.eref = 0;
                ci.colscale = a.wscale[n];
            }
        }
        cinfo[t] = ci;
    } else if (amx) {
        const int r = t - BN;
        const int m = m0 + r;
        int mx = 0;
        if (m < a.M)
            for (int b = 0; b < K / 32; ++b) mx = max(mx, (int)a.xe8[(int64_t)m * (K / 32) + b]);
        rowE[r] = mx - 127;
    }
    __syncthreads();

    const int lane = t & 63, wave = t >> 6;
    const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;
    float4v acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = float4v{0.f, 0.f, 0.f, 0.f};

    const int dr = t >> 1, dh = (t & 1) * 16;  // decode assignment: row/channel dr, k-half dh
    const ColInfo ci = cinfo[dr];
    const int my_rowE = amx ? rowE[dr] : 0;

    for (int k0 = 0; k0 < K; k0 += BK) {
        // ---- decode A: row dr, 16 codes
        {
            const int m = m0 + dr;
            _Float16 h[16];
            if (m < a.M) {
                const uint4 c4 = *reinterpret_cast<const uint4*>(a.xc + (int64_t)m * K + k0 + dh);
                const uint32_t cw[4] = {c4.x, c4.y, c4.z, c4.w};
                const int kb = amx ? (int)a.xe8[(int64_t)m * (K / 32) + (k0 >> 5)] - 127 : 0;
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    uint32_t c = (cw[j >> 2] >> (8 * (j & 3))) & 0xFFu;
                    h[j] = (_Float16)adecode(a.afmt, c, az, kb, my_rowE);
                }
            } else {
#pragma unroll
                for (int j = 0; j < 16; ++j) h[j] = (_Float16)0.0f;
            }
#pragma unroll
            for (int j = 0; j < 16; ++j) As[dr][dh + j] = h[j];
        }
        // ---- decode B: channel dr, 16 codes
        {
            const int n = n0 + dr;
            _Float16 h[16];
            if (n < a.N && ci.colscale != 0.0f) {
                uint32_t cw[4];
                if (CODE_BITS == 4) {
                    const uint2 c2 = *reinterpret_cast<const uint2*>(a.wc + (int64_t)n * (K / 2) + (k0 + dh) / 2);
                    cw[0] = c2.x; cw[1] = c2.y; cw[2] = 0; cw[3] = 0;
                } else {
                    const uint4 c4 = *reinterpret_cast<const uint4*>(a.wc + (int64_t)n * K + k0 + dh);
                    cw[0] = c4.x; cw[1] = c4.y; cw[2] = c4.z; cw[3] = c4.w;
                }
                int kb = 0;
                float nf = 0.0f;
                if (ci.fmt == CHAM_W_MXINT8 || ci.fmt == CHAM_W_MXINT4 || ci.fmt == CHAM_W_MXFP4)
                    kb = (int)a.we8[(int64_t)n * (K / 32) + (k0 >> 5)] - 127;
                if (ci.fmt == CHAM_W_NF4) nf = a.wnf4[(int64_t)n * (K / 64) + (k0 >> 6)];
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    uint32_t c = CODE_BITS == 4 ? (cw[j >> 3] >> (4 * (j & 7))) & 0xFu
                                                : (cw[j >> 2] >> (8 * (j & 3))) & 0xFFu;
                    h[j] = (_Float16)wdecode(ci.fmt, c, ci.zero, kb, nf, ci.eref);
                }
            } else {
#pragma unroll
                for (int j = 0; j < 16; ++j) h[j] = (_Float16)0.0f;
            }
#pragma unroll
            for (int j = 0; j < 16; ++j) Bs[dr][dh + j] = h[j];
        }
        __syncthreads();
        // ---- MFMA: each wave 64x64 = 4x4 tiles of 16x16, one K=32 step
        const int li = lane & 15, lk = (lane >> 4) * 8;
        half8 af[4], bf[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const half8*>(&As[wm + i * 16 + li][lk]);
#pragma unroll
        for (int j = 0; j < 4; ++j) bf[j] = *reinterpret_cast<const half8*>(&Bs[wn + j * 16 + li][lk]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[i], bf[j], acc[i][j], 0, 0, 0);
        __syncthreads();
    }

    // ---- epilogue: D[i][j] of a 16x16 tile: column lane%16, rows 4*(lane/16) + r
    const float xs = *a.xs;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int nl = wn + j * 16 + (lane & 15);
            const int n = n0 + nl;
            if (n >= a.N) continue;
            const float cs = cinfo[nl].colscale;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int ml = wm + i * 16 + (lane >> 4) * 4 + r;
                const int m = m0 + ml;
                if (m >= a.M) continue;
                const float rs = amx ? ldexpf(1.0f, rowE[ml]) : xs;
                a.Y[(int64_t)m * a.N + n] = (acc[i][j][r] * rs) * cs;
            }
        }
    }
}

}  // namespace
}  // namespace cham

using namespace cham;

extern "C" int cham_mixed_linear(const cham_aq* xq, const cham_wq* wq, float* Y, void* ws, size_t ws_bytes,
                                 void* stream) {
    (void)ws;
    (void)ws_bytes;
    if (!xq || !wq || !Y || !xq->codes || !xq->scale || !xq->zero) return CHAM_EINVAL;
    if (!wq->fmt || !wq->codes || !wq->scale || !wq->zero) return CHAM_EINVAL;
    if (xq->M < 1 || wq->N < 1 || xq->K < 1 || xq->K != wq->K) return CHAM_EINVAL;
    if (xq->M > INT32_MAX || wq->N > INT32_MAX || xq->K > INT32_MAX) return CHAM_EINVAL;
    if (xq->fmt < 0 || xq->fmt >= CHAM_A_NFMT) return CHAM_EFORMAT;
    const uint32_t mask = wq->palette_mask;
    if (mask == 0u || (mask >> CHAM_W_NFMT) != 0u) return CHAM_EFORMAT;
    const int code_bits = (mask & 0x7u) ? 8 : 4;
    if (wq->code_bits != code_bits) return CHAM_EFORMAT;
    if (xq->K % 32 != 0) return CHAM_ESHAPE;
    const bool nf4 = (mask >> CHAM_W_NF4) & 1u;
    const bool wmx = (mask & ((1u << CHAM_W_MXINT8) | (1u << CHAM_W_MXINT4) | (1u << CHAM_W_MXFP4))) != 0u;
    if (nf4 && xq->K % 64 != 0) return CHAM_ESHAPE;
    if ((nf4 && !wq->nf4_absmax) || (wmx && !wq->e8m0)) return CHAM_EINVAL;
    const bool amx = xq->fmt == CHAM_A_MXFP8_E4M3 || xq->fmt == CHAM_A_MXINT8;
    if (amx && !xq->e8m0) return CHAM_EINVAL;
    if (((uintptr_t)xq->codes & 15u) || ((uintptr_t)wq->codes & 15u)) return CHAM_EINVAL;
    GemmArgs a;
    a.mask = mask;
    a.xc = xq->codes;
    a.xe8 = xq->e8m0;
    a.xs = xq->scale;
    a.xz = xq->zero;
    a.afmt = xq->fmt;
    a.wfmt = wq->fmt;
    a.wc = wq->codes;
    a.wscale = wq->scale;
    a.wzero = wq->zero;
    a.wnf4 = wq->nf4_absmax;
    a.we8 = wq->e8m0;
    a.Y = Y;
    a.M = (int)xq->M;
    a.N = (int)wq->N;
    a.K = (int)xq->K;
    dim3 grid((unsigned)((a.N + BN - 1) / BN), (unsigned)((a.M + BM - 1) / BM));
    hipStream_t s = (hipStream_t)stream;
    if (code_bits == 4) hipLaunchKernelGGL(gemm_f16_kernel<4>, grid, dim3(kThreads), 0, s, a);
    else hipLaunchKernelGGL(gemm_f16_kernel<8>, grid, dim3(kThreads), 0, s, a);
    CHAM_CHECK_LAUNCH();
    return CHAM_OK;
}
