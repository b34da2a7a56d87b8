// DiT joint (group size, format) weight search (Sec. 4.6 (i)): for every tuple (g, f) of the
// group sizes {32, 64, 128, 192, 288} and the enabled formats, each output row is quantized
// in groups of g consecutive input channels, each with its own scale (and zero point), and
// the layer's input-aware error sum_n sum_k E[x_k^2] (w - w^)^2 is formed; the tuple with
// the smallest error (ties: the lowest index t = group index * 9 + format) is emitted.  MX
// formats carry their own 32-element blocks and are evaluated at g = 32 only.  Also the
// calibration pre-pass that gives E[x_k^2]: per-input-channel sums of squares.
//
// Three launches: (1) one wavefront per output channel stages its row in LDS and, for each
// enabled (g, f), computes the group parameters (one lane per group) and the channel's
// weighted error in binary64; (2) one workgroup sums the channels' errors per tuple in a
// fixed order and selects the tuple on the device; (3) one wavefront per channel re-derives
// the chosen tuple's group parameters and writes the codes and group metadata.  The host
// never reads the choice, so the search and a later GEMM need no synchronization.
#include <algorithm>

#include "cham_device.h"

namespace cham {
namespace {

constexpr int kGroupSizes[CHAM_NGROUPS] = {32, 64, 128, 192, 288};
constexpr int kTuples = CHAM_NGROUPS * CHAM_W_NFMT;
constexpr int kGWaves = 4;           // channels (wavefronts) per workgroup at most
constexpr int kGLdsMax = 64 * 1024;  // LDS per workgroup the launches stay within

CHAM_DEV bool mx_fmt(int f) { return f == CHAM_W_MXINT8 || f == CHAM_W_MXINT4 || f == CHAM_W_MXFP4; }

// Parameters of one group in one format: scale s, its reciprocal r, zero point z; for MX
// formats the block exponent in z.
struct GParam {
    float s, r, z;
};

CHAM_DEV GParam group_param(int f, float lo, float hi) {
    const float amax = fmaxf(fabsf(lo), fabsf(hi));
    GParam p{0.0f, 0.0f, 0.0f};
    switch (f) {
    case CHAM_W_INT8_SYM: p.s = floor_scale(amax / 127.0f); p.r = 1.0f / p.s; break;
    case CHAM_W_INT4_SYM: p.s = floor_scale(amax / 7.0f); p.r = 1.0f / p.s; break;
    case CHAM_W_INT8_ASYM: int_asym_scale_zp(lo, hi, 255.0f, &p.s, &p.z); p.r = 1.0f / p.s; break;
    case CHAM_W_INT4_ASYM: int_asym_scale_zp(lo, hi, 15.0f, &p.s, &p.z); p.r = 1.0f / p.s; break;
    case CHAM_W_FP4: p.s = floor_scale(amax / 6.0f); p.r = 1.0f / p.s; break;
    case CHAM_W_NF4: p.s = floor_scale(amax); p.r = 1.0f / p.s; break;
    case CHAM_W_MXINT8:
    case CHAM_W_MXINT4: p.z = (float)mx_exponent(amax, 0); break;
    default: p.z = (float)mx_exponent(amax, 2); break;  // MXFP4: OCP emax(E2M1) = 2
    }
    return p;
}

// Code and reconstruction of w in format f with its group's parameters (each step one
// binary32 operation, as the format defines it).
CHAM_DEV uint32_t group_quant(int f, float w, const GParam& p, float* wh) {
    switch (f) {
    case CHAM_W_INT8_SYM:
    case CHAM_W_INT4_SYM: {
        const float Q = f == CHAM_W_INT8_SYM ? 127.0f : 7.0f;
        const float q = clampf(rne(w * p.r), -Q, Q);
        *wh = q * p.s;
        return (uint32_t)(int)q & (f == CHAM_W_INT8_SYM ? 0xFFu : 0xFu);
    }
    case CHAM_W_INT8_ASYM:
    case CHAM_W_INT4_ASYM: {
        const float L = f == CHAM_W_INT8_ASYM ? 255.0f : 15.0f;
        const float q = clampf(rne(w * p.r) + p.z, 0.0f, L);
        *wh = (q - p.z) * p.s;
        return (uint32_t)q;
    }
    case CHAM_W_FP4: {
        float e;
        const uint32_t c = e2m1_encode(clampf(w * p.r, -6.0f, 6.0f), &e);
        *wh = e * p.s;
        return c;
    }
    case CHAM_W_NF4: {
        const uint32_t c = nf4_encode(w * p.r);
        *wh = nf4_level(c) * p.s;
        return c;
    }
    case CHAM_W_MXINT8:
    case CHAM_W_MXINT4: {
        const int E = (int)p.z, F = f == CHAM_W_MXINT8 ? 6 : 2;
        const float Q = f == CHAM_W_MXINT8 ? 127.0f : 7.0f;
        const float k = clampf(rne(ldexpf(w, F - E)), -Q, Q);
        *wh = ldexpf(k, E - F);
        return (uint32_t)(int)k & (f == CHAM_W_MXINT8 ? 0xFFu : 0xFu);
    }
    default: {  // MXFP4
        const int E = (int)p.z;
        float e;
        const uint32_t c = e2m1_encode(clampf(ldexpf(w, -E), -6.0f, 6.0f), &e);
        *wh = ldexpf(e, E);
        return c;
    }
    }
}

struct GSArgs {
    int waves;            // channels (wavefronts) per workgroup
    const float* W;
    const float* energy;  // [K]
    int N, K;
    uint32_t mask, gmask;
    int code_bits;
    double* cerr;          // [N][kTuples] per-channel errors (workspace)
    const int32_t* choice; // emit: {g, f}
    uint8_t* fmt;
    uint8_t* codes;
    float* gscale;
    float* gzero;
    uint8_t* e8;
};

// LDS of one wavefront: its row, then the parameters of up to K/32 groups (a stride rounded
// to 16 bytes so every row is float4-aligned).
__host__ __device__ inline int wave_lds_floats(int K) { return (K + 3 * (K / 32) + 3) & ~3; }
CHAM_DEV float* wave_row(float* lds, int K) { return lds + (threadIdx.x >> 6) * wave_lds_floats(K); }

// Row of channel n into LDS (float4), group parameters of (g, f) into LDS.
CHAM_DEV void stage_row(const GSArgs& a, int n, float* row) {
    const int lane = threadIdx.x & 63;
    const float4* src = reinterpret_cast<const float4*>(a.W + (int64_t)n * a.K);
    for (int q = lane; q < a.K / 4; q += 64) reinterpret_cast<float4*>(row)[q] = src[q];
}

CHAM_DEV void group_params(const float* row, int K, int g, int f, GParam* gp) {
    const int lane = threadIdx.x & 63;
    const int G = (K + g - 1) / g;
    for (int j = lane; j < G; j += 64) {
        const int k0 = j * g, k1 = min(k0 + g, K);
        float lo = INFINITY, hi = -INFINITY;
        for (int k = k0; k < k1; ++k) {
            lo = fminf(lo, row[k]);
            hi = fmaxf(hi, row[k]);
        }
        gp[j] = group_param(f, lo, hi);
    }
}

// (1) per-channel weighted errors of every enabled tuple
__global__ __launch_bounds__(256) void gsearch_err_kernel(GSArgs a) {
    extern __shared__ float lds[];
    const int lane = threadIdx.x & 63;
    const int n = blockIdx.x * a.waves + (threadIdx.x >> 6);
    if (n >= a.N) return;  // wavefront-uniform; no workgroup barrier below
    const int K = a.K;
    float* row = wave_row(lds, K);
    GParam* gp = reinterpret_cast<GParam*>(row + K);
    stage_row(a, n, row);
    __builtin_amdgcn_wave_barrier();
    double* out = a.cerr + (int64_t)n * kTuples;
    for (int gi = 0; gi < CHAM_NGROUPS; ++gi) {
        if (!((a.gmask >> gi) & 1u)) continue;
        const int g = kGroupSizes[gi];
        for (int f = 0; f < CHAM_W_NFMT; ++f) {
            if (!((a.mask >> f) & 1u) || (mx_fmt(f) && g != 32)) continue;
            group_params(row, K, g, f, gp);
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
            double e = 0.0;
            for (int k0 = 4 * lane; k0 < K; k0 += 256) {
                const float4 w4 = reinterpret_cast<const float4*>(row)[k0 >> 2];
                const float4 e4 = reinterpret_cast<const float4*>(a.energy)[k0 >> 2];
                const GParam p = gp[k0 / g];  // 4 consecutive elements share a group (g % 4 == 0)
                const float w[4] = {w4.x, w4.y, w4.z, w4.w}, ek[4] = {e4.x, e4.y, e4.z, e4.w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    float wh;
                    (void)group_quant(f, w[j], p, &wh);
                    const double d = (double)(w[j] - wh);
                    e = fma((double)ek[j], d * d, e);
                }
            }
            e = wave_sum(e);
            if (lane == 0) out[gi * CHAM_W_NFMT + f] = e;
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        }
    }
}

// (2) layer error of each tuple (channels added in a fixed order) and the choice
__global__ __launch_bounds__(256) void gsearch_select_kernel(const double* cerr, int N, uint32_t mask, uint32_t gmask,
                                                             int32_t* choice, double* err_out) {
    __shared__ double tot[kTuples];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int t = wave; t < kTuples; t += 4) {
        const int gi = t / CHAM_W_NFMT, f = t % CHAM_W_NFMT;
        const bool on = ((gmask >> gi) & 1u) && ((mask >> f) & 1u) && !(mx_fmt(f) && kGroupSizes[gi] != 32);
        double s = 0.0;
        if (on)
            for (int n = lane; n < N; n += 64) s += cerr[(int64_t)n * kTuples + t];
        s = wave_sum(s);
        if (lane == 0) tot[t] = on ? s : -1.0;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int best = -1;
        for (int t = 0; t < kTuples; ++t)
            if (tot[t] >= 0.0 && (best < 0 || tot[t] < tot[best])) best = t;
        choice[0] = best >= 0 ? kGroupSizes[best / CHAM_W_NFMT] : 0;
        choice[1] = best >= 0 ? best % CHAM_W_NFMT : CHAM_W_NFMT;
    }
    if (err_out)
        for (int t = threadIdx.x; t < kTuples; t += 256) err_out[t] = tot[t];
}

// (3) codes and group metadata of the chosen tuple
__global__ __launch_bounds__(256) void gsearch_emit_kernel(GSArgs a) {
    extern __shared__ float lds[];
    const int lane = threadIdx.x & 63;
    const int n = blockIdx.x * a.waves + (threadIdx.x >> 6);
    if (n >= a.N) return;
    const int K = a.K;
    const int g = a.choice[0], f = a.choice[1];
    float* row = wave_row(lds, K);
    GParam* gp = reinterpret_cast<GParam*>(row + K);
    stage_row(a, n, row);
    if (f >= CHAM_W_NFMT || g < 32) return;  // nothing was selected (checked on the host)
    __builtin_amdgcn_wave_barrier();
    group_params(row, K, g, f, gp);
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    const int G = (K + g - 1) / g;
    for (int j = lane; j < K / 32; j += 64) {
        const bool mx = mx_fmt(f);
        const GParam p = j < G ? gp[j] : GParam{0.0f, 0.0f, 0.0f};
        a.gscale[(int64_t)n * (K / 32) + j] = mx || j >= G ? 0.0f : p.s;
        a.gzero[(int64_t)n * (K / 32) + j] = mx || j >= G ? 0.0f : p.z;
        if (a.e8) a.e8[(int64_t)n * (K / 32) + j] = mx ? (uint8_t)((int)gp[j].z + 127) : (uint8_t)0;
    }
    if (lane == 0) a.fmt[n] = (uint8_t)f;
    for (int k0 = 4 * lane; k0 < K; k0 += 256) {
        const float4 w4 = reinterpret_cast<const float4*>(row)[k0 >> 2];
        const GParam p = gp[k0 / g];
        const float w[4] = {w4.x, w4.y, w4.z, w4.w};
        uint32_t cw = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float wh;
            const uint32_t c = group_quant(f, w[j], p, &wh);
            cw |= a.code_bits == 4 ? (c & 15u) << (4 * j) : (c & 255u) << (8 * j);
        }
        if (a.code_bits == 4) reinterpret_cast<uint16_t*>(a.codes + (int64_t)n * (K / 2))[k0 >> 2] = (uint16_t)cw;
        else reinterpret_cast<uint32_t*>(a.codes + (int64_t)n * K)[k0 >> 2] = cw;
    }
}

// ---- per-input-channel sums of squares: partials over row chunks, then a fixed-order sum
constexpr int kColChunks = 64;

__global__ __launch_bounds__(256) void colsq_partial_kernel(const float* X, int64_t M, int K, double* part) {
    const int k = blockIdx.x * 256 + threadIdx.x;
    const int c = blockIdx.y;
    if (k >= K) return;
    const int64_t m0 = M * c / kColChunks, m1 = M * (c + 1) / kColChunks;
    double s = 0.0;
    for (int64_t m = m0; m < m1; ++m) {
        const double x = (double)X[m * K + k];
        s = fma(x, x, s);
    }
    part[(int64_t)c * K + k] = s;
}

__global__ __launch_bounds__(256) void colsq_sum_kernel(const double* part, int K, double* colsq) {
    const int k = blockIdx.x * 256 + threadIdx.x;
    if (k >= K) return;
    double s = colsq[k];
    for (int c = 0; c < kColChunks; ++c) s += part[(int64_t)c * K + k];
    colsq[k] = s;
}

}  // namespace
}  // namespace cham

using namespace cham;

int cham_pack_grouped(const cham_gwq* gq, hipStream_t s);  // the GEMM's record pre-pass

// wavefronts per workgroup so that their rows and group parameters fit kGLdsMax
static int gsearch_waves(int64_t K) {
    const size_t per = (size_t)wave_lds_floats((int)K) * 4;
    return (int)std::max<size_t>(1, std::min<size_t>(kGWaves, kGLdsMax / per));
}

size_t cham_gselect_workspace_bytes(int64_t N) { return N > 0 ? (size_t)N * kTuples * sizeof(double) : 0; }
size_t cham_colsq_workspace_bytes(int64_t K) { return K > 0 ? (size_t)kColChunks * (size_t)K * sizeof(double) : 0; }

extern "C" int cham_select_group_formats(const float* W, const float* energy, cham_gwq* gq, void* ws, size_t ws_bytes,
                                         void* stream) {
    if (!W || !energy || !gq) return CHAM_EINVAL;
    const uint32_t mask = gq->palette_mask, gmask = gq->group_mask;
    if (mask == 0u || (mask >> CHAM_W_NFMT) != 0u || gmask == 0u || (gmask >> CHAM_NGROUPS) != 0u) return CHAM_EFORMAT;
    const uint32_t mxm = (1u << CHAM_W_MXINT8) | (1u << CHAM_W_MXINT4) | (1u << CHAM_W_MXFP4);
    if ((mask & ~mxm) == 0u && !(gmask & 1u)) return CHAM_EFORMAT;  // MX formats only, without g = 32
    if (gq->N < 1 || gq->K < 1 || gq->N > (int64_t)INT32_MAX - kGWaves) return CHAM_EINVAL;
    const int64_t K = gq->K;
    if (K % 32 != 0 || K > 8192) return CHAM_ESHAPE;
    if (!gq->choice || !gq->fmt || !gq->codes || !gq->gscale || !gq->gzero) return CHAM_EINVAL;
    if ((mask & mxm) && !gq->e8m0) return CHAM_EINVAL;
    if (((uintptr_t)W & 15u) || ((uintptr_t)energy & 15u) || ((uintptr_t)gq->codes & 3u)) return CHAM_EINVAL;
    const int code_bits = (mask & 0x7u) ? 8 : 4;
    if (gq->packed) {
        if (code_bits != 4 || K % 64 != 0) return CHAM_ESHAPE;  // the GEMM layout: 4-bit codes, 64-wide k-steps
        if (((uintptr_t)gq->packed & 255u) || gq->N * (K / 64) * 128 > (int64_t)INT32_MAX) return CHAM_EINVAL;
    }
    if (!ws || ws_bytes < cham_gselect_workspace_bytes(gq->N)) return CHAM_EWORKSPACE;
    gq->code_bits = code_bits;
    hipStream_t s = (hipStream_t)stream;
    GSArgs a;
    a.W = W;
    a.energy = energy;
    a.N = (int)gq->N;
    a.K = (int)K;
    a.mask = mask;
    a.gmask = gmask;
    a.code_bits = code_bits;
    a.cerr = (double*)ws;
    a.choice = gq->choice;
    a.fmt = gq->fmt;
    a.codes = gq->codes;
    a.gscale = gq->gscale;
    a.gzero = gq->gzero;
    a.e8 = (mask & mxm) ? gq->e8m0 : nullptr;
    a.waves = gsearch_waves(K);
    const dim3 grid((unsigned)((gq->N + a.waves - 1) / a.waves)), block((unsigned)(64 * a.waves));
    const size_t lds = (size_t)a.waves * (size_t)wave_lds_floats((int)K) * 4;
    hipLaunchKernelGGL(gsearch_err_kernel, grid, block, lds, s, a);
    CHAM_CHECK_LAUNCH();
    hipLaunchKernelGGL(gsearch_select_kernel, dim3(1), dim3(256), 0, s, (const double*)ws, a.N, mask, gmask,
                       gq->choice, gq->err);
    CHAM_CHECK_LAUNCH();
    hipLaunchKernelGGL(gsearch_emit_kernel, grid, block, lds, s, a);
    CHAM_CHECK_LAUNCH();
    if (gq->packed) return cham_pack_grouped(gq, s);
    return CHAM_OK;
}

extern "C" int cham_act_colsq_accumulate(const float* X, int64_t M, int64_t K, double* colsq, void* ws, size_t ws_bytes,
                                         void* stream) {
    if (!X || !colsq || M < 1 || K < 1 || K > INT32_MAX) return CHAM_EINVAL;
    if (!ws || ws_bytes < cham_colsq_workspace_bytes(K)) return CHAM_EWORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    const unsigned bx = (unsigned)((K + 255) / 256);
    hipLaunchKernelGGL(colsq_partial_kernel, dim3(bx, kColChunks), dim3(256), 0, s, X, M, (int)K, (double*)ws);
    CHAM_CHECK_LAUNCH();
    hipLaunchKernelGGL(colsq_sum_kernel, dim3(bx), dim3(256), 0, s, (const double*)ws, (int)K, colsq);
    CHAM_CHECK_LAUNCH();
    return CHAM_OK;
}
