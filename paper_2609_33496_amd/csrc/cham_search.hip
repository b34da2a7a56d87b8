// Per-output-channel weight-format search (Sec. 4.5, Eq. weight-argmax) and the stable
// grouping of channels by chosen format.
//
// One wavefront owns one output channel.  The row is read from HBM once (coalesced
// float4 loads) and held in registers; lane l holds elements 4(l + 64c) .. +3 of chunk c,
// so an MX block (32 elements) is 8 consecutive lanes and an NF4 block (64) 16 lanes.
// Row and block statistics come from shuffle reductions; every enabled format's round
// trip is evaluated from the registers, its squared error summed in binary64, and the
// winner's codes and metadata are written packed.  Nothing is re-read.
#include "cham_device.h"

namespace cham {
namespace {

struct SearchArgs {
    const float* W;
    int64_t N;
    int K;
    uint32_t mask;
    int code_bits;
    uint8_t* fmt;
    uint8_t* codes;
    float* scale;
    int32_t* zero;
    float* nf4a;
    uint8_t* e8;
    double* err;
};

// per-channel parameters of every format, computed from the row statistics
struct RowParams {
    float s_sym8, r_sym8, s_sym4, r_sym4;  // INT-sym
    float s_as8, r_as8, z_as8;             // INT-asym 8
    float s_as4, r_as4, z_as4;             // INT-asym 4
    float s_fp4, r_fp4;                    // FP4
};

// Quantize-dequantize of one element in format f.  blk32 = the element's 32-block absmax,
// blk64 = its 64-block absmax.  Returns the code (low bits) and writes the reconstruction.
template <int F>
CHAM_DEV uint32_t quant_one(float w, const RowParams& p, float blk32, float blk64, float* wh) {
    switch (F) {
    case CHAM_W_INT8_SYM: {
        float q = clampf(rne(w * p.r_sym8), -127.0f, 127.0f);
        *wh = q * p.s_sym8;
        return (uint32_t)(int)q & 0xFFu;
    }
    case CHAM_W_INT4_SYM: {
        float q = clampf(rne(w * p.r_sym4), -7.0f, 7.0f);
        *wh = q * p.s_sym4;
        return (uint32_t)(int)q & 0xFu;
    }
    case CHAM_W_INT8_ASYM: {
        float q = clampf(rne(w * p.r_as8) + p.z_as8, 0.0f, 255.0f);
        *wh = (q - p.z_as8) * p.s_as8;
        return (uint32_t)q;
    }
    case CHAM_W_INT4_ASYM: {
        float q = clampf(rne(w * p.r_as4) + p.z_as4, 0.0f, 15.0f);
        *wh = (q - p.z_as4) * p.s_as4;
        return (uint32_t)q;
    }
    case CHAM_W_FP4: {
        float y = clampf(w * p.r_fp4, -6.0f, 6.0f);
        float e;
        uint32_t c = e2m1_encode(y, &e);
        *wh = e * p.s_fp4;
        return c;
    }
    case CHAM_W_NF4: {
        float a = floor_scale(blk64);
        float r = 1.0f / a;
        uint32_t c = nf4_encode(w * r);
        *wh = nf4_level(c) * a;
        return c;
    }
    case CHAM_W_MXINT8: {
        int E = mx_exponent(blk32, 0);
        float k = clampf(rne(ldexpf(w, 6 - E)), -127.0f, 127.0f);
        *wh = ldexpf(k, E - 6);
        return (uint32_t)(int)k & 0xFFu;
    }
    case CHAM_W_MXINT4: {
        int E = mx_exponent(blk32, 0);
        float k = clampf(rne(ldexpf(w, 2 - E)), -7.0f, 7.0f);
        *wh = ldexpf(k, E - 2);
        return (uint32_t)(int)k & 0xFu;
    }
    default: {  // CHAM_W_MXFP4
        int E = mx_exponent(blk32, 2);
        float y = clampf(ldexpf(w, -E), -6.0f, 6.0f);
        float e;
        uint32_t c = e2m1_encode(y, &e);
        *wh = ldexpf(e, E);
        return c;
    }
    }
}

template <int F, int NCH>
CHAM_DEV void row_codes(const float (&v)[NCH][4], const RowParams& p, const float (&b32)[NCH],
                        const float (&b64)[NCH], int code_bits, uint32_t (&cws)[NCH]) {
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        uint32_t cw = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float wh;
            uint32_t code = quant_one<F>(v[c][j], p, b32[c], b64[c], &wh);
            cw |= code_bits == 4 ? (code & 15u) << (4 * j) : (code & 255u) << (8 * j);
        }
        cws[c] = cw;
    }
}

// Squared reconstruction error of one element in format F, accumulated in binary64.  The
// square of a binary32 difference is exact in binary64, so fma(d, d, e) == e + d*d.
template <int F>
CHAM_DEV void acc_err(float w, const RowParams& p, float blk32, float blk64, double& e) {
    float wh;
    (void)quant_one<F>(w, p, blk32, blk64, &wh);
    const double d = (double)(w - wh);
    e = fma(d, d, e);
}

CHAM_DEV float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }

template <uint32_t MASK, int NCH>
__global__ __launch_bounds__(256) void search_kernel(SearchArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t n = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (n >= a.N) return;  // wave-uniform
    const int K = a.K;
    const int nq = K >> 2;  // float4 per row
    const float* row = a.W + n * (int64_t)K;

    float v[NCH][4];
    bool valid[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        int q = c * 64 + lane;
        valid[c] = q < nq;
        float4 t = valid[c] ? ld4(row + 4 * q) : make_float4(0.f, 0.f, 0.f, 0.f);
        v[c][0] = t.x; v[c][1] = t.y; v[c][2] = t.z; v[c][3] = t.w;
    }

    // ---- row and block statistics
    float lo = INFINITY, hi = -INFINITY;
    float b32[NCH], b64[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        float m = 0.0f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            m = fmaxf(m, fabsf(v[c][j]));
            if (valid[c]) { lo = fminf(lo, v[c][j]); hi = fmaxf(hi, v[c][j]); }
        }
        b32[c] = group_max<8>(m);
        b64[c] = fmaxf(b32[c], __shfl_xor(b32[c], 8, kWave));
    }
    lo = wave_min(lo);
    hi = wave_max(hi);
    const float amax = fmaxf(fabsf(lo), fabsf(hi));

    RowParams p;
    p.s_sym8 = floor_scale(amax / 127.0f); p.r_sym8 = 1.0f / p.s_sym8;
    p.s_sym4 = floor_scale(amax / 7.0f);   p.r_sym4 = 1.0f / p.s_sym4;
    {
        float l0 = fminf(lo, 0.0f), h0 = fmaxf(hi, 0.0f);
        p.s_as8 = floor_scale((h0 - l0) / 255.0f); p.r_as8 = 1.0f / p.s_as8;
        p.z_as8 = clampf(rne(-l0 / p.s_as8), 0.0f, 255.0f);
        p.s_as4 = floor_scale((h0 - l0) / 15.0f);  p.r_as4 = 1.0f / p.s_as4;
        p.z_as4 = clampf(rne(-l0 / p.s_as4), 0.0f, 15.0f);
    }
    p.s_fp4 = floor_scale(amax / 6.0f); p.r_fp4 = 1.0f / p.s_fp4;

    // ---- error of every enabled format: one fused pass over the row held in registers
    const uint32_t mask = MASK ? MASK : a.mask;
    double e[CHAM_W_NFMT];
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) e[f] = 0.0;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (!valid[c]) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float w = v[c][j];
            if (mask & (1u << 0)) acc_err<0>(w, p, b32[c], b64[c], e[0]);
            if (mask & (1u << 1)) acc_err<1>(w, p, b32[c], b64[c], e[1]);
            if (mask & (1u << 2)) acc_err<2>(w, p, b32[c], b64[c], e[2]);
            if (mask & (1u << 3)) acc_err<3>(w, p, b32[c], b64[c], e[3]);
            if (mask & (1u << 4)) acc_err<4>(w, p, b32[c], b64[c], e[4]);
            if (mask & (1u << 5)) acc_err<5>(w, p, b32[c], b64[c], e[5]);
            if (mask & (1u << 6)) acc_err<6>(w, p, b32[c], b64[c], e[6]);
            if (mask & (1u << 7)) acc_err<7>(w, p, b32[c], b64[c], e[7]);
            if (mask & (1u << 8)) acc_err<8>(w, p, b32[c], b64[c], e[8]);
        }
    }
    int best = -1;
    double best_err = 0.0;
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) {
        if (!(mask & (1u << f))) {
            if (a.err && lane == 0) a.err[n * CHAM_W_NFMT + f] = -1.0;
            continue;
        }
        const double ef = wave_sum(e[f]);
        if (a.err && lane == 0) a.err[n * CHAM_W_NFMT + f] = ef;
        if (best < 0 || ef < best_err) { best = f; best_err = ef; }
    }

    // ---- emit the winner's codes and metadata
    const int f = best;
    if (lane == 0) {
        a.fmt[n] = (uint8_t)f;
        float s = 0.0f;
        int32_t z = 0;
        if (f == CHAM_W_INT8_SYM) s = p.s_sym8;
        else if (f == CHAM_W_INT4_SYM) s = p.s_sym4;
        else if (f == CHAM_W_INT8_ASYM) { s = p.s_as8; z = (int32_t)p.z_as8; }
        else if (f == CHAM_W_INT4_ASYM) { s = p.s_as4; z = (int32_t)p.z_as4; }
        else if (f == CHAM_W_FP4) s = p.s_fp4;
        a.scale[n] = s;
        a.zero[n] = z;
    }
    const bool is_mx = f == CHAM_W_MXINT8 || f == CHAM_W_MXINT4 || f == CHAM_W_MXFP4;
    uint32_t cws[NCH];
    switch (f) {
    case 0: row_codes<0, NCH>(v, p, b32, b64, a.code_bits, cws); break;
    case 1: row_codes<1, NCH>(v, p, b32, b64, a.code_bits, cws); break;
    case 2: row_codes<2, NCH>(v, p, b32, b64, a.code_bits, cws); break;
    case 3: row_codes<3, NCH>(v, p, b32, b64, a.code_bits, cws); break;
    case 4: row_codes<4, NCH>(v, p, b32, b64, a.code_bits, cws); break;
    case 5: row_codes<5, NCH>(v, p, b32, b64, a.code_bits, cws); break;
    case 6: row_codes<6, NCH>(v, p, b32, b64, a.code_bits, cws); break;
    case 7: row_codes<7, NCH>(v, p, b32, b64, a.code_bits, cws); break;
    default: row_codes<8, NCH>(v, p, b32, b64, a.code_bits, cws); break;
    }
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (!valid[c]) continue;
        const int q = c * 64 + lane;
        const uint32_t cw = cws[c];
        if (a.code_bits == 4) {
            reinterpret_cast<uint16_t*>(a.codes + n * (int64_t)(K / 2))[q] = (uint16_t)cw;
        } else {
            reinterpret_cast<uint32_t*>(a.codes + n * (int64_t)K)[q] = cw;
        }
        if (a.e8 && (lane & 7) == 0) {
            int E = f == CHAM_W_MXFP4 ? mx_exponent(b32[c], 2) : mx_exponent(b32[c], 0);
            a.e8[n * (int64_t)(K / 32) + (q >> 3)] = is_mx ? (uint8_t)(E + 127) : (uint8_t)0;
        }
        if (a.nf4a && (lane & 15) == 0) {
            a.nf4a[n * (int64_t)(K / 64) + (q >> 4)] = f == CHAM_W_NF4 ? floor_scale(b64[c]) : 0.0f;
        }
    }
}

// Stable counting sort of channels by format, in one workgroup: thread t owns rows
// [t*R, (t+1)*R); per-format counts are prefix-summed across threads in LDS.
__global__ __launch_bounds__(1024) void group_kernel(const uint8_t* fmt, int64_t N, int32_t* perm,
                                                     int32_t* group_off) {
    __shared__ int32_t cnt[CHAM_W_NFMT][1024];
    __shared__ int32_t tot[CHAM_W_NFMT + 1];
    const int t = threadIdx.x;
    const int64_t R = (N + 1023) / 1024;
    const int64_t r0 = t * R, r1 = r0 + R < N ? r0 + R : N;
    int32_t c[CHAM_W_NFMT];
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) c[f] = 0;
    for (int64_t r = r0; r < r1; ++r) {
        int f = fmt[r];
#pragma unroll
        for (int g = 0; g < CHAM_W_NFMT; ++g) c[g] += (f == g);
    }
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) cnt[f][t] = c[f];
    __syncthreads();
    // inclusive scan over threads for each format (Hillis-Steele)
    for (int o = 1; o < 1024; o <<= 1) {
        int32_t add[CHAM_W_NFMT];
#pragma unroll
        for (int f = 0; f < CHAM_W_NFMT; ++f) add[f] = t >= o ? cnt[f][t - o] : 0;
        __syncthreads();
#pragma unroll
        for (int f = 0; f < CHAM_W_NFMT; ++f) cnt[f][t] += add[f];
        __syncthreads();
    }
    if (t == 0) {
        int32_t acc = 0;
        for (int f = 0; f < CHAM_W_NFMT; ++f) { tot[f] = acc; acc += cnt[f][1023]; }
        tot[CHAM_W_NFMT] = acc;
    }
    __syncthreads();
    if (group_off && t <= CHAM_W_NFMT) group_off[t] = tot[t];
    if (perm) {
        int32_t pos[CHAM_W_NFMT];
#pragma unroll
        for (int f = 0; f < CHAM_W_NFMT; ++f) pos[f] = tot[f] + cnt[f][t] - c[f];
        for (int64_t r = r0; r < r1; ++r) {
            int f = fmt[r];
            int32_t p = 0;
#pragma unroll
            for (int g = 0; g < CHAM_W_NFMT; ++g) {
                if (f == g) { p = pos[g]; pos[g]++; }
            }
            perm[p] = (int32_t)r;
        }
    }
}

template <int NCH>
void launch_search(const SearchArgs& a, hipStream_t s) {
    dim3 grid((unsigned)((a.N + 3) / 4));
    if (a.mask == CHAM_MASK_W4) hipLaunchKernelGGL((search_kernel<CHAM_MASK_W4, NCH>), grid, dim3(256), 0, s, a);
    else if (a.mask == CHAM_MASK_W8) hipLaunchKernelGGL((search_kernel<CHAM_MASK_W8, NCH>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((search_kernel<0u, NCH>), grid, dim3(256), 0, s, a);
}

}  // namespace
}  // namespace cham

using namespace cham;

static int mask_code_bits(uint32_t mask) {
    return (mask & 0x7u) ? 8 : 4;  // formats 0..2 are the 8-bit ones
}

extern "C" int cham_select_weight_formats(const float* W, cham_wq* wq, void* stream) {
    if (!W || !wq) return CHAM_EINVAL;
    const uint32_t mask = wq->palette_mask;
    if (mask == 0u || (mask >> CHAM_W_NFMT) != 0u) return CHAM_EFORMAT;
    if (wq->N < 1 || wq->K < 1 || wq->N > (int64_t)INT32_MAX) return CHAM_EINVAL;
    const int64_t K = wq->K;
    if (K % 32 != 0) return CHAM_ESHAPE;
    const bool nf4 = (mask >> CHAM_W_NF4) & 1u;
    const bool mx = (mask & ((1u << CHAM_W_MXINT8) | (1u << CHAM_W_MXINT4) | (1u << CHAM_W_MXFP4))) != 0u;
    if (nf4 && K % 64 != 0) return CHAM_ESHAPE;
    if (!wq->fmt || !wq->codes || !wq->scale || !wq->zero) return CHAM_EINVAL;
    if ((nf4 && !wq->nf4_absmax) || (mx && !wq->e8m0)) return CHAM_EINVAL;
    if (K > 32 * 256) return CHAM_ESHAPE;  // rows up to 8192 are held in registers
    wq->code_bits = mask_code_bits(mask);

    SearchArgs a;
    a.W = W;
    a.N = wq->N;
    a.K = (int)K;
    a.mask = mask;
    a.code_bits = wq->code_bits;
    a.fmt = wq->fmt;
    a.codes = wq->codes;
    a.scale = wq->scale;
    a.zero = wq->zero;
    a.nf4a = nf4 ? wq->nf4_absmax : nullptr;  // block metadata is written only when its format is enabled
    a.e8 = mx ? wq->e8m0 : nullptr;
    a.err = wq->err;
    hipStream_t s = (hipStream_t)stream;
    const int nch = (int)((K + 255) / 256);
    if (nch <= 3) launch_search<3>(a, s);
    else if (nch <= 5) launch_search<5>(a, s);
    else if (nch <= 10) launch_search<10>(a, s);
    else if (nch <= 20) launch_search<20>(a, s);
    else launch_search<32>(a, s);
    CHAM_CHECK_LAUNCH();
    if (wq->perm || wq->group_off) {
        hipLaunchKernelGGL(group_kernel, dim3(1), dim3(1024), 0, s, wq->fmt, wq->N, wq->perm, wq->group_off);
        CHAM_CHECK_LAUNCH();
    }
    return CHAM_OK;
}
