// Per-output-channel weight-format search (Sec. 4.5, Eq. weight-argmax) and the stable
// grouping of channels by chosen format.
//
// One wavefront owns one output channel.  The row is read from HBM once (coalesced float4
// loads) and held in registers: lane l holds elements 4(l + 64c) .. +3 of chunk c, so an MX
// block (32 elements) is 8 consecutive lanes and an NF4 block (64) 16 lanes.  Row and block
// statistics come from DPP reductions.  One fused pass round-trips every element through
// every enabled format and accumulates the squared reconstruction errors in binary32; the
// per-element reconstructions are the exact binary32 values the format defines (E2M1 via
// the gfx950 FP4 converters, which round to nearest even and saturate exactly as the format
// requires; NF4 through a 33-cell table in LDS plus one exact threshold comparison).  If
// the two smallest error sums are within 2^-15 of each other -- above the binary32
// summation error -- the errors of every enabled format are recomputed with binary64 sums,
// so the choice is always the binary64 argmin.  The winner's codes and metadata are then
// written packed.  Nothing is re-read from HBM.
#include <algorithm>
#include <vector>

#include "cham_device.h"
#include "cham_group.h"

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
    float* zero;
    float* nf4a;
    uint8_t* e8;
    double* err;
    int split;  // wavefronts per channel: 1, or 4 (a quarter of the row each)
    int lpc;    // 16, 32 or 64: lanes per channel of the 8-elements-per-lane kernel; 0: not used
};

// per-channel parameters of the per-channel formats
struct RowParams {
    float s_sym8, r_sym8, s_sym4, r_sym4;  // INT-sym
    float s_as8, r_as8, z_as8;             // INT-asym 8
    float s_as4, r_as4, z_as4;             // INT-asym 4
    float s_fp4, r_fp4;                    // FP4
};

// ------------------------------------------------------------------------------------
// DPP reductions
// ------------------------------------------------------------------------------------
// Every control used here reads a lane of the same wavefront row, so no lane is invalid and
// bound_ctrl is free to set: it lets the compiler fold the move into the consuming min/max/add.
template <int CTRL>
CHAM_DEV float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}
// max over the aligned 8-lane group (quad_perm 1,0,3,2; quad_perm 2,3,0,1; row_half_mirror)
CHAM_DEV float max8(float v) {
    v = fmaxf(v, dpp<0xB1>(v));
    v = fmaxf(v, dpp<0x4E>(v));
    return fmaxf(v, dpp<0x141>(v));
}
CHAM_DEV float max16_from8(float v) { return fmaxf(v, dpp<0x140>(v)); }  // row_mirror
// reductions over the wave: within rows of 16 by DPP, then the 4 rows by readlane
CHAM_DEV float row_sum16(float v) {
    v += dpp<0xB1>(v);
    v += dpp<0x4E>(v);
    v += dpp<0x141>(v);
    return v + dpp<0x140>(v);
}
CHAM_DEV float lane_f(float v, int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l)); }
CHAM_DEV float wave_sum_dpp(float v) {
    v = row_sum16(v);
    return (lane_f(v, 0) + lane_f(v, 16)) + (lane_f(v, 32) + lane_f(v, 48));
}
CHAM_DEV float wave_min_dpp(float v) {
    v = fminf(v, dpp<0xB1>(v));
    v = fminf(v, dpp<0x4E>(v));
    v = fminf(v, dpp<0x141>(v));
    v = fminf(v, dpp<0x140>(v));
    return fminf(fminf(lane_f(v, 0), lane_f(v, 16)), fminf(lane_f(v, 32), lane_f(v, 48)));
}
CHAM_DEV float wave_max_dpp(float v) {
    v = max16_from8(max8(v));
    return fmaxf(fmaxf(lane_f(v, 0), lane_f(v, 16)), fmaxf(lane_f(v, 32), lane_f(v, 48)));
}

// ------------------------------------------------------------------------------------
// NF4 lookup: cell i of [-1, 1] (width 1/16) holds cnt = number of decision thresholds
// below the cell's lower bound, the first threshold at or above it (+inf if none), and
// the levels cnt and cnt+1.  Consecutive thresholds are more than 1/16 apart and none is
// within 1e-3 of a cell boundary, so for y in the cell the nearest level is
// cnt + (y > thr); an index computed one cell off near a boundary gives the same code.
// ------------------------------------------------------------------------------------
struct NF4Cell {
    float thr, vlo, vhi;
    uint32_t cnt;
};

CHAM_DEV void nf4_cells_init(NF4Cell* cells) {
    const int i = threadIdx.x;
    if (i < 33) {
        const float b = -1.0f + (float)i * 0.0625f;
        uint32_t cnt = 0;
#pragma unroll
        for (int j = 0; j < 15; ++j) cnt += (__uint_as_float(kNF4ThrBits[j]) < b) ? 1u : 0u;
        NF4Cell c;
        c.cnt = cnt;
        c.thr = cnt < 15 ? __uint_as_float(kNF4ThrBits[cnt]) : INFINITY;
        c.vlo = nf4_level(cnt);
        c.vhi = nf4_level(cnt < 15 ? cnt + 1 : 15);
        cells[i] = c;
    }
}

// y = w fl(1/a) with |w| <= a, so |y| <= 1 + 2^-23: 16 y + 16 truncates to 0 .. 32.
CHAM_DEV NF4Cell nf4_cell(const NF4Cell* cells, float y) {
    return cells[(int)__builtin_fmaf(y, 16.0f, 16.0f)];
}

// ------------------------------------------------------------------------------------
// exact per-element quantize-dequantize of format F (used for the emitted codes and for
// the binary64 re-check); blk32 / blk64 = the element's 32- / 64-block absmax
// ------------------------------------------------------------------------------------
template <int F>
CHAM_DEV uint32_t quant_one(float w, const RowParams& p, float blk32, float blk64, const NF4Cell* cells, float* wh) {
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
        float y = w * rcp_rn(a);
        const NF4Cell cl = nf4_cell(cells, y);
        const bool up = y > cl.thr;
        *wh = (up ? cl.vhi : cl.vlo) * a;
        return cl.cnt + (up ? 1u : 0u);
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

// ------------------------------------------------------------------------------------
// fast binary32 error accumulation of one chunk (4 elements) in format F
// ------------------------------------------------------------------------------------
typedef float v2f __attribute__((ext_vector_type(2)));

// 2^E as the binary32 scale operand of the FP4 converters (they read its exponent field)
CHAM_DEV float e8m0_scale(int E) { return __uint_as_float((uint32_t)(E + 127) << 23); }

// E2M1 round trip of four values through the hardware converter with a power-of-two scale:
// the two pairs' codes go to bytes 0 and 1 of one register.  `old` is any value that is
// dead after the call (the converter only replaces the selected byte).
CHAM_DEV void fp4_quad(float y0, float y1, float y2, float y3, float scale, uint32_t old, v2f& lo, v2f& hi) {
    uint32_t c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, y0, y1, scale, 0);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, y2, y3, scale, 1);
    lo = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, scale, 0);
    hi = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, scale, 1);
}

// e0 / e2: the chunk's MX block exponent for emax 0 (MXINT) and 2 (MXFP4)
template <int F>
CHAM_DEV float chunk_err(const float (&w)[4], const RowParams& p, float blk32, float blk64, const NF4Cell* cells,
                         int e0, int e2) {
    float e = 0.0f;
    if (F == CHAM_W_INT8_ASYM || F == CHAM_W_INT4_ASYM) {
        const float r = F == CHAM_W_INT8_ASYM ? p.r_as8 : p.r_as4;
        const float s = F == CHAM_W_INT8_ASYM ? p.s_as8 : p.s_as4;
        const float z = F == CHAM_W_INT8_ASYM ? p.z_as8 : p.z_as4;
        const float L = F == CHAM_W_INT8_ASYM ? 255.0f : 15.0f;
        if (fabsf(z) <= 0x1p23f) {  // wavefront-uniform (one channel per wavefront)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                // clamp(round(w r) + z, 0, L) - z == clamp(round(w r), -z, L - z): with |z| <= 2^23
                // every integer here is exact in binary32
                const float u = __builtin_amdgcn_fmed3f(rne(w[j] * r), -z, L - z);
                const float d = w[j] - u * s;
                e = __builtin_fmaf(d, d, e);
            }
        } else {  // a zero point beyond 2^23: the sums round, so each step as the format states it
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float q = __builtin_amdgcn_fmed3f(rne(w[j] * r) + z, 0.0f, L);
                const float d = w[j] - (q - z) * s;
                e = __builtin_fmaf(d, d, e);
            }
        }
    } else if (F == CHAM_W_INT8_SYM || F == CHAM_W_INT4_SYM) {
        const float r = F == CHAM_W_INT8_SYM ? p.r_sym8 : p.r_sym4;
        const float s = F == CHAM_W_INT8_SYM ? p.s_sym8 : p.s_sym4;
        const float Q = F == CHAM_W_INT8_SYM ? 127.0f : 7.0f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float q = __builtin_amdgcn_fmed3f(rne(w[j] * r), -Q, Q);
            const float d = w[j] - q * s;
            e = __builtin_fmaf(d, d, e);
        }
    } else if (F == CHAM_W_FP4) {
        const float y0 = w[0] * p.r_fp4;
        v2f v[2];
        fp4_quad(y0, w[1] * p.r_fp4, w[2] * p.r_fp4, w[3] * p.r_fp4, 1.0f, __float_as_uint(y0), v[0], v[1]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float d = w[j] - v[j >> 1][j & 1] * p.s_fp4;
            e = __builtin_fmaf(d, d, e);
        }
    } else if (F == CHAM_W_MXFP4) {
        const float sc = e8m0_scale(e2);
        v2f v[2];
        fp4_quad(w[0], w[1], w[2], w[3], sc, 0u, v[0], v[1]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float d = w[j] - v[j >> 1][j & 1];
            e = __builtin_fmaf(d, d, e);
        }
    } else if (F == CHAM_W_MXINT4 || F == CHAM_W_MXINT8) {
        // in the block's scaled domain: y = w 2^(F-E) exactly, d = y - k exactly
        const int Fb = F == CHAM_W_MXINT8 ? 6 : 2;
        const float Q = F == CHAM_W_MXINT8 ? 127.0f : 7.0f;
        const int E = e0;
        float es = 0.0f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float y = ldexpf(w[j], Fb - E);
            const float k = __builtin_amdgcn_fmed3f(rne(y), -Q, Q);
            const float d = y - k;
            es = __builtin_fmaf(d, d, es);
        }
        e = ldexpf(es, 2 * (E - Fb));
    } else {  // NF4
        const float a = floor_scale(blk64);
        const float r = rcp_rn(a);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float y = w[j] * r;
            const NF4Cell cl = nf4_cell(cells, y);
            const float d = w[j] - (y > cl.thr ? cl.vhi : cl.vlo) * a;
            e = __builtin_fmaf(d, d, e);
        }
    }
    return e;
}

// NF4 error of one chunk, and the chunk's NF4 codes packed as the emitted layout has them
// (4 bits per code, or one byte per code with 8-bit codes): the error pass already finds
// each code, so a channel that chooses NF4 needs no second quantization pass.
CHAM_DEV float chunk_err_nf4(const float (&w)[4], float blk64, const NF4Cell* cells, int code_bits, uint32_t& cw) {
    const float a = floor_scale(blk64);
    const float r = rcp_rn(a);
    float e = 0.0f;
    cw = 0u;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const float y = w[j] * r;
        const NF4Cell cl = nf4_cell(cells, y);
        const bool up = y > cl.thr;
        const float d = w[j] - (up ? cl.vhi : cl.vlo) * a;
        e = __builtin_fmaf(d, d, e);
        cw |= (cl.cnt + (up ? 1u : 0u)) << (code_bits == 4 ? 4 * j : 8 * j);
    }
    return e;
}

template <int F, int NCH>
CHAM_DEV void row_codes(const float (&v)[NCH][4], const RowParams& p, const float (&b32)[NCH],
                        const float (&b64)[NCH], const NF4Cell* cells, int code_bits, uint32_t (&cws)[NCH]) {
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        uint32_t cw = 0;
        if (F == CHAM_W_MXFP4 || F == CHAM_W_FP4) {
            // hardware converter: two codes per byte, even element in the low nibble
            uint32_t c01, c23;
            if (F == CHAM_W_MXFP4) {
                const float sc = e8m0_scale(mx_exponent(b32[c], 2));
                c01 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, v[c][0], v[c][1], sc, 0) & 0xFFu;
                c23 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, v[c][2], v[c][3], sc, 0) & 0xFFu;
            } else {
                c01 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, v[c][0] * p.r_fp4, v[c][1] * p.r_fp4, 1.0f, 0) & 0xFFu;
                c23 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, v[c][2] * p.r_fp4, v[c][3] * p.r_fp4, 1.0f, 0) & 0xFFu;
            }
            if (code_bits == 4) cw = c01 | (c23 << 8);
            else cw = (c01 & 15u) | ((c01 >> 4) << 8) | ((c23 & 15u) << 16) | ((c23 >> 4) << 24);
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                float wh;
                uint32_t code = quant_one<F>(v[c][j], p, b32[c], b64[c], cells, &wh);
                cw |= code_bits == 4 ? (code & 15u) << (4 * j) : (code & 255u) << (8 * j);
            }
        }
        cws[c] = cw;
    }
}

template <int F, int NCH>
CHAM_DEV double row_err64(const float (&v)[NCH][4], const bool (&valid)[NCH], const RowParams& p,
                          const float (&b32)[NCH], const float (&b64)[NCH], const NF4Cell* cells) {
    double e = 0.0;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (!valid[c]) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float wh;
            (void)quant_one<F>(v[c][j], p, b32[c], b64[c], cells, &wh);
            const double d = (double)(v[c][j] - wh);
            e = fma(d, d, e);
        }
    }
    return wave_sum(e);
}

CHAM_DEV float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }

// Cross-wavefront sums when `split` wavefronts share a channel (split = 4: the whole
// workgroup); partial values are combined in wavefront order, so the result is fixed.
struct SplitLDS {
    float lohi[4][2];
    float e[4][CHAM_W_NFMT];
    double ed[4][CHAM_W_NFMT];
};

// Search of channel n by `split` wavefronts; this wavefront holds part `part` of the row
// (K / split consecutive elements, a multiple of 64).  split is the same for the whole
// workgroup, so the barriers below are reached by all of its wavefronts.
template <uint32_t MASK, int NCH>
CHAM_DEV void search_row(const SearchArgs& a, const NF4Cell* cells, int64_t n, int part, SplitLDS* sl) {
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int K = a.K;
    const int SPLIT = a.split;
    // elements [sp, sp + lp) of the row: split rows are cut at 64-element block boundaries
    // (K % 64 == 0), the quarters within one block of each other
    const int nblk = K / 64;
    const int sp = SPLIT > 1 ? (part * nblk / SPLIT) * 64 : 0;
    const int lp = SPLIT > 1 ? ((part + 1) * nblk / SPLIT) * 64 - sp : K;
    const int nq = lp >> 2;  // float4 of this wavefront
    const float* row = a.W + n * (int64_t)K + sp;
    const uint32_t mask = MASK ? MASK : a.mask;

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
        float m = fmaxf(fmaxf(fabsf(v[c][0]), fabsf(v[c][1])), fmaxf(fabsf(v[c][2]), fabsf(v[c][3])));
        if (valid[c]) {
            lo = fminf(lo, fminf(fminf(v[c][0], v[c][1]), fminf(v[c][2], v[c][3])));
            hi = fmaxf(hi, fmaxf(fmaxf(v[c][0], v[c][1]), fmaxf(v[c][2], v[c][3])));
        }
        b32[c] = max8(m);
        b64[c] = max16_from8(b32[c]);
    }
    lo = wave_min_dpp(lo);
    hi = wave_max_dpp(hi);
    if (SPLIT > 1) {
        if (lane == 0) { sl->lohi[wv][0] = lo; sl->lohi[wv][1] = hi; }
        __syncthreads();
#pragma unroll
        for (int w = 0; w < 4; ++w) { lo = fminf(lo, sl->lohi[w][0]); hi = fmaxf(hi, sl->lohi[w][1]); }
    }
    const float amax = fmaxf(fabsf(lo), fabsf(hi));

    RowParams p;
    p.s_sym8 = floor_scale(amax / 127.0f); p.r_sym8 = rcp_rn(p.s_sym8);
    p.s_sym4 = floor_scale(amax / 7.0f);   p.r_sym4 = rcp_rn(p.s_sym4);
    int_asym_scale_zp(lo, hi, 255.0f, &p.s_as8, &p.z_as8);
    p.r_as8 = rcp_rn(p.s_as8);
    int_asym_scale_zp(lo, hi, 15.0f, &p.s_as4, &p.z_as4);
    p.r_as4 = rcp_rn(p.s_as4);
    p.s_fp4 = floor_scale(amax / 6.0f); p.r_fp4 = rcp_rn(p.s_fp4);

    // ---- binary32 error sums of every enabled format, one fused pass
    float e[CHAM_W_NFMT];
    uint32_t nf4cw[NCH];  // NF4 codes of each chunk, kept from the error pass
#pragma unroll
    for (int c = 0; c < NCH; ++c) nf4cw[c] = 0u;
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) e[f] = 0.0f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (!valid[c]) continue;
        // the block exponent of both MX emax values from one floor(log2 amax): the exponent
        // of frexp (mantissa in [1/2, 1)) less one, subnormal blocks included
        const bool nz32 = b32[c] > 0.0f;
        const int fl32 = __builtin_amdgcn_frexp_expf(b32[c]) - 1;
        const int e0 = mx_exponent_fl(fl32, nz32, 0), e2 = mx_exponent_fl(fl32, nz32, 2);
        if (mask & (1u << 0)) e[0] += chunk_err<0>(v[c], p, b32[c], b64[c], cells, e0, e2);
        if (mask & (1u << 1)) e[1] += chunk_err<1>(v[c], p, b32[c], b64[c], cells, e0, e2);
        if (mask & (1u << 2)) e[2] += chunk_err<2>(v[c], p, b32[c], b64[c], cells, e0, e2);
        if (mask & (1u << 3)) e[3] += chunk_err<3>(v[c], p, b32[c], b64[c], cells, e0, e2);
        if (mask & (1u << 4)) e[4] += chunk_err<4>(v[c], p, b32[c], b64[c], cells, e0, e2);
        if (mask & (1u << 5)) e[5] += chunk_err_nf4(v[c], b64[c], cells, a.code_bits, nf4cw[c]);
        if (mask & (1u << 6)) e[6] += chunk_err<6>(v[c], p, b32[c], b64[c], cells, e0, e2);
        if (mask & (1u << 7)) e[7] += chunk_err<7>(v[c], p, b32[c], b64[c], cells, e0, e2);
        if (mask & (1u << 8)) e[8] += chunk_err<8>(v[c], p, b32[c], b64[c], cells, e0, e2);
    }
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) {
        if (!(mask & (1u << f))) continue;
        e[f] = wave_sum_dpp(e[f]);
        if (SPLIT > 1 && lane == 0) sl->e[wv][f] = e[f];
    }
    if (SPLIT > 1) {
        __syncthreads();
#pragma unroll
        for (int f = 0; f < CHAM_W_NFMT; ++f) {
            if (!(mask & (1u << f))) continue;
            float t = sl->e[0][f];
#pragma unroll
            for (int w = 1; w < 4; ++w) t += sl->e[w][f];
            e[f] = t;
        }
    }
    int best = -1, second = -1;
    float eb = 0.0f, es = 0.0f;
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) {
        if (!(mask & (1u << f))) continue;
        if (best < 0 || e[f] < eb) {
            second = best; es = eb;
            best = f; eb = e[f];
        } else if (second < 0 || e[f] < es) {
            second = f; es = e[f];
        }
    }
    double ed[CHAM_W_NFMT];
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) ed[f] = (double)e[f];
    // ---- near tie (or exact tie), or sums outside binary32's comfortable range (tiny or
    // huge rows): binary64 re-check of every enabled format.  Each binary32 sum carries a
    // relative error below (n + 9) 2^-24 for the n <= 160 roundings of a lane's serial sum
    // (128 elements at most, MX chunks one more per 4) and the 9 of the reductions, so two
    // sums more than 2^-15 apart are in the order of their exact values.
    if (second >= 0 && (!(es - eb > 0x1p-15f * es) || !(eb > 0x1p-100f) || !(es < 0x1p100f))) {
#pragma unroll
        for (int f = 0; f < CHAM_W_NFMT; ++f) {
            if (!(mask & (1u << f))) continue;
            switch (f) {
            case 0: ed[0] = row_err64<0, NCH>(v, valid, p, b32, b64, cells); break;
            case 1: ed[1] = row_err64<1, NCH>(v, valid, p, b32, b64, cells); break;
            case 2: ed[2] = row_err64<2, NCH>(v, valid, p, b32, b64, cells); break;
            case 3: ed[3] = row_err64<3, NCH>(v, valid, p, b32, b64, cells); break;
            case 4: ed[4] = row_err64<4, NCH>(v, valid, p, b32, b64, cells); break;
            case 5: ed[5] = row_err64<5, NCH>(v, valid, p, b32, b64, cells); break;
            case 6: ed[6] = row_err64<6, NCH>(v, valid, p, b32, b64, cells); break;
            case 7: ed[7] = row_err64<7, NCH>(v, valid, p, b32, b64, cells); break;
            default: ed[8] = row_err64<8, NCH>(v, valid, p, b32, b64, cells); break;
            }
            if (SPLIT > 1 && lane == 0) sl->ed[wv][f] = ed[f];
        }
        if (SPLIT > 1) {  // the condition above is the same in every wavefront of the channel
            __syncthreads();
#pragma unroll
            for (int f = 0; f < CHAM_W_NFMT; ++f) {
                if (!(mask & (1u << f))) continue;
                double t = sl->ed[0][f];
#pragma unroll
                for (int w = 1; w < 4; ++w) t += sl->ed[w][f];
                ed[f] = t;
            }
        }
        best = -1;
        double bd = 0.0;
#pragma unroll
        for (int f = 0; f < CHAM_W_NFMT; ++f) {
            if (!(mask & (1u << f))) continue;
            if (best < 0 || ed[f] < bd) { best = f; bd = ed[f]; }
        }
    }
    if (a.err && lane == 0 && part == 0) {
#pragma unroll
        for (int f = 0; f < CHAM_W_NFMT; ++f) a.err[n * CHAM_W_NFMT + f] = (mask & (1u << f)) ? ed[f] : -1.0;
    }

    // ---- emit the winner's codes and metadata
    const int f = best;
    if (lane == 0 && part == 0) {
        a.fmt[n] = (uint8_t)f;
        float s = 0.0f, z = 0.0f;
        if (f == CHAM_W_INT8_SYM) s = p.s_sym8;
        else if (f == CHAM_W_INT4_SYM) s = p.s_sym4;
        else if (f == CHAM_W_INT8_ASYM) { s = p.s_as8; z = p.z_as8; }
        else if (f == CHAM_W_INT4_ASYM) { s = p.s_as4; z = p.z_as4; }
        else if (f == CHAM_W_FP4) s = p.s_fp4;
        a.scale[n] = s;
        a.zero[n] = z;
    }
    const bool is_mx = f == CHAM_W_MXINT8 || f == CHAM_W_MXINT4 || f == CHAM_W_MXFP4;
    uint32_t cws[NCH];
    switch (f) {
    case 0: row_codes<0, NCH>(v, p, b32, b64, cells, a.code_bits, cws); break;
    case 1: row_codes<1, NCH>(v, p, b32, b64, cells, a.code_bits, cws); break;
    case 2: row_codes<2, NCH>(v, p, b32, b64, cells, a.code_bits, cws); break;
    case 3: row_codes<3, NCH>(v, p, b32, b64, cells, a.code_bits, cws); break;
    case 4: row_codes<4, NCH>(v, p, b32, b64, cells, a.code_bits, cws); break;
    case 5:
#pragma unroll
        for (int c = 0; c < NCH; ++c) cws[c] = nf4cw[c];
        break;
    case 6: row_codes<6, NCH>(v, p, b32, b64, cells, a.code_bits, cws); break;
    case 7: row_codes<7, NCH>(v, p, b32, b64, cells, a.code_bits, cws); break;
    default: row_codes<8, NCH>(v, p, b32, b64, cells, a.code_bits, cws); break;
    }
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (!valid[c]) continue;
        const int q = c * 64 + lane + (sp >> 2);  // float4 index in the row
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

// ------------------------------------------------------------------------------------
// Rows of at most 5120 elements in layers with many channels: LPC (16, 32 or 64) lanes per
// channel, so a wavefront searches 64 / LPC channels at once, and each lane holds 8
// consecutive elements per chunk (an MX block is 4 lanes, an NF4 block 8).  The per-row
// work (reductions, scales, the choice, the metadata) is shared by 4 or 2 channels and
// the per-block work (block maxima, MX exponents, the NF4 reciprocal) by 8 elements.
// Every reduction stays inside the channel's aligned lane group, so channels may branch
// apart; the binary64 re-check re-reads its row from memory (it is rare).
// ------------------------------------------------------------------------------------
template <int LPC>
CHAM_DEV float grp_sum(float v) {
    v = row_sum16(v);  // every lane of the row ends with the same sum (each step adds a pair)
    if (LPC >= 32) v += __shfl_xor(v, 16, kWave);
    if (LPC >= 64) v += __shfl_xor(v, 32, kWave);
    return v;
}
template <int LPC>
CHAM_DEV float grp_min(float v) {
    v = fminf(v, dpp<0xB1>(v));
    v = fminf(v, dpp<0x4E>(v));
    v = fminf(v, dpp<0x141>(v));
    v = fminf(v, dpp<0x140>(v));
    if (LPC >= 32) v = fminf(v, __shfl_xor(v, 16, kWave));
    if (LPC >= 64) v = fminf(v, __shfl_xor(v, 32, kWave));
    return v;
}
template <int LPC>
CHAM_DEV float grp_max(float v) {
    v = max16_from8(max8(v));
    if (LPC >= 32) v = fmaxf(v, __shfl_xor(v, 16, kWave));
    if (LPC >= 64) v = fmaxf(v, __shfl_xor(v, 32, kWave));
    return v;
}
template <int LPC>
CHAM_DEV double grp_sumd(double v) {
#pragma unroll
    for (int o = LPC / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

// binary32 squared error of 8 consecutive elements in format F (as chunk_err)
template <int F>
CHAM_DEV float oct_err(const float (&w)[8], const RowParams& p, float blk64, const NF4Cell* cells, int e0, int e2) {
    const float lo[4] = {w[0], w[1], w[2], w[3]};
    const float hi[4] = {w[4], w[5], w[6], w[7]};
    if (F == CHAM_W_MXINT4 || F == CHAM_W_MXINT8) {  // one rescale for the 8 elements
        const int Fb = F == CHAM_W_MXINT8 ? 6 : 2;
        const float Q = F == CHAM_W_MXINT8 ? 127.0f : 7.0f;
        float es = 0.0f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float y = ldexpf(w[j], Fb - e0);
            const float d = y - __builtin_amdgcn_fmed3f(rne(y), -Q, Q);
            es = __builtin_fmaf(d, d, es);
        }
        return ldexpf(es, 2 * (e0 - Fb));
    }
    // the other formats' per-element work is that of chunk_err, on two quads
    return chunk_err<F>(lo, p, 0.0f, blk64, cells, e0, e2) + chunk_err<F>(hi, p, 0.0f, blk64, cells, e0, e2);
}

// NF4 error of 8 consecutive elements and their codes (4 bits each, or a byte each in
// cw[0..1] with 8-bit codes)
CHAM_DEV float oct_err_nf4(const float (&w)[8], float blk64, const NF4Cell* cells, int code_bits, uint32_t (&cw)[2]) {
    const float a = floor_scale(blk64);
    const float r = rcp_rn(a);
    float e = 0.0f;
    cw[0] = cw[1] = 0u;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const float y = w[j] * r;
        const NF4Cell cl = nf4_cell(cells, y);
        const bool up = y > cl.thr;
        const float d = w[j] - (up ? cl.vhi : cl.vlo) * a;
        e = __builtin_fmaf(d, d, e);
        const uint32_t c = cl.cnt + (up ? 1u : 0u);
        if (code_bits == 4) cw[0] |= c << (4 * j);
        else cw[j >> 2] |= c << (8 * (j & 3));
    }
    return e;
}

// codes of 8 consecutive elements in the winning format F (layout as oct_err_nf4)
template <int F>
CHAM_DEV void oct_codes(const float (&w)[8], const RowParams& p, float b32, float b64, const NF4Cell* cells,
                        int code_bits, uint32_t (&cw)[2]) {
    cw[0] = cw[1] = 0u;
    if (F == CHAM_W_MXFP4 || F == CHAM_W_FP4) {
        // hardware converter: byte k holds elements 2k (low nibble) and 2k + 1
        const float sc = F == CHAM_W_MXFP4 ? e8m0_scale(mx_exponent(b32, 2)) : 1.0f;
        const float m = F == CHAM_W_MXFP4 ? 1.0f : p.r_fp4;
        uint32_t c = 0u;
        c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, w[0] * m, w[1] * m, sc, 0);
        c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, w[2] * m, w[3] * m, sc, 1);
        c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, w[4] * m, w[5] * m, sc, 2);
        c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, w[6] * m, w[7] * m, sc, 3);
        if (code_bits == 4) {
            cw[0] = c;
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) cw[j >> 2] |= ((c >> (4 * j)) & 15u) << (8 * (j & 3));
        }
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float wh;
            const uint32_t code = quant_one<F>(w[j], p, b32, b64, cells, &wh);
            if (code_bits == 4) cw[0] |= (code & 15u) << (4 * j);
            else cw[j >> 2] |= (code & 255u) << (8 * (j & 3));
        }
    }
}

// binary64 errors of every enabled format over the lane's elements, re-read from the row
// (the rare near-tie path): per chunk the block maxima by the same lane exchanges, each
// element through the exact quantize-dequantize, summed over the channel's lanes.
template <int NCH, int LPC>
CHAM_DEV void recheck_oct(const float* row, int K, int ll, uint32_t mask, const RowParams& p, const NF4Cell* cells,
                          double (&ed)[CHAM_W_NFMT]) {
    double acc[CHAM_W_NFMT];
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) acc[f] = 0.0;
#pragma unroll 1
    for (int c = 0; c < NCH; ++c) {
        const int e0 = 8 * (ll + LPC * c);
        const bool valid = e0 < K;
        float w[8];
        const float4 t0 = valid ? ld4(row + e0) : make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 t1 = valid ? ld4(row + e0 + 4) : make_float4(0.f, 0.f, 0.f, 0.f);
        w[0] = t0.x; w[1] = t0.y; w[2] = t0.z; w[3] = t0.w; w[4] = t1.x; w[5] = t1.y; w[6] = t1.z; w[7] = t1.w;
        float m = 0.0f;
#pragma unroll
        for (int j = 0; j < 8; ++j) m = fmaxf(m, fabsf(w[j]));
        m = fmaxf(m, dpp<0xB1>(m));
        const float b32 = fmaxf(m, dpp<0x4E>(m));
        const float b64 = fmaxf(b32, dpp<0x141>(b32));
        if (!valid) continue;
#pragma unroll
        for (int f = 0; f < CHAM_W_NFMT; ++f) {
            if (!(mask & (1u << f))) continue;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                float wh;
                switch (f) {
                case 0: quant_one<0>(w[j], p, b32, b64, cells, &wh); break;
                case 1: quant_one<1>(w[j], p, b32, b64, cells, &wh); break;
                case 2: quant_one<2>(w[j], p, b32, b64, cells, &wh); break;
                case 3: quant_one<3>(w[j], p, b32, b64, cells, &wh); break;
                case 4: quant_one<4>(w[j], p, b32, b64, cells, &wh); break;
                case 5: quant_one<5>(w[j], p, b32, b64, cells, &wh); break;
                case 6: quant_one<6>(w[j], p, b32, b64, cells, &wh); break;
                case 7: quant_one<7>(w[j], p, b32, b64, cells, &wh); break;
                default: quant_one<8>(w[j], p, b32, b64, cells, &wh); break;
                }
                const double d = (double)(w[j] - wh);
                acc[f] = fma(d, d, acc[f]);
            }
        }
    }
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f)
        if (mask & (1u << f)) ed[f] = grp_sumd<LPC>(acc[f]);
}

// Search of channel n by its LPC lanes (lane ll of the group); n < N for the whole group.
template <uint32_t MASK, int NCH, int LPC>
CHAM_DEV void search_oct(const SearchArgs& a, const NF4Cell* cells, int64_t n, int ll) {
    const int K = a.K;
    const float* row = a.W + n * (int64_t)K;
    const uint32_t mask = MASK ? MASK : a.mask;
    const int code_bits = MASK == CHAM_MASK_W4 ? 4 : (MASK == CHAM_MASK_W8 ? 8 : a.code_bits);

    float v[NCH][8];
    bool valid[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int e0 = 8 * (ll + LPC * c);
        valid[c] = e0 < K;
        const float4 t0 = valid[c] ? ld4(row + e0) : make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 t1 = valid[c] ? ld4(row + e0 + 4) : make_float4(0.f, 0.f, 0.f, 0.f);
        v[c][0] = t0.x; v[c][1] = t0.y; v[c][2] = t0.z; v[c][3] = t0.w;
        v[c][4] = t1.x; v[c][5] = t1.y; v[c][6] = t1.z; v[c][7] = t1.w;
    }

    // ---- row and block statistics (invalid chunks are zeros: no effect on block maxima,
    // and they stay out of lo / hi)
    float lo = INFINITY, hi = -INFINITY;
    float b32[NCH], b64[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        float m = 0.0f, l = INFINITY, h = -INFINITY;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            m = fmaxf(m, fabsf(v[c][j]));
            l = fminf(l, v[c][j]);
            h = fmaxf(h, v[c][j]);
        }
        if (valid[c]) { lo = fminf(lo, l); hi = fmaxf(hi, h); }
        m = fmaxf(m, dpp<0xB1>(m));
        b32[c] = fmaxf(m, dpp<0x4E>(m));
        b64[c] = fmaxf(b32[c], dpp<0x141>(b32[c]));
    }
    lo = grp_min<LPC>(lo);
    hi = grp_max<LPC>(hi);
    const float amax = fmaxf(fabsf(lo), fabsf(hi));

    RowParams p;
    p.s_sym8 = floor_scale(amax / 127.0f); p.r_sym8 = rcp_rn(p.s_sym8);
    p.s_sym4 = floor_scale(amax / 7.0f);   p.r_sym4 = rcp_rn(p.s_sym4);
    int_asym_scale_zp(lo, hi, 255.0f, &p.s_as8, &p.z_as8);
    p.r_as8 = rcp_rn(p.s_as8);
    int_asym_scale_zp(lo, hi, 15.0f, &p.s_as4, &p.z_as4);
    p.r_as4 = rcp_rn(p.s_as4);
    p.s_fp4 = floor_scale(amax / 6.0f); p.r_fp4 = rcp_rn(p.s_fp4);

    // ---- binary32 error sums of every enabled format, one fused pass
    float e[CHAM_W_NFMT];
    uint32_t nf4cw[NCH][2];
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) e[f] = 0.0f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        nf4cw[c][0] = nf4cw[c][1] = 0u;
        if (!valid[c]) continue;
        const bool nz32 = b32[c] > 0.0f;
        const int fl32 = __builtin_amdgcn_frexp_expf(b32[c]) - 1;
        const int e0 = mx_exponent_fl(fl32, nz32, 0), e2 = mx_exponent_fl(fl32, nz32, 2);
        if (mask & (1u << 0)) e[0] += oct_err<0>(v[c], p, b64[c], cells, e0, e2);
        if (mask & (1u << 1)) e[1] += oct_err<1>(v[c], p, b64[c], cells, e0, e2);
        if (mask & (1u << 2)) e[2] += oct_err<2>(v[c], p, b64[c], cells, e0, e2);
        if (mask & (1u << 3)) e[3] += oct_err<3>(v[c], p, b64[c], cells, e0, e2);
        if (mask & (1u << 4)) e[4] += oct_err<4>(v[c], p, b64[c], cells, e0, e2);
        if (mask & (1u << 5)) e[5] += oct_err_nf4(v[c], b64[c], cells, code_bits, nf4cw[c]);
        if (mask & (1u << 6)) e[6] += oct_err<6>(v[c], p, b64[c], cells, e0, e2);
        if (mask & (1u << 7)) e[7] += oct_err<7>(v[c], p, b64[c], cells, e0, e2);
        if (mask & (1u << 8)) e[8] += oct_err<8>(v[c], p, b64[c], cells, e0, e2);
    }
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f)
        if (mask & (1u << f)) e[f] = grp_sum<LPC>(e[f]);
    int best = -1, second = -1;
    float eb = 0.0f, es = 0.0f;
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) {
        if (!(mask & (1u << f))) continue;
        if (best < 0 || e[f] < eb) {
            second = best; es = eb;
            best = f; eb = e[f];
        } else if (second < 0 || e[f] < es) {
            second = f; es = e[f];
        }
    }
    double ed[CHAM_W_NFMT];
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) ed[f] = (double)e[f];
    // the re-check rule of search_row (the same binary32 error bound: a lane's serial sum
    // runs over at most 80 elements here, plus the reductions)
    if (second >= 0 && (!(es - eb > 0x1p-15f * es) || !(eb > 0x1p-100f) || !(es < 0x1p100f))) {
        recheck_oct<NCH, LPC>(row, K, ll, mask, p, cells, ed);
        best = -1;
        double bd = 0.0;
#pragma unroll
        for (int f = 0; f < CHAM_W_NFMT; ++f) {
            if (!(mask & (1u << f))) continue;
            if (best < 0 || ed[f] < bd) { best = f; bd = ed[f]; }
        }
    }
    if (a.err && ll == 0) {
#pragma unroll
        for (int f = 0; f < CHAM_W_NFMT; ++f) a.err[n * CHAM_W_NFMT + f] = (mask & (1u << f)) ? ed[f] : -1.0;
    }

    // ---- emit the winner's codes and metadata
    const int f = best;
    if (ll == 0) {
        a.fmt[n] = (uint8_t)f;
        float s = 0.0f, z = 0.0f;
        if (f == CHAM_W_INT8_SYM) s = p.s_sym8;
        else if (f == CHAM_W_INT4_SYM) s = p.s_sym4;
        else if (f == CHAM_W_INT8_ASYM) { s = p.s_as8; z = p.z_as8; }
        else if (f == CHAM_W_INT4_ASYM) { s = p.s_as4; z = p.z_as4; }
        else if (f == CHAM_W_FP4) s = p.s_fp4;
        a.scale[n] = s;
        a.zero[n] = z;
    }
    const bool is_mx = f == CHAM_W_MXINT8 || f == CHAM_W_MXINT4 || f == CHAM_W_MXFP4;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (!valid[c]) continue;
        uint32_t cw[2];
        switch (f) {
        case 0: oct_codes<0>(v[c], p, b32[c], b64[c], cells, code_bits, cw); break;
        case 1: oct_codes<1>(v[c], p, b32[c], b64[c], cells, code_bits, cw); break;
        case 2: oct_codes<2>(v[c], p, b32[c], b64[c], cells, code_bits, cw); break;
        case 3: oct_codes<3>(v[c], p, b32[c], b64[c], cells, code_bits, cw); break;
        case 4: oct_codes<4>(v[c], p, b32[c], b64[c], cells, code_bits, cw); break;
        case 5: cw[0] = nf4cw[c][0]; cw[1] = nf4cw[c][1]; break;
        case 6: oct_codes<6>(v[c], p, b32[c], b64[c], cells, code_bits, cw); break;
        case 7: oct_codes<7>(v[c], p, b32[c], b64[c], cells, code_bits, cw); break;
        default: oct_codes<8>(v[c], p, b32[c], b64[c], cells, code_bits, cw); break;
        }
        const int e0 = 8 * (ll + LPC * c);  // first element of the lane's 8
        if (code_bits == 4) {
            reinterpret_cast<uint32_t*>(a.codes + n * (int64_t)(K / 2))[e0 >> 3] = cw[0];
        } else {
            uint32_t* dst = reinterpret_cast<uint32_t*>(a.codes + n * (int64_t)K) + (e0 >> 2);
            dst[0] = cw[0];
            dst[1] = cw[1];
        }
        if (a.e8 && (ll & 3) == 0) {
            const int E = f == CHAM_W_MXFP4 ? mx_exponent(b32[c], 2) : mx_exponent(b32[c], 0);
            a.e8[n * (int64_t)(K / 32) + (e0 >> 5)] = is_mx ? (uint8_t)(E + 127) : (uint8_t)0;
        }
        if (a.nf4a && (ll & 7) == 0) {
            a.nf4a[n * (int64_t)(K / 64) + (e0 >> 6)] = f == CHAM_W_NF4 ? floor_scale(b64[c]) : 0.0f;
        }
    }
}

constexpr int kGroupThreads = 1024;
constexpr int kGroupLdsChannels = 16000;  // with the static arrays, within 64 KB of LDS

// layers per launch of a batched call (the descriptors travel in the kernel arguments)
constexpr int kBatchMax = 16;
struct GroupBatch {
    int nl;
    GroupArgs g[kBatchMax];
};

// workgroup i groups layer i of the batch (permutation staged in LDS when it fits)
__global__ __launch_bounds__(kGroupThreads) void group_kernel(GroupBatch B) {
    const GroupArgs& a = B.g[blockIdx.x];
    extern __shared__ int32_t lperm[];  // [N] when N <= kGroupLdsChannels
    group_channels<kGroupThreads>(a, a.perm && a.N <= kGroupLdsChannels ? lperm : nullptr);
}

struct SearchBatch {
    int nl;
    int64_t wg_end[kBatchMax];  // workgroups of layers 0..i
    SearchArgs l[kBatchMax];
};

// split = 1: four channels per workgroup, one per wavefront.  split = 4: one channel per
// workgroup, a quarter of the row per wavefront (more wavefronts in flight when the
// layer has few channels).  The workgroups of the batch's layers follow each other.
template <uint32_t MASK, int NCH>
__global__ __launch_bounds__(256) void search_kernel(SearchBatch B) {
    __shared__ NF4Cell cells[33];
    __shared__ SplitLDS sl;
    nf4_cells_init(cells);
    __syncthreads();
    const int64_t b = blockIdx.x;
    int i = 0;
    while (i + 1 < B.nl && b >= B.wg_end[i]) ++i;
    const SearchArgs& a = B.l[i];
    const int64_t lb = b - (i ? B.wg_end[i - 1] : 0);
    const int wv = threadIdx.x >> 6;
    const int64_t n = a.split == 1 ? lb * 4 + wv : lb;
    if (n < a.N) search_row<MASK, NCH>(a, cells, n, a.split == 1 ? 0 : wv, &sl);  // workgroup-uniform for split 4
}

// LPC lanes per channel, 256 / LPC channels per workgroup.
template <uint32_t MASK, int NCH, int LPC>
__global__ __launch_bounds__(256) void search_oct_kernel(SearchBatch B) {
    __shared__ NF4Cell cells[33];
    nf4_cells_init(cells);
    __syncthreads();
    const int64_t b = blockIdx.x;
    int i = 0;
    while (i + 1 < B.nl && b >= B.wg_end[i]) ++i;
    const SearchArgs& a = B.l[i];
    const int64_t lb = b - (i ? B.wg_end[i - 1] : 0);
    const int64_t n = lb * (256 / LPC) + (int)threadIdx.x / LPC;
    if (n < a.N) search_oct<MASK, NCH, LPC>(a, cells, n, (int)threadIdx.x % LPC);  // uniform per lane group
}

template <int NCH, int LPC>
void launch_oct(const SearchBatch& B, uint32_t mask, hipStream_t s) {
    const dim3 grid((unsigned)B.wg_end[B.nl - 1]);
    if (mask == CHAM_MASK_W4) hipLaunchKernelGGL((search_oct_kernel<CHAM_MASK_W4, NCH, LPC>), grid, dim3(256), 0, s, B);
    else if (mask == CHAM_MASK_W8) hipLaunchKernelGGL((search_oct_kernel<CHAM_MASK_W8, NCH, LPC>), grid, dim3(256), 0, s, B);
    else hipLaunchKernelGGL((search_oct_kernel<0u, NCH, LPC>), grid, dim3(256), 0, s, B);
}

template <int NCH>
void launch_search(const SearchBatch& B, uint32_t mask, hipStream_t s) {
    const dim3 grid((unsigned)B.wg_end[B.nl - 1]);
    if (mask == CHAM_MASK_W4) hipLaunchKernelGGL((search_kernel<CHAM_MASK_W4, NCH>), grid, dim3(256), 0, s, B);
    else if (mask == CHAM_MASK_W8) hipLaunchKernelGGL((search_kernel<CHAM_MASK_W8, NCH>), grid, dim3(256), 0, s, B);
    else hipLaunchKernelGGL((search_kernel<0u, NCH>), grid, dim3(256), 0, s, B);
}

// Layers with few channels and long rows split each row over the four wavefronts of a
// workgroup, so at least ~4 wavefronts per SIMD are in flight.
constexpr int64_t kSplitBelowChannels = 4096;

// Kernel variant of a layer: rows split over 4 wavefronts or not, and the register
// chunks (256 elements) per wavefront, rounded up to an instantiated count.
struct Variant {
    int split, nch, lpc;
};
// Rows up to 5120 elements in layers of at least this many channels (512 for rows longer
// than 1280) take the 8-elements-per-lane kernel: 16 lanes per channel up to 640 elements,
// 32 up to 2560 (two channels per wavefront), a whole wavefront up to 5120 (at most 10
// chunks; at most 5 up to 1280, which keeps the kernel at four wavefronts per SIMD).
constexpr int64_t kOctMinChannels = 1024;
Variant variant_of(int64_t N, int64_t K) {
    if (K > 2560 && K <= 5120 && N >= kOctMinChannels) return Variant{1, 10, 64};
    if (K <= 2560 && N >= (K > 1280 ? kOctMinChannels / 2 : kOctMinChannels)) {
        const int lpc = K <= 640 ? 16 : 32;
        const int nch = (int)((K + 8 * lpc - 1) / (8 * lpc));
        return Variant{1, nch <= 2 ? 2 : (nch <= 3 ? 3 : (nch <= 5 ? 5 : 10)), lpc};
    }
    // split when the quarter rows fill their 256-element chunks to at least 85 %, and
    // always for rows longer than one wavefront holds (8192)
    const int64_t qc = K / 4;
    const bool fill = K % 256 == 0 && qc * 100 >= 85 * ((qc + 255) / 256 * 256);
    const int split = K > 8192 || (fill && K >= 1024 && N < kSplitBelowChannels) ? 4 : 1;
    // the longest quarter: ceil(blocks / 4) 64-element blocks
    const int64_t kp = split == 1 ? K : (K / 64 + 3) / 4 * 64;
    const int nch = (int)((kp + 255) / 256);
    static const int counts[] = {2, 3, 5, 8, 10, 20, 32};
    int r = 32;
    for (int c : counts)
        if (nch <= c) { r = c; break; }
    return Variant{split, r, 0};
}

void launch_variant(const Variant& v, const SearchBatch& B, uint32_t mask, hipStream_t s) {
    if (v.lpc == 16) {
        switch (v.nch) {
        case 2: launch_oct<2, 16>(B, mask, s); break;
        case 3: launch_oct<3, 16>(B, mask, s); break;
        case 5: launch_oct<5, 16>(B, mask, s); break;
        default: launch_oct<10, 16>(B, mask, s); break;
        }
        return;
    }
    if (v.lpc == 64) {
        launch_oct<10, 64>(B, mask, s);
        return;
    }
    if (v.lpc == 32) {
        switch (v.nch) {
        case 2: launch_oct<2, 32>(B, mask, s); break;
        case 3: launch_oct<3, 32>(B, mask, s); break;
        case 5: launch_oct<5, 32>(B, mask, s); break;
        default: launch_oct<10, 32>(B, mask, s); break;
        }
        return;
    }
    switch (v.nch) {
    case 2: launch_search<2>(B, mask, s); break;
    case 3: launch_search<3>(B, mask, s); break;
    case 5: launch_search<5>(B, mask, s); break;
    case 8: launch_search<8>(B, mask, s); break;
    case 10: launch_search<10>(B, mask, s); break;
    case 20: launch_search<20>(B, mask, s); break;
    default: launch_search<32>(B, mask, s); break;
    }
}

}  // namespace
}  // namespace cham

using namespace cham;

int cham_pack_weights(const cham_wq* const* wqs, int n, hipStream_t s);  // the GEMM's record pre-pass

static int mask_code_bits(uint32_t mask) {
    return (mask & 0x7u) ? 8 : 4;  // formats 0..2 are the 8-bit ones
}

// Checks one layer's arguments and fills its search descriptor.
static int prepare_layer(const float* W, cham_wq* wq, SearchArgs& a) {
    if (!W || !wq) return CHAM_EINVAL;
    const uint32_t mask = wq->palette_mask;
    if (mask == 0u || (mask >> CHAM_W_NFMT) != 0u) return CHAM_EFORMAT;
    if (wq->N < 1 || wq->K < 1 || wq->N > (int64_t)INT32_MAX - 4096) return CHAM_EINVAL;
    const int64_t K = wq->K;
    if (K % 32 != 0) return CHAM_ESHAPE;
    const bool nf4 = (mask >> CHAM_W_NF4) & 1u;
    const bool mx = (mask & ((1u << CHAM_W_MXINT8) | (1u << CHAM_W_MXINT4) | (1u << CHAM_W_MXFP4))) != 0u;
    if (nf4 && K % 64 != 0) return CHAM_ESHAPE;
    if (!wq->fmt || !wq->codes || !wq->scale || !wq->zero) return CHAM_EINVAL;
    if ((nf4 && !wq->nf4_absmax) || (mx && !wq->e8m0)) return CHAM_EINVAL;
    if (((uintptr_t)W & 15u) || ((uintptr_t)wq->codes & 3u)) return CHAM_EINVAL;
    // rows up to 8192 are held in one wavefront's registers, up to 32768 in four (cut at
    // 64-element blocks)
    if (K > 4 * 32 * 256 || (K > 32 * 256 && K % 64 != 0)) return CHAM_ESHAPE;
    if (wq->packed) {  // the packed GEMM layout: 64-wide k-steps, 32-bit record offsets
        if (K % 64 != 0) return CHAM_ESHAPE;
        if (((uintptr_t)wq->packed & 255u) || wq->N * (K / 64) * 128 > (int64_t)INT32_MAX) return CHAM_EINVAL;
    }
    a.W = W;
    a.N = wq->N;
    a.K = (int)K;
    a.mask = mask;
    a.code_bits = mask_code_bits(mask);
    a.fmt = wq->fmt;
    a.codes = wq->codes;
    a.scale = wq->scale;
    a.zero = wq->zero;
    a.nf4a = nf4 ? wq->nf4_absmax : nullptr;  // block metadata is written only when its format is enabled
    a.e8 = mx ? wq->e8m0 : nullptr;
    a.err = wq->err;
    return CHAM_OK;
}

extern "C" int cham_select_weight_formats_batch(const float* const* W, cham_wq* wq, int32_t nlayers, void* stream) {
    if (!W || !wq || nlayers < 1) return CHAM_EINVAL;
    std::vector<SearchArgs> args((size_t)nlayers);
    for (int i = 0; i < nlayers; ++i) {
        const int rc = prepare_layer(W[i], &wq[i], args[i]);
        if (rc != CHAM_OK) return rc;
    }
    hipStream_t s = (hipStream_t)stream;
    // one launch per register-chunk count (and palette), up to kBatchMax layers each
    std::vector<bool> done((size_t)nlayers, false);
    for (int i = 0; i < nlayers; ++i) {
        if (done[i]) continue;
        const Variant v = variant_of(args[i].N, args[i].K);
        args[i].split = v.split;
        const uint32_t key = args[i].mask == CHAM_MASK_W4 || args[i].mask == CHAM_MASK_W8 ? args[i].mask : 0u;
        SearchBatch B;
        B.nl = 0;
        int64_t wgs = 0;
        for (int j = i; j < nlayers; ++j) {
            if (done[j]) continue;
            const Variant vj = variant_of(args[j].N, args[j].K);
            const uint32_t kj = args[j].mask == CHAM_MASK_W4 || args[j].mask == CHAM_MASK_W8 ? args[j].mask : 0u;
            if (vj.nch != v.nch || vj.lpc != v.lpc || kj != key) continue;
            args[j].split = vj.split;
            args[j].lpc = vj.lpc;
            const int64_t per_wg = vj.lpc ? 256 / vj.lpc : (vj.split == 1 ? 4 : 1);  // channels per workgroup
            wgs += (args[j].N + per_wg - 1) / per_wg;
            B.l[B.nl] = args[j];
            B.wg_end[B.nl] = wgs;
            ++B.nl;
            done[j] = true;
            if (B.nl == kBatchMax) break;
        }
        // a mixed palette (key 0) reads each layer's mask at run time
        launch_variant(v, B, key ? key : 0u, s);
        CHAM_CHECK_LAUNCH();
    }
    for (int i = 0; i < nlayers; ++i) wq[i].code_bits = args[i].code_bits;
    // packed layouts (and the grouping of those layers) in the packing launch
    std::vector<const cham_wq*> pk;
    for (int i = 0; i < nlayers; ++i)
        if (wq[i].packed) pk.push_back(&wq[i]);
    if (!pk.empty() && cham_pack_weights(pk.data(), (int)pk.size(), s) != CHAM_OK) return CHAM_EHIP;
    // grouping of the other layers: one workgroup per layer that asks for it
    GroupBatch G;
    G.nl = 0;
    size_t lds = 0;
    for (int i = 0; i <= nlayers; ++i) {
        if (i < nlayers && !wq[i].packed && (wq[i].perm || wq[i].group_off)) {
            G.g[G.nl++] = GroupArgs{wq[i].fmt, (int)wq[i].N, wq[i].perm, wq[i].group_off};
            if (wq[i].perm && wq[i].N <= kGroupLdsChannels) lds = std::max(lds, (size_t)wq[i].N * 4);
        }
        if (G.nl > 0 && (G.nl == kBatchMax || i == nlayers)) {
            hipLaunchKernelGGL(group_kernel, dim3((unsigned)G.nl), dim3(kGroupThreads), lds, s, G);
            CHAM_CHECK_LAUNCH();
            G.nl = 0;
            lds = 0;
        }
    }
    return CHAM_OK;
}

extern "C" int cham_select_weight_formats(const float* W, cham_wq* wq, void* stream) {
    return cham_select_weight_formats_batch(&W, wq, 1, stream);
}
