// Device-side building blocks shared by the HIP kernels of the library: exact binary32
// quantizer arithmetic for the paper's number formats (App. A.11), wavefront reductions,
// and launch-argument plumbing.  Every quantizer step is a single IEEE binary32 operation
// (the library is compiled with -ffp-contract=off), so codes are bitwise reproducible.
#pragma once

#include <hip/hip_runtime.h>
#include <float.h>
#include <stdint.h>

#include "../../include/chameleon.h"

#define CHAM_DEV __device__ __forceinline__

namespace cham {

constexpr int kWave = 64;

// ------------------------------------------------------------------------------------
// scalar helpers
// ------------------------------------------------------------------------------------
CHAM_DEV float rne(float x) { return __builtin_rintf(x); }

CHAM_DEV float clampf(float x, float lo, float hi) { return fminf(fmaxf(x, lo), hi); }

// Every floating group scale is floored at the smallest normal number (finite reciprocal).
CHAM_DEV float floor_scale(float s) { return s < FLT_MIN ? FLT_MIN : s; }

// ScaleZP of the INT-asym formats (App. A.7; App. A.11: L + 1 evenly spaced levels from min
// to max): s = (hi - lo)/L, z = round(-lo/s) with no clamp, so a one-sided range keeps its
// own end points and z lies outside [0, L].  A constant group (hi == lo) takes s = |lo|
// (1 if lo = 0), z = -sign(lo): every element is reconstructed exactly.
CHAM_DEV void int_asym_scale_zp(float lo, float hi, float L, float* s, float* z) {
    const float d = hi - lo;
    const float sc = d == 0.0f ? (lo != 0.0f ? fabsf(lo) : 1.0f) : floor_scale(d / L);
    *s = sc;
    *z = rne(-lo / sc);
}

// floor(log2(a)) for finite a > 0, from the binary32 fields (subnormals included).
CHAM_DEV int floor_log2(float a) {
    uint32_t u = __float_as_uint(a) & 0x7fffffffu;
    int e = (int)(u >> 23);
    if (e != 0) return e - 127;
    return (31 - __clz((int)u)) - 149;
}

// Shared exponent of an MX block with absolute maximum a: floor(log2 a) - emax, clamped to
// the E8M0 range [-127, 127]; -127 for an all-zero block.
CHAM_DEV int mx_exponent(float a, int emax) {
    if (!(a > 0.0f)) return -127;
    int e = floor_log2(a) - emax;
    return e < -127 ? -127 : (e > 127 ? 127 : e);
}

// The same from fl = floor_log2(a) computed once for several emax (fl is ignored when the
// block is all zero); branch-free.
CHAM_DEV int mx_exponent_fl(int fl, bool nonzero, int emax) {
    const int e = fl - emax;
    return nonzero ? (e < -127 ? -127 : (e > 127 ? 127 : e)) : -127;
}

// Correctly rounded 1/a for a >= FLT_MIN: the hardware estimate refined by one
// Newton-Raphson step with a fused multiply-add (Markstein's reciprocal iteration).  It
// equals the IEEE quotient 1/a for every binary32 a in [2^-126, 2^126) (checked
// exhaustively on gfx950); larger a, whose reciprocal is subnormal, take the division.
CHAM_DEV float rcp_rn(float a) {
    if (a >= 0x1p126f) return 1.0f / a;
    const float r0 = __builtin_amdgcn_rcpf(a);
    return __builtin_fmaf(__builtin_fmaf(-a, r0, 1.0f), r0, r0);
}

// ------------------------------------------------------------------------------------
// E2M1 (FP4): magnitudes {0, .5, 1, 1.5, 2, 3, 4, 6}; round to nearest, ties to the even
// code.  Adding 2^22 / 2^23 / 2^24 rounds to the format's step (0.5 below 2, 1 in [2, 4),
// 2 in [4, 6]) with IEEE ties-to-even, which is ties-to-even-code on this grid.
// ------------------------------------------------------------------------------------
CHAM_DEV float e2m1_round_mag(float a) {  // 0 <= a <= 6
    float c = a < 2.0f ? 4194304.0f : (a < 4.0f ? 8388608.0f : 16777216.0f);
    return (a + c) - c;
}

CHAM_DEV uint32_t e2m1_mag_code(float v) {  // v on the grid
    return v < 2.0f ? (uint32_t)(v * 2.0f) : (v < 4.0f ? (uint32_t)v + 2u : (uint32_t)(v * 0.5f) + 4u);
}

CHAM_DEV float e2m1_mag_value(uint32_t m) {  // m = code & 7
    return m < 4u ? (float)m * 0.5f : (m < 6u ? (float)m - 2.0f : (float)(m - 4u) * 2.0f);
}

// y already clamped to [-6, 6]; returns the 4-bit code (sign bit kept) and its value.
CHAM_DEV uint32_t e2m1_encode(float y, float* val) {
    float v = e2m1_round_mag(fabsf(y));
    uint32_t sgn = (__float_as_uint(y) >> 31) << 3;
    *val = __uint_as_float(__float_as_uint(v) | ((__float_as_uint(y) & 0x80000000u)));
    return sgn | e2m1_mag_code(v);
}

CHAM_DEV float e2m1_decode(uint32_t c) {
    float v = e2m1_mag_value(c & 7u);
    return (c & 8u) ? -v : v;
}

// ------------------------------------------------------------------------------------
// FP8 E4M3 (OCP "FN", bias 7, max 448) and E5M2 (bias 15, max 57344) decoding, subnormals
// and the sign of zero included.
// ------------------------------------------------------------------------------------
CHAM_DEV float e4m3_decode(uint32_t c) {
    uint32_t e = (c >> 3) & 15u, m = c & 7u;
    float v = e == 0u ? (float)m * 0.001953125f : ldexpf((float)(8u + m), (int)e - 10);
    return (c & 0x80u) ? -v : v;
}

CHAM_DEV float e5m2_decode(uint32_t c) {
    uint32_t e = (c >> 2) & 31u, m = c & 3u;
    float v = e == 0u ? (float)m * 1.52587890625e-05f : ldexpf((float)(4u + m), (int)e - 17);
    return (c & 0x80u) ? -v : v;
}

// ------------------------------------------------------------------------------------
// NF4 levels (QLoRA's normal-quantile construction, binary64 rounded to binary32) and the
// decision thresholds between neighbours: the largest binary32 number <= the exact
// midpoint, so that "y > t_i" holds exactly when y is strictly nearer level i+1 (a tie
// goes to the lower level).
// ------------------------------------------------------------------------------------
__device__ __constant__ const uint32_t kNF4Bits[16] = {
    0xbf800000u, 0xbf3239b1u, 0xbf066b2eu, 0xbeca329eu, 0xbe91a24bu, 0xbe3d353du,
    0xbdba7869u, 0x00000000u, 0x3da2fb01u, 0x3e24cadfu, 0x3e7c04dau, 0x3ead0336u,
    0x3ee1a4b5u, 0x3f1007a9u, 0x3f3913b0u, 0x3f800000u};
__device__ __constant__ const uint32_t kNF4ThrBits[15] = {
    0xbf591cd9u, 0xbf1c5270u, 0xbeeb847du, 0xbeadea75u, 0xbe703ceau, 0xbe0d38b9u,
    0xbd3a7869u, 0x3d22fb01u, 0x3df6485fu, 0x3e5067dcu, 0x3e9582d1u, 0x3ec753f5u,
    0x3f006d01u, 0x3f248dacu, 0x3f5c89d8u};

CHAM_DEV float nf4_level(uint32_t c) { return __uint_as_float(kNF4Bits[c & 15u]); }

CHAM_DEV uint32_t nf4_encode(float y) {
    uint32_t c = 0;
#pragma unroll
    for (int i = 0; i < 15; ++i) c += (y > __uint_as_float(kNF4ThrBits[i])) ? 1u : 0u;
    return c;
}

// ------------------------------------------------------------------------------------
// wavefront reductions (64 lanes)
// ------------------------------------------------------------------------------------
CHAM_DEV float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}
CHAM_DEV float wave_min(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o, kWave));
    return v;
}
CHAM_DEV double wave_sum(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}
CHAM_DEV float wave_sumf(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}
// max over aligned groups of G lanes (G = 8, 16)
template <int G>
CHAM_DEV float group_max(float v) {
#pragma unroll
    for (int o = G / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

// ------------------------------------------------------------------------------------
// activation codes of one float4 (App. A.11; the quantize pass and the fused
// quantize-and-accumulate pass share this arithmetic, so their codes are the same bits)
// ------------------------------------------------------------------------------------
// Four codes (already scaled, in range) packed into one word, element j in byte j.  FP8:
// the gfx950 converters (round to nearest even, subnormals included; the operands are
// clamped to the largest finite value first, so no saturation rule applies).
template <int FMT>
CHAM_DEV uint32_t pack_codes(float y0, float y1, float y2, float y3, float z) {
    if (FMT == CHAM_A_INT8_ASYM) {
        const float e[4] = {y0, y1, y2, y3};
        uint32_t w = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) w |= (uint32_t)clampf(rne(e[j]) + z, 0.0f, 255.0f) << (8 * j);
        return w;
    } else {
        typedef short v2s __attribute__((ext_vector_type(2)));
        v2s c = {0, 0};
        if (FMT == CHAM_A_FP8_E4M3) {
            c = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(c, y0, y1, 1.0f, false);
            c = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(c, y2, y3, 1.0f, true);
        } else {
            c = __builtin_amdgcn_cvt_scalef32_pk_bf8_f32(c, y0, y1, 1.0f, false);
            c = __builtin_amdgcn_cvt_scalef32_pk_bf8_f32(c, y2, y3, 1.0f, true);
        }
        return __builtin_bit_cast(uint32_t, c);
    }
}

// Per-tensor formats (INT8-asym, E4M3, E5M2): x r with r = fl(1/s), FP8 clamped to the
// format's largest finite value, INT8-asym rne(x r) + z clamped to [0, 255].
template <int FMT>
CHAM_DEV uint32_t act_codes4(const float4& t, float r, float z) {
    if (FMT == CHAM_A_INT8_ASYM) return pack_codes<FMT>(t.x * r, t.y * r, t.z * r, t.w * r, z);
    const float ymax = FMT == CHAM_A_FP8_E4M3 ? 448.0f : 57344.0f;
    return pack_codes<FMT>(clampf(t.x * r, -ymax, ymax), clampf(t.y * r, -ymax, ymax), clampf(t.z * r, -ymax, ymax),
                           clampf(t.w * r, -ymax, ymax), 0.0f);
}

// MX formats: the float4 is one eighth of a 32-block held by 8 consecutive lanes, which
// must all be active; returns the codes and the block's exponent E (its E8M0
// byte is E + 127).
template <int FMT>
CHAM_DEV uint32_t act_codes4_mx(const float4& t, int* Eout) {
    const float e[4] = {t.x, t.y, t.z, t.w};
    float m = fmaxf(fmaxf(fabsf(e[0]), fabsf(e[1])), fmaxf(fabsf(e[2]), fabsf(e[3])));
    m = group_max<8>(m);
    const int E = mx_exponent(m, 0);
    uint32_t w = 0;
    if (FMT == CHAM_A_MXFP8_E4M3) {
        float y[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) y[j] = clampf(ldexpf(e[j], -E), -448.0f, 448.0f);
        w = pack_codes<CHAM_A_FP8_E4M3>(y[0], y[1], y[2], y[3], 0.0f);
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float k = clampf(rne(ldexpf(e[j], 6 - E)), -127.0f, 127.0f);
            w |= ((uint32_t)(int)k & 0xFFu) << (8 * j);
        }
    }
    *Eout = E;
    return w;
}

}  // namespace cham

// host-side helpers shared by the entry points
#define CHAM_CHECK_LAUNCH()                                     \
    do {                                                        \
        if (hipGetLastError() != hipSuccess) return CHAM_EHIP; \
    } while (0)
