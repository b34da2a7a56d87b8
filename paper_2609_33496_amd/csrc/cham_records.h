// GEMM-ready layout of a searched weight ("records"), written by the record pre-pass (into
// the weight's packed buffer when the search asks for it, else into the linear layer's
// workspace) and read by the GEMM: per output channel a ColPrep, and per
// (k-step of 64, channel, half k-step of 32) a record of the half's codes followed by a
// 16-entry half-precision decode table (base value x block factor relative to the channel's
// largest block, rounded to binary32 and then to half precision) as two byte planes; and per
// channel the sum of its dequantized weights (the zero-point correction of INT8-asym
// activations whose zero point lies beyond what the half-precision decode holds exactly).
#ifndef CHAM_RECORDS_H_
#define CHAM_RECORDS_H_

#include "cham_device.h"

namespace cham {

typedef _Float16 half2v __attribute__((ext_vector_type(2)));

CHAM_DEV bool is_mx(int f) { return f == CHAM_W_MXINT8 || f == CHAM_W_MXINT4 || f == CHAM_W_MXFP4; }
CHAM_DEV bool is_8bit(int f) { return f == CHAM_W_INT8_SYM || f == CHAM_W_INT8_ASYM || f == CHAM_W_MXINT8; }
CHAM_DEV int mx_F(int f) { return f == CHAM_W_MXINT8 ? 6 : (f == CHAM_W_MXINT4 ? 2 : 0); }

// Per-channel parameters of the layout.
struct ColPrep {
    int fmt;         // CHAM_W_NFMT: not a valid format of the palette (decodes as zero)
    int eref;        // exponent removed from the decoded values: block-scaled formats (NF4,
                     // MX) that of the channel's largest block; INT-asym the power of two
                     // that keeps (q - z) 2^-eref within half precision's range; else 0
    float zero;      // INT-asym zero point (integral binary32, not limited to [0, L])
    float colscale;  // epilogue factor: INT/FP4 scale (times 2^eref), or 2^eref
};

// INT-asym: the exponent that brings every level q - z (q = 0..L) below 2^15 in magnitude.
CHAM_DEV int int_asym_eref(float zero, float L) {
    const float m = fmaxf(fabsf(zero), fabsf(L - zero));
    return m < 32768.0f ? 0 : floor_log2(m) - 14;
}

// 16-entry half-precision table as byte planes: lo[j] holds the low bytes of entries
// 4j..4j+3, hi[j] the high bytes.  8-bit integer formats use the same 32 bytes for
// {xor mask, then as half pairs the offset a, the factor f and the offset b}: a code c
// decodes as fma((1024 + (c ^ mask)) + a, f, b) in half precision.
struct Table {
    uint32_t lo[4], hi[4];
};

CHAM_DEV float e2m1_value(int c) {
    const float m[8] = {0.0f, 0.5f, 1.0f, 1.5f, 2.0f, 3.0f, 4.0f, 6.0f};
    return (c & 8) ? -m[c & 7] : m[c & 7];
}

// entry c of the table of a 4-bit-coded format: base value times block factor, rounded to
// binary32 (then, by the caller, to half precision).  The empty asm keeps the product a
// binary32 value, so the compiler cannot fuse the multiply with the conversion to half
// (a mixed-precision FMA rounds once instead of twice) in some tables and not in others:
// every table is built with the same two roundings.
CHAM_DEV float table_value(int f, int c, float zero, float factor) {
    float b;
    if (f == CHAM_W_NF4) b = nf4_level(c);
    else if (f == CHAM_W_FP4 || f == CHAM_W_MXFP4) b = e2m1_value(c);
    else if (f == CHAM_W_INT4_ASYM) b = (float)c - zero;
    else b = (float)(c < 8 ? c : c - 16);  // INT4-sym, MXINT4
    float v = b * factor;
    __asm__ volatile("" : "+v"(v));
    return v;
}

CHAM_DEV uint32_t half_pair2(float a, float b) {
    half2v p;
    p.x = (_Float16)a;
    p.y = (_Float16)b;
    return __builtin_bit_cast(uint32_t, p);
}

template <int F>
CHAM_DEV Table table_fmt(float zero, float factor) {
    Table t;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint32_t w01 = half_pair2(table_value(F, 4 * j, zero, factor), table_value(F, 4 * j + 1, zero, factor));
        const uint32_t w23 = half_pair2(table_value(F, 4 * j + 2, zero, factor), table_value(F, 4 * j + 3, zero, factor));
        t.lo[j] = __builtin_amdgcn_perm(w23, w01, 0x06040200u);
        t.hi[j] = __builtin_amdgcn_perm(w23, w01, 0x07050301u);
    }
    return t;
}

CHAM_DEV uint32_t half_pair(float v) {
    __asm__ volatile("" : "+v"(v));
    return half_pair2(v, v);
}

// Symmetric 8-bit codes (INT8-sym, MXINT8): (c ^ 0x80) is c + 128, so a = -1152 gives c
// exactly, times the block factor (a power of two), b = 0.
CHAM_DEV Table int8_sym_record(float factor) {
    return Table{{0x80808080u, half_pair(-1152.0f), half_pair(factor), 0u}, {0u, 0u, 0u, 0u}};
}

// INT8-asym: the level (c - z) 2^-e in half precision.  zr is z 2^-e rounded to half
// precision and base = zr 2^e - z (an integer, exact in binary32, |base| <= 8 2^e): then
// (1024 + c) + (base - 1024) = c + base exactly, and fma(c + base, 2^-e, -zr) is
// (c - z) 2^-e with one rounding.  For |z| <= 2048, e = 0 and zr = z, so every level with
// |c - z| <= 2048 is exact.  Beyond |z| = 2^22 (e >= 8) base is clamped to +-1024 so the
// offset stays a half-precision number; the level then carries up to one half-precision
// ulp (relative 2^-10) -- such a channel's values agree to 6e-5 of their magnitude.
CHAM_DEV Table int8_asym_record(float zero, int e) {
    const float zs = ldexpf(zero, -e);
    const float zr = (float)(_Float16)zs;
    const float base = clampf(ldexpf(zr, e) - zero, -1024.0f, 1024.0f);
    return Table{{0u, half_pair(base - 1024.0f), half_pair(ldexpf(1.0f, -e)), half_pair(-zr)}, {0u, 0u, 0u, 0u}};
}

// block factor of a record: the NF4 block absmax, or the MX block scale, over 2^eref
CHAM_DEV float record_factor(const ColPrep& c, float nf4a, int e8) {
    if (c.fmt == CHAM_W_NF4) return ldexpf(nf4a, -c.eref);
    if (is_mx(c.fmt)) return ldexpf(1.0f, e8 - 127 - mx_F(c.fmt) - c.eref);
    return 1.0f;
}

CHAM_DEV Table record_table(const ColPrep& c, float nf4a, int e8) {
    Table tb;
    switch (c.fmt) {
    case CHAM_W_NF4: tb = table_fmt<CHAM_W_NF4>(0.0f, record_factor(c, nf4a, e8)); break;
    case CHAM_W_MXFP4: tb = table_fmt<CHAM_W_MXFP4>(0.0f, record_factor(c, nf4a, e8)); break;
    case CHAM_W_MXINT4: tb = table_fmt<CHAM_W_MXINT4>(0.0f, record_factor(c, nf4a, e8)); break;
    case CHAM_W_MXINT8: tb = int8_sym_record(record_factor(c, nf4a, e8)); break;
    case CHAM_W_FP4: tb = table_fmt<CHAM_W_FP4>(0.0f, 1.0f); break;
    case CHAM_W_INT4_ASYM: tb = table_fmt<CHAM_W_INT4_ASYM>(c.zero, ldexpf(1.0f, -c.eref)); break;
    case CHAM_W_INT4_SYM: tb = table_fmt<CHAM_W_INT4_SYM>(0.0f, 1.0f); break;
    case CHAM_W_INT8_SYM: tb = int8_sym_record(1.0f); break;
    case CHAM_W_INT8_ASYM: tb = int8_asym_record(c.zero, c.eref); break;
    default: tb = Table{{0u, 0u, 0u, 0u}, {0u, 0u, 0u, 0u}}; break;
    }
    return tb;
}

// Table of a half k-step of a group-scaled 4-bit weight (the DiT search): the base values
// of the channel's format times the group's scale (NF4: absmax) over 2^eref; INT-asym with
// the group's zero point.
CHAM_DEV Table group_table(const ColPrep& c, float gscale, float gzero) {
    const float factor = ldexpf(gscale, -c.eref);
    switch (c.fmt) {
    case CHAM_W_NF4: return table_fmt<CHAM_W_NF4>(0.0f, factor);
    case CHAM_W_FP4: return table_fmt<CHAM_W_FP4>(0.0f, factor);
    case CHAM_W_INT4_ASYM: return table_fmt<CHAM_W_INT4_ASYM>(gzero, factor);
    case CHAM_W_INT4_SYM: return table_fmt<CHAM_W_INT4_SYM>(0.0f, factor);
    default: return Table{{0u, 0u, 0u, 0u}, {0u, 0u, 0u, 0u}};
    }
}

}  // namespace cham

#endif  // CHAM_RECORDS_H_
