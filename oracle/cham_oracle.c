/*
 * cham_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, scalar CPU implementation of what the Chameleon quantized-linear
 * path computes (arXiv 2609.33496, "Chameleon: Dynamic Format Adapter for Efficient
 * Diffusion").  It exists to check the HIP library against; nothing in the product
 * path may link, load or call it.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg use it.  It shares no code, header, table or constant
 * with the HIP library: every number format below is rebuilt here from its bit-level
 * definition, and the NF4 levels from their normal-quantile construction.
 *
 * Arithmetic conventions (the paper fake-quantizes with PyTorch casts; its inputs here
 * are binary32):
 *   - every quantizer step is one IEEE binary32 operation, round-to-nearest-even, with
 *     no FMA contraction (build with -ffp-contract=off, no fast-math);
 *   - "round" is round-half-to-even (nearbyintf in the default rounding mode);
 *   - floor(log2 a) is read exactly from the binary32 number (frexpf), never from a
 *     floating log2;
 *   - powers of two are applied with ldexpf (exact unless the result is subnormal);
 *   - error sums, moments, SNR and the GEMM reference are binary64.
 *
 * Readings of points the paper leaves open are marked READING and listed in the
 * design notes.  Parity of every function here is pinned by tests/test_oracle_*.py
 * against code tables enumerated from bits, brute force, closed forms, invariants
 * stated by the paper and the SNR values it prints (App. A.9, Tab. lutstats).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#include <float.h>
#include <fenv.h>

/* ------------------------------------------------------------------------- */
/* format identifiers (palette order of Sec. 4.2)                             */
/* ------------------------------------------------------------------------- */
enum { W_INT8_SYM = 0, W_INT8_ASYM = 1, W_MXINT8 = 2, W_INT4_SYM = 3, W_INT4_ASYM = 4,
       W_NF4 = 5, W_FP4 = 6, W_MXINT4 = 7, W_MXFP4 = 8, W_NFMT = 9 };
/* activation codes of the runtime LUT (Sec. 4.2): 0..4 */
enum { A_INT8_ASYM = 0, A_FP8_E4M3 = 1, A_FP8_E5M2 = 2, A_MXFP8 = 3, A_MXINT8 = 4 };

int orc_rounding_ok(void) { return fegetround() == FE_TONEAREST; }

/* ------------------------------------------------------------------------- */
/* exact helpers                                                               */
/* ------------------------------------------------------------------------- */

/* round half to even */
static float rne(float x) { return nearbyintf(x); }

static float clampf(float x, float lo, float hi) {
    if (x < lo) return lo;
    if (x > hi) return hi;
    return x;
}

/* floor(log2(a)) for finite a > 0, exact (frexp: a = f * 2^e, f in [0.5, 1)). */
static int floor_log2(float a) {
    int e;
    (void)frexpf(a, &e);
    return e - 1;
}

/* READING: every per-group floating scale is floored at the smallest normal binary32
 * number, so that its reciprocal is finite.  This only changes groups whose range is
 * below ~1e-36 (it also gives all-zero groups a defined scale). */
static float floor_scale(float s) { return s < FLT_MIN ? FLT_MIN : s; }

/* ------------------------------------------------------------------------- */
/* minifloat codes (App. A.11): value of a code from its sign/exponent/mantissa  */
/* fields, and nearest-value encoding with ties to the even code                */
/* ------------------------------------------------------------------------- */
typedef struct { int ebits, mbits, bias; unsigned max_mag; } minifloat;

/* E2M1: 1 sign, 2 exponent (bias 1), 1 mantissa; magnitudes {0,.5,1,1.5,2,3,4,6} */
static const minifloat MF_E2M1 = { 2, 1, 1, 0x7u };
/* E4M3 (OCP "FN"): bias 7, max 448, no infinities; code 0x7F is NaN */
static const minifloat MF_E4M3 = { 4, 3, 7, 0x7Eu };
/* E5M2: bias 15, max 57344; exponent field 31 is Inf/NaN */
static const minifloat MF_E5M2 = { 5, 2, 15, 0x7Bu };

static double mf_decode(const minifloat* f, unsigned code) {
    unsigned s = (code >> (f->ebits + f->mbits)) & 1u;
    unsigned e = (code >> f->mbits) & ((1u << f->ebits) - 1u);
    unsigned m = code & ((1u << f->mbits) - 1u);
    double v;
    if (e == 0) v = ldexp((double)m, 1 - f->bias - f->mbits);                 /* subnormal */
    else v = ldexp((double)((1u << f->mbits) + m), (int)e - f->bias - f->mbits); /* normal */
    return s ? -v : v;
}

/* nearest representable magnitude, ties to the code with an even mantissa LSB; the sign
 * bit is kept (so -0 encodes as the negative-zero code).  Caller clamps |y| <= max. */
static unsigned mf_encode(const minifloat* f, float y) {
    unsigned sbit = signbit(y) ? (1u << (f->ebits + f->mbits)) : 0u;
    double a = fabs((double)y);
    unsigned best = 0;
    double bd = INFINITY;
    for (unsigned c = 0; c <= f->max_mag; ++c) {
        double d = fabs(mf_decode(f, c) - a);
        if (d < bd || (d == bd && (c & 1u) == 0u)) { best = c; bd = d; }
    }
    return sbit | best;
}

double orc_mf_decode(int which, unsigned code) {
    const minifloat* f = which == 0 ? &MF_E2M1 : which == 1 ? &MF_E4M3 : &MF_E5M2;
    return mf_decode(f, code);
}
unsigned orc_mf_encode(int which, float y) {
    const minifloat* f = which == 0 ? &MF_E2M1 : which == 1 ? &MF_E4M3 : &MF_E5M2;
    return mf_encode(f, y);
}

/* ------------------------------------------------------------------------- */
/* NF4 (App. A.11, citing QLoRA).  READING: the 16 levels are QLoRA's construction:  */
/* 8 positive quantiles of N(0,1) at probabilities linspace(d, 1/2, 9)[:8], 7        */
/* negative ones at linspace(d, 1/2, 8)[:7], and an exact zero, with                 */
/* d = 1 - (1/30 + 1/32)/2, normalized by the largest; evaluated in binary64 and       */
/* rounded once to binary32.                                                          */
/* ------------------------------------------------------------------------- */
static double norm_cdf(double x) { return 0.5 * erfc(-x / sqrt(2.0)); }

/* inverse normal CDF for p in [1/2, 1): bisection on the CDF to binary64 resolution */
static double norm_ppf_upper(double p) {
    double lo = 0.0, hi = 10.0;
    for (int it = 0; it < 200; ++it) {
        double mid = 0.5 * (lo + hi);
        if (mid == lo || mid == hi) break;
        if (norm_cdf(mid) < p) lo = mid; else hi = mid;
    }
    return 0.5 * (lo + hi);
}

static float NF4[16];
static int nf4_ready = 0;

static void nf4_build(void) {
    if (nf4_ready) return;
    const double d = 1.0 - 0.5 * (1.0 / 30.0 + 1.0 / 32.0);
    double v[16];
    int n = 0;
    for (int j = 0; j < 7; ++j) v[n++] = -norm_ppf_upper(d + (0.5 - d) * j / 7.0);
    v[n++] = 0.0;
    for (int i = 7; i >= 0; --i) v[n++] = norm_ppf_upper(d + (0.5 - d) * i / 8.0);
    /* v is ascending: most negative first, largest positive last */
    double mx = v[15];
    for (int i = 0; i < 16; ++i) NF4[i] = (float)(v[i] / mx);
    nf4_ready = 1;
}

void orc_nf4_table(float* out16) { nf4_build(); memcpy(out16, NF4, sizeof(NF4)); }

/* nearest NF4 level to y (exact comparison in binary64), ties to the lower code */
static unsigned nf4_encode(float y) {
    unsigned best = 0;
    double bd = INFINITY;
    for (unsigned c = 0; c < 16; ++c) {
        double dd = fabs((double)NF4[c] - (double)y);
        if (dd < bd) { best = c; bd = dd; }
    }
    return best;
}

/* ------------------------------------------------------------------------- */
/* per-group quantizers.  Each takes one scale group of n values, writes one code    */
/* per element (unpacked, low bits of a byte), the group metadata, and the            */
/* dequantized values DQ_f(Q_f(x)).                                                   */
/* ------------------------------------------------------------------------- */

/* INT-sym, Q = 127 or 7: s = amax/Q, q = clamp(round(x/s), -Q, Q) (READING: symmetric
 * range, -2^(b-1) unused).  Codes are two's complement in b bits. */
static void q_int_sym(const float* x, int64_t n, int Q, unsigned bits, uint8_t* code,
                      float* xh, float* scale) {
    float amax = 0.0f;
    for (int64_t i = 0; i < n; ++i) amax = fmaxf(amax, fabsf(x[i]));
    float s = floor_scale(amax / (float)Q);
    float r = 1.0f / s;
    for (int64_t i = 0; i < n; ++i) {
        float q = clampf(rne(x[i] * r), (float)-Q, (float)Q);
        code[i] = (uint8_t)((int)q & ((1 << bits) - 1));
        xh[i] = q * s;
    }
    *scale = s;
}

/* INT-asym, L = 255 or 15 (App. A.7 ScaleZP; App. A.11: L + 1 evenly spaced levels from
 * min to max): s = (hi - lo)/L, z = round(-lo/s), both taken literally -- the range is the
 * observed one and z is not clamped, so for a one-sided range z lies outside [0, L] and the
 * levels (q - z) s, q = 0..L, run from lo to hi.  Quantization q = clamp(round(x/s) + z,
 * 0, L), x^ = (q - z) s, each step one binary32 operation (x/s as x * (1/s)).
 * READING: a constant group (hi == lo) has no spread to divide; it takes s = |lo| (1 if
 * lo = 0), so z = -sign(lo) and every element is reconstructed exactly. */
static void scalezp_int_asym(float lo, float hi, int L, float* s_out, float* z_out) {
    float d = hi - lo;
    float s;
    if (d == 0.0f) s = lo != 0.0f ? fabsf(lo) : 1.0f;
    else s = floor_scale(d / (float)L);
    *s_out = s;
    *z_out = rne(-lo / s);
}

static void q_int_asym_with(const float* x, int64_t n, int L, float s, float z, uint8_t* code,
                            float* xh) {
    float r = 1.0f / s;
    for (int64_t i = 0; i < n; ++i) {
        float q = clampf(rne(x[i] * r) + z, 0.0f, (float)L);
        code[i] = (uint8_t)(int)q;
        if (xh) xh[i] = (q - z) * s;
    }
}

static void q_int_asym(const float* x, int64_t n, int L, uint8_t* code, float* xh,
                       float* scale, float* zero) {
    float lo = INFINITY, hi = -INFINITY;
    for (int64_t i = 0; i < n; ++i) { lo = fminf(lo, x[i]); hi = fmaxf(hi, x[i]); }
    float s, z;
    scalezp_int_asym(lo, hi, L, &s, &z);
    q_int_asym_with(x, n, L, s, z, code, xh);
    *scale = s;
    *zero = z;
}

/* FP4 E2M1 with one scale per output channel (READING: s = amax/6, saturating at +-6). */
static void q_fp4(const float* x, int64_t n, uint8_t* code, float* xh, float* scale) {
    float amax = 0.0f;
    for (int64_t i = 0; i < n; ++i) amax = fmaxf(amax, fabsf(x[i]));
    float s = floor_scale(amax / 6.0f);
    float r = 1.0f / s;
    for (int64_t i = 0; i < n; ++i) {
        float y = clampf(x[i] * r, -6.0f, 6.0f);
        unsigned c = mf_encode(&MF_E2M1, y);
        code[i] = (uint8_t)c;
        xh[i] = (float)mf_decode(&MF_E2M1, c) * s;
    }
    *scale = s;
}

/* NF4 on one 64-element block: a = block absmax, y = x/a, code = nearest level. */
static void q_nf4_block(const float* x, int64_t n, uint8_t* code, float* xh, float* absmax) {
    nf4_build();
    float a = 0.0f;
    for (int64_t i = 0; i < n; ++i) a = fmaxf(a, fabsf(x[i]));
    a = floor_scale(a);
    float r = 1.0f / a;
    for (int64_t i = 0; i < n; ++i) {
        unsigned c = nf4_encode(x[i] * r);
        code[i] = (uint8_t)c;
        xh[i] = NF4[c] * a;
    }
    *absmax = a;
}

/* Shared block exponent of an MX block (App. A.11: E = floor(log2 max|x|)), minus the
 * element type's emax, clamped to the E8M0 range; an all-zero block takes -127
 * (READING; the E8M0 NaN byte 0xFF is never produced). */
static int mx_exponent(const float* x, int64_t n, int emax_elem) {
    float a = 0.0f;
    for (int64_t i = 0; i < n; ++i) a = fmaxf(a, fabsf(x[i]));
    if (a == 0.0f) return -127;
    int e = floor_log2(a) - emax_elem;
    if (e < -127) e = -127;
    if (e > 127) e = 127;
    return e;
}

/* MX integer block (MXINT8: 1.6 fixed point, MXINT4: 1.2 fixed point by analogy; READING:
 * symmetric clamp +-Q).  x^ = k * 2^(E - F). */
static void q_mxint_block(const float* x, int64_t n, int F, int Q, unsigned bits, uint8_t* code,
                          float* xh, uint8_t* e8) {
    int E = mx_exponent(x, n, 0);
    for (int64_t i = 0; i < n; ++i) {
        float k = clampf(rne(ldexpf(x[i], F - E)), (float)-Q, (float)Q);
        code[i] = (uint8_t)((int)k & ((1 << bits) - 1));
        xh[i] = ldexpf(k, E - F);
    }
    *e8 = (uint8_t)(E + 127);
}

/* MX minifloat block: E = floor(log2 amax) - emax_offset; element = f(x / 2^E) with
 * saturation at the element's max; x^ = f * 2^E.
 *  - weights, MXFP4: OCP MX v1.0 offset emax(E2M1) = 2 (the paper is silent on
 *    weight-side MX exponents; READING);
 *  - activations, MXFP8: the paper's own exponent floor(log2 amax), offset 0, so block
 *    values land in (-2, 2) (Sec. 4.7, App. A.12). */
static void q_mxfp_block(const float* x, int64_t n, const minifloat* mf, int emax_offset,
                         float satmax, uint8_t* code, float* xh, uint8_t* e8) {
    int E = mx_exponent(x, n, emax_offset);
    for (int64_t i = 0; i < n; ++i) {
        float y = clampf(ldexpf(x[i], -E), -satmax, satmax);
        unsigned c = mf_encode(mf, y);
        code[i] = (uint8_t)c;
        if (xh) xh[i] = ldexpf((float)mf_decode(mf, c), E);
    }
    *e8 = (uint8_t)(E + 127);
}

static int wfmt_bits(int f) { return (f == W_INT8_SYM || f == W_INT8_ASYM || f == W_MXINT8) ? 8 : 4; }

/* Quantize-dequantize one weight row of K values in format f (Sec. 4.5 round trip).
 * codes[K] unpacked; scale/zero per row; nf4a[K/64]; e8[K/32]; wh[K] = DQ_f(Q_f(w)).
 * Metadata a format does not use is written as 0. */
static void wq_row(int f, const float* w, int64_t K, uint8_t* codes, float* wh, float* scale,
                   float* zero, float* nf4a, uint8_t* e8) {
    *scale = 0.0f;
    *zero = 0.0f;
    if (nf4a) for (int64_t b = 0; b < K / 64; ++b) nf4a[b] = 0.0f;
    if (e8) for (int64_t b = 0; b < K / 32; ++b) e8[b] = 0;
    switch (f) {
    case W_INT8_SYM: q_int_sym(w, K, 127, 8, codes, wh, scale); break;
    case W_INT4_SYM: q_int_sym(w, K, 7, 4, codes, wh, scale); break;
    case W_INT8_ASYM: q_int_asym(w, K, 255, codes, wh, scale, zero); break;
    case W_INT4_ASYM: q_int_asym(w, K, 15, codes, wh, scale, zero); break;
    case W_FP4: q_fp4(w, K, codes, wh, scale); break;
    case W_NF4:
        for (int64_t b = 0; b < K / 64; ++b)
            q_nf4_block(w + 64 * b, 64, codes + 64 * b, wh + 64 * b, &nf4a[b]);
        break;
    case W_MXINT8:
        for (int64_t b = 0; b < K / 32; ++b)
            q_mxint_block(w + 32 * b, 32, 6, 127, 8, codes + 32 * b, wh + 32 * b, &e8[b]);
        break;
    case W_MXINT4:
        for (int64_t b = 0; b < K / 32; ++b)
            q_mxint_block(w + 32 * b, 32, 2, 7, 4, codes + 32 * b, wh + 32 * b, &e8[b]);
        break;
    case W_MXFP4:
        for (int64_t b = 0; b < K / 32; ++b)
            q_mxfp_block(w + 32 * b, 32, &MF_E2M1, 2, 6.0f, codes + 32 * b, wh + 32 * b, &e8[b]);
        break;
    }
}

/* Decode one weight row from codes + metadata (the same DQ_f as above, from the stored
 * representation).  codes unpacked. */
static void wdq_row(int f, const uint8_t* c, int64_t K, float scale, float zero,
                    const float* nf4a, const uint8_t* e8, float* wh) {
    nf4_build();
    for (int64_t k = 0; k < K; ++k) {
        unsigned u = c[k];
        float v = 0.0f;
        switch (f) {
        case W_INT8_SYM: v = (float)(int8_t)u * scale; break;
        case W_INT4_SYM: v = (float)((int)(u << 28) >> 28) * scale; break;
        case W_INT8_ASYM:
        case W_INT4_ASYM: v = ((float)u - zero) * scale; break;
        case W_FP4: v = (float)mf_decode(&MF_E2M1, u) * scale; break;
        case W_NF4: v = NF4[u & 15u] * nf4a[k / 64]; break;
        case W_MXINT8: v = ldexpf((float)(int8_t)u, (int)e8[k / 32] - 127 - 6); break;
        case W_MXINT4: v = ldexpf((float)((int)(u << 28) >> 28), (int)e8[k / 32] - 127 - 2); break;
        case W_MXFP4: v = ldexpf((float)mf_decode(&MF_E2M1, u), (int)e8[k / 32] - 127); break;
        }
        wh[k] = v;
    }
}

/* ------------------------------------------------------------------------- */
/* weight-format search (Sec. 4.5, Eq. weight-argmax)                            */
/* ------------------------------------------------------------------------- */
/* For each output channel n: err_f = sum_k (w - DQ_f(Q_f(w)))^2 over the enabled formats
 * (each difference a binary32 op, squared and summed in binary64); the chosen format is
 * argmin err_f, i.e. argmax SQNR (the row energy is common to all f), ties to the lowest
 * palette id.  The codes and metadata of the chosen format are emitted:
 *   codes : two 4-bit codes per byte (even k in the low nibble) when every enabled
 *           format is 4-bit, otherwise one code per byte; row-major [N][K/2] or [N][K].
 *   scale[N], zero[N] (integral binary32), nf4a[N][K/64] (may be NULL if NF4 disabled),
 *   e8[N][K/32] (may be NULL if no MX format enabled), err[N][9] (may be NULL; -1 for
 *   disabled formats).
 * perm / group_off: stable sort of channels by chosen format (may be NULL).
 * scratch: caller buffer of at least 4*K floats + 2*K bytes + K/64 floats + K/32 bytes.
 * Returns 0, or -1 on a bad mask/shape. */
int orc_select_weight_formats(const float* W, int64_t N, int64_t K, uint32_t mask, uint8_t* fmt,
                              uint8_t* codes, float* scale, float* zero, float* nf4a,
                              uint8_t* e8, int32_t* perm, int32_t* group_off, double* err) {
    if (N < 0 || K <= 0 || (mask & ~0x1FFu) || mask == 0) return -1;
    int code_bits = 4;
    for (int f = 0; f < W_NFMT; ++f)
        if ((mask >> f) & 1u) { if (wfmt_bits(f) == 8) code_bits = 8; }
    if ((mask & (1u << W_NF4)) && (K % 64)) return -1;
    if ((mask & ((1u << W_MXINT8) | (1u << W_MXINT4) | (1u << W_MXFP4))) && (K % 32)) return -1;
    if (K % 2) return -1;

    static float wh[1 << 16];
    static uint8_t cbuf[1 << 16], cbest[1 << 16];
    static float nfa[1 << 10], nfa_best[1 << 10];
    static uint8_t eb[1 << 11], eb_best[1 << 11];
    if (K > (1 << 16)) return -1;

    for (int64_t n = 0; n < N; ++n) {
        const float* w = W + n * K;
        int best = -1;
        double best_err = 0.0;
        float bs = 0.0f;
        float bz = 0.0f;
        for (int f = 0; f < W_NFMT; ++f) {
            if (!((mask >> f) & 1u)) { if (err) err[n * W_NFMT + f] = -1.0; continue; }
            float s, z;
            wq_row(f, w, K, cbuf, wh, &s, &z, nfa, eb);
            double e = 0.0;
            for (int64_t k = 0; k < K; ++k) {
                float d = w[k] - wh[k];
                e += (double)d * (double)d;
            }
            if (err) err[n * W_NFMT + f] = e;
            if (best < 0 || e < best_err) {
                best = f;
                best_err = e;
                bs = s;
                bz = z;
                memcpy(cbest, cbuf, (size_t)K);
                memcpy(nfa_best, nfa, sizeof(float) * (size_t)(K / 64));
                memcpy(eb_best, eb, (size_t)(K / 32));
            }
        }
        fmt[n] = (uint8_t)best;
        scale[n] = bs;
        zero[n] = bz;
        if (nf4a) for (int64_t b = 0; b < K / 64; ++b) nf4a[n * (K / 64) + b] = nfa_best[b];
        if (e8) for (int64_t b = 0; b < K / 32; ++b) e8[n * (K / 32) + b] = eb_best[b];
        if (code_bits == 4) {
            uint8_t* dst = codes + n * (K / 2);
            for (int64_t k = 0; k < K; k += 2)
                dst[k / 2] = (uint8_t)((cbest[k] & 15u) | ((cbest[k + 1] & 15u) << 4));
        } else {
            memcpy(codes + n * K, cbest, (size_t)K);
        }
    }
    if (perm || group_off) {
        int32_t cnt[W_NFMT] = { 0 }, off[W_NFMT + 1];
        for (int64_t n = 0; n < N; ++n) cnt[fmt[n]]++;
        off[0] = 0;
        for (int f = 0; f < W_NFMT; ++f) off[f + 1] = off[f] + cnt[f];
        if (group_off) for (int f = 0; f <= W_NFMT; ++f) group_off[f] = off[f];
        if (perm) {
            int32_t pos[W_NFMT];
            for (int f = 0; f < W_NFMT; ++f) pos[f] = off[f];
            for (int64_t n = 0; n < N; ++n) perm[pos[fmt[n]]++] = (int32_t)n;
        }
    }
    return 0;
}

/* Dequantize a whole packed weight matrix (as emitted above) to binary32. */
int orc_dequant_weights(int64_t N, int64_t K, int code_bits, const uint8_t* fmt,
                        const uint8_t* codes, const float* scale, const float* zero,
                        const float* nf4a, const uint8_t* e8, float* Wh) {
    static uint8_t cb[1 << 16];
    if (K > (1 << 16)) return -1;
    for (int64_t n = 0; n < N; ++n) {
        if (code_bits == 4) {
            const uint8_t* src = codes + n * (K / 2);
            for (int64_t k = 0; k < K; k += 2) {
                cb[k] = src[k / 2] & 15u;
                cb[k + 1] = src[k / 2] >> 4;
            }
        } else {
            memcpy(cb, codes + n * K, (size_t)K);
        }
        wdq_row(fmt[n], cb, K, scale[n], zero[n], nf4a ? nf4a + n * (K / 64) : NULL,
                e8 ? e8 + n * (K / 32) : NULL, Wh + n * K);
    }
    return 0;
}

/* Round-trip one row in one format (diagnostics and pins). codes unpacked. */
void orc_wq_row(int f, const float* w, int64_t K, uint8_t* codes, float* wh, float* scale,
                float* zero, float* nf4a, uint8_t* e8) {
    wq_row(f, w, K, codes, wh, scale, zero, nf4a, e8);
}

/* ------------------------------------------------------------------------- */
/* activations: ScaleZP (App. A.7) and the quantizers of Alg. 2 / Alg. 3           */
/* ------------------------------------------------------------------------- */
void orc_minmax(const float* X, int64_t n, float* lo, float* hi) {
    float a = INFINITY, b = -INFINITY;
    for (int64_t i = 0; i < n; ++i) { a = fminf(a, X[i]); b = fmaxf(b, X[i]); }
    *lo = a;
    *hi = b;
}

/* ScaleZP(f, lo, hi): INT8-asym s = (hi-lo)/255, z = round(-lo/s); E4M3 s = amax/448;
 * E5M2 s = amax/57344, z = 0; MX formats s = 1, z = 0. */
void orc_scale_zp(int fmt, float lo, float hi, float* s, float* z) {
    switch (fmt) {
    case A_INT8_ASYM: scalezp_int_asym(lo, hi, 255, s, z); return;
    case A_FP8_E4M3: *s = floor_scale(fmaxf(fabsf(lo), fabsf(hi)) / 448.0f); *z = 0.0f; return;
    case A_FP8_E5M2: *s = floor_scale(fmaxf(fabsf(lo), fabsf(hi)) / 57344.0f); *z = 0.0f; return;
    default: *s = 1.0f; *z = 0.0f; return;
    }
}

/* Quantize X [M][K] to format fmt with per-tensor (s, z) (formats 0-2) or per-32-block
 * shared exponents along K (formats 3-4).  codes [M][K]: INT8-asym unsigned q; FP8 codes;
 * MXINT8 two's complement.  e8 [M][K/32] for MX (may be NULL otherwise).  xh optional:
 * the dequantized values.  FP8 values are clamped to the format's range before the cast
 * (App. A.7, implementation note ii). */
int orc_quantize_act(const float* X, int64_t M, int64_t K, int fmt, float s, float z,
                     uint8_t* codes, uint8_t* e8, float* xh) {
    int64_t n = M * K;
    if (fmt == A_INT8_ASYM) {
        q_int_asym_with(X, n, 255, s, z, codes, xh);
        return 0;
    }
    if (fmt == A_FP8_E4M3 || fmt == A_FP8_E5M2) {
        const minifloat* mf = fmt == A_FP8_E4M3 ? &MF_E4M3 : &MF_E5M2;
        float mx = fmt == A_FP8_E4M3 ? 448.0f : 57344.0f;
        float r = 1.0f / s;
        for (int64_t i = 0; i < n; ++i) {
            float y = clampf(X[i] * r, -mx, mx);
            unsigned c = mf_encode(mf, y);
            codes[i] = (uint8_t)c;
            if (xh) xh[i] = (float)mf_decode(mf, c) * s;
        }
        return 0;
    }
    if (K % 32) return -1;
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t b = 0; b < K / 32; ++b) {
            const float* x = X + m * K + 32 * b;
            uint8_t* c = codes + m * K + 32 * b;
            float* h = xh ? xh + m * K + 32 * b : NULL;
            uint8_t* eb = &e8[m * (K / 32) + b];
            if (fmt == A_MXFP8) {
                q_mxfp_block(x, 32, &MF_E4M3, 0, 448.0f, c, h, eb);
            } else {
                float tmp[32];
                q_mxint_block(x, 32, 6, 127, 8, c, h ? h : tmp, eb);
            }
        }
    }
    return 0;
}

/* Decode activation codes back to binary32. */
int orc_dequant_act(int64_t M, int64_t K, int fmt, const uint8_t* codes, const uint8_t* e8,
                    float s, float z, float* xh) {
    int64_t n = M * K;
    for (int64_t i = 0; i < n; ++i) {
        unsigned u = codes[i];
        float v;
        switch (fmt) {
        case A_INT8_ASYM: v = ((float)u - z) * s; break;
        case A_FP8_E4M3: v = (float)mf_decode(&MF_E4M3, u) * s; break;
        case A_FP8_E5M2: v = (float)mf_decode(&MF_E5M2, u) * s; break;
        case A_MXFP8: v = ldexpf((float)mf_decode(&MF_E4M3, u), (int)e8[i / 32] - 127); break;
        case A_MXINT8: v = ldexpf((float)(int8_t)u, (int)e8[i / 32] - 127 - 6); break;
        default: return -1;
        }
        xh[i] = v;
    }
    return 0;
}

/* ------------------------------------------------------------------------- */
/* calibration statistics and the LUT (Sec. 4.3, Sec. 4.4, App. A.7 Alg. 1)       */
/* ------------------------------------------------------------------------- */
/* nS[5] = n, S1..S4 (binary64 power sums), lohi[2] = running min / max (binary32). */
void orc_stats_accumulate(const float* X, int64_t n, double* nS, float* lohi) {
    double s1 = 0, s2 = 0, s3 = 0, s4 = 0;
    float lo = lohi[0], hi = lohi[1];
    for (int64_t i = 0; i < n; ++i) {
        double d = (double)X[i];
        double d2 = d * d;
        s1 += d;
        s2 += d2;
        s3 += d2 * d;
        s4 += d2 * d2;
        lo = fminf(lo, X[i]);
        hi = fmaxf(hi, X[i]);
    }
    nS[0] += (double)n;
    nS[1] += s1;
    nS[2] += s2;
    nS[3] += s3;
    nS[4] += s4;
    lohi[0] = lo;
    lohi[1] = hi;
}

/* Pearson kurtosis m4 / m2^2 from raw power sums (App. A.3, Eq. kurt; Sec. 4.4). */
double orc_kurtosis(const double* nS) {
    double n = nS[0];
    double mu = nS[1] / n;
    double e2 = nS[2] / n, e3 = nS[3] / n, e4 = nS[4] / n;
    double m2 = e2 - mu * mu;
    double m4 = e4 - 4.0 * mu * e3 + 6.0 * mu * mu * e2 - 3.0 * mu * mu * mu * mu;
    return m4 / (m2 * m2);
}

/* Noise schedule (Sec. 3.1, Eq. snr): alpha_bar_t = prod_{s<=t} (1 - beta_s), t = 0..T-1,
 * SNR(t) = alpha_bar_t / (1 - alpha_bar_t).  kind 0: scaled-linear betas
 * (sqrt(b0) + (sqrt(b1)-sqrt(b0)) s/(T-1))^2; kind 1: linear b0 + (b1-b0) s/(T-1). */
void orc_snr_table(int T, double b0, double b1, int kind, double* snr) {
    double ab = 1.0;
    double r0 = sqrt(b0), r1 = sqrt(b1);
    for (int s = 0; s < T; ++s) {
        double frac = T > 1 ? (double)s / (double)(T - 1) : 0.0;
        double beta;
        if (kind == 0) { double r = r0 + (r1 - r0) * frac; beta = r * r; }
        else beta = b0 + (b1 - b0) * frac;
        ab *= (1.0 - beta);
        snr[s] = ab / (1.0 - ab);
    }
}

/* bucket of timestep t (Alg. 2): min(floor(t B / T), B - 1) */
int orc_bucket(int t, int T, int B) {
    long b = ((long)t * B) / T;
    return (int)(b < B - 1 ? b : B - 1);
}

/* bucket midpoint t_b = b T/B + T/(2B), floored to an integer timestep (Sec. 4.3) */
int orc_bucket_mid(int b, int T, int B) { return (int)(((long)(2 * b + 1) * T) / (2L * B)); }

/* Routing rule of Sec. 4.3. gates: kappa_lo, kappa_hi, snr_lo, snr_hi; snr_gate_on = 0
 * disables the SNR conditions (the kurtosis-only arm). */
int orc_route(double kappa, double snr, int is_shortcut, double k_lo, double k_hi, double s_lo,
              double s_hi, int snr_gate_on) {
    if (is_shortcut) return A_MXFP8;
    int snr_low = snr_gate_on ? (snr < s_lo) : 0;
    int snr_high = snr_gate_on ? (snr > s_hi) : 1;
    if (kappa > k_hi || snr_low) return A_FP8_E5M2;
    if (kappa <= k_lo && snr_high) return A_INT8_ASYM;
    return A_FP8_E4M3;
}

/* Alg. 1 second loop: for each (l, b): kappa, SNR(t_b), Route, ScaleZP.
 * nS [L*B*5], lohi [L*B*2]; is_shortcut [L] or NULL; outputs F [L*B] u8, S, Z [L*B] f32,
 * kappa [L*B] f64 (may be NULL).  An empty bucket (n = 0) gets s = 1, z = 0 (READING). */
void orc_build_lut(int L, int B, const double* nS, const float* lohi, int T, double b0,
                   double b1, int kind, double k_lo, double k_hi, double s_lo, double s_hi,
                   int snr_gate_on, const uint8_t* is_shortcut, uint8_t* F, float* S,
                   float* Z, double* kappa_out) {
    static double snr[1 << 16];
    orc_snr_table(T, b0, b1, kind, snr);
    for (int l = 0; l < L; ++l) {
        for (int b = 0; b < B; ++b) {
            int i = l * B + b;
            double kap = orc_kurtosis(nS + 5 * i);
            double sn = snr[orc_bucket_mid(b, T, B)];
            int f = orc_route(kap, sn, is_shortcut ? is_shortcut[l] : 0, k_lo, k_hi, s_lo, s_hi,
                              snr_gate_on);
            float s, z;
            if (nS[5 * i] == 0.0) { s = 1.0f; z = 0.0f; }
            else orc_scale_zp(f, lohi[2 * i], lohi[2 * i + 1], &s, &z);
            F[i] = (uint8_t)f;
            S[i] = s;
            Z[i] = z;
            if (kappa_out) kappa_out[i] = kap;
        }
    }
}

/* ------------------------------------------------------------------------- */
/* the linear layer on dequantized operands (binary64 reference)                 */
/* ------------------------------------------------------------------------- */
/* Y[m][n] = sum_k Xh[m][k] Wh[n][k]; Babs[m][n] = sum_k |Xh Wh| (the tolerance scale). */
void orc_linear(int64_t M, int64_t N, int64_t K, const float* Xh, const float* Wh, double* Y,
                double* Babs) {
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < N; ++n) {
            double acc = 0.0, ab = 0.0;
            for (int64_t k = 0; k < K; ++k) {
                double p = (double)Xh[m * K + k] * (double)Wh[n * K + k];
                acc += p;
                ab += fabs(p);
            }
            Y[m * N + n] = acc;
            if (Babs) Babs[m * N + n] = ab;
        }
}

/* The same on a list of (m, n) pairs. */
void orc_linear_pairs(int64_t K, int64_t npairs, const int64_t* mm, const int64_t* nn,
                      const float* Xh, const float* Wh, double* Y, double* Babs) {
    for (int64_t p = 0; p < npairs; ++p) {
        double acc = 0.0, ab = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            double v = (double)Xh[mm[p] * K + k] * (double)Wh[nn[p] * K + k];
            acc += v;
            ab += fabs(v);
        }
        Y[p] = acc;
        Babs[p] = ab;
    }
}

/* ------------------------------------------------------------------------- */
/* DiT joint (group size, format) weight search (Sec. 4.6 (i), Fig. dit caption;  */
/* App. A.11).  For every tuple (g, f) of the group sizes G = {32, 64, 128, 192,   */
/* 288} and the enabled formats, every output row is quantized in groups of g      */
/* consecutive input channels (the last group holds K mod g when g does not divide */
/* K; READING), each group with its own scale as the format's per-channel           */
/* quantizer defines it (INT-sym/asym ScaleZP on the group's range, FP4 amax/6, NF4 */
/* the group absmax); MX formats carry their own 32-element blocks and are         */
/* evaluated at g = 32 only.  The input-aware error of a tuple is                   */
/* sum_n sum_k e_k (w - w^)^2 with e_k = E[x_k^2] (the SQNR of the paper weights     */
/* each input channel's squared error by its activation energy; the signal term is */
/* common to all tuples, so the argmax SQNR is this argmin).  Ties go to the lowest  */
/* tuple index t = gi * 9 + f (group sizes in the listed order, formats in palette  */
/* order; READING).                                                                 */
/* ------------------------------------------------------------------------- */
static const int GROUP_SIZES[5] = { 32, 64, 128, 192, 288 };

static int is_mx_fmt(int f) { return f == W_MXINT8 || f == W_MXINT4 || f == W_MXFP4; }

/* Round trip one row in groups of g with format f; scale / zero per group into gs / gz
 * (index j of group j; NF4: the group absmax), e8 per 32-block for MX formats. */
static void gq_row(int f, int g, const float* w, int64_t K, uint8_t* code, float* wh, float* gs,
                   float* gz, uint8_t* e8) {
    nf4_build();
    for (int64_t b = 0; b < K / 32; ++b) { gs[b] = 0.0f; gz[b] = 0.0f; if (e8) e8[b] = 0; }
    if (is_mx_fmt(f)) {  /* its own 32-blocks */
        float s;
        float z;
        wq_row(f, w, K, code, wh, &s, &z, NULL, e8);
        return;
    }
    for (int64_t j = 0; j * g < K; ++j) {
        const int64_t k0 = j * g, n = (k0 + g <= K) ? g : K - k0;
        float s = 0.0f;
        float z = 0.0f;
        switch (f) {
        case W_INT8_SYM: q_int_sym(w + k0, n, 127, 8, code + k0, wh + k0, &s); break;
        case W_INT4_SYM: q_int_sym(w + k0, n, 7, 4, code + k0, wh + k0, &s); break;
        case W_INT8_ASYM: q_int_asym(w + k0, n, 255, code + k0, wh + k0, &s, &z); break;
        case W_INT4_ASYM: q_int_asym(w + k0, n, 15, code + k0, wh + k0, &s, &z); break;
        case W_FP4: q_fp4(w + k0, n, code + k0, wh + k0, &s); break;
        case W_NF4: q_nf4_block(w + k0, n, code + k0, wh + k0, &s); break;
        }
        gs[j] = s;
        gz[j] = z;
    }
}

/* The search over a layer W [N][K] (K % 32 == 0, K <= 65536).  mask: formats; gmask: group
 * sizes (bit i enables GROUP_SIZES[i]); energy [K] (binary32).  Outputs: choice[2] = {g, f},
 * err[45] = the layer error of each tuple (-1 when not evaluated), fmt [N] (= f), codes
 * ([N][K/2] when every enabled format is 4-bit, else [N][K]), gscale / gzero [N][K/32]
 * (group j at j, 0 past the last group), e8 [N][K/32] (MX; may be NULL).
 * Returns 0, or -1 on a bad argument. */
int orc_select_group_formats(const float* W, int64_t N, int64_t K, uint32_t mask, uint32_t gmask,
                             const float* energy, int32_t* choice, double* err, uint8_t* fmt,
                             uint8_t* codes, float* gscale, float* gzero, uint8_t* e8) {
    if (N < 1 || K <= 0 || K % 32 || K > (1 << 16) || mask == 0 || (mask & ~0x1FFu) || gmask == 0 ||
        (gmask & ~0x1Fu))
        return -1;
    static float wh[1 << 16], gs[1 << 11], gz[1 << 11];
    static uint8_t cb[1 << 16], eb[1 << 11];
    int code_bits = 4;
    for (int f = 0; f < W_NFMT; ++f)
        if (((mask >> f) & 1u) && wfmt_bits(f) == 8) code_bits = 8;
    for (int t = 0; t < 45; ++t) err[t] = -1.0;
    int best = -1;
    for (int gi = 0; gi < 5; ++gi) {
        if (!((gmask >> gi) & 1u)) continue;
        for (int f = 0; f < W_NFMT; ++f) {
            if (!((mask >> f) & 1u)) continue;
            if (is_mx_fmt(f) && GROUP_SIZES[gi] != 32) continue;
            double e = 0.0;
            for (int64_t n = 0; n < N; ++n) {
                gq_row(f, GROUP_SIZES[gi], W + n * K, K, cb, wh, gs, gz, eb);
                for (int64_t k = 0; k < K; ++k) {
                    float d = W[n * K + k] - wh[k];
                    e += (double)energy[k] * ((double)d * (double)d);
                }
            }
            const int t = gi * 9 + f;
            err[t] = e;
            if (best < 0 || e < err[best]) best = t;
        }
    }
    if (best < 0) return -1;  /* only MX formats enabled without g = 32 */
    const int g = GROUP_SIZES[best / 9], f = best % 9;
    choice[0] = g;
    choice[1] = f;
    for (int64_t n = 0; n < N; ++n) {
        gq_row(f, g, W + n * K, K, cb, wh, gs, gz, eb);
        fmt[n] = (uint8_t)f;
        for (int64_t b = 0; b < K / 32; ++b) {
            gscale[n * (K / 32) + b] = gs[b];
            gzero[n * (K / 32) + b] = gz[b];
            if (e8) e8[n * (K / 32) + b] = is_mx_fmt(f) ? eb[b] : 0;
        }
        if (code_bits == 4) {
            for (int64_t k = 0; k < K; k += 2)
                codes[n * (K / 2) + k / 2] = (uint8_t)((cb[k] & 15u) | ((cb[k + 1] & 15u) << 4));
        } else {
            memcpy(codes + n * K, cb, (size_t)K);
        }
    }
    return 0;
}

/* Decode a grouped weight (as emitted above) to binary32. */
int orc_dequant_grouped(int64_t N, int64_t K, int code_bits, int g, int f, const uint8_t* codes,
                        const float* gscale, const float* gzero, const uint8_t* e8, float* Wh) {
    nf4_build();
    if (K % 32 || K > (1 << 16)) return -1;
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t k = 0; k < K; ++k) {
            unsigned u = code_bits == 4 ? ((codes[n * (K / 2) + k / 2] >> (4 * (k & 1))) & 15u)
                                        : codes[n * K + k];
            const float s = gscale[n * (K / 32) + k / g], z = gzero[n * (K / 32) + k / g];
            float v = 0.0f;
            switch (f) {
            case W_INT8_SYM: v = (float)(int8_t)u * s; break;
            case W_INT4_SYM: v = (float)((int)(u << 28) >> 28) * s; break;
            case W_INT8_ASYM:
            case W_INT4_ASYM: v = ((float)u - z) * s; break;
            case W_FP4: v = (float)mf_decode(&MF_E2M1, u) * s; break;
            case W_NF4: v = NF4[u & 15u] * s; break;
            case W_MXINT8: v = ldexpf((float)(int8_t)u, (int)e8[n * (K / 32) + k / 32] - 127 - 6); break;
            case W_MXINT4: v = ldexpf((float)((int)(u << 28) >> 28), (int)e8[n * (K / 32) + k / 32] - 127 - 2); break;
            case W_MXFP4: v = ldexpf((float)mf_decode(&MF_E2M1, u), (int)e8[n * (K / 32) + k / 32] - 127); break;
            }
            Wh[n * K + k] = v;
        }
    }
    return 0;
}

/* Round trip one row in groups (diagnostics and pins). */
void orc_gq_row(int f, int g, const float* w, int64_t K, uint8_t* codes, float* wh, float* gs,
                float* gz, uint8_t* e8) {
    gq_row(f, g, w, K, codes, wh, gs, gz, e8);
}

/* ------------------------------------------------------------------------- */
/* 3x3 convolution (stride 1, zero padding 1) on dequantized operands -- the UNet   */
/* path's conv layers, e.g. the up-block resnet conv1 downstream of a shortcut     */
/* concatenation that Sec. 4.6 routes to MXFP8 -- in binary64.  Xh [B][H][W][C]      */
/* (channels last), Wh [Co][3][3][C] (tap-major rows of 9C, the linear layer's      */
/* [N][K] with K = 9C), Y [B][H][W][Co]; Babs the sum of |products| (tolerance).    */
/* ------------------------------------------------------------------------- */
void orc_conv3x3(int64_t B, int64_t H, int64_t W, int64_t C, int64_t Co, const float* Xh,
                 const float* Wh, double* Y, double* Babs) {
    for (int64_t b = 0; b < B; ++b)
        for (int64_t y = 0; y < H; ++y)
            for (int64_t x = 0; x < W; ++x)
                for (int64_t o = 0; o < Co; ++o) {
                    double acc = 0.0, ab = 0.0;
                    for (int64_t ky = 0; ky < 3; ++ky)
                        for (int64_t kx = 0; kx < 3; ++kx) {
                            const int64_t yy = y + ky - 1, xx = x + kx - 1;
                            if (yy < 0 || yy >= H || xx < 0 || xx >= W) continue;
                            const float* xp = Xh + ((b * H + yy) * W + xx) * C;
                            const float* wp = Wh + o * 9 * C + (ky * 3 + kx) * C;
                            for (int64_t c = 0; c < C; ++c) {
                                const double p = (double)xp[c] * (double)wp[c];
                                acc += p;
                                ab += fabs(p);
                            }
                        }
                    const int64_t i = ((b * H + y) * W + x) * Co + o;
                    Y[i] = acc;
                    if (Babs) Babs[i] = ab;
                }
}
