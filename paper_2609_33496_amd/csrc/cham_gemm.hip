// Mixed-format linear layer: Y = DQ(X codes) . DQ(W codes)^T with a per-output-channel
// weight format (Sec. 4.5) and one activation format per call (Sec. 4.3).
//
// Per-channel formats do not map onto one native MFMA operand type (Sec. 6), so the
// weights are dequantized on the fly into a common half-precision operand: every code of
// every 4-bit format becomes an entry of a 16-value table built per (channel, scale block)
// -- base value (NF4 level, E2M1 value, integer, q - z) times the block factor (NF4 block
// absmax, MX 2^E) relative to the channel's largest block, rounded once to half precision.
// The table lives in registers as two byte planes and is read with v_perm_b32, so decoding
// needs no LDS traffic.  Integers, E2M1 values and MX mantissas are exact in half precision;
// NF4 levels times their block absmax carry one rounding (relative error <= 2^-11).  8-bit
// integer formats are decoded arithmetically (1024 + c trick, exact).
//
// Activations are decoded once per call by a small pre-pass into a half-precision copy in
// the workspace (exact for every activation format), with the per-row scale.  The main
// kernel tiles BM x BN x 64 over 4 wavefronts (2 x 2), runs v_mfma_f32_32x32x16_f16 with
// binary32 accumulation, streams the activation tile through double-buffered LDS, and keeps
// each wavefront's weight operand in registers.  Inside a tile the output channels are
// sorted by format, so a 32-channel MFMA column block almost always decodes one format
// (wave-uniform branches); every output line of the tile is still written by the tile.
//
// The MFMA contracts over k in any order as long as both operands agree: a lane's 8 values
// of one k-step are the codes of 8 consecutive k in the order (0,2,4,6,1,3,5,7) when codes
// are packed two per byte (even/odd nibbles), and the activation copy stores its columns in
// that same order.
#include "cham_device.h"

namespace cham {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float16v __attribute__((ext_vector_type(16)));

constexpr int BK = 64;
constexpr int LDA = BK + 8;  // LDS row stride of the activation tile (halves)

// ------------------------------------------------------------------------------------
// activation pre-pass: codes -> half precision (exact), k permuted within groups of 8
// ------------------------------------------------------------------------------------
struct DecodeArgs {
    const uint8_t* xc;
    const uint8_t* xe8;
    const float* xs;
    const float* xz;
    int afmt;
    int M, K;
    int perm4;  // 1: store each group of 8 columns in the order 0,2,4,6,1,3,5,7
    _Float16* Xh;
    float* rowscale;
};

CHAM_DEV float adecode(int afmt, uint32_t c, float z, int kblk_e, int eref) {
    switch (afmt) {
    case CHAM_A_INT8_ASYM: return (float)c - z;
    case CHAM_A_FP8_E4M3: return e4m3_decode(c);
    case CHAM_A_FP8_E5M2: return e5m2_decode(c);
    case CHAM_A_MXFP8_E4M3: return ldexpf(e4m3_decode(c), kblk_e - eref);
    default: return ldexpf((float)(int8_t)c, kblk_e - 6 - eref);  // MXINT8
    }
}

// Per-channel decode parameters, computed by the pre-pass for every output channel.
struct ColPrep {
    int fmt;         // CHAM_W_NFMT: not a valid format of the palette (decodes as zero)
    int eref;        // exponent removed from block-scaled values (NF4 / MX), 0 otherwise
    float zero;      // INT-asym zero point
    float colscale;  // epilogue factor: INT/FP4 scale, or 2^eref
};

struct PrepArgs {
    DecodeArgs d;
    const uint8_t* wfmt;
    const float* wscale;
    const int32_t* wzero;
    const float* wnf4;
    const uint8_t* we8;
    int N;
    uint32_t mask;
    ColPrep* cols;
};

// Workgroups [0, M): activation row m -> half precision.  Workgroups [M, M + ceil(N/256)):
// one thread per output channel computes its ColPrep.
__global__ __launch_bounds__(256) void prep_kernel(PrepArgs p) {
    const DecodeArgs& a = p.d;
    if ((int)blockIdx.x >= a.M) {
        const int n = ((int)blockIdx.x - a.M) * 256 + (int)threadIdx.x;
        if (n >= p.N) return;
        const int K = a.K;
        ColPrep c{CHAM_W_NFMT, 0, 0.0f, 0.0f};
        const int f = p.wfmt[n];
        if (f < CHAM_W_NFMT && ((p.mask >> f) & 1u)) {
            c.fmt = f;
            c.zero = (float)p.wzero[n];
            if (f == CHAM_W_NF4) {
                float mx = 0.0f;
                const float* r = p.wnf4 + (int64_t)n * (K / 64);
#pragma unroll 8
                for (int b = 0; b < K / 64; ++b) mx = fmaxf(mx, r[b]);
                c.eref = floor_log2(floor_scale(mx));
                c.colscale = ldexpf(1.0f, c.eref);
            } else if (f == CHAM_W_MXINT8 || f == CHAM_W_MXINT4 || f == CHAM_W_MXFP4) {
                int mx = 0;
                const uint32_t* r = reinterpret_cast<const uint32_t*>(p.we8 + (int64_t)n * (K / 32));
#pragma unroll 8
                for (int b = 0; b < K / 128; ++b) {
                    const uint32_t w = r[b];
                    mx = max(mx, (int)max(max(w & 255u, (w >> 8) & 255u), max((w >> 16) & 255u, w >> 24)));
                }
                for (int b = (K / 128) * 4; b < K / 32; ++b) mx = max(mx, (int)p.we8[(int64_t)n * (K / 32) + b]);
                const int F = f == CHAM_W_MXINT8 ? 6 : (f == CHAM_W_MXINT4 ? 2 : 0);
                c.eref = mx - 127 - F;
                c.colscale = ldexpf(1.0f, c.eref);
            } else {
                c.colscale = p.wscale[n];
            }
        }
        p.cols[n] = c;
        return;
    }
    const int m = blockIdx.x;
    const int K = a.K;
    const bool mx = a.afmt == CHAM_A_MXFP8_E4M3 || a.afmt == CHAM_A_MXINT8;
    __shared__ int sh_e;
    int eref = 0;
    if (mx) {
        int mx_e = 0;
        for (int b = threadIdx.x; b < K / 32; b += blockDim.x) mx_e = max(mx_e, (int)a.xe8[(int64_t)m * (K / 32) + b]);
        for (int o = 32; o > 0; o >>= 1) mx_e = max(mx_e, __shfl_xor(mx_e, o, kWave));
        if (threadIdx.x == 0) sh_e = 0;
        __syncthreads();
        if ((threadIdx.x & 63) == 0) atomicMax(&sh_e, mx_e);
        __syncthreads();
        eref = sh_e - 127;
    }
    const float z = *a.xz;
    const uint8_t* row = a.xc + (int64_t)m * K;
    _Float16* out = a.Xh + (int64_t)m * K;
    for (int g = threadIdx.x; g < K / 8; g += blockDim.x) {
        const uint2 c2 = *reinterpret_cast<const uint2*>(row + 8 * g);
        const int kb = mx ? (int)a.xe8[(int64_t)m * (K / 32) + (g >> 2)] - 127 : 0;
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            uint32_t c = ((j < 4 ? c2.x : c2.y) >> (8 * (j & 3))) & 0xFFu;
            v[j] = adecode(a.afmt, c, z, kb, eref);
        }
        half8 h;
        if (a.perm4) {
            h[0] = (_Float16)v[0]; h[1] = (_Float16)v[2]; h[2] = (_Float16)v[4]; h[3] = (_Float16)v[6];
            h[4] = (_Float16)v[1]; h[5] = (_Float16)v[3]; h[6] = (_Float16)v[5]; h[7] = (_Float16)v[7];
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) h[j] = (_Float16)v[j];
        }
        *reinterpret_cast<half8*>(out + 8 * g) = h;
    }
    if (threadIdx.x == 0) a.rowscale[m] = mx ? ldexpf(1.0f, eref) : *a.xs;
}

// ------------------------------------------------------------------------------------
// main kernel
// ------------------------------------------------------------------------------------
struct GemmArgs {
    const _Float16* Xh;      // [M][K] (column order as above)
    const float* rowscale;   // [M]
    const ColPrep* cols;     // [N]
    const uint8_t* wc;       // codes
    const float* wnf4;       // [N][K/64]
    const uint8_t* we8;      // [N][K/32]
    float* Y;
    int M, N, K;
};

struct ColInfo {
    int n;           // channel index (-1: padding / invalid)
    int fmt;
    int eref;
    float zero;
    float colscale;
};

CHAM_DEV bool is_mx(int f) { return f == CHAM_W_MXINT8 || f == CHAM_W_MXINT4 || f == CHAM_W_MXFP4; }
CHAM_DEV bool is_8bit(int f) { return f == CHAM_W_INT8_SYM || f == CHAM_W_INT8_ASYM || f == CHAM_W_MXINT8; }

// 16-entry half-precision table as byte planes: lo[j] holds the low bytes of entries
// 4j..4j+3, hi[j] the high bytes.
struct Table {
    uint32_t lo[4], hi[4];
};

CHAM_DEV void table_from_values(Table& t, const float (&v)[16]) {
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        h2 a01, a23;
        a01.x = (_Float16)v[4 * j + 0]; a01.y = (_Float16)v[4 * j + 1];
        a23.x = (_Float16)v[4 * j + 2]; a23.y = (_Float16)v[4 * j + 3];
        const uint32_t w01 = __builtin_bit_cast(uint32_t, a01), w23 = __builtin_bit_cast(uint32_t, a23);
        t.lo[j] = __builtin_amdgcn_perm(w23, w01, 0x06040200u);
        t.hi[j] = __builtin_amdgcn_perm(w23, w01, 0x07050301u);
    }
}

// Base values of the 4-bit codes of each format (before the block factor).
CHAM_DEV float e2m1_value(int c) {
    const float m[8] = {0.0f, 0.5f, 1.0f, 1.5f, 2.0f, 3.0f, 4.0f, 6.0f};
    return (c & 8) ? -m[c & 7] : m[c & 7];
}

template <int F>
CHAM_DEV void table_fmt(Table& t, float zero, float factor) {
    float v[16];
#pragma unroll
    for (int c = 0; c < 16; ++c) {
        float b;
        if (F == CHAM_W_NF4) b = nf4_level(c);
        else if (F == CHAM_W_FP4 || F == CHAM_W_MXFP4) b = e2m1_value(c);
        else if (F == CHAM_W_INT4_ASYM) b = (float)c - zero;
        else b = (float)(c < 8 ? c : c - 16);  // INT4-sym, MXINT4
        v[c] = b * factor;
    }
    table_from_values(t, v);
}

// Table of channel format f (4-bit) with block factor `factor` (branches are wave-uniform
// whenever the 32 channels of an MFMA column block share a format).
CHAM_DEV void build_table(Table& t, int f, float zero, float factor) {
    switch (f) {
    case CHAM_W_NF4: table_fmt<CHAM_W_NF4>(t, zero, factor); break;
    case CHAM_W_FP4: table_fmt<CHAM_W_FP4>(t, zero, factor); break;
    case CHAM_W_MXFP4: table_fmt<CHAM_W_MXFP4>(t, zero, factor); break;
    case CHAM_W_INT4_ASYM: table_fmt<CHAM_W_INT4_ASYM>(t, zero, factor); break;
    default: table_fmt<CHAM_W_INT4_SYM>(t, zero, factor); break;
    }
}

// Look up 4 codes (one per byte, values 0..15); returns the low and high bytes.
CHAM_DEV void lookup4(const Table& t, uint32_t codes, uint32_t& lo, uint32_t& hi) {
    const uint32_t sel = codes & 0x07070707u;
    const uint32_t sel2 = 0x03020100u | ((codes >> 1) & 0x04040404u);
    const uint32_t l0 = __builtin_amdgcn_perm(t.lo[1], t.lo[0], sel);
    const uint32_t l1 = __builtin_amdgcn_perm(t.lo[3], t.lo[2], sel);
    const uint32_t h0 = __builtin_amdgcn_perm(t.hi[1], t.hi[0], sel);
    const uint32_t h1 = __builtin_amdgcn_perm(t.hi[3], t.hi[2], sel);
    lo = __builtin_amdgcn_perm(l1, l0, sel2);
    hi = __builtin_amdgcn_perm(h1, h0, sel2);
}

union H8 {
    half8 h;
    uint32_t u[4];
};

// 8 codes of one k-step from a word of 8 nibbles -> order (0,2,4,6,1,3,5,7)
CHAM_DEV half8 decode_nibbles(const Table& t, uint32_t w) {
    uint32_t lo_e, hi_e, lo_o, hi_o;
    lookup4(t, w & 0x0F0F0F0Fu, lo_e, hi_e);
    lookup4(t, (w >> 4) & 0x0F0F0F0Fu, lo_o, hi_o);
    H8 r;
    r.u[0] = __builtin_amdgcn_perm(hi_e, lo_e, 0x05010400u);
    r.u[1] = __builtin_amdgcn_perm(hi_e, lo_e, 0x07030602u);
    r.u[2] = __builtin_amdgcn_perm(hi_o, lo_o, 0x05010400u);
    r.u[3] = __builtin_amdgcn_perm(hi_o, lo_o, 0x07030602u);
    return r.h;
}

// 8 codes in natural order from two words of 4 byte-codes (4-bit formats in 8-bit layout)
CHAM_DEV half8 decode_bytes_table(const Table& t, uint32_t w0, uint32_t w1) {
    uint32_t lo0, hi0, lo1, hi1;
    lookup4(t, w0, lo0, hi0);
    lookup4(t, w1, lo1, hi1);
    H8 r;
    r.u[0] = __builtin_amdgcn_perm(hi0, lo0, 0x05010400u);
    r.u[1] = __builtin_amdgcn_perm(hi0, lo0, 0x07030602u);
    r.u[2] = __builtin_amdgcn_perm(hi1, lo1, 0x05010400u);
    r.u[3] = __builtin_amdgcn_perm(hi1, lo1, 0x07030602u);
    return r.h;
}

// 8-bit integer codes: value = ((c ^ x) - zoff) * factor, through 1024 + c in half precision
CHAM_DEV half8 decode_bytes_int(uint32_t w0, uint32_t w1, uint32_t xmask, _Float16 negoff, _Float16 factor) {
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    w0 ^= xmask;
    w1 ^= xmask;
    H8 r;
    r.u[0] = __builtin_amdgcn_perm(0x64646464u, w0, 0x04010400u);
    r.u[1] = __builtin_amdgcn_perm(0x64646464u, w0, 0x04030402u);
    r.u[2] = __builtin_amdgcn_perm(0x64646464u, w1, 0x04010400u);
    r.u[3] = __builtin_amdgcn_perm(0x64646464u, w1, 0x04030402u);
    h2 off = {negoff, negoff}, fac = {factor, factor};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        h2 v = __builtin_bit_cast(h2, r.u[i]);
        v = (v + off) * fac;
        r.u[i] = __builtin_bit_cast(uint32_t, v);
    }
    return r.h;
}

CHAM_DEV int mx_F(int f) { return f == CHAM_W_MXINT8 ? 6 : (f == CHAM_W_MXINT4 ? 2 : 0); }

template <int BM, int BN, int WAVES_M, int WAVES_N, int CODE_BITS>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N, 1) void gemm_kernel(GemmArgs a) {
    constexpr int kThreads = 64 * WAVES_M * WAVES_N;
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;  // wavefront tile
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int A_CHUNKS = BM * BK * 2 / 16 / kThreads;  // 16-byte chunks per thread
    static_assert(A_CHUNKS >= 1 && BN <= kThreads, "tile / workgroup mismatch");
    __shared__ _Float16 As[2][BM][LDA];
    __shared__ ColInfo cinfo[BN];
    __shared__ uint64_t ballots[CHAM_W_NFMT + 1][kThreads / kWave];

    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const int K = a.K;

    // ---- prologue: sort this tile's channels by format (ballot ranks, deterministic)
    ColPrep cp{CHAM_W_NFMT, 0, 0.0f, 0.0f};
    if (t < BN && n0 + t < a.N) cp = a.cols[n0 + t];
    const int myf = t < BN ? cp.fmt : CHAM_W_NFMT + 1;
    for (int f = 0; f <= CHAM_W_NFMT; ++f) {
        const uint64_t b = __ballot(myf == f);
        if (lane == 0) ballots[f][wave] = b;
    }
    __syncthreads();
    if (t < BN) {
        int pos = __popcll(ballots[myf][wave] & ((1ull << lane) - 1ull));
        for (int w = 0; w < wave; ++w) pos += __popcll(ballots[myf][w]);
        for (int f = 0; f < myf; ++f)
            for (int w = 0; w < kThreads / kWave; ++w) pos += __popcll(ballots[f][w]);
        ColInfo ci{-1, CHAM_W_INT4_SYM, 0, 0.0f, 0.0f};
        if (myf < CHAM_W_NFMT) ci = ColInfo{n0 + t, myf, cp.eref, cp.zero, cp.colscale};
        cinfo[pos] = ci;
    }
    __syncthreads();

    const int wm = (wave / WAVES_N) * WM, wn = (wave % WAVES_N) * WN;
    const int g = lane >> 5;  // k-half of the lane within a k-step
    ColInfo my[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) my[j] = cinfo[wn + j * 32 + (lane & 31)];

    // channels whose table does not depend on the k-block: build once
    Table tab[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j)
        if (!is_mx(my[j].fmt) && my[j].fmt != CHAM_W_NF4 && !is_8bit(my[j].fmt))
            build_table(tab[j], my[j].fmt, my[j].zero, 1.0f);

    float16v acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    // activation tile loads: chunk c -> row c / 8, 16-byte column c % 8
    uint4 areg[A_CHUNKS];
    auto load_a = [&](int k0) {
#pragma unroll
        for (int i = 0; i < A_CHUNKS; ++i) {
            const int c = i * kThreads + t;
            const int r = c >> 3, col = (c & 7) * 8;
            const int m = m0 + r;
            areg[i] = m < a.M ? *reinterpret_cast<const uint4*>(a.Xh + (int64_t)m * K + k0 + col)
                              : make_uint4(0u, 0u, 0u, 0u);
        }
    };
    auto store_a = [&](int buf) {
#pragma unroll
        for (int i = 0; i < A_CHUNKS; ++i) {
            const int c = i * kThreads + t;
            const int r = c >> 3, col = (c & 7) * 8;
            *reinterpret_cast<uint4*>(&As[buf][r][col]) = areg[i];
        }
    };
    // weight codes of a k-step (32 consecutive k of each of the lane's TN channels) and the
    // block metadata of those k (NF4 absmax bits, or the E8M0 byte)
    constexpr int CW = CODE_BITS == 4 ? 4 : 8;  // 32-bit words per channel per k-step
    uint32_t wreg[TN][CW];
    uint32_t mreg[TN];
    auto load_w = [&](int k0) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int n = my[j].n;
            if (n < 0) {
#pragma unroll
                for (int q = 0; q < CW; ++q) wreg[j][q] = 0u;
                mreg[j] = 0u;
                continue;
            }
            if (CODE_BITS == 4) {
                const uint4 v = *reinterpret_cast<const uint4*>(a.wc + (int64_t)n * (K / 2) + (k0 + 32 * g) / 2);
                wreg[j][0] = v.x; wreg[j][1] = v.y; wreg[j][2] = v.z; wreg[j][3] = v.w;
            } else {
                const uint4* p = reinterpret_cast<const uint4*>(a.wc + (int64_t)n * K + k0 + 32 * g);
                const uint4 v0 = p[0], v1 = p[1];
                wreg[j][0] = v0.x; wreg[j][1] = v0.y; wreg[j][2] = v0.z; wreg[j][3] = v0.w;
                wreg[j][4] = v1.x; wreg[j][5] = v1.y; wreg[j][6] = v1.z; wreg[j][7] = v1.w;
            }
            if (my[j].fmt == CHAM_W_NF4) mreg[j] = __float_as_uint(a.wnf4[(int64_t)n * (K / 64) + (k0 >> 6)]);
            else if (is_mx(my[j].fmt)) mreg[j] = a.we8[(int64_t)n * (K / 32) + ((k0 + 32 * g) >> 5)];
            else mreg[j] = 0u;
        }
    };

    const int nsteps = K / BK;
    load_a(0);
    load_w(0);
    store_a(0);
    __syncthreads();

    for (int step = 0; step < nsteps; ++step) {
        const int k0 = step * BK;
        const int buf = step & 1;
        uint32_t wcur[TN][CW];
        _Float16 bfac[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
#pragma unroll
            for (int q = 0; q < CW; ++q) wcur[j][q] = wreg[j][q];
            const ColInfo& ci = my[j];
            bfac[j] = (_Float16)1.0f;
            if (ci.fmt == CHAM_W_NF4) {
                build_table(tab[j], CHAM_W_NF4, 0.0f, ldexpf(__uint_as_float(mreg[j]), -ci.eref));
            } else if (is_mx(ci.fmt)) {
                const float factor = ldexpf(1.0f, (int)mreg[j] - 127 - mx_F(ci.fmt) - ci.eref);
                if (ci.fmt == CHAM_W_MXINT8) bfac[j] = (_Float16)factor;
                else build_table(tab[j], ci.fmt, 0.0f, factor);
            }
        }
        // prefetch the next k-step
        if (step + 1 < nsteps) {
            load_a(k0 + BK);
            load_w(k0 + BK);
        }
        // 4 sub-steps of 16 k: lane group g covers k = 32g + 8s .. +7
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            half8 af[TM];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                af[i] = *reinterpret_cast<const half8*>(&As[buf][wm + i * 32 + (lane & 31)][32 * g + 8 * s]);
            half8 bf[TN];
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                if (CODE_BITS == 4) {
                    bf[j] = decode_nibbles(tab[j], wcur[j][s]);
                } else {
                    const ColInfo& ci = my[j];
                    if (is_8bit(ci.fmt)) {
                        const bool sgn = ci.fmt != CHAM_W_INT8_ASYM;
                        bf[j] = decode_bytes_int(wcur[j][2 * s], wcur[j][2 * s + 1], sgn ? 0x80808080u : 0u,
                                                 (_Float16)(-(1024.0f + (sgn ? 128.0f : ci.zero))), bfac[j]);
                    } else {
                        bf[j] = decode_bytes_table(tab[j], wcur[j][2 * s], wcur[j][2 * s + 1]);
                    }
                }
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[i], bf[j], acc[i][j], 0, 0, 0);
        }
        if (step + 1 < nsteps) {
            store_a(buf ^ 1);
            __syncthreads();
        }
    }

    // ---- epilogue: 32x32 tile, lane holds column lane%32, rows 8*(r/4) + 4*(lane/32) + r%4
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        float rs[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int m = m0 + wm + i * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
            rs[r] = m < a.M ? a.rowscale[m] : 0.0f;
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const ColInfo& ci = my[j];
            if (ci.n < 0) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = m0 + wm + i * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
                if (m < a.M) a.Y[(int64_t)m * a.N + ci.n] = (acc[i][j][r] * rs[r]) * ci.colscale;
            }
        }
    }
}

template <int BM, int BN, int WAVES_M, int WAVES_N>
void launch_gemm(const GemmArgs& a, int code_bits, hipStream_t s) {
    dim3 grid((unsigned)((a.N + BN - 1) / BN), (unsigned)((a.M + BM - 1) / BM));
    dim3 block(64 * WAVES_M * WAVES_N);
    if (code_bits == 4) hipLaunchKernelGGL((gemm_kernel<BM, BN, WAVES_M, WAVES_N, 4>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((gemm_kernel<BM, BN, WAVES_M, WAVES_N, 8>), grid, block, 0, s, a);
}

}  // namespace
}  // namespace cham

using namespace cham;

size_t cham_linear_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    const size_t xh = (((size_t)M * (size_t)K * 2) + 255) & ~(size_t)255;
    const size_t rs = (((size_t)M * 4) + 255) & ~(size_t)255;
    return xh + rs + (size_t)N * sizeof(ColPrep);
}

extern "C" int cham_mixed_linear(const cham_aq* xq, const cham_wq* wq, float* Y, void* ws, size_t ws_bytes,
                                 void* stream) {
    if (!xq || !wq || !Y || !xq->codes || !xq->scale || !xq->zero) return CHAM_EINVAL;
    if (!wq->fmt || !wq->codes || !wq->scale || !wq->zero) return CHAM_EINVAL;
    if (xq->M < 1 || wq->N < 1 || xq->K < 1 || xq->K != wq->K) return CHAM_EINVAL;
    if (xq->M > INT32_MAX / 2 || wq->N > INT32_MAX / 2 || xq->K > INT32_MAX / 2) return CHAM_EINVAL;
    if (xq->fmt < 0 || xq->fmt >= CHAM_A_NFMT) return CHAM_EFORMAT;
    const uint32_t mask = wq->palette_mask;
    if (mask == 0u || (mask >> CHAM_W_NFMT) != 0u) return CHAM_EFORMAT;
    const int code_bits = (mask & 0x7u) ? 8 : 4;
    if (wq->code_bits != code_bits) return CHAM_EFORMAT;
    if (xq->K % 64 != 0) return CHAM_ESHAPE;
    const bool nf4 = (mask >> CHAM_W_NF4) & 1u;
    const bool wmx = (mask & ((1u << CHAM_W_MXINT8) | (1u << CHAM_W_MXINT4) | (1u << CHAM_W_MXFP4))) != 0u;
    if ((nf4 && !wq->nf4_absmax) || (wmx && !wq->e8m0)) return CHAM_EINVAL;
    const bool amx = xq->fmt == CHAM_A_MXFP8_E4M3 || xq->fmt == CHAM_A_MXINT8;
    if (amx && !xq->e8m0) return CHAM_EINVAL;
    if (((uintptr_t)xq->codes & 15u) || ((uintptr_t)wq->codes & 15u)) return CHAM_EINVAL;
    const size_t need = cham_linear_workspace_bytes(xq->M, wq->N, xq->K);
    if (!ws || ws_bytes < need || ((uintptr_t)ws & 255u)) return CHAM_EWORKSPACE;
    hipStream_t s = (hipStream_t)stream;

    char* w = (char*)ws;
    _Float16* Xh = (_Float16*)w;
    w += (((size_t)xq->M * (size_t)xq->K * 2) + 255) & ~(size_t)255;
    float* rowscale = (float*)w;
    w += (((size_t)xq->M * 4) + 255) & ~(size_t)255;
    ColPrep* cols = (ColPrep*)w;

    PrepArgs p;
    p.d.xc = xq->codes;
    p.d.xe8 = xq->e8m0;
    p.d.xs = xq->scale;
    p.d.xz = xq->zero;
    p.d.afmt = xq->fmt;
    p.d.M = (int)xq->M;
    p.d.K = (int)xq->K;
    p.d.perm4 = code_bits == 4;
    p.d.Xh = Xh;
    p.d.rowscale = rowscale;
    p.wfmt = wq->fmt;
    p.wscale = wq->scale;
    p.wzero = wq->zero;
    p.wnf4 = wq->nf4_absmax;
    p.we8 = wq->e8m0;
    p.N = (int)wq->N;
    p.mask = mask;
    p.cols = cols;
    const unsigned nprep = (unsigned)(p.d.M + (p.N + 255) / 256);
    hipLaunchKernelGGL(prep_kernel, dim3(nprep), dim3(256), 0, s, p);
    CHAM_CHECK_LAUNCH();

    GemmArgs a;
    a.Xh = Xh;
    a.rowscale = rowscale;
    a.cols = cols;
    a.wc = wq->codes;
    a.wnf4 = wq->nf4_absmax;
    a.we8 = wq->e8m0;
    a.Y = Y;
    a.M = (int)xq->M;
    a.N = (int)wq->N;
    a.K = (int)xq->K;
    // tile choice: the largest tile that still gives about one wave of workgroups on 256 CUs
    const int64_t t256 = ((a.M + 255) / 256) * (int64_t)((a.N + 255) / 256);
    const int64_t t128x256 = ((a.M + 127) / 128) * (int64_t)((a.N + 255) / 256);
    if (t256 >= 240) launch_gemm<256, 256, 2, 4>(a, code_bits, s);
    else if (t128x256 >= 200) launch_gemm<128, 256, 2, 4>(a, code_bits, s);
    else launch_gemm<128, 128, 2, 4>(a, code_bits, s);
    CHAM_CHECK_LAUNCH();
    return CHAM_OK;
}
