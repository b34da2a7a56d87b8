// Mixed-format linear layer: Y = DQ(X codes) . DQ(W codes)^T with a per-output-channel
// weight format (Sec. 4.5) and one activation format per call (Sec. 4.3).
//
// Per-channel formats do not map onto one native MFMA operand type (Sec. 6), so the
// weights are dequantized on the fly into a common half-precision operand.  Every 4-bit
// code of every format is an entry of a 16-value decode table per (k-step of 64, channel,
// half k-step of 32): base value (NF4 level, E2M1 value, integer, q - z) times the block
// factor (NF4 block absmax, MX 2^E) relative to the channel's largest block, rounded to
// binary32 and then to half precision.  A pre-pass packs, per (k-step, channel, half), the
// codes and this table (two byte planes) into one record (layout in cham_records.h); the
// main kernel decodes with v_perm_b32, so every 4-bit format decodes with the same
// instructions.  Integers, E2M1 values and MX mantissas are exact in half precision; NF4
// levels times their block absmax carry the two roundings (relative error <= 2^-11 +
// 2^-24).  8-bit integer formats are decoded arithmetically
// (1024 + c trick, exact) with parameters from the same table slot.
//
// Activations in a per-tensor format (INT8, E4M3, E5M2) are decoded to half precision
// while they are staged into LDS (exact); MX activations are decoded by a pre-pass into a
// half-precision copy relative to the row's largest block exponent, with a row scale.
//
// Main kernel: BM x 256 output tiles (BM = 256, 128 or 64), or 128 x 128 for layers whose
// full-width tiles leave CUs idle; k-steps of 64; four wavefronts that each own BM rows x
// 32 TN channels (BM/32 x TN blocks of v_mfma_f32_32x32x16_f16, binary32 accumulation), so
// a decoded weight feeds BM/32 MFMAs per k sub-step.
// Activation tiles and weight records go global -> registers with coalesced 16-byte
// buffer loads one or more k-steps ahead (deeper register rings for the short steps of
// small tiles); the activation tile is stored into one of two LDS buffers with its
// 16-byte chunks XOR-swizzled per row pair, so all LDS accesses are free of bank
// conflicts, and the weight records stay in registers.  Barriers fence LDS only, so the
// prefetch stays in flight across them.  Layers with too few output tiles to fill the
// CUs split k over several workgroups that write partial outputs, summed in split order
// by a second kernel; every output element is produced by plain stores (no atomics), so
// results do not depend on scheduling.
//
// The MFMA contracts over k in any order as long as both operands agree: lane half h of a
// k-step takes k = 32h .. 32h+31, sub-step s the 8 k at 32h + 8s, and with two codes per
// byte those 8 values come in the order (0,4,1,5,2,6,3,7); the activation operand is
// staged with its columns in that same order.
#include <atomic>
#include <cmath>
#include <vector>

#include "cham_device.h"
#include "cham_group.h"
#include "cham_records.h"

namespace cham {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float16v __attribute__((ext_vector_type(16)));

constexpr int BK = 64;
constexpr int kThreads = 256;
// TN = 32-channel MFMA blocks per wavefront: a tile is 128 TN channels wide (four wavefronts)
constexpr int tile_width(int TN) { return 128 * TN; }
constexpr int kBufferFlags = 0x00020000;  // buffer descriptor word 3: 32-bit data, raw
constexpr int kStoreNonTemporal = 2;      // cache-policy operand of a buffer store: nt

// ------------------------------------------------------------------------------------
// pre-pass for MX activation formats: codes -> half precision relative to the row's
// largest block exponent (exact for blocks within 2^28 of it), the row scale separately
// ------------------------------------------------------------------------------------
struct PrepArgs {
    const uint8_t* xc;
    const uint8_t* xe8;
    int afmt;
    int M, K;
    int perm4;  // 1: store each group of 8 columns in the order 0,4,1,5,2,6,3,7
    _Float16* Xh;
    float* rowscale;
};

// One workgroup per activation row.
__global__ __launch_bounds__(256) void prep_kernel(PrepArgs p) {
    const int K = p.K;
    const int m = blockIdx.x;
    __shared__ int sh_e;
    int mx_e = 0;
    for (int b = threadIdx.x; b < K / 32; b += blockDim.x) mx_e = max(mx_e, (int)p.xe8[(int64_t)m * (K / 32) + b]);
    for (int o = 32; o > 0; o >>= 1) mx_e = max(mx_e, __shfl_xor(mx_e, o, kWave));
    if (threadIdx.x == 0) sh_e = 0;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) atomicMax(&sh_e, mx_e);
    __syncthreads();
    // the row's largest block lands at [2^14, 2^15): blocks down to 2^-28 of it stay normal
    // in half precision (values are below 2 times 2^(block exponent - eref))
    const int eref = sh_e - 127 - 14;
    const uint8_t* row = p.xc + (int64_t)m * K;
    _Float16* out = p.Xh + (int64_t)m * K;
    for (int g = threadIdx.x; g < K / 8; g += blockDim.x) {
        const uint2 c2 = *reinterpret_cast<const uint2*>(row + 8 * g);
        const int kb = (int)p.xe8[(int64_t)m * (K / 32) + (g >> 2)] - 127;
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t c = ((j < 4 ? c2.x : c2.y) >> (8 * (j & 3))) & 0xFFu;
            v[j] = p.afmt == CHAM_A_MXFP8_E4M3 ? ldexpf(e4m3_decode(c), kb - eref)
                                               : ldexpf((float)(int8_t)c, kb - 6 - eref);
        }
        half8 h;
        if (p.perm4) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                h[2 * j] = (_Float16)v[j];
                h[2 * j + 1] = (_Float16)v[j + 4];
            }
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) h[j] = (_Float16)v[j];
        }
        *reinterpret_cast<half8*>(out + 8 * g) = h;
    }
    if (threadIdx.x == 0) p.rowscale[m] = ldexpf(1.0f, eref);
}

// ------------------------------------------------------------------------------------
// pre-pass of the 3x3 convolution: the activation codes -> a zero-padded half-precision
// copy [B][H+2][W+2][C] (the border is the padding) that the GEMM gathers per output pixel
// and tap.  MX formats relative to the tensor's largest block exponent (every output row
// gathers nine pixels, so they need one reference), per-tensor formats as code values
// (E4M3, E5M2 exact) or q - z (INT8-asym) with the sample's scale as the row scale.
// ------------------------------------------------------------------------------------
struct PrepConvArgs {
    const uint8_t* xc;
    const uint8_t* xe8;
    int afmt;
    int B, H, W, C;
    int perm4;
    const float* xs;  // per-sample scale / zero point (per-tensor formats)
    const float* xz;
    int rps;          // rows (pixels) per sample
    int* emax;        // MX: the largest biased block exponent of the tensor (device)
    _Float16* Xh;
    float* rowscale;  // [B*H*W]
};

// One workgroup: the largest E8M0 byte of n (a plain maximum, so the order is free).
__global__ __launch_bounds__(1024) void emax_kernel(const uint8_t* e8, int64_t n, int* out) {
    int m = 0;
    for (int64_t i = threadIdx.x; i < n; i += 1024) m = max(m, (int)e8[i]);
    for (int o = 32; o > 0; o >>= 1) m = max(m, __shfl_xor(m, o, kWave));
    __shared__ int wm[16];
    if ((threadIdx.x & 63) == 0) wm[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int i = 1; i < 16; ++i) m = max(m, wm[i]);
        *out = max(m, wm[0]);
    }
}

// One workgroup per padded pixel.
__global__ __launch_bounds__(256) void prep_conv_kernel(PrepConvArgs p) {
    const int C = p.C, Wp = p.W + 2, Hp = p.H + 2;
    const int pp = blockIdx.x, xp = pp % Wp, yb = pp / Wp, yp = yb % Hp, b = yb / Hp;
    _Float16* out = p.Xh + (int64_t)pp * C;
    const bool border = xp == 0 || yp == 0 || xp == Wp - 1 || yp == Hp - 1;
    if (border) {
        for (int g = threadIdx.x; g < C / 8; g += blockDim.x) *reinterpret_cast<uint4*>(out + 8 * g) = make_uint4(0u, 0u, 0u, 0u);
        return;
    }
    const int64_t m = ((int64_t)b * p.H + (yp - 1)) * p.W + (xp - 1);  // source = output row
    const bool mx = p.afmt == CHAM_A_MXFP8_E4M3 || p.afmt == CHAM_A_MXINT8;
    const float z = mx ? 0.0f : p.xz[m / p.rps];
    // MX: the tensor's reference exponent; INT8-asym: the power of two that keeps q - z
    // within half precision's range
    const float zm = fabsf(z) + 255.0f;
    const int eref = mx ? *p.emax - 127 - 14
                        : (p.afmt == CHAM_A_INT8_ASYM && zm >= 32768.0f ? floor_log2(zm) - 14 : 0);
    const uint8_t* row = p.xc + m * C;
    for (int g = threadIdx.x; g < C / 8; g += blockDim.x) {
        const uint2 c2 = *reinterpret_cast<const uint2*>(row + 8 * g);
        const int kb = mx ? (int)p.xe8[m * (C / 32) + (g >> 2)] - 127 : 0;
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t c = ((j < 4 ? c2.x : c2.y) >> (8 * (j & 3))) & 0xFFu;
            switch (p.afmt) {
            case CHAM_A_MXFP8_E4M3: v[j] = ldexpf(e4m3_decode(c), kb - eref); break;
            case CHAM_A_MXINT8: v[j] = ldexpf((float)(int8_t)c, kb - 6 - eref); break;
            case CHAM_A_FP8_E4M3: v[j] = e4m3_decode(c); break;
            case CHAM_A_FP8_E5M2: v[j] = e5m2_decode(c); break;
            default: v[j] = ldexpf((float)c - z, -eref); break;  // INT8-asym
            }
        }
        half8 h;
        if (p.perm4) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                h[2 * j] = (_Float16)v[j];
                h[2 * j + 1] = (_Float16)v[j + 4];
            }
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) h[j] = (_Float16)v[j];
        }
        *reinterpret_cast<half8*>(out + 8 * g) = h;
    }
    if (threadIdx.x == 0) p.rowscale[m] = mx ? ldexpf(1.0f, eref) : ldexpf(p.xs[m / p.rps], eref);
}

// ------------------------------------------------------------------------------------
// weight decode in the main kernel
// ------------------------------------------------------------------------------------

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

// 8 codes of one sub-step from a word of 8 nibbles -> order (0,4,1,5,2,6,3,7)
CHAM_DEV half8 decode_nibbles(const Table& t, uint32_t w) {
    uint32_t lo_e, hi_e, lo_o, hi_o;
    lookup4(t, w & 0x0F0F0F0Fu, lo_e, hi_e);         // k = 0, 2, 4, 6
    lookup4(t, (w >> 4) & 0x0F0F0F0Fu, lo_o, hi_o);  // k = 1, 3, 5, 7
    H8 r;
    r.u[0] = __builtin_amdgcn_perm(hi_e, lo_e, 0x06020400u);  // k0, k4
    r.u[1] = __builtin_amdgcn_perm(hi_o, lo_o, 0x06020400u);  // k1, k5
    r.u[2] = __builtin_amdgcn_perm(hi_e, lo_e, 0x07030501u);  // k2, k6
    r.u[3] = __builtin_amdgcn_perm(hi_o, lo_o, 0x07030501u);  // k3, k7
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

// 8-bit integer codes: value = fma((1024 + (c ^ x)) + a, f, b) in half precision, 1024 + c
// formed by placing c in the mantissa; x, a, f and b come from the table slot.
CHAM_DEV half8 decode_bytes_int(const Table& t, uint32_t w0, uint32_t w1) {
    w0 ^= t.lo[0];
    w1 ^= t.lo[0];
    H8 r;
    r.u[0] = __builtin_amdgcn_perm(0x64646464u, w0, 0x04010400u);
    r.u[1] = __builtin_amdgcn_perm(0x64646464u, w0, 0x04030402u);
    r.u[2] = __builtin_amdgcn_perm(0x64646464u, w1, 0x04010400u);
    r.u[3] = __builtin_amdgcn_perm(0x64646464u, w1, 0x04030402u);
    const half2v off = __builtin_bit_cast(half2v, t.lo[1]), fac = __builtin_bit_cast(half2v, t.lo[2]),
                 off2 = __builtin_bit_cast(half2v, t.lo[3]);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        half2v v = __builtin_bit_cast(half2v, r.u[i]);
        v = __builtin_elementwise_fma(v + off, fac, off2);
        r.u[i] = __builtin_bit_cast(uint32_t, v);
    }
    return r.h;
}

// ------------------------------------------------------------------------------------
// pre-pass 2: weight records (layout in cham_records.h), one per (k-step, channel, half
// k-step): the half's codes (16 bytes at 4 bits, 32 at 8 bits), then its decode table
// ------------------------------------------------------------------------------------
struct RecArgs {
    const uint8_t* wfmt;
    const float* wscale;
    const float* wzero;
    const float* wnf4;
    const uint8_t* we8;
    const uint8_t* wc;
    uint32_t mask;
    int N, K, code_bits;
    int kchunk;  // k-steps per workgroup
    ColPrep* cols;
    float* colsum;  // [k-chunks][N] per workgroup chunk of k-steps: the sum of the channel's
                    // decoded weights (the GEMM adds the chunks in order)
    uint4* rec;     // [K/64][N][2][pieces]
    // group-scaled weights (the DiT search): the chosen group size on the device (NULL: the
    // per-channel formats above), per-group scale / NF4 absmax and zero point [N][K/32]
    const int32_t* gsel;
    const float* gscale;
    const float* gzero;
};

// Workgroup b handles 32 channels (block b % nblk) and the k-steps of chunk b / nblk.
// 8 threads per channel compute its ColPrep (the reference exponent is the largest NF4
// block absmax or MX block exponent of the whole channel); thread t builds the records of
// channel t/2 % 32, half t % 2, at k-steps congruent to t/64 mod 4, so each wavefront
// stores 64 consecutive records (coalesced).  The codes and block metadata of the
// thread's first kRecPrefetch records are loaded before the ColPrep pass, so both
// passes' loads are in flight together.
constexpr int kRecChannels = 32;
constexpr int kRecPrefetch = 3;

// Several weights' records in one launch: the workgroups of the batch's layers follow
// each other (descriptors in the kernel arguments); before them, one workgroup per entry
// of g groups a searched weight's channels by format (the search's grouping, run here when
// the search also packs the weights, to save a launch; first, so its longer serial work
// overlaps the records instead of trailing them).
constexpr int kRecBatchMax = 16;
struct RecBatch {
    int nl, ng;
    int wg_end[kRecBatchMax];  // record workgroups of layers 0..i
    RecArgs r[kRecBatchMax];
    GroupArgs g[kRecBatchMax];
};

__global__ __launch_bounds__(256) void record_kernel(RecBatch B) {
    __shared__ ColPrep cp[kRecChannels];
    if ((int)blockIdx.x < B.ng) {  // workgroup-uniform
        group_channels<256>(B.g[blockIdx.x], nullptr);
        return;
    }
    const int rb = (int)blockIdx.x - B.ng;  // record workgroup index
    int li = 0;
    while (li + 1 < B.nl && rb >= B.wg_end[li]) ++li;
    const RecArgs& a = B.r[li];
    const int bid = rb - (li ? B.wg_end[li - 1] : 0);
    const int t = threadIdx.x;
    const int K = a.K, nst = K / BK;
    const int nblk = (a.N + kRecChannels - 1) / kRecChannels;
    const int cb = bid % nblk, kc = bid / nblk;
    const int n0 = cb * kRecChannels;
    const int cw = a.code_bits / 4;  // 16-byte code pieces per half k-step
    const int64_t cstride = (int64_t)K * a.code_bits / 8;

    // this thread's records: channel n, half h, k-steps kb, kb + 4, ... below ke
    const int n = n0 + ((t & 63) >> 1), h = t & 1;
    const bool live = n < a.N;
    const int kb = kc * a.kchunk + (t >> 6), ke = min(nst, (kc + 1) * a.kchunk);
    const int gsz = a.gsel ? *a.gsel : 0;  // group size of group-scaled weights, else 0
    // block parameters of a record: NF4 absmax (or the group's scale / absmax) in nfa, the
    // group's zero point in gz, the MX exponent in e8
    auto load_rec = [&](int k, uint4 (&code)[2], float& nfa, float& gz, int& e8) __attribute__((always_inline)) {
        const uint4* src = reinterpret_cast<const uint4*>(a.wc + n * cstride + (int64_t)k * (16 * a.code_bits / 2) +
                                                          (int64_t)h * 16 * cw);
        code[0] = src[0];
        code[1] = cw > 1 ? src[1] : make_uint4(0u, 0u, 0u, 0u);
        if (gsz) {
            const int64_t j = (int64_t)n * (K / 32) + (64 * k + 32 * h) / gsz;
            nfa = a.gscale[j];
            gz = a.gzero[j];
        } else {
            nfa = a.wnf4 ? a.wnf4[(int64_t)n * (K / 64) + k] : 0.0f;
            gz = 0.0f;
        }
        e8 = a.we8 ? (int)a.we8[(int64_t)n * (K / 32) + 2 * k + h] : 0;
    };
    auto store_rec = [&](int k, const uint4 (&code)[2], const Table& tb) __attribute__((always_inline)) {
        uint4* dst = a.rec + (((int64_t)k * a.N + n) * 2 + h) * (cw + 2);
        dst[0] = code[0];
        if (cw > 1) dst[1] = code[1];
        dst[cw] = make_uint4(tb.lo[0], tb.lo[1], tb.lo[2], tb.lo[3]);
        dst[cw + 1] = make_uint4(tb.hi[0], tb.hi[1], tb.hi[2], tb.hi[3]);
    };
    uint4 pc[kRecPrefetch][2];
    float pn[kRecPrefetch], pz[kRecPrefetch];
    int pe[kRecPrefetch];
#pragma unroll
    for (int i = 0; i < kRecPrefetch; ++i)
        if (live && kb + 4 * i < ke) load_rec(kb + 4 * i, pc[i], pn[i], pz[i], pe[i]);

    {
        const int ch = t >> 3, sub = t & 7;
        const int nn = n0 + ch;
        const int f = nn < a.N ? a.wfmt[nn] : CHAM_W_NFMT;
        const bool ok = f < CHAM_W_NFMT && ((a.mask >> f) & 1u);
        // the block metadata of every enabled kind is read without waiting for the format
        // (it is zero for channels of other formats), so these loads overlap the format load
        float mxf = 0.0f;
        int mxe = 0;
        if (nn < a.N && a.wnf4) {
            const float* r = a.wnf4 + (int64_t)nn * (K / 64);
#pragma unroll 4
            for (int b = sub; b < K / 64; b += 8) mxf = fmaxf(mxf, r[b]);
        }
        if (nn < a.N && a.we8) {
            const uint8_t* r = a.we8 + (int64_t)nn * (K / 32);
#pragma unroll 4
            for (int b = sub; b < K / 32; b += 8) mxe = max(mxe, (int)r[b]);
        }
        if (gsz && nn < a.N && ok && !is_mx(f)) {
            // group-scaled: the largest decoded magnitude over the channel's groups
            const int G = (K + gsz - 1) / gsz;
            const float* gs = a.gscale + (int64_t)nn * (K / 32);
            const float* gzr = a.gzero + (int64_t)nn * (K / 32);
            for (int j = sub; j < G; j += 8) {
                float m = gs[j];  // NF4: the group absmax
                if (f == CHAM_W_FP4) m = 6.0f * gs[j];
                else if (f == CHAM_W_INT4_SYM) m = 7.0f * gs[j];
                else if (f == CHAM_W_INT8_SYM) m = 127.0f * gs[j];
                else if (f == CHAM_W_INT4_ASYM || f == CHAM_W_INT8_ASYM) {
                    const float L = f == CHAM_W_INT4_ASYM ? 15.0f : 255.0f;
                    m = fmaxf(fabsf(gzr[j]), fabsf(L - gzr[j])) * gs[j];
                }
                mxf = fmaxf(mxf, m);
            }
        } else if (!(ok && f == CHAM_W_NF4)) {
            mxf = 0.0f;
        }
        if (!(ok && is_mx(f))) mxe = 0;
#pragma unroll
        for (int o = 1; o < 8; o <<= 1) {
            mxf = fmaxf(mxf, __shfl_xor(mxf, o, kWave));
            mxe = max(mxe, __shfl_xor(mxe, o, kWave));
        }
        ColPrep c{CHAM_W_NFMT, 0, 0.0f, 0.0f};
        if (ok && gsz && !is_mx(f)) {
            // group-scaled: every table is relative to the channel's largest decoded magnitude
            c.fmt = f;
            c.eref = floor_log2(floor_scale(mxf)) - 14;
            c.colscale = ldexpf(1.0f, c.eref);
        } else if (ok) {
            c.fmt = f;
            c.zero = a.wzero[nn];
            if (f == CHAM_W_NF4) {
                // levels (|v| <= 1) times the block absmax over 2^eref stay below 2^15, and a
                // block 2^-28 below the largest is still a normal half-precision number
                c.eref = floor_log2(floor_scale(mxf)) - 14;
                c.colscale = ldexpf(1.0f, c.eref);
            } else if (is_mx(f)) {
                // element magnitudes up to 127 (MXINT8) times 2^8 stay below 2^15
                c.eref = mxe - 127 - mx_F(f) - 8;
                c.colscale = ldexpf(1.0f, c.eref);
            } else if (f == CHAM_W_INT8_ASYM || f == CHAM_W_INT4_ASYM) {
                c.eref = int_asym_eref(c.zero, f == CHAM_W_INT8_ASYM ? 255.0f : 15.0f);
                c.colscale = ldexpf(a.wscale[nn], c.eref);
            } else {
                c.colscale = a.wscale[nn];
            }
        }
        if (sub == 0) {
            cp[ch] = c;
            if (kc == 0 && nn < a.N) a.cols[nn] = c;
        }
    }
    __syncthreads();
    const ColPrep c = cp[(t & 63) >> 1];
    auto table = [&](float nfa, float gz, int e8) __attribute__((always_inline)) {
        return gsz && !is_mx(c.fmt) ? group_table(c, nfa, gz) : record_table(c, nfa, e8);
    };
    // the sum of the record's decoded weights (the half-precision values the GEMM uses,
    // relative to colscale), through the GEMM's own decode and binary32 dot products
    const bool int8c = a.code_bits == 8 && is_8bit(c.fmt);
    auto record_sum = [&](const uint4 (&code)[2], const Table& tb) __attribute__((always_inline)) {
        float sum = 0.0f;
        const half2v one = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            H8 v;
            if (a.code_bits == 4) {
                const uint32_t w = q == 0 ? code[0].x : q == 1 ? code[0].y : q == 2 ? code[0].z : code[0].w;
                v.h = decode_nibbles(tb, w);
            } else {
                const uint4& cc = code[q >> 1];
                const uint32_t w0 = (q & 1) ? cc.z : cc.x, w1 = (q & 1) ? cc.w : cc.y;
                v.h = int8c ? decode_bytes_int(tb, w0, w1) : decode_bytes_table(tb, w0, w1);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) sum = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2v, v.u[r]), one, sum, false);
        }
        return sum;
    };
    double psum = 0.0;
    if (live) {
#pragma unroll
        for (int i = 0; i < kRecPrefetch; ++i)
            if (kb + 4 * i < ke) {
                const Table tb = table(pn[i], pz[i], pe[i]);
                store_rec(kb + 4 * i, pc[i], tb);
                psum += (double)record_sum(pc[i], tb);
            }
        for (int k = kb + 4 * kRecPrefetch; k < ke; k += 4) {
            uint4 code[2];
            float nfa, gz;
            int e8;
            load_rec(k, code, nfa, gz, e8);
            const Table tb = table(nfa, gz, e8);
            store_rec(k, code, tb);
            psum += (double)record_sum(code, tb);
        }
    }
    // the channel's sum over this workgroup's k-steps: its 8 threads (2 halves x 4 k-phases)
    // added in a fixed order, times the channel's scale
    __shared__ double part[4][64];
    part[t >> 6][t & 63] = psum;
    __syncthreads();
    if (t < kRecChannels && n0 + t < a.N) {
        double s2 = 0.0;
#pragma unroll
        for (int p = 0; p < 4; ++p) s2 += part[p][2 * t] + part[p][2 * t + 1];
        a.colsum[(int64_t)kc * a.N + n0 + t] = (float)(s2 * (double)cp[t].colscale);
    }
}

// Workgroup barrier that orders LDS accesses only: outstanding global loads (the
// prefetch) stay in flight.
CHAM_DEV void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// ------------------------------------------------------------------------------------
// main kernel
// ------------------------------------------------------------------------------------
struct GemmArgs {
    const _Float16* Xh;      // [M][K] (column order as above), MX activation formats
    const float* rowscale;   // [M], MX activation formats
    const uint8_t* xc;       // [M][K] activation codes, per-tensor formats
    const float* xs;         // activation scale per sample [M / rps] (per-tensor formats)
    const float* xz;         // activation zero point per sample
    int rps;                 // rows per sample
    const ColPrep* cols;     // [N]
    const float* colsum;     // [nkc][N] per k-chunk sums of the decoded weights
    int nkc;
    const uint4* rec;        // [K/64][N][2][pieces]
    float* Y;
    int M, N, K;
    int row0, row1;  // rows [row0, row1) of this launch
    int tn;          // tile columns
    int gm;          // tile rows per group of the XCD-aware tile order, 0: row-major (launch_gemm)
    int splits;      // k-splits: workgroup b takes tile b % tiles and k-steps of split b / tiles
    int kchunk;      // k-steps per split
    float* part;     // splits > 1: [splits][M][N] partial outputs, summed by reduce_kernel
    // 3x3 convolution (implicit GEMM): Xh is the zero-padded activation [B][H+2][W+2][C] in
    // half precision; row m = (b, y, x) of the output, k = (ky * 3 + kx) * C + c
    int H, W, C;
    uint32_t xh_bytes;
};

// Activation operand source: the half-precision copy of the pre-pass (MX formats), the
// per-tensor codes, decoded while they are staged into LDS, or (3x3 convolution) the
// pre-pass's zero-padded half-precision copy, gathered per output pixel and tap.
constexpr int kAF16 = 0, kAInt8 = 1, kAE4M3 = 2, kAE5M2 = 3, kAConv = 4;

// 8 activation codes (k0..k3 in w0, k4..k7 in w1) -> 8 halves, in the order
// (0,4,1,5,2,6,3,7) when perm4, else natural; exact for all three per-tensor formats.
template <int AF>
CHAM_DEV uint4 decode_act8(uint32_t w0, uint32_t w1, bool perm4, half2v negz) {
    // byte selectors of v_perm_b32(w1, w0, sel): 0..3 -> k0..k3, 4..7 -> k4..k7, 12 -> 0
    uint32_t d[4];
    if (AF == kAE5M2) {  // E5M2 is the top byte of binary16
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t a = perm4 ? j : 2 * j, b = perm4 ? j + 4 : 2 * j + 1;
            d[j] = __builtin_amdgcn_perm(w1, w0, 0x0Cu | (a << 8) | (0x0Cu << 16) | (b << 24));
        }
    } else if (AF == kAE4M3) {  // hardware E4M3 -> binary16 conversion, unit scale
        const uint32_t p0 = perm4 ? __builtin_amdgcn_perm(w1, w0, 0x05010400u) : w0;
        const uint32_t p1 = perm4 ? __builtin_amdgcn_perm(w1, w0, 0x07030602u) : w1;
        d[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(p0, 1.0f, false));
        d[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(p0, 1.0f, true));
        d[2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(p1, 1.0f, false));
        d[3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(p1, 1.0f, true));
    } else {  // INT8-asym: (1024 + c) - (1024 + z) in binary16
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t a = perm4 ? j : 2 * j, b = perm4 ? j + 4 : 2 * j + 1;
            const uint32_t v = __builtin_amdgcn_perm(w1, w0, a | (0x0Cu << 8) | (b << 16) | (0x0Cu << 24)) | 0x64006400u;
            d[j] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, v) + negz);
        }
    }
    return make_uint4(d[0], d[1], d[2], d[3]);
}

template <int CODE_BITS, int TM, int AF, int TN>
__global__ __launch_bounds__(kThreads, TN == 1 ? 3 : (TM == 4 && CODE_BITS == 4) ? 2 : 1) void gemm_kernel(GemmArgs a) {
    constexpr int BM = 32 * TM;
    constexpr int BN = tile_width(TN);
    constexpr int CW = CODE_BITS / 4;  // 16-byte code pieces per record
    constexpr int P = CW + 2;          // 16-byte pieces per record (codes + two table planes)
    constexpr bool HALF = AF == kAF16 || AF == kAConv;   // the operand comes in half precision
    constexpr int AQ = HALF ? TM : (TM + 1) / 2;  // activation loads per thread per k-step
    // codes: every load of the workgroup falls inside the tile (even TM), no range test
    constexpr bool AFULL = HALF || AQ * kThreads == BM * 4;
    constexpr int A_CH = BM * BK * 2 / 16;      // 16-byte chunks of an activation tile
    __shared__ uint4 lds[2][A_CH];
    __shared__ __align__(16) float Rs[BM];
    __shared__ __align__(16) float Rc[AF == kAInt8 ? BM : 4];

    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int l32 = lane & 31, h = lane >> 5;
    const int K = a.K, N = a.N;
    // Workgroup -> (split, tile).  gm = 0: tiles in row-major order, workgroup b taking
    // tile b % tiles of split b / tiles.  gm > 0, the XCD-aware order: the dispatcher deals
    // a launch's workgroups to the chip's 8 XCDs in turn (workgroup b runs on XCD b % 8, as
    // its (b / 8)-th), and each XCD has its own L2, so each XCD takes a contiguous run of a
    // logical order that walks groups of gm tile rows column by column: an XCD's tiles form
    // a block of about gm rows by a few columns, whose activation rows and weight columns
    // its L2 serves.  Both maps are bijections of [0, grid), whatever the grid.
    const int mt = (a.row1 - a.row0 + BM - 1) / BM;
    const int tiles = mt * a.tn;
    const int G = (int)gridDim.x, b = (int)blockIdx.x, xcd = b & 7;
    const int lin = a.gm > 0 ? xcd * (G >> 3) + (xcd < (G & 7) ? xcd : (G & 7)) + (b >> 3) : b;
    const int tile = lin % tiles, split = lin / tiles;
    int m0, n0;
    if (a.gm > 0) {
        const int g0 = (tile / (a.gm * a.tn)) * a.gm;    // first tile row of the group
        const int gm = a.gm < mt - g0 ? a.gm : mt - g0;  // its tile rows (the last may be short)
        const int in = tile - g0 * a.tn;
        m0 = a.row0 + (g0 + in % gm) * BM;
        n0 = (in / gm) * BN;
    } else {
        m0 = a.row0 + (tile / a.tn) * BM;
        n0 = (tile % a.tn) * BN;
    }
    const int rows = a.row1 - m0 < BM ? a.row1 - m0 : BM;
    // k-steps [kb, kb + nsteps) of this workgroup; the operand bases below start at kb
    const int kb = split * a.kchunk;
    const int nsteps = K / BK - kb < a.kchunk ? K / BK - kb : a.kchunk;

    // per-row activation scale (the row's sample's s; MX: the pre-pass's row scale).
    // INT8-asym: codes are decoded as (1024 + c) - (1024 + z1) with z1 the sample's zero point
    // clamped to [-1024, 1024] (exact in half precision); the rest z - z1 (an integer, exact
    // in binary32) is taken out in the epilogue as -(z - z1) s times the channel's weight sum
    // (split 0 only).
    if (t < BM) {
        const int m = t < rows ? m0 + t : m0;
        if (HALF) {
            Rs[t] = a.rowscale[m];
        } else {
            Rs[t] = a.xs[m / a.rps];
            if (AF == kAInt8) {
                const float za = a.xz[m / a.rps], z1 = clampf(za, -1024.0f, 1024.0f);
                Rc[t] = split == 0 ? -((za - z1) * a.xs[m / a.rps]) : 0.0f;
            }
        }
    }
    // the staging rows of this thread (row q >> 2 of load q = 256 i + t): their -(1024 + z1)
    constexpr int AQ0 = HALF ? 1 : (TM + 1) / 2;
    half2v negz[AQ0];
#pragma unroll
    for (int i = 0; i < AQ0; ++i) {
        negz[i] = half2v{(_Float16)0.0f, (_Float16)0.0f};
        if (AF == kAInt8) {
            const int r = (i * 256 + t) >> 2;
            const int m = r < rows ? m0 + r : m0;
            const _Float16 nz = (_Float16)(-(1024.0f + clampf(a.xz[m / a.rps], -1024.0f, 1024.0f)));
            negz[i] = half2v{nz, nz};
        }
    }

    // ---- activation tile: global -> registers two k-steps ahead -> LDS, 16-byte loads
    // through a buffer resource whose range check returns zeros past the last row.  The
    // tile is stored as rows of 8 logical 16-byte chunks (8 k each), chunk c of row r at
    // slot c ^ ((r >> 1) & 7).
    //  half-precision copy: load q = 256 i + t is row q >> 3, chunk q & 7;
    //  codes: load q is row q >> 2, codes 16 (q & 3) .. + 15 = chunks 2 (q & 3), + 1.
    const bool perm4 = CODE_BITS == 4;
    const __amdgpu_buffer_rsrc_t ra =
        AF == kAConv ? __builtin_amdgcn_make_buffer_rsrc((void*)a.Xh, (short)0, (int)a.xh_bytes, kBufferFlags)
        : AF == kAF16 ? __builtin_amdgcn_make_buffer_rsrc((void*)(a.Xh + (int64_t)m0 * K + kb * BK), (short)0,
                                                          (rows * K - kb * BK) * 2, kBufferFlags)
                      : __builtin_amdgcn_make_buffer_rsrc((void*)(a.xc + (int64_t)m0 * K + kb * BK), (short)0,
                                                          rows * K - kb * BK, kBufferFlags);
    const uint32_t aoff0 = HALF ? (uint32_t)((t >> 3) * K * 2 + (((t & 7) ^ ((t >> 4) & 7)) << 4))
                                : (uint32_t)((t >> 2) * K + ((t & 3) << 4));
    // convolution: the padded pixel of each staging row (row (t >> 3) + 32 i) at tap (0, 0);
    // rows past the tile's last take an offset past the buffer (loads return zeros)
    int pix[AF == kAConv ? AQ : 1];
#pragma unroll
    for (int i = 0; i < (AF == kAConv ? AQ : 1); ++i) {
        pix[i] = -1;
        if (AF == kAConv) {
            const int r = (t >> 3) + 32 * i;
            if (r < rows) {
                const int m = m0 + r, x = m % a.W, yb = m / a.W, y = yb % a.H, b = yb / a.H;
                pix[i] = (b * (a.H + 2) + y) * (a.W + 2) + x;
            }
        }
    }
    struct AStage {
        uint4 v[AQ];
    };
    auto load_a = [&](AStage& S, int k) __attribute__((always_inline)) {
        int tapoff = 0, ci0 = 0;
        if (AF == kAConv) {  // k-step -> tap (ky, kx) and channel offset (C % 64 == 0)
            const int kk = (kb + k) * BK, tap = kk / a.C;
            ci0 = kk - tap * a.C;
            tapoff = (tap / 3) * (a.W + 2) + tap % 3;
        }
#pragma unroll
        for (int i = 0; i < AQ; ++i) {
            uint32_t off;
            if (AF == kAConv)
                off = pix[i] < 0 ? 0x7FFFFFF0u
                                 : (uint32_t)(((pix[i] + tapoff) * a.C + ci0) * 2) + (aoff0 - (uint32_t)((t >> 3) * K * 2));
            else
                off = HALF ? aoff0 + (uint32_t)(i * 64 * K + k * BK * 2) : aoff0 + (uint32_t)(i * 64 * K + k * BK);
            S.v[i] = (!AFULL && i * 256 + t >= BM * 4)
                         ? make_uint4(0u, 0u, 0u, 0u)
                         : __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(ra, (int)off, 0, 0));
        }
    };
    auto store_a = [&](const AStage& S, int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < AQ; ++i) {
            if (HALF) {
                lds[buf][i * 256 + t] = S.v[i];
            } else {
                const int q = i * 256 + t;
                if (AFULL || q < BM * 4) {
                    const int r = q >> 2, c = 2 * (q & 3), sw = (r >> 1) & 7;
                    lds[buf][r * 8 + (c ^ sw)] = decode_act8<AF>(S.v[i].x, S.v[i].y, perm4, negz[i]);
                    lds[buf][r * 8 + ((c + 1) ^ sw)] = decode_act8<AF>(S.v[i].z, S.v[i].w, perm4, negz[i]);
                }
            }
        }
    };

    // ---- weight records of the lane's channels (column l32 of the wave's TN 32-channel
    // blocks, half h): global -> registers one k-step ahead; past the last channel the
    // range check returns zeros (zero codes, zero table)
    const int nl = 32 * TN * wave + l32;
    const int chans = N - n0 < BN ? N - n0 : BN;
    const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(a.rec + ((int64_t)kb * N + n0) * 2 * P), (short)0, (int)(((int64_t)(K / BK - kb) * N - n0) * 2 * P * 16),
        kBufferFlags);
    const uint32_t rstep = (uint32_t)N * 2u * P * 16u;  // record bytes per k-step
    struct Rec {
        uint4 c[CW];
        Table tb;
    };
    struct WStage {
        Rec r[TN];
    };
    auto load_w = [&](WStage& W, int k) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = nl + 32 * j;
            const uint32_t off = col < chans ? (uint32_t)k * rstep + (uint32_t)((col * 2 + h) * P) * 16u : 0x7FFFFF00u;
            uint4 v[P];
#pragma unroll
            for (int q = 0; q < P; ++q)
                v[q] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rr, (int)(off + 16u * q), 0, 0));
#pragma unroll
            for (int q = 0; q < CW; ++q) W.r[j].c[q] = v[q];
            W.r[j].tb = Table{{v[CW].x, v[CW].y, v[CW].z, v[CW].w}, {v[CW + 1].x, v[CW + 1].y, v[CW + 1].z, v[CW + 1].w}};
        }
    };

    // per-channel parameters of the lane's TN channels: 8-bit code layout decoded
    // arithmetically, epilogue factor (loaded here, off the tail of the kernel)
    bool int8[TN];
    float cs[TN], csum[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int n = n0 + nl + 32 * j;
        const ColPrep cp = n < N ? a.cols[n] : ColPrep{CHAM_W_NFMT, 0, 0.0f, 0.0f};
        int8[j] = CODE_BITS == 8 && is_8bit(cp.fmt);
        cs[j] = cp.colscale;
        csum[j] = 0.0f;
        if (AF == kAInt8 && n < N)
            for (int q = 0; q < a.nkc; ++q) csum[j] += a.colsum[(int64_t)q * N + n];
    }
    auto decode = [&](const Rec& r, int j, int s) __attribute__((always_inline)) -> half8 {
        if (CODE_BITS == 4) {
            const uint32_t w = s == 0 ? r.c[0].x : s == 1 ? r.c[0].y : s == 2 ? r.c[0].z : r.c[0].w;
            return decode_nibbles(r.tb, w);
        } else {
            const uint4& cc = r.c[(s >> 1) & (CW - 1)];
            const uint32_t w0 = (s & 1) ? cc.z : cc.x, w1 = (s & 1) ? cc.w : cc.y;
            return int8[j] ? decode_bytes_int(r.tb, w0, w1) : decode_bytes_table(r.tb, w0, w1);
        }
    };

    // LDS chunk offset of the lane's activation operand in sub-step s (row l32 of block i
    // at + 256 i chunks)
    int aoff[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) aoff[s] = l32 * 8 + ((4 * h + s) ^ ((l32 >> 1) & 7));

    float16v acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    // ---- main loop.  Step k computes from LDS buffer k & 1.  At its start it stores the
    // activation tile of step k + 1 (loaded DA steps earlier) into the other buffer and
    // issues the loads of step k + 1 + DA (activations) and k + DW (weights) into register
    // rings of DA and DW + 1 stages.  Short steps (64-row tiles) take deeper rings so the
    // loads have more than one memory latency to arrive.  Half-width tiles keep 2-stage
    // rings, which fit three workgroups per CU (at most 168 registers): with a 4-stage ring
    // they fit two, which was 3-7 % faster than two workgroups with 2 stages, but three
    // workgroups with 2 stages beat both (the QKV layers at 1280 4 % faster, the step 1 %,
    // where the search shares the CUs).  Sub-steps 0-2 run with the
    // operand reads and weight decode one sub-step ahead; then one barrier makes the new
    // tile visible (and retires every read of this step's buffer), and the first operands
    // of step k + 1 are read and decoded behind the MFMAs of sub-step 3.  Step indices past
    // the end are clamped (harmless reloads); scheduling barriers keep the compiler from
    // sinking the reads next to their uses.  The loop is unrolled by a multiple of both
    // ring lengths and of the two LDS buffers, so every ring and buffer index is a constant.
    constexpr int DW = TM == 2 ? 3 : 1;
    constexpr int DA = TM == 2 ? 2 : 1;
    constexpr int U = (DW + 1) > 2 ? (DW + 1) : 2;
    static_assert(U % DA == 0 && U % 2 == 0, "the unrolled steps must repeat every ring and buffer index");
    const int klast = nsteps - 1;
    AStage R[DA];
    WStage W[DW + 1];
    half8 af[TM], an[TM], bf[TN], bn[TN];
#pragma unroll
    for (int d = 0; d < DW; ++d) load_w(W[d], d < klast ? d : klast);
    load_a(R[0], 0);
    store_a(R[0], 0);
#pragma unroll
    for (int d = 1; d <= DA; ++d) load_a(R[d % DA], d < klast ? d : klast);
    lds_barrier();
#pragma unroll
    for (int i = 0; i < TM; ++i) af[i] = __builtin_bit_cast(half8, lds[0][i * 256 + aoff[0]]);
#pragma unroll
    for (int j = 0; j < TN; ++j) bf[j] = decode(W[0].r[j], j, 0);

    auto mfmas = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[i], bf[j], acc[i][j], 0, 0, 0);
    };
    auto step = [&](int k, int buf, const WStage& Wc, const WStage& Wn, WStage& Wl, AStage& Ra)
                    __attribute__((always_inline)) {
        if (k + 1 < nsteps) store_a(Ra, buf ^ 1);
        load_a(Ra, k + 1 + DA < klast ? k + 1 + DA : klast);
        load_w(Wl, k + DW < klast ? k + DW : klast);
        const uint4* L = lds[buf];
#pragma unroll
        for (int s = 0; s < 3; ++s) {
#pragma unroll
            for (int i = 0; i < TM; ++i) an[i] = __builtin_bit_cast(half8, L[i * 256 + aoff[s + 1]]);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int j = 0; j < TN; ++j) bn[j] = decode(Wc.r[j], j, s + 1);
            mfmas();
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < TM; ++i) af[i] = an[i];
#pragma unroll
            for (int j = 0; j < TN; ++j) bf[j] = bn[j];
        }
        lds_barrier();
        const uint4* Ln = lds[buf ^ 1];
#pragma unroll
        for (int i = 0; i < TM; ++i) an[i] = __builtin_bit_cast(half8, Ln[i * 256 + aoff[0]]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < TN; ++j) bn[j] = decode(Wn.r[j], j, 0);
        mfmas();
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < TM; ++i) af[i] = an[i];
#pragma unroll
        for (int j = 0; j < TN; ++j) bf[j] = bn[j];
    };
    int k = 0;
    for (; k + U <= nsteps; k += U) {
#pragma unroll
        for (int u = 0; u < U; ++u)
            step(k + u, u & 1, W[u % (DW + 1)], W[(u + 1) % (DW + 1)], W[(u + DW) % (DW + 1)], R[(u + 1) % DA]);
    }
#pragma unroll
    for (int u = 0; u + 1 < U; ++u)
        if (k + u < nsteps)
            step(k + u, u & 1, W[u % (DW + 1)], W[(u + 1) % (DW + 1)], W[(u + DW) % (DW + 1)], R[(u + 1) % DA]);

    // ---- epilogue: 32x32 block, lane holds column l32, rows 8*(r/4) + 4*h + r%4; the
    // lane's 16 row scales of block i are 4 aligned float4 in LDS.  Stores go through a
    // buffer resource over the tile's rows of the output: the lane's offset is one VGPR per
    // block, each row's offset a wave-uniform SGPR, and the range check drops the rows past
    // the last of a ragged tile (the lane skips columns past the last).  The output is not
    // read again here, so it is stored non-temporally (the L2 stays with the operand tiles
    // other workgroups still read); k-split partials, which the reduction reads back at
    // once, take ordinary stores.
    float* const out = a.splits > 1 ? a.part + (int64_t)split * a.M * N : a.Y;
    const __amdgpu_buffer_rsrc_t ro =
        __builtin_amdgcn_make_buffer_rsrc((void*)(out + (int64_t)m0 * N), (short)0, rows * N * 4, kBufferFlags);
    const bool partial = a.splits > 1;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        float rs[16], rc[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 v = *reinterpret_cast<const float4*>(&Rs[32 * i + 8 * q + 4 * h]);
            rs[4 * q] = v.x; rs[4 * q + 1] = v.y; rs[4 * q + 2] = v.z; rs[4 * q + 3] = v.w;
            if (AF == kAInt8) {
                const float4 c = *reinterpret_cast<const float4*>(&Rc[32 * i + 8 * q + 4 * h]);
                rc[4 * q] = c.x; rc[4 * q + 1] = c.y; rc[4 * q + 2] = c.z; rc[4 * q + 3] = c.w;
            }
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int n = n0 + nl + 32 * j;
            if (n < N) {
                const int voff = ((32 * i + 4 * h) * N + n) * 4;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    // (acc rs) cs, plus the zero-point correction of INT8-asym activations
                    float v = (acc[i][j][r] * rs[r]) * cs[j];
                    if (AF == kAInt8) v = v + rc[r] * csum[j];
                    const uint32_t bits = __builtin_bit_cast(uint32_t, v);
                    const int soff = (8 * (r >> 2) + (r & 3)) * N * 4;
                    if (partial) __builtin_amdgcn_raw_buffer_store_b32(bits, ro, voff, soff, 0);
                    else __builtin_amdgcn_raw_buffer_store_b32(bits, ro, voff, soff, kStoreNonTemporal);
                }
            }
        }
    }
}

// Sum of the k-split partial outputs in split order (the result does not depend on the
// order in which workgroups ran); 4 outputs per thread when M N is a multiple of 4.
constexpr int kMaxSplits = 8;
typedef float f32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void reduce_kernel(const float* __restrict__ part, float* __restrict__ Y,
                                                     int64_t MN, int splits) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    if ((MN & 3) == 0) {
        const float4* p4 = reinterpret_cast<const float4*>(part);
        float4* y4 = reinterpret_cast<float4*>(Y);
        const int64_t n4 = MN >> 2;
        for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
            // every split's load issued before the first sum (splits <= kMaxSplits)
            float4 v[kMaxSplits];
#pragma unroll
            for (int sp = 0; sp < kMaxSplits; ++sp)
                v[sp] = sp < splits ? p4[(int64_t)sp * n4 + i] : make_float4(0.f, 0.f, 0.f, 0.f);
            float4 acc = v[0];
#pragma unroll
            for (int sp = 1; sp < kMaxSplits; ++sp) {
                if (sp < splits) { acc.x += v[sp].x; acc.y += v[sp].y; acc.z += v[sp].z; acc.w += v[sp].w; }
            }
            const f32x4 o = {acc.x, acc.y, acc.z, acc.w};
            __builtin_nontemporal_store(o, reinterpret_cast<f32x4*>(&y4[i]));
        }
    } else {
        for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < MN; i += stride) {
            float acc = part[i];
            for (int sp = 1; sp < splits; ++sp) acc += part[(int64_t)sp * MN + i];
            Y[i] = acc;
        }
    }
}

// ---- launch plan.  A launch covers rows [row0, row1) with one tile shape.  The plan is
// either one launch, optionally split along k into partial outputs that reduce_kernel
// sums (for layers with too few output tiles to fill the CUs), or two launches of
// different tile shapes: one for whole rounds of workgroups, the other for the rows left,
// so the last round does not leave most CUs idle.
// CU count of the current device, queried once per device (every thread that races to
// fill the cache stores the same value, so relaxed atomics suffice)
int cu_count() {
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int n = cached[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
        cached[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

// Modeled time (us) of a launch of one tile shape, fitted to measurements on MI355X: one
// fixed cost (prologue, output write) per launch -- the workgroups of later rounds start
// while earlier ones finish -- plus the k-steps of the rounds of workgroups, each at the
// k-step time of as many workgroups per CU as the round puts there.  Tiles 128 high fit two
// workgroups on a CU, the half-width tile (128 x 128) three.
struct TileCost {
    int bm, tn, occ;                   // tile height, 32-channel blocks per wavefront, workgroups per CU
    double step1, step2, step3, fixed;  // us: k-step with 1, 2, 3 workgroups on the CU; per launch
};
constexpr int kNumTiles = 4;
constexpr TileCost kTileCosts[kNumTiles] = {{256, 2, 1, 2.13, 2.13, 2.13, 8.0},
                                            {128, 2, 2, 1.21, 1.89, 1.89, 9.0},
                                            {128, 1, 3, 0.715, 1.26, 1.64, 6.0},
                                            {64, 2, 1, 0.82, 0.82, 0.82, 6.2}};

double step_cost(const TileCost& c, int64_t per_cu) {
    return per_cu <= 1 ? c.step1 : per_cu == 2 ? c.step2 : c.step3;
}

double launch_cost(int64_t wgs, int nsteps, const TileCost& c, int P) {
    if (wgs <= 0) return 0.0;
    const int64_t slots = (int64_t)c.occ * P;
    const int64_t full = wgs / slots, rem = wgs % slots;
    return c.fixed + (double)full * nsteps * step_cost(c, c.occ) +
           (rem == 0 ? 0.0 : nsteps * step_cost(c, (rem + P - 1) / P));
}

struct Launch {
    int row0, row1, bm, tn;
};
struct Plan {
    int n;       // launches
    int splits;  // k-splits of a single launch (1: none)
    Launch l[2];
};
// k-split: the GEMM writes one binary32 partial output per split (≈ 5 TB/s, on top of its
// k-steps), and one extra launch reads them back and writes the output (measured ≈ 7 TB/s:
// the partials come back from the last-level cache in part)
double reduce_cost(int64_t M, int64_t N, int splits) {
    return splits > 1 ? 2.0 + (double)(splits + 1) * (double)(M * N * 4) / 7.0e6 +
                            (double)splits * (double)(M * N * 4) / 5.0e6
                      : 0.0;
}

int col_tiles(int N, int tn) { return (N + tile_width(tn) - 1) / tile_width(tn); }

Plan plan_gemm(int M, int N, int K, int code_bits) {
    const int P = cu_count();
    const int nsteps = K / BK;
    TileCost costs[kNumTiles];
    for (int b = 0; b < kNumTiles; ++b) costs[b] = kTileCosts[b];
    if (code_bits != 4) {  // the full-width 128-high tile with 8-bit codes: one per CU
        costs[1].occ = 1;
        costs[1].step2 = costs[1].step3 = costs[1].step1;
    }
    // half-width tiles: with 4-bit codes wherever the model prefers them; with 8-bit codes
    // (the costs are fitted on 4-bit codes) only where the full-width tiles leave CUs idle
    const bool half_ok = code_bits == 4 || (int64_t)((M + 127) / 128) * col_tiles(N, 2) < P;
    // 64 x 128 tiles (three per CU), outside the model: for short 4-bit layers whose
    // 128 x 128 tiles fill at most half the CUs and whose 64 x 128 tiles fill at least half,
    // they beat every plan the model offers (1024 x 1280 x 1280: 12.5 us against 18.3 us for
    // 3 k-splits of 128 x 128 tiles); on the shapes measured outside that range they lost
    const int64_t t128 = (int64_t)((M + 127) / 128) * col_tiles(N, 1), t64 = (int64_t)((M + 63) / 64) * col_tiles(N, 1);
    if (code_bits == 4 && nsteps <= 20 && 2 * t128 <= P && 2 * t64 >= P)
        return Plan{1, 1, {Launch{0, M, 64, 1}, Launch{0, 0, 0, 0}}};
    double best = 1e300;
    Plan plan{1, 1, {Launch{0, M, 64, 2}, Launch{0, 0, 0, 0}}};
    for (int b = 0; b < kNumTiles; ++b) {
        if (costs[b].tn == 1 && !half_ok) continue;
        const int tn = col_tiles(N, costs[b].tn);
        for (int sp = 1; sp <= kMaxSplits && sp <= nsteps; ++sp) {
            const int kchunk = (nsteps + sp - 1) / sp;
            if (sp > 1 && (sp - 1) * kchunk >= nsteps) continue;  // an empty split
            const int64_t tiles = (int64_t)((M + costs[b].bm - 1) / costs[b].bm) * tn;
            const double c = launch_cost(tiles * sp, kchunk, costs[b], P) + reduce_cost(M, N, sp);
            if (c < best) { best = c; plan = Plan{1, sp, {Launch{0, M, costs[b].bm, costs[b].tn}, Launch{0, 0, 0, 0}}}; }
        }
    }
    // one tile shape for whole rounds of full tile rows, another for the rows left
    for (int b = 0; b < kNumTiles; ++b) {
        if (costs[b].tn == 1 && !half_ok) continue;
        const TileCost& c1 = costs[b];
        const int tn1 = col_tiles(N, c1.tn);
        const int rows_per_round = (c1.occ * P / tn1) * c1.bm;
        if (rows_per_round <= 0) continue;
        const int r1 = (M / rows_per_round) * rows_per_round;
        if (r1 <= 0 || r1 >= M) continue;
        for (int b2 = 0; b2 < kNumTiles; ++b2) {
            if (b2 == b || (costs[b2].tn == 1 && !half_ok)) continue;
            const TileCost& c2 = costs[b2];
            const double c = launch_cost((int64_t)(r1 / c1.bm) * tn1, nsteps, c1, P) +
                             launch_cost((int64_t)((M - r1 + c2.bm - 1) / c2.bm) * col_tiles(N, c2.tn), nsteps, c2, P);
            if (c < best) { best = c; plan = Plan{2, 1, {Launch{0, r1, c1.bm, c1.tn}, Launch{r1, M, c2.bm, c2.tn}}}; }
        }
    }
    return plan;
}

// partial-output bytes of the plan for these sizes (the larger of the two code widths)
size_t split_bytes(int64_t M, int64_t N, int64_t K) {
    size_t b = 0;
    for (int bits = 4; bits <= 8; bits += 4) {
        const Plan p = plan_gemm((int)M, (int)N, (int)K, bits);
        if (p.splits > 1) b = std::max(b, (size_t)p.splits * (size_t)M * (size_t)N * 4);
    }
    return b;
}

template <int CODE_BITS, int AF>
void launch_gemm_af(const GemmArgs& a, const Launch& l, hipStream_t s) {
    const unsigned grid = (unsigned)(((l.row1 - l.row0 + l.bm - 1) / l.bm) * a.tn * a.splits);
    if (l.bm == 256) hipLaunchKernelGGL((gemm_kernel<CODE_BITS, 8, AF, 2>), dim3(grid), dim3(kThreads), 0, s, a);
    else if (l.bm == 128 && l.tn == 1)
        hipLaunchKernelGGL((gemm_kernel<CODE_BITS, 4, AF, 1>), dim3(grid), dim3(kThreads), 0, s, a);
    else if (l.bm == 128) hipLaunchKernelGGL((gemm_kernel<CODE_BITS, 4, AF, 2>), dim3(grid), dim3(kThreads), 0, s, a);
    else if (l.tn == 1) hipLaunchKernelGGL((gemm_kernel<CODE_BITS, 2, AF, 1>), dim3(grid), dim3(kThreads), 0, s, a);
    else hipLaunchKernelGGL((gemm_kernel<CODE_BITS, 2, AF, 2>), dim3(grid), dim3(kThreads), 0, s, a);
}

// Tile rows per group of the XCD-aware order, or 0 for row-major order.  The XCD-aware
// order is taken where a workgroup runs at least 24 k-steps: there one tile's operand slabs
// are large enough that the row-major order's share of an XCD (most tile rows, several
// columns) overflows its L2; measured on the sweep stack's FF-out layers, 3-5 % faster,
// while the shorter layers ran 2-4 % slower in it.  An XCD's block of tiles (T of them,
// about r rows by T / r columns) reads r activation row tiles and T / r weight column
// tiles, so r = sqrt(T x column-tile bytes / row-tile bytes) reads the least; the divisor
// of the tile rows nearest to it (in ratio) keeps the groups whole.
int group_rows(int mt, int tn, int splits, int kchunk, int bm, int bn, bool half_act, int code_bits) {
    if (kchunk < 24) return 0;
    const double T = std::ceil((double)mt * tn * splits / 8.0);
    const double row_bytes = (double)bm * (half_act ? 2.0 : 1.0);
    const double col_bytes = (double)bn * (code_bits == 4 ? 1.5 : 2.0);
    const double r = std::sqrt(T * col_bytes / row_bytes);
    int best = 1;
    for (int d = 1; d <= mt; ++d)
        if (mt % d == 0 && std::fabs(std::log((double)d / r)) < std::fabs(std::log((double)best / r))) best = d;
    return best;
}

template <int CODE_BITS>
void launch_gemm(GemmArgs a, const Launch& l, int af, hipStream_t s) {
    a.row0 = l.row0;
    a.row1 = l.row1;
    a.tn = col_tiles(a.N, l.tn);
    a.gm = group_rows((l.row1 - l.row0 + l.bm - 1) / l.bm, a.tn, a.splits, a.kchunk, l.bm, tile_width(l.tn),
                      af == kAF16 || af == kAConv, CODE_BITS);
    switch (af) {
    case kAInt8: launch_gemm_af<CODE_BITS, kAInt8>(a, l, s); break;
    case kAE4M3: launch_gemm_af<CODE_BITS, kAE4M3>(a, l, s); break;
    case kAE5M2: launch_gemm_af<CODE_BITS, kAE5M2>(a, l, s); break;
    case kAConv: launch_gemm_af<CODE_BITS, kAConv>(a, l, s); break;
    default: launch_gemm_af<CODE_BITS, kAF16>(a, l, s); break;
    }
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }
// weight record slots (48 or 64 bytes used) per (k-step, channel, half)
int64_t record_bytes(int64_t N, int64_t K) { return N * (K / BK) * 2 * 64; }

}  // namespace
}  // namespace cham

using namespace cham;

// Chunks of k-steps the record pre-pass splits a weight into: about one workgroup per CU per
// layer (all of a batch resident at once), at least 4 k-steps each.
static void rec_chunks(int64_t N, int64_t K, int* nkc, int* rchunk) {
    const int nblk = (int)((N + kRecChannels - 1) / kRecChannels), nst = (int)(K / BK);
    const int n = std::max(1, std::min((256 + nblk - 1) / nblk, (nst + 3) / 4));
    *rchunk = (nst + n - 1) / n;
    *nkc = (nst + *rchunk - 1) / *rchunk;
}

// The packed layout: ColPrep[N], the column-sum partials [k-chunks][N], then the records.
extern "C" size_t cham_packed_bytes(int64_t N, int64_t K) {
    if (N < 1 || K < 64) return 0;
    int nkc, rchunk;
    rec_chunks(N, K, &nkc, &rchunk);
    return align256((size_t)N * sizeof(ColPrep)) + align256((size_t)nkc * (size_t)N * 4) + (size_t)record_bytes(N, K);
}

struct Layout {
    ColPrep* cols;
    float* colsum;
    uint4* rec;
};
static Layout layout_at(void* p, int64_t N, int64_t K) {
    int nkc, rchunk;
    rec_chunks(N, K, &nkc, &rchunk);
    char* c = (char*)p;
    Layout l;
    l.cols = (ColPrep*)c;
    c += align256((size_t)N * sizeof(ColPrep));
    l.colsum = (float*)c;
    c += align256((size_t)nkc * (size_t)N * 4);
    l.rec = (uint4*)c;
    return l;
}

// One searched weight as the record pre-pass and the GEMM see it: per-channel formats
// (cham_wq) or group-scaled weights of one format (cham_gwq).
struct WView {
    int64_t N, K;
    uint32_t mask;
    int code_bits;
    const uint8_t* fmt;
    const float* scale;
    const float* zero;
    const float* nf4;
    const uint8_t* e8;
    const uint8_t* codes;
    void* packed;
    const int32_t* gsel;
    const float* gscale;
    const float* gzero;
};

static WView view_of(const cham_wq* wq) {
    return WView{wq->N, wq->K, wq->palette_mask, wq->code_bits, wq->fmt, wq->scale, wq->zero, wq->nf4_absmax,
                 wq->e8m0, wq->codes, wq->packed, nullptr, nullptr, nullptr};
}

static WView view_of(const cham_gwq* gq) {
    return WView{gq->N, gq->K, gq->palette_mask, gq->code_bits, gq->fmt, nullptr, nullptr, nullptr,
                 gq->e8m0, gq->codes, gq->packed, gq->choice, gq->gscale, gq->gzero};
}

// Record pre-pass arguments of one searched weight writing into the layout L (device),
// and the workgroups it takes.
static RecArgs record_args(const WView& v, const Layout& L, int* wgs) {
    const uint32_t mask = v.mask;
    const int N = (int)v.N, K = (int)v.K;
    const bool nf4 = (mask >> CHAM_W_NF4) & 1u;
    const bool wmx = (mask & ((1u << CHAM_W_MXINT8) | (1u << CHAM_W_MXINT4) | (1u << CHAM_W_MXFP4))) != 0u;
    const int nblk = (N + kRecChannels - 1) / kRecChannels;
    int nkc, rchunk;
    rec_chunks(N, K, &nkc, &rchunk);
    *wgs = nblk * nkc;
    // block metadata only of the enabled formats (the pre-pass reads it ahead of the format)
    return RecArgs{v.fmt, v.scale, v.zero, nf4 && !v.gsel ? v.nf4 : nullptr, wmx ? v.e8 : nullptr, v.codes,
                   mask, N, K, v.code_bits, rchunk, L.cols, L.colsum, L.rec, v.gsel, v.gscale, v.gzero};
}

static void launch_records(const WView& v, const Layout& L, hipStream_t s) {
    RecBatch B;
    B.nl = 1;
    B.ng = 0;
    int wgs = 0;
    B.r[0] = record_args(v, L, &wgs);
    B.wg_end[0] = wgs;
    hipLaunchKernelGGL(record_kernel, dim3((unsigned)wgs), dim3(256), 0, s, B);
}

// Writes the packed layout of n searched weights (the arguments checked and code_bits set),
// and with `group` also groups the channels of those that ask for perm / group_off; one
// launch per kRecBatchMax weights.
static int pack_weights(const cham_wq* const* wqs, int n, bool group, hipStream_t s) {
    for (int i0 = 0; i0 < n; i0 += kRecBatchMax) {
        RecBatch B;
        B.nl = std::min(kRecBatchMax, n - i0);
        B.ng = 0;
        int total = 0;
        for (int j = 0; j < B.nl; ++j) {
            const cham_wq* wq = wqs[i0 + j];
            int wgs = 0;
            B.r[j] = record_args(view_of(wq), layout_at(wq->packed, wq->N, wq->K), &wgs);
            total += wgs;
            B.wg_end[j] = total;
            if (group && (wq->perm || wq->group_off))
                B.g[B.ng++] = GroupArgs{wq->fmt, (int)wq->N, wq->perm, wq->group_off};
        }
        hipLaunchKernelGGL(record_kernel, dim3((unsigned)(total + B.ng)), dim3(256), 0, s, B);
        CHAM_CHECK_LAUNCH();
    }
    return CHAM_OK;
}

// The search entry points' packing step (they have checked the arguments and set code_bits).
int cham_pack_weights(const cham_wq* const* wqs, int n, hipStream_t s) { return pack_weights(wqs, n, true, s); }

extern "C" int cham_pack_weights_batch(const cham_wq* wq, int32_t n, void* stream) {
    if (!wq || n < 1) return CHAM_EINVAL;
    std::vector<const cham_wq*> p((size_t)n);
    for (int i = 0; i < n; ++i) {
        const cham_wq& w = wq[i];
        if (!w.fmt || !w.codes || !w.scale || !w.zero || !w.packed || w.N < 1) return CHAM_EINVAL;
        if ((uintptr_t)w.packed & 255u) return CHAM_EINVAL;
        const uint32_t mask = w.palette_mask;
        if (mask == 0u || (mask >> CHAM_W_NFMT) != 0u) return CHAM_EFORMAT;
        if (w.code_bits != ((mask & 0x7u) ? 8 : 4)) return CHAM_EINVAL;
        if (w.K < 64 || w.K % 64 != 0 || w.K > (1 << 20)) return CHAM_ESHAPE;
        if (((mask >> CHAM_W_NF4) & 1u) && !w.nf4_absmax) return CHAM_EINVAL;
        if ((mask & ((1u << CHAM_W_MXINT8) | (1u << CHAM_W_MXINT4) | (1u << CHAM_W_MXFP4))) && !w.e8m0)
            return CHAM_EINVAL;
        if (w.N * (w.K / 64) * 128 > (int64_t)INT32_MAX) return CHAM_EINVAL;
        p[(size_t)i] = &w;
    }
    return pack_weights(p.data(), n, false, (hipStream_t)stream);
}

// The packed layout of a group-scaled weight (called by the grouped search after its
// launches, which have checked the arguments).
int cham_pack_grouped(const cham_gwq* gq, hipStream_t s) {
    launch_records(view_of(gq), layout_at(gq->packed, gq->N, gq->K), s);
    CHAM_CHECK_LAUNCH();
    return CHAM_OK;
}

size_t cham_linear_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    return align256((size_t)M * (size_t)K * 2) + align256((size_t)M * 4) + align256(cham_packed_bytes(N, K)) +
           split_bytes(M, N, K);
}

extern "C" int cham_linear_plan(int64_t M, int64_t N, int64_t K, int32_t code_bits, int32_t* out, int32_t out_len) {
    if (!out || out_len < 10 || M < 1 || N < 1 || K < 1 || M > INT32_MAX || N > INT32_MAX || K > INT32_MAX ||
        (code_bits != 4 && code_bits != 8))
        return CHAM_EINVAL;
    const Plan p = plan_gemm((int)M, (int)N, (int)K, code_bits);
    for (int i = 0; i < 10; ++i) out[i] = 0;
    out[0] = p.n;
    out[1] = p.splits;
    for (int i = 0; i < p.n; ++i) {
        out[2 + 4 * i] = p.l[i].row0;
        out[3 + 4 * i] = p.l[i].row1;
        out[4 + 4 * i] = p.l[i].bm;
        out[5 + 4 * i] = tile_width(p.l[i].tn);
    }
    return CHAM_OK;
}

// 3x3 convolution geometry (images B x H x W, channels last)
struct ConvSpec {
    int B, H, W;
};

// Workspace of the convolution: the padded half-precision copy, the row scales, the block
// exponent maximum, the weights' layout (no packed layout given) and the k-split partials.
static size_t conv_workspace(int64_t B, int64_t H, int64_t W, int64_t C, int64_t Co) {
    const int64_t M = B * H * W;
    return align256((size_t)(B * (H + 2) * (W + 2) * C) * 2) + align256((size_t)M * 4) + 256 +
           align256(cham_packed_bytes(Co, 9 * C)) + split_bytes(M, Co, 9 * C);
}

// What one call uses of its workspace, in this order: the half-precision activation copy
// and row scales (MX activations and the convolution only), the block exponent maximum
// (convolution), the weight layout (when no packed layout comes with the weight) and the
// k-split partials (when the plan splits).
struct WsLayout {
    size_t xh, rs, emax, rec, part, total;
};
static WsLayout ws_layout(bool half_copy, size_t xh_bytes, bool conv, bool packed, int64_t M, int64_t N, int64_t K,
                          int splits) {
    WsLayout l;
    l.xh = 0;
    l.rs = l.xh + (half_copy ? align256(xh_bytes) : 0);
    l.emax = l.rs + (half_copy ? align256((size_t)M * 4) : 0);
    l.rec = l.emax + (conv ? 256 : 0);
    l.part = l.rec + (packed ? 0 : align256(cham_packed_bytes(N, K)));
    l.total = l.part + (splits > 1 ? (size_t)splits * (size_t)M * (size_t)N * 4 : 0);
    return l;
}

// ws_need != NULL: only report the workspace bytes these operands need (Y and ws unused).
static int mixed_linear_impl(const cham_aq* xq, const WView& v, float* Y, void* ws, size_t ws_bytes, void* stream,
                             const ConvSpec* cv = nullptr, size_t* ws_need = nullptr) {
    const WView* wq = &v;
    if (!xq || (!Y && !ws_need) || !xq->codes || !xq->scale || !xq->zero) return CHAM_EINVAL;
    if (!wq->fmt || !wq->codes) return CHAM_EINVAL;
    if (!wq->gsel && (!wq->scale || !wq->zero)) return CHAM_EINVAL;
    if (wq->gsel && (!wq->gscale || !wq->gzero)) return CHAM_EINVAL;
    if (xq->M < 1 || wq->N < 1 || xq->K < 1 || (cv ? 9 * xq->K : xq->K) != wq->K) return CHAM_EINVAL;
    if (cv) {
        if (cv->B < 1 || cv->H < 1 || cv->W < 1 || (int64_t)cv->B * cv->H * cv->W != xq->M) return CHAM_EINVAL;
        if (xq->K % 64 != 0) return CHAM_ESHAPE;  // a k-step never straddles two taps
        const int64_t xb = (int64_t)cv->B * (cv->H + 2) * (cv->W + 2) * xq->K * 2;
        if (xb > (int64_t)INT32_MAX - 4096) return CHAM_ESHAPE;  // 32-bit buffer offsets
        if (xq->nsamples != 1 && xq->nsamples != cv->B) return CHAM_EINVAL;  // a sample is whole images
    }
    if (xq->fmt < 0 || xq->fmt >= CHAM_A_NFMT) return CHAM_EFORMAT;
    if (xq->nsamples < 1 || xq->M % xq->nsamples != 0) return CHAM_EINVAL;
    const uint32_t mask = wq->mask;
    if (mask == 0u || (mask >> CHAM_W_NFMT) != 0u) return CHAM_EFORMAT;
    const int code_bits = (mask & 0x7u) ? 8 : 4;
    if (wq->code_bits != code_bits) return CHAM_EFORMAT;
    if (wq->gsel && code_bits != 4) return CHAM_EFORMAT;  // the 8-bit group-scaled decode is not built
    if (wq->K % 64 != 0) return CHAM_ESHAPE;
    // 32-bit buffer offsets: a 256-row activation tile, a 256-row output tile and the
    // weight records stay below 2^31 bytes
    if (xq->M > INT32_MAX / 2 || wq->N > INT32_MAX / 1024 || wq->K > (1 << 20) ||
        record_bytes(wq->N, wq->K) > (int64_t)INT32_MAX)
        return CHAM_ESHAPE;
    const bool nf4 = (mask >> CHAM_W_NF4) & 1u;
    const bool wmx = (mask & ((1u << CHAM_W_MXINT8) | (1u << CHAM_W_MXINT4) | (1u << CHAM_W_MXFP4))) != 0u;
    if ((nf4 && !wq->gsel && !wq->nf4) || (wmx && !wq->e8)) return CHAM_EINVAL;
    const bool amx = xq->fmt == CHAM_A_MXFP8_E4M3 || xq->fmt == CHAM_A_MXINT8;
    if (amx && !xq->e8m0) return CHAM_EINVAL;
    if (((uintptr_t)xq->codes & 15u) || ((uintptr_t)wq->codes & 15u) || ((uintptr_t)wq->packed & 255u))
        return CHAM_EINVAL;
    const int M = (int)xq->M, N = (int)wq->N, K = (int)wq->K;
    const Plan plan = plan_gemm(M, N, K, code_bits);
    const int kchunk = (K / BK + plan.splits - 1) / plan.splits;
    // every split holds at least one k-step (the operand ranges of the kernel rely on it)
    if (plan.splits < 1 || (plan.splits - 1) * kchunk >= K / BK) return CHAM_ESHAPE;
    const size_t xh_bytes = cv ? (size_t)cv->B * (cv->H + 2) * (cv->W + 2) * xq->K * 2 : (size_t)M * (size_t)K * 2;
    const WsLayout wl = ws_layout(amx || cv, xh_bytes, cv != nullptr, wq->packed != nullptr, M, N, K, plan.splits);
    if (ws_need) {  // the size query: nothing is checked against a buffer, nothing launched
        *ws_need = wl.total;
        return CHAM_OK;
    }
    if (wl.total > 0 && (!ws || ws_bytes < wl.total || ((uintptr_t)ws & 255u))) return CHAM_EWORKSPACE;
    hipStream_t s = (hipStream_t)stream;

    char* w = (char*)ws;
    _Float16* Xh = (_Float16*)(w + wl.xh);
    float* rowscale = (float*)(w + wl.rs);
    int* emax = (int*)(w + wl.emax);
    // the search's packed layout replaces the pre-pass
    const Layout lay = layout_at(wq->packed ? wq->packed : (void*)(w + wl.rec), N, K);
    float* part = (float*)(w + wl.part);

    if (cv) {
        if (amx) {
            hipLaunchKernelGGL(emax_kernel, dim3(1), dim3(1024), 0, s, xq->e8m0, xq->M * (xq->K / 32), emax);
            CHAM_CHECK_LAUNCH();
        }
        PrepConvArgs p{xq->codes, xq->e8m0, xq->fmt, cv->B, cv->H, cv->W, (int)xq->K, code_bits == 4, xq->scale,
                       xq->zero, (int)(xq->M / xq->nsamples), emax, Xh, rowscale};
        hipLaunchKernelGGL(prep_conv_kernel, dim3((unsigned)(cv->B * (cv->H + 2) * (cv->W + 2))), dim3(256), 0, s, p);
        CHAM_CHECK_LAUNCH();
    } else if (amx) {
        PrepArgs p{xq->codes, xq->e8m0, xq->fmt, M, K, code_bits == 4, Xh, rowscale};
        hipLaunchKernelGGL(prep_kernel, dim3((unsigned)M), dim3(256), 0, s, p);
        CHAM_CHECK_LAUNCH();
    }

    if (!wq->packed) launch_records(v, lay, s);
    CHAM_CHECK_LAUNCH();

    GemmArgs a;
    a.Xh = Xh;
    a.rowscale = rowscale;
    a.xc = xq->codes;
    a.xs = xq->scale;
    a.xz = xq->zero;
    a.rps = M / xq->nsamples;
    a.cols = lay.cols;
    a.colsum = lay.colsum;
    {
        int rchunk;
        rec_chunks(N, K, &a.nkc, &rchunk);
    }
    a.rec = lay.rec;
    a.Y = Y;
    a.M = M;
    a.N = N;
    a.K = K;
    a.row0 = 0;
    a.row1 = M;
    a.part = part;
    a.H = cv ? cv->H : 0;
    a.W = cv ? cv->W : 0;
    a.C = cv ? (int)xq->K : 0;
    a.xh_bytes = (uint32_t)xh_bytes;
    const int af = cv ? kAConv
                 : amx ? kAF16
                       : (xq->fmt == CHAM_A_INT8_ASYM ? kAInt8 : (xq->fmt == CHAM_A_FP8_E4M3 ? kAE4M3 : kAE5M2));
    a.splits = plan.splits;
    a.kchunk = kchunk;
    for (int i = 0; i < plan.n; ++i) {
        if (code_bits == 4) launch_gemm<4>(a, plan.l[i], af, s);
        else launch_gemm<8>(a, plan.l[i], af, s);
        CHAM_CHECK_LAUNCH();
    }
    if (plan.splits > 1) {
        const int64_t MN = (int64_t)M * N;
        const int64_t per = (MN & 3) == 0 ? MN / 4 : MN;
        const unsigned grid = (unsigned)std::min<int64_t>((per + 255) / 256, 4096);
        hipLaunchKernelGGL(reduce_kernel, dim3(grid), dim3(256), 0, s, part, Y, MN, plan.splits);
        CHAM_CHECK_LAUNCH();
    }
    return CHAM_OK;
}

extern "C" int cham_mixed_linear(const cham_aq* xq, const cham_wq* wq, float* Y, void* ws, size_t ws_bytes,
                                 void* stream) {
    if (!wq) return CHAM_EINVAL;
    return mixed_linear_impl(xq, view_of(wq), Y, ws, ws_bytes, stream);
}

extern "C" int cham_mixed_linear_workspace_query(const cham_aq* xq, const cham_wq* wq, size_t* bytes) {
    if (!wq || !bytes) return CHAM_EINVAL;
    return mixed_linear_impl(xq, view_of(wq), nullptr, nullptr, 0, nullptr, nullptr, bytes);
}

extern "C" int cham_mixed_linear_grouped_workspace_query(const cham_aq* xq, const cham_gwq* gq, size_t* bytes) {
    if (!gq || !gq->choice || !bytes) return CHAM_EINVAL;
    return mixed_linear_impl(xq, view_of(gq), nullptr, nullptr, 0, nullptr, nullptr, bytes);
}

extern "C" int cham_mixed_linear_grouped(const cham_aq* xq, const cham_gwq* gq, float* Y, void* ws, size_t ws_bytes,
                                         void* stream) {
    if (!gq || !gq->choice) return CHAM_EINVAL;
    return mixed_linear_impl(xq, view_of(gq), Y, ws, ws_bytes, stream);
}

extern "C" int cham_conv3x3_mixed(const cham_aq* xq, int32_t B, int32_t H, int32_t W, const cham_wq* wq, float* Y,
                                  void* ws, size_t ws_bytes, void* stream) {
    if (!wq) return CHAM_EINVAL;
    const ConvSpec cv{B, H, W};
    return mixed_linear_impl(xq, view_of(wq), Y, ws, ws_bytes, stream, &cv);
}

extern "C" size_t cham_conv3x3_workspace_bytes(int64_t B, int64_t H, int64_t W, int64_t C, int64_t Co) {
    if (B < 1 || H < 1 || W < 1 || C < 64 || Co < 1) return 0;
    return conv_workspace(B, H, W, C, Co);
}

