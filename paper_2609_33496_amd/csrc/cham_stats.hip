// Calibration statistics (Sec. 4.4; App. A.7, Alg. 1 first loop) and the LUT build
// (Sec. 4.3 routing, Sec. 3.1 Eq. snr, App. A.3 Eq. kurt, App. A.7 ScaleZP).
//
// Accumulation is HBM-bound: one pass over X with float4 loads, binary64 power sums and
// binary32 min/max per thread, a workgroup reduction, and per-workgroup partials in the
// workspace.  A one-workgroup finalize kernel adds the partials in a fixed order into the
// (layer, bucket) accumulator, so the result is bitwise reproducible run to run (no
// floating atomics).  The LUT build runs in one workgroup (B <= 1024 buckets).
#include <math.h>

#include <algorithm>

#include "cham_moments.h"

namespace cham {
namespace {

// Tensors of one accumulate call (several for the batched call): workgroups of tensor i are
// [blk_end[i-1], blk_end[i]); partials are stored at the workgroup index.
constexpr int kStatsBatchMax = 64;
struct StatsBatch {
    int n;
    int blk_end[kStatsBatchMax];
    const float* X[kStatsBatchMax];
    int64_t numel[kStatsBatchMax];
};

// the batch entry (tensor) of workgroup blockIdx.x, its first workgroup and its count
CHAM_DEV int batch_entry(const int* blk_end, int n, int* lb, int* nb) {
    int ti = 0;
    while (ti + 1 < n && (int)blockIdx.x >= blk_end[ti]) ++ti;
    const int b0 = ti ? blk_end[ti - 1] : 0;
    *lb = (int)blockIdx.x - b0;
    *nb = blk_end[ti] - b0;
    return ti;
}

__global__ __launch_bounds__(kStatsThreads) void stats_partial_kernel(StatsBatch B, Partial* part) {
    int lb, nb;
    const int ti = batch_entry(B.blk_end, B.n, &lb, &nb);
    moments_block(B.X[ti], B.numel[ti], lb, nb, [](const float4&, int64_t) {}, part + blockIdx.x);
}

// The fused pass: each tensor quantized with its static scale (as the quantize pass does it,
// App. A.7 Alg. 2 with the LUT's (s, z)) while its moments are gathered exactly as the
// statistics pass gathers them.  One read of X serves both.
constexpr int kQSBatchMax = 32;
struct QSBatch {
    int n;
    int blk_end[kQSBatchMax];
    const float* X[kQSBatchMax];
    int64_t numel[kQSBatchMax];
    int fmt[kQSBatchMax];
    int nsamples[kQSBatchMax];
    const float* s_dev[kQSBatchMax];  // the LUT's (s, z) of the tensor's (layer, bucket)
    const float* z_dev[kQSBatchMax];
    uint32_t* codes[kQSBatchMax];
    uint8_t* e8[kQSBatchMax];
    float* scale_out[kQSBatchMax];
    float* zero_out[kQSBatchMax];
};

template <int FMT>
CHAM_DEV void quant_stats_tensor(const QSBatch& B, int ti, int lb, int nb, Partial* out) {
    uint32_t* C4 = B.codes[ti];
    if (FMT == CHAM_A_MXFP8_E4M3 || FMT == CHAM_A_MXINT8) {
        if (lb == 0)
            for (int q = threadIdx.x; q < B.nsamples[ti]; q += kStatsThreads) {
                B.scale_out[ti][q] = 1.0f;
                B.zero_out[ti][q] = 0.0f;
            }
        uint8_t* e8 = B.e8[ti];
        moments_block(B.X[ti], B.numel[ti], lb, nb,
                      [&](const float4& t, int64_t i) {
                          int E;
                          C4[i] = act_codes4_mx<FMT>(t, &E);
                          if ((threadIdx.x & 7) == 0) e8[i >> 3] = (uint8_t)(E + 127);
                      },
                      out);
    } else {
        const float s = *B.s_dev[ti], z = *B.z_dev[ti];
        if (lb == 0)
            for (int q = threadIdx.x; q < B.nsamples[ti]; q += kStatsThreads) {
                B.scale_out[ti][q] = s;
                B.zero_out[ti][q] = z;
            }
        const float r = 1.0f / s;
        moments_block(B.X[ti], B.numel[ti], lb, nb, [&](const float4& t, int64_t i) { C4[i] = act_codes4<FMT>(t, r, z); },
                      out);
    }
}

__global__ __launch_bounds__(kStatsThreads) void quant_stats_kernel(QSBatch B, Partial* part) {
    int lb, nb;
    const int ti = batch_entry(B.blk_end, B.n, &lb, &nb);
    Partial* out = part + blockIdx.x;
    switch (B.fmt[ti]) {  // workgroup-uniform
    case CHAM_A_INT8_ASYM: quant_stats_tensor<CHAM_A_INT8_ASYM>(B, ti, lb, nb, out); break;
    case CHAM_A_FP8_E4M3: quant_stats_tensor<CHAM_A_FP8_E4M3>(B, ti, lb, nb, out); break;
    case CHAM_A_FP8_E5M2: quant_stats_tensor<CHAM_A_FP8_E5M2>(B, ti, lb, nb, out); break;
    case CHAM_A_MXFP8_E4M3: quant_stats_tensor<CHAM_A_MXFP8_E4M3>(B, ti, lb, nb, out); break;
    default: quant_stats_tensor<CHAM_A_MXINT8>(B, ti, lb, nb, out); break;
    }
}

// Finalize of a batch: workgroup j owns accumulator target j and adds the sums of its
// tensors in batch order (each tensor's partials in index order, as one call would), so
// a batch gives the bits that one call per tensor would.
struct FinBatch {
    int ntgt;
    int first[kStatsBatchMax], count[kStatsBatchMax];  // per target: its tensors in order[]
    int order[kStatsBatchMax];                          // tensor indices grouped by target
    int pbeg[kStatsBatchMax], pcnt[kStatsBatchMax];     // per tensor: its partials
    int64_t numel[kStatsBatchMax];
    double* nS[kStatsBatchMax];  // per target
    float* lohi[kStatsBatchMax];
};

__global__ __launch_bounds__(kStatsThreads) void stats_finalize_kernel(FinBatch F, const Partial* part) {
    const int j = blockIdx.x;
    double* nS = F.nS[j];
    float* lohi = F.lohi[j];
    // the accumulator is read at the start so its latency overlaps the partial loads
    double acc[5] = {0.0, 0.0, 0.0, 0.0, 0.0};
    float alo = 0.0f, ahi = 0.0f;
    if (threadIdx.x == 0) {
#pragma unroll
        for (int k = 0; k < 5; ++k) acc[k] = nS[k];
        alo = lohi[0];
        ahi = lohi[1];
    }
    __shared__ Partial wp[kStatsThreads / kWave];
    for (int q = 0; q < F.count[j]; ++q) {
        const int ti = F.order[F.first[j] + q];
        const Partial* pt = part + F.pbeg[ti];
        const int nparts = F.pcnt[ti];
        double s1 = 0.0, s2 = 0.0, s3 = 0.0, s4 = 0.0;
        float lo = INFINITY, hi = -INFINITY;
#pragma unroll 4
        for (int i = threadIdx.x; i < nparts; i += kStatsThreads) {  // loads of 4 partials in flight
            Partial p = pt[i];
            s1 += p.s1; s2 += p.s2; s3 += p.s3; s4 += p.s4;
            lo = fminf(lo, p.lo); hi = fmaxf(hi, p.hi);
        }
        s1 = wave_sum(s1); s2 = wave_sum(s2); s3 = wave_sum(s3); s4 = wave_sum(s4);
        lo = wave_min(lo); hi = wave_max(hi);
        if ((threadIdx.x & 63) == 0) wp[threadIdx.x >> 6] = Partial{s1, s2, s3, s4, lo, hi, 0.f, 0.f};
        __syncthreads();
        if (threadIdx.x == 0) {
            Partial r = wp[0];
            for (int i = 1; i < kStatsThreads / kWave; ++i) {
                r.s1 += wp[i].s1; r.s2 += wp[i].s2; r.s3 += wp[i].s3; r.s4 += wp[i].s4;
                r.lo = fminf(r.lo, wp[i].lo); r.hi = fmaxf(r.hi, wp[i].hi);
            }
            acc[0] = acc[0] + (double)F.numel[ti];
            acc[1] = acc[1] + r.s1;
            acc[2] = acc[2] + r.s2;
            acc[3] = acc[3] + r.s3;
            acc[4] = acc[4] + r.s4;
            alo = fminf(alo, r.lo);
            ahi = fmaxf(ahi, r.hi);
        }
        __syncthreads();  // wp is reused by the next tensor
    }
    if (threadIdx.x == 0) {
#pragma unroll
        for (int k = 0; k < 5; ++k) nS[k] = acc[k];
        lohi[0] = alo;
        lohi[1] = ahi;
    }
}

__global__ void stats_reset_kernel(double* nS, float* lohi, int n) {
    int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) {
        for (int k = 0; k < 5; ++k) nS[5 * i + k] = 0.0;
        lohi[2 * i] = INFINITY;
        lohi[2 * i + 1] = -INFINITY;
    }
}

struct LutArgs {
    const double* nS;
    const float* lohi;
    const uint8_t* is_shortcut;
    uint8_t* F;
    float* S;
    float* Z;
    double* kappa;
    int L, B, T, kind;
    double b0, b1, r0, r1;  // r0, r1 = sqrt(b0), sqrt(b1), correctly rounded on the host
    double k_lo, k_hi, s_lo, s_hi;
    int snr_gate_on;
};

constexpr int kLutThreads = 256;

// One workgroup.  First the SNR at every bucket midpoint: alpha_bar_t = prod_{s<=t}
// (1 - beta_s) as a tree product over the workgroup (binary64; its rounding differs from a
// sequential product only in the last bits, so only an SNR within ~1e-15 of a gate could
// route differently).  Then one thread per (layer, bucket): kurtosis, route, ScaleZP.
constexpr int kLutMaxBuckets = 1024;

__global__ __launch_bounds__(kLutThreads) void lut_kernel(LutArgs a) {
    __shared__ double red[kLutThreads / kWave];
    __shared__ double snr_ws[kLutMaxBuckets];
    for (int b = 0; b < a.B; ++b) {
        const int tb = (int)(((int64_t)(2 * b + 1) * a.T) / (2LL * a.B));
        double prod = 1.0;
        for (int s = threadIdx.x; s <= tb; s += kLutThreads) {
            const double frac = a.T > 1 ? (double)s / (double)(a.T - 1) : 0.0;
            double beta;
            if (a.kind == CHAM_SCHED_SCALED_LINEAR) {
                const double r = a.r0 + (a.r1 - a.r0) * frac;
                beta = r * r;
            } else {
                beta = a.b0 + (a.b1 - a.b0) * frac;
            }
            prod *= (1.0 - beta);
        }
        // product tree: within each wavefront by shuffles, then the wavefronts' products
        for (int o = 32; o > 0; o >>= 1) prod *= __shfl_xor(prod, o, kWave);
        if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = prod;
        __syncthreads();
        if (threadIdx.x == 0) {
            const double ab = (red[0] * red[1]) * (red[2] * red[3]);
            snr_ws[b] = ab / (1.0 - ab);
        }
        __syncthreads();
    }
    for (int i = threadIdx.x; i < a.L * a.B; i += kLutThreads) {
        const int l = i / a.B, b = i % a.B;
        // kurtosis from raw power sums (population moments)
        const double* p = a.nS + 5 * (int64_t)i;
        const double n = p[0];
        const double mu = p[1] / n;
        const double e2 = p[2] / n, e3 = p[3] / n, e4 = p[4] / n;
        const double m2 = e2 - mu * mu;
        const double m4 = e4 - 4.0 * mu * e3 + 6.0 * mu * mu * e2 - 3.0 * mu * mu * mu * mu;
        const double kap = m4 / (m2 * m2);
        const double snr = snr_ws[b];
        int f;
        const int sc = a.is_shortcut ? a.is_shortcut[l] : 0;
        const bool snr_low = a.snr_gate_on ? (snr < a.s_lo) : false;
        const bool snr_high = a.snr_gate_on ? (snr > a.s_hi) : true;
        if (sc) f = CHAM_A_MXFP8_E4M3;
        else if (kap > a.k_hi || snr_low) f = CHAM_A_FP8_E5M2;
        else if (kap <= a.k_lo && snr_high) f = CHAM_A_INT8_ASYM;
        else f = CHAM_A_FP8_E4M3;
        // ScaleZP on the bucket range
        float s = 1.0f, z = 0.0f;
        if (n != 0.0) {
            const float lo = a.lohi[2 * i], hi = a.lohi[2 * i + 1];
            if (f == CHAM_A_INT8_ASYM) {
                int_asym_scale_zp(lo, hi, 255.0f, &s, &z);
            } else if (f == CHAM_A_FP8_E4M3) {
                s = floor_scale(fmaxf(fabsf(lo), fabsf(hi)) / 448.0f);
            } else if (f == CHAM_A_FP8_E5M2) {
                s = floor_scale(fmaxf(fabsf(lo), fabsf(hi)) / 57344.0f);
            }
        }
        a.F[i] = (uint8_t)f;
        a.S[i] = s;
        a.Z[i] = z;
        if (a.kappa) a.kappa[i] = kap;
    }
}

}  // namespace
}  // namespace cham

using namespace cham;

extern "C" int cham_act_stats_reset(cham_act_stats* st, void* stream) {
    if (!st || !st->nS || !st->lohi || st->L < 1 || st->B < 1) return CHAM_EINVAL;
    const int n = st->L * st->B;
    hipLaunchKernelGGL(stats_reset_kernel, dim3((n + 255) / 256), dim3(256), 0, (hipStream_t)stream,
                       st->nS, st->lohi, n);
    CHAM_CHECK_LAUNCH();
    return CHAM_OK;
}

static int stats_blocks(int64_t numel) {
    int64_t nq = numel >> 2;
    int64_t b = (nq + kStatsThreads * kStatsLoads - 1) / (kStatsThreads * kStatsLoads);  // >= kStatsLoads float4 per thread
    if (b < 1) b = 1;
    if (b > kStatsMaxBlocks) b = kStatsMaxBlocks;
    return (int)b;
}

size_t cham_stats_workspace_bytes(int64_t numel) { return sizeof(Partial) * (size_t)stats_blocks(numel); }

// The finalize launch of batch tensors [i0, i0 + m): per tensor its partials (counts nb[q])
// and numel, and the accumulator targets (layer, bucket) in order of first appearance, each
// with its tensors in batch order.
static FinBatch fin_batch(const int64_t* numel, const int* nb, const int32_t* layer, const int32_t* bucket, int m,
                          const cham_act_stats* st) {
    FinBatch F;
    F.ntgt = 0;
    int blk = 0;
    for (int q = 0; q < m; ++q) {
        F.pbeg[q] = blk;
        F.pcnt[q] = nb[q];
        F.numel[q] = numel[q];
        blk += nb[q];
    }
    int tgt_of[kStatsBatchMax];
    for (int q = 0; q < m; ++q) {
        const int64_t ti = (int64_t)layer[q] * st->B + bucket[q];
        int j = 0;
        while (j < F.ntgt && F.nS[j] != st->nS + 5 * ti) ++j;
        if (j == F.ntgt) {
            F.nS[j] = st->nS + 5 * ti;
            F.lohi[j] = st->lohi + 2 * ti;
            F.count[j] = 0;
            ++F.ntgt;
        }
        tgt_of[q] = j;
        ++F.count[j];
    }
    for (int j = 0, o = 0; j < F.ntgt; ++j) {
        F.first[j] = o;
        for (int q = 0; q < m; ++q)
            if (tgt_of[q] == j) F.order[o++] = q;
    }
    return F;
}

extern "C" int cham_act_stats_accumulate_batch(const float* const* X, const int64_t* numel, const int32_t* layer,
                                               const int32_t* bucket, int32_t n, cham_act_stats* st, void* ws,
                                               size_t ws_bytes, void* stream) {
    if (!X || !numel || !layer || !bucket || n < 1 || !st || !st->nS || !st->lohi) return CHAM_EINVAL;
    size_t parts = 0;
    for (int i = 0; i < n; ++i) {
        if (!X[i] || numel[i] < 1 || ((uintptr_t)X[i] & 15u) != 0) return CHAM_EINVAL;
        if (layer[i] < 0 || layer[i] >= st->L || bucket[i] < 0 || bucket[i] >= st->B) return CHAM_EINVAL;
        parts += (size_t)stats_blocks(numel[i]);
    }
    if (!ws || ws_bytes < sizeof(Partial) * parts) return CHAM_EWORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    Partial* part = (Partial*)ws;
    for (int i0 = 0; i0 < n; i0 += kStatsBatchMax) {  // launches in order: the accumulation order holds
        const int m = std::min(kStatsBatchMax, n - i0);
        StatsBatch B;
        int nb[kStatsBatchMax];
        B.n = m;
        int blk = 0;
        for (int q = 0; q < m; ++q) {
            nb[q] = stats_blocks(numel[i0 + q]);
            B.X[q] = X[i0 + q];
            B.numel[q] = numel[i0 + q];
            blk += nb[q];
            B.blk_end[q] = blk;
        }
        const FinBatch F = fin_batch(numel + i0, nb, layer + i0, bucket + i0, m, st);
        hipLaunchKernelGGL(stats_partial_kernel, dim3(blk), dim3(kStatsThreads), 0, s, B, part);
        CHAM_CHECK_LAUNCH();
        hipLaunchKernelGGL(stats_finalize_kernel, dim3(F.ntgt), dim3(kStatsThreads), 0, s, F, part);
        CHAM_CHECK_LAUNCH();
        part += blk;
    }
    return CHAM_OK;
}

// Bucket b of timestep t for every tensor; formats from the host mirror of the LUT's F.
extern "C" int cham_quantize_act_lut_accumulate_batch(const float* const* X, const int32_t* layer, int32_t n,
                                                      int32_t t, const cham_lut* lut, const uint8_t* F_host,
                                                      cham_aq* out, cham_act_stats* st, void* ws, size_t ws_bytes,
                                                      void* stream) {
    if (!X || !layer || n < 1 || !lut || !F_host || !lut->S || !lut->Z || !out) return CHAM_EINVAL;
    if (!st || !st->nS || !st->lohi || st->L != lut->L || st->B != lut->B) return CHAM_EINVAL;
    const int32_t b = cham_bucket(t, lut->T, lut->B);
    if (b < 0) return CHAM_EINVAL;
    size_t parts = 0;
    for (int i = 0; i < n; ++i) {
        if (layer[i] < 0 || layer[i] >= lut->L) return CHAM_EINVAL;
        const cham_aq& o = out[i];
        if (!X[i] || !o.codes || !o.scale || !o.zero || o.M < 1 || o.K < 1) return CHAM_EINVAL;
        if (o.nsamples < 1 || o.M % o.nsamples != 0) return CHAM_EINVAL;
        if (((uintptr_t)X[i] & 15u) != 0 || ((uintptr_t)o.codes & 3u) != 0) return CHAM_EINVAL;
        const int fmt = F_host[(int64_t)layer[i] * lut->B + b];
        if (fmt < 0 || fmt >= CHAM_A_NFMT) return CHAM_EFORMAT;
        if (o.K % 32 != 0) return CHAM_ESHAPE;
        if ((fmt == CHAM_A_MXFP8_E4M3 || fmt == CHAM_A_MXINT8) && !o.e8m0) return CHAM_EINVAL;
        parts += (size_t)stats_blocks(o.M * o.K);
    }
    if (!ws || ws_bytes < sizeof(Partial) * parts) return CHAM_EWORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    Partial* part = (Partial*)ws;
    for (int i0 = 0; i0 < n; i0 += kQSBatchMax) {  // launches in order: the accumulation order holds
        const int m = std::min(kQSBatchMax, n - i0);
        QSBatch B;
        int nb[kQSBatchMax];
        int64_t numel[kQSBatchMax];
        int32_t bucket[kQSBatchMax];
        B.n = m;
        int blk = 0;
        for (int q = 0; q < m; ++q) {
            cham_aq& o = out[i0 + q];
            const int64_t li = (int64_t)layer[i0 + q] * lut->B + b;
            o.fmt = F_host[li];
            numel[q] = o.M * o.K;
            bucket[q] = b;
            nb[q] = stats_blocks(numel[q]);
            B.X[q] = X[i0 + q];
            B.numel[q] = numel[q];
            B.fmt[q] = o.fmt;
            B.nsamples[q] = o.nsamples;
            B.s_dev[q] = lut->S + li;
            B.z_dev[q] = lut->Z + li;
            B.codes[q] = (uint32_t*)o.codes;
            B.e8[q] = o.e8m0;
            B.scale_out[q] = o.scale;
            B.zero_out[q] = o.zero;
            blk += nb[q];
            B.blk_end[q] = blk;
        }
        const FinBatch F = fin_batch(numel, nb, layer + i0, bucket, m, st);
        hipLaunchKernelGGL(quant_stats_kernel, dim3(blk), dim3(kStatsThreads), 0, s, B, part);
        CHAM_CHECK_LAUNCH();
        hipLaunchKernelGGL(stats_finalize_kernel, dim3(F.ntgt), dim3(kStatsThreads), 0, s, F, part);
        CHAM_CHECK_LAUNCH();
        part += blk;
    }
    return CHAM_OK;
}

extern "C" int cham_act_stats_accumulate(const float* X, int64_t numel, int32_t layer, int32_t bucket,
                                         cham_act_stats* st, void* ws, size_t ws_bytes, void* stream) {
    return cham_act_stats_accumulate_batch(&X, &numel, &layer, &bucket, 1, st, ws, ws_bytes, stream);
}

extern "C" void cham_schedule_default(cham_schedule* s) {
    if (!s) return;
    s->T = 1000;
    s->beta0 = 0.00085;
    s->beta1 = 0.012;
    s->kind = CHAM_SCHED_SCALED_LINEAR;
    s->kappa_lo = 3.0;
    s->kappa_hi = 5.0;
    s->snr_lo = 0.2;
    s->snr_hi = 2.0;
    s->snr_gate_on = 1;
}

extern "C" int32_t cham_bucket(int32_t t, int32_t T, int32_t B) {
    if (t < 0 || T < 1 || B < 1) return -1;
    int64_t b = ((int64_t)t * B) / T;
    return (int32_t)(b < B - 1 ? b : B - 1);
}

extern "C" int cham_build_act_lut(const cham_act_stats* st, const cham_schedule* sch, const uint8_t* is_shortcut,
                                  cham_lut* lut, double* kappa, void* stream) {
    if (!st || !sch || !lut || !st->nS || !st->lohi || !lut->F || !lut->S || !lut->Z) return CHAM_EINVAL;
    if (st->L < 1 || st->B < 1 || lut->L != st->L || lut->B != st->B) return CHAM_EINVAL;
    if (sch->T < 1 || sch->T > (1 << 20) || st->B > sch->T || st->B > kLutMaxBuckets) return CHAM_EINVAL;
    if (!(sch->beta0 >= 0.0 && sch->beta0 < 1.0 && sch->beta1 >= 0.0 && sch->beta1 < 1.0)) return CHAM_EINVAL;
    if (sch->kind != CHAM_SCHED_SCALED_LINEAR && sch->kind != CHAM_SCHED_LINEAR) return CHAM_EINVAL;
    lut->T = sch->T;
    LutArgs a;
    a.nS = st->nS;
    a.lohi = st->lohi;
    a.is_shortcut = is_shortcut;
    a.F = lut->F;
    a.S = lut->S;
    a.Z = lut->Z;
    a.kappa = kappa;
    a.L = st->L;
    a.B = st->B;
    a.T = sch->T;
    a.kind = sch->kind;
    a.b0 = sch->beta0;
    a.b1 = sch->beta1;
    a.r0 = sqrt(sch->beta0);
    a.r1 = sqrt(sch->beta1);
    a.k_lo = sch->kappa_lo;
    a.k_hi = sch->kappa_hi;
    a.s_lo = sch->snr_lo;
    a.s_hi = sch->snr_hi;
    a.snr_gate_on = sch->snr_gate_on;
    const int n = st->L * st->B;
    (void)n;
    hipLaunchKernelGGL(lut_kernel, dim3(1), dim3(kLutThreads), 0, (hipStream_t)stream, a);
    CHAM_CHECK_LAUNCH();
    return CHAM_OK;
}
