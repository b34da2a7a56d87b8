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

#include "cham_device.h"

namespace cham {
namespace {

constexpr int kStatsThreads = 256;
constexpr int kStatsMaxBlocks = 1024;
constexpr int kStatsLoads = 16;  // 16-byte loads in flight per thread

struct Partial {
    double s1, s2, s3, s4;
    float lo, hi;
    float pad0, pad1;
};

// Tensors of one accumulate call (several for the batched call): workgroups of tensor i are
// [blk_end[i-1], blk_end[i]); partials are stored at the workgroup index.
constexpr int kStatsBatchMax = 64;
struct StatsBatch {
    int n;
    int blk_end[kStatsBatchMax];
    const float* X[kStatsBatchMax];
    int64_t numel[kStatsBatchMax];
};

__global__ __launch_bounds__(kStatsThreads) void stats_partial_kernel(StatsBatch B, Partial* part) {
    int ti = 0;
    while (ti + 1 < B.n && (int)blockIdx.x >= B.blk_end[ti]) ++ti;
    const int b0 = ti ? B.blk_end[ti - 1] : 0;
    const int lb = (int)blockIdx.x - b0, nb = B.blk_end[ti] - b0;  // this tensor's workgroups
    const float* X = B.X[ti];
    const int64_t numel = B.numel[ti];
    double s1 = 0.0, s2 = 0.0, s3 = 0.0, s4 = 0.0;
    float lo = INFINITY, hi = -INFINITY;
    const int64_t nq = numel >> 2;
    const int64_t stride = (int64_t)nb * blockDim.x;
    const float4* X4 = reinterpret_cast<const float4*>(X);
    auto add = [&](const float4& t) {
        const float e[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            double d = (double)e[j];
            double d2 = d * d;
            s1 += d;
            s2 += d2;
            s3 += d2 * d;
            s4 += d2 * d2;
            lo = fminf(lo, e[j]);
            hi = fmaxf(hi, e[j]);
        }
    };
    // kStatsLoads loads in flight per thread, then their sums in index order
    int64_t i = (int64_t)lb * blockDim.x + threadIdx.x;
    for (; i + (kStatsLoads - 1) * stride < nq; i += kStatsLoads * stride) {
        float4 t[kStatsLoads];
#pragma unroll
        for (int q = 0; q < kStatsLoads; ++q) t[q] = X4[i + q * stride];
#pragma unroll
        for (int q = 0; q < kStatsLoads; ++q) add(t[q]);
    }
    // the last few: all loads issued first, then the sums in index order
    {
        float4 t[kStatsLoads - 1];
#pragma unroll
        for (int q = 0; q < kStatsLoads - 1; ++q) t[q] = i + q * stride < nq ? X4[i + q * stride] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int q = 0; q < kStatsLoads - 1; ++q)
            if (i + q * stride < nq) add(t[q]);
    }
    // scalar tail (numel % 4), handled by the first threads of the tensor's workgroup 0
    if (lb == 0 && threadIdx.x < (numel & 3)) {
        float x = X[(nq << 2) + threadIdx.x];
        double d = (double)x, d2 = d * d;
        s1 += d; s2 += d2; s3 += d2 * d; s4 += d2 * d2;
        lo = fminf(lo, x); hi = fmaxf(hi, x);
    }
    s1 = wave_sum(s1); s2 = wave_sum(s2); s3 = wave_sum(s3); s4 = wave_sum(s4);
    lo = wave_min(lo); hi = wave_max(hi);
    __shared__ Partial wp[kStatsThreads / kWave];
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) wp[w] = Partial{s1, s2, s3, s4, lo, hi, 0.f, 0.f};
    __syncthreads();
    if (threadIdx.x == 0) {
        Partial r = wp[0];
        for (int i = 1; i < kStatsThreads / kWave; ++i) {
            r.s1 += wp[i].s1; r.s2 += wp[i].s2; r.s3 += wp[i].s3; r.s4 += wp[i].s4;
            r.lo = fminf(r.lo, wp[i].lo); r.hi = fmaxf(r.hi, wp[i].hi);
        }
        part[blockIdx.x] = r;
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
        FinBatch F;
        B.n = m;
        F.ntgt = 0;
        int blk = 0;
        for (int q = 0; q < m; ++q) {
            const int i = i0 + q;
            const int nb = stats_blocks(numel[i]);
            B.X[q] = X[i];
            B.numel[q] = numel[i];
            F.pbeg[q] = blk;
            F.pcnt[q] = nb;
            F.numel[q] = numel[i];
            blk += nb;
            B.blk_end[q] = blk;
        }
        // targets in order of first appearance, each with its tensors in batch order
        int tgt_of[kStatsBatchMax];
        for (int q = 0; q < m; ++q) {
            const int64_t ti = (int64_t)layer[i0 + q] * st->B + bucket[i0 + q];
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
        hipLaunchKernelGGL(stats_partial_kernel, dim3(blk), dim3(kStatsThreads), 0, s, B, part);
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
