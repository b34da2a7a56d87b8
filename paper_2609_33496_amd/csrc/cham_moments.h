// One workgroup's share of an activation tensor's moments (Sec. 4.4; App. A.3 Eq. kurt):
// binary64 power sums x, x^2, x^3, x^4 and binary32 min / max over the float4s it owns.
// Shared by the statistics pass and the fused quantize-and-accumulate pass, so both give a
// tensor the same partial sums, bit for bit, and the same finalize turns them into the
// same accumulator bits.
#ifndef CHAM_MOMENTS_H_
#define CHAM_MOMENTS_H_

#include "cham_device.h"

namespace cham {

constexpr int kStatsThreads = 256;
constexpr int kStatsMaxBlocks = 1024;
constexpr int kStatsLoads = 16;  // 16-byte loads in flight per thread

struct Partial {
    double s1, s2, s3, s4;
    float lo, hi;
    float pad0, pad1;
};

// Workgroup lb of nb over X[numel]: thread t owns float4s lb * 256 + t + j * nb * 256 (so
// consecutive lanes hold consecutive float4s and an aligned 8-lane group holds a whole
// 32-element block), issues kStatsLoads of them at once and adds them in index order.
// visit(t, i) runs on every float4 with its index, right after it is added, with the
// whole 8-lane group active.  Thread 0 writes the workgroup's partial to *out.
template <class Visit>
CHAM_DEV void moments_block(const float* X, int64_t numel, int lb, int nb, Visit&& visit, Partial* out) {
    double s1 = 0.0, s2 = 0.0, s3 = 0.0, s4 = 0.0;
    float lo = INFINITY, hi = -INFINITY;
    const int64_t nq = numel >> 2;
    const int64_t stride = (int64_t)nb * blockDim.x;
    const float4* X4 = reinterpret_cast<const float4*>(X);
    // x^3 and x^4 are added with fused multiply-adds (one rounding each instead of two)
    auto add = [&](const float4& t) {
        const float e[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            double d = (double)e[j];
            double d2 = d * d;
            s1 += d;
            s2 += d2;
            s3 = __builtin_fma(d2, d, s3);
            s4 = __builtin_fma(d2, d2, s4);
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
        for (int q = 0; q < kStatsLoads; ++q) {
            add(t[q]);
            visit(t[q], i + q * stride);
        }
    }
    // the last few: all loads issued first, then the sums in index order (a float4 is in
    // or out with its whole aligned 8-lane group when nq is a multiple of 8)
    {
        float4 t[kStatsLoads - 1];
#pragma unroll
        for (int q = 0; q < kStatsLoads - 1; ++q) t[q] = i + q * stride < nq ? X4[i + q * stride] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int q = 0; q < kStatsLoads - 1; ++q)
            if (i + q * stride < nq) {
                add(t[q]);
                visit(t[q], i + q * stride);
            }
    }
    // scalar tail (numel % 4), handled by the first threads of the tensor's workgroup 0
    if (lb == 0 && threadIdx.x < (numel & 3)) {
        float x = X[(nq << 2) + threadIdx.x];
        double d = (double)x, d2 = d * d;
        s1 += d; s2 += d2; s3 = __builtin_fma(d2, d, s3); s4 = __builtin_fma(d2, d2, s4);
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
        for (int k = 1; k < kStatsThreads / kWave; ++k) {
            r.s1 += wp[k].s1; r.s2 += wp[k].s2; r.s3 += wp[k].s3; r.s4 += wp[k].s4;
            r.lo = fminf(r.lo, wp[k].lo); r.hi = fmaxf(r.hi, wp[k].hi);
        }
        *out = r;
    }
}

}  // namespace cham

#endif  // CHAM_MOMENTS_H_
