// Activation quantization (App. A.7: Alg. 2 static scales, Alg. 3 dynamic per-tensor
// scales; ScaleZP) to the five activation formats of Sec. 4.2.
//
// HBM-bound elementwise pass: float4 loads, one packed 32-bit store of four codes per
// float4; each thread issues its kQLoads loads (a workgroup's consecutive float4 runs)
// before it converts any of them, so they are in flight together.  MX formats: a 32-element block is 8 consecutive lanes; its amax comes from a
// shuffle reduction and one lane writes the E8M0 byte.  Dynamic mode first reduces
// min/max into per-workgroup partials (workspace); the quantize kernel folds them (min
// and max are exact, so the result does not depend on the order).
#include <algorithm>
#include <atomic>

#include "cham_device.h"

namespace cham {
namespace {

constexpr int kQThreads = 256;
constexpr int kQMaxBlocks = 1024;
constexpr int kQLoads = 4;  // float4 loads in flight per thread

// Per-sample launches: the grid is nbs workgroups per sample, sample-major; workgroup
// j = blockIdx.x % nbs of sample blockIdx.x / nbs strides over that sample's float4s.
// float4 index of load u of the thread's run starting at i0 (workgroup-strided)
CHAM_DEV int64_t qidx(int64_t i0, int u) { return i0 + (int64_t)u * kQThreads; }
CHAM_DEV int64_t qfirst(int nbs) { return (int64_t)(blockIdx.x % nbs) * kQThreads * kQLoads + threadIdx.x; }
CHAM_DEV int64_t qstep(int nbs) { return (int64_t)nbs * kQThreads * kQLoads; }

// n: elements per sample (a multiple of 4)
__global__ __launch_bounds__(kQThreads) void minmax_partial_kernel(const float* X, int64_t n, int nbs, float2* part) {
    float lo = INFINITY, hi = -INFINITY;
    const int64_t nq = n >> 2;
    const float4* X4 = reinterpret_cast<const float4*>(X) + (int64_t)(blockIdx.x / nbs) * nq;
    for (int64_t i0 = qfirst(nbs); i0 < nq; i0 += qstep(nbs)) {
        float4 t[kQLoads];
#pragma unroll
        for (int u = 0; u < kQLoads; ++u) {
            const int64_t i = qidx(i0, u);
            t[u] = X4[i < nq ? i : i0];  // past the end: a repeat of the first (i0 < nq)
        }
#pragma unroll
        for (int u = 0; u < kQLoads; ++u) {
            lo = fminf(fminf(lo, t[u].x), fminf(fminf(t[u].y, t[u].z), t[u].w));
            hi = fmaxf(fmaxf(hi, t[u].x), fmaxf(fmaxf(t[u].y, t[u].z), t[u].w));
        }
    }
    lo = wave_min(lo);
    hi = wave_max(hi);
    __shared__ float2 wp[kQThreads / kWave];
    if ((threadIdx.x & 63) == 0) wp[threadIdx.x >> 6] = make_float2(lo, hi);
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int i = 1; i < kQThreads / kWave; ++i) { lo = fminf(lo, wp[i].x); hi = fmaxf(hi, wp[i].y); }
        lo = fminf(lo, wp[0].x);
        hi = fmaxf(hi, wp[0].y);
        part[blockIdx.x] = make_float2(lo, hi);
    }
}

// ScaleZP (App. A.7) for the per-tensor formats.
CHAM_DEV void scale_zp(int fmt, float lo, float hi, float* s, float* z) {
    if (fmt == CHAM_A_INT8_ASYM) {
        int_asym_scale_zp(lo, hi, 255.0f, s, z);
    } else if (fmt == CHAM_A_FP8_E4M3) {
        *s = floor_scale(fmaxf(fabsf(lo), fabsf(hi)) / 448.0f);
        *z = 0.0f;
    } else if (fmt == CHAM_A_FP8_E5M2) {
        *s = floor_scale(fmaxf(fabsf(lo), fabsf(hi)) / 57344.0f);
        *z = 0.0f;
    } else {
        *s = 1.0f;
        *z = 0.0f;
    }
}

struct QArgs {
    const float* X;
    int64_t n;          // elements per sample (M/S * K), multiple of 4
    int nbs;            // workgroups per sample
    int fmt;
    const float* s_dev;  // static
    const float* z_dev;
    const float2* part;  // dynamic: nbs partials per sample (or NULL)
    uint8_t* codes;
    float* scale_out;    // [S]
    float* zero_out;
};

// The first loads of every thread are issued before the workgroup learns the scale (its
// fetch, or the fold of the dynamic partials, would otherwise stand in front of them), and
// each iteration issues the next run's loads before it converts the current one.
template <int FMT>
__global__ __launch_bounds__(kQThreads) void quant_tensor_kernel(QArgs a) {
    __shared__ float sh_s, sh_z;
    const int sample = (int)blockIdx.x / a.nbs;
    const int64_t nq = a.n >> 2;
    const float4* X4 = reinterpret_cast<const float4*>(a.X) + (int64_t)sample * nq;
    uint32_t* C4 = reinterpret_cast<uint32_t*>(a.codes) + (int64_t)sample * nq;
    auto load = [&](float4 (&t)[kQLoads], int64_t i0) {
#pragma unroll
        for (int u = 0; u < kQLoads; ++u) {
            const int64_t i = qidx(i0, u);
            t[u] = i < nq ? X4[i] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    };
    int64_t i0 = qfirst(a.nbs);
    float4 t[kQLoads];
    load(t, i0);
    if (threadIdx.x < kWave) {
        float s, z;
        if (a.part) {
            float lo = INFINITY, hi = -INFINITY;
            for (int i = threadIdx.x; i < a.nbs; i += kWave) {
                float2 p = a.part[(int64_t)sample * a.nbs + i];
                lo = fminf(lo, p.x);
                hi = fmaxf(hi, p.y);
            }
            lo = wave_min(lo);
            hi = wave_max(hi);
            scale_zp(FMT, lo, hi, &s, &z);
        } else {
            s = *a.s_dev;
            z = *a.z_dev;
        }
        if (threadIdx.x == 0) {
            sh_s = s;
            sh_z = z;
            if ((int)blockIdx.x % a.nbs == 0) { a.scale_out[sample] = s; a.zero_out[sample] = z; }
        }
    }
    __syncthreads();
    const float s = sh_s, z = sh_z;
    const float r = 1.0f / s;
    for (; i0 < nq; i0 += qstep(a.nbs)) {
        float4 tn[kQLoads];
        if (i0 + qstep(a.nbs) < nq) load(tn, i0 + qstep(a.nbs));
#pragma unroll
        for (int u = 0; u < kQLoads; ++u) {
            const uint32_t w = act_codes4<FMT>(t[u], r, z);
            const int64_t i = qidx(i0, u);
            if (i < nq) C4[i] = w;
        }
#pragma unroll
        for (int u = 0; u < kQLoads; ++u) t[u] = tn[u];
    }
}

// MX formats: one 32-block = 8 lanes x float4.  Grid-stride over float4 index i; the
// 8-lane groups stay aligned because the stride is a multiple of 64.
template <int FMT>
__global__ __launch_bounds__(kQThreads) void quant_mx_kernel(const float* X, int64_t n, uint8_t* codes, uint8_t* e8,
                                                             float* scale_out, float* zero_out, int nsamples) {
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < nsamples; i += kQThreads) { scale_out[i] = 1.0f; zero_out[i] = 0.0f; }
    const int nbs = gridDim.x;  // the block exponents need no per-sample scale: one range
    const int64_t nq = n >> 2;  // multiple of 8
    const float4* X4 = reinterpret_cast<const float4*>(X);
    uint32_t* C4 = reinterpret_cast<uint32_t*>(codes);
    // the same trip count for every lane: the 8-lane reductions run with whole wavefronts
    const int64_t iters = (nq + qstep(nbs) - 1) / qstep(nbs);
    for (int64_t it = 0; it < iters; ++it) {
        const int64_t i0 = qfirst(nbs) + it * qstep(nbs);
        float4 t[kQLoads];
#pragma unroll
        for (int u = 0; u < kQLoads; ++u) {
            const int64_t i = qidx(i0, u);
            t[u] = i < nq ? X4[i] : make_float4(0.f, 0.f, 0.f, 0.f);  // whole 8-lane groups are in or out
        }
#pragma unroll
        for (int u = 0; u < kQLoads; ++u) {
            int E;
            const uint32_t w = act_codes4_mx<FMT>(t[u], &E);
            const int64_t i = qidx(i0, u);
            if (i < nq) {
                C4[i] = w;
                if ((threadIdx.x & 7) == 0) e8[i >> 3] = (uint8_t)(E + 127);
            }
        }
    }
}

int qblocks(int64_t nq) {
    int64_t b = (nq + kQThreads * kQLoads - 1) / (kQThreads * kQLoads);
    if (b < 1) b = 1;
    if (b > kQMaxBlocks) b = kQMaxBlocks;
    return (int)b;
}

}  // namespace
}  // namespace cham

using namespace cham;

// dynamic scales: at most kQMaxBlocks min/max partials in all (float2 each)
size_t cham_quant_workspace_bytes(int64_t n) { return n > 0 ? sizeof(float2) * (size_t)kQMaxBlocks : 0; }

// Checks the arguments of a quantize call (no launch).
static int quant_check(const float* X, int32_t fmt, int32_t dynamic, const float* s_dev, const float* z_dev,
                       const cham_aq* out) {
    if (!X || !out || !out->codes || !out->scale || !out->zero) return CHAM_EINVAL;
    if (out->M < 1 || out->K < 1) return CHAM_EINVAL;
    if (out->nsamples < 1 || out->nsamples > kQMaxBlocks || out->M % out->nsamples != 0) return CHAM_EINVAL;
    if (fmt < 0 || fmt >= CHAM_A_NFMT) return CHAM_EFORMAT;
    if (out->K % 32 != 0) return CHAM_ESHAPE;
    if (((uintptr_t)X & 15u) != 0 || ((uintptr_t)out->codes & 3u) != 0) return CHAM_EINVAL;
    const bool mx = fmt == CHAM_A_MXFP8_E4M3 || fmt == CHAM_A_MXINT8;
    if (mx && !out->e8m0) return CHAM_EINVAL;
    if (!mx && !dynamic && (!s_dev || !z_dev)) return CHAM_EINVAL;
    return CHAM_OK;
}

// The launches of a checked quantize call; part: kQMaxBlocks float2 of device scratch
// (used when dynamic).
static int quant_launch(const float* X, int32_t fmt, int32_t dynamic, const float* s_dev, const float* z_dev,
                        cham_aq* out, float2* part, hipStream_t s) {
    const int64_t n = out->M * out->K;
    const int S = out->nsamples;
    out->fmt = fmt;
    if (fmt == CHAM_A_MXFP8_E4M3 || fmt == CHAM_A_MXINT8) {
        const int nb = qblocks(n >> 2);
        if (fmt == CHAM_A_MXFP8_E4M3)
            hipLaunchKernelGGL(quant_mx_kernel<CHAM_A_MXFP8_E4M3>, dim3(nb), dim3(kQThreads), 0, s, X, n, out->codes,
                               out->e8m0, out->scale, out->zero, S);
        else
            hipLaunchKernelGGL(quant_mx_kernel<CHAM_A_MXINT8>, dim3(nb), dim3(kQThreads), 0, s, X, n, out->codes,
                               out->e8m0, out->scale, out->zero, S);
        CHAM_CHECK_LAUNCH();
        return CHAM_OK;
    }
    const int64_t ns = n / S;  // elements per sample, a multiple of 32
    const int nbs = std::max(1, std::min(qblocks(ns >> 2), kQMaxBlocks / S));
    QArgs a;
    a.X = X;
    a.n = ns;
    a.nbs = nbs;
    a.fmt = fmt;
    a.s_dev = s_dev;
    a.z_dev = z_dev;
    a.part = nullptr;
    a.codes = out->codes;
    a.scale_out = out->scale;
    a.zero_out = out->zero;
    const dim3 grid((unsigned)(nbs * S));
    if (dynamic) {
        hipLaunchKernelGGL(minmax_partial_kernel, grid, dim3(kQThreads), 0, s, X, ns, nbs, part);
        CHAM_CHECK_LAUNCH();
        a.part = part;
    }
    if (fmt == CHAM_A_INT8_ASYM)
        hipLaunchKernelGGL(quant_tensor_kernel<CHAM_A_INT8_ASYM>, grid, dim3(kQThreads), 0, s, a);
    else if (fmt == CHAM_A_FP8_E4M3)
        hipLaunchKernelGGL(quant_tensor_kernel<CHAM_A_FP8_E4M3>, grid, dim3(kQThreads), 0, s, a);
    else
        hipLaunchKernelGGL(quant_tensor_kernel<CHAM_A_FP8_E5M2>, grid, dim3(kQThreads), 0, s, a);
    CHAM_CHECK_LAUNCH();
    return CHAM_OK;
}

// ---- allocation-free variant: the dynamic min/max partials go to a file-scope device array
// (kQMaxBlocks float2 = 8 KB on every device the library runs on, held until the process
// ends), addressed through hipGetSymbolAddress once per device.
static __device__ __align__(256) float2 scratch[kQMaxBlocks];

// Device address of this device's copy of scratch (queried on the first call on each
// device, with that device current; concurrent first calls store the same address).
static float2* scratch_ptr() {
    static std::atomic<void*> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
    void* p = cached[dev].load(std::memory_order_acquire);
    if (!p) {
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        cached[dev].store(p, std::memory_order_release);
    }
    return (float2*)p;
}

extern "C" int cham_quantize_act_noalloc(const float* X, int32_t fmt, int32_t dynamic, const float* s_dev,
                                         const float* z_dev, cham_aq* out, void* stream) {
    const int rc = quant_check(X, fmt, dynamic, s_dev, z_dev, out);
    if (rc != CHAM_OK) return rc;
    float2* part = scratch_ptr();
    if (!part) return CHAM_EHIP;
    // every call needs at most kQMaxBlocks partials (the launch caps its workgroups), so no
    // size exceeds the array
    return quant_launch(X, fmt, dynamic, s_dev, z_dev, out, part, (hipStream_t)stream);
}

extern "C" int cham_quantize_act(const float* X, int32_t fmt, int32_t dynamic, const float* s_dev, const float* z_dev,
                                 cham_aq* out, void* ws, size_t ws_bytes, void* stream) {
    const int rc = quant_check(X, fmt, dynamic, s_dev, z_dev, out);
    if (rc != CHAM_OK) return rc;
    const bool mx = fmt == CHAM_A_MXFP8_E4M3 || fmt == CHAM_A_MXINT8;
    if (dynamic && !mx && (!ws || ws_bytes < cham_quant_workspace_bytes(out->M * out->K))) return CHAM_EWORKSPACE;
    return quant_launch(X, fmt, dynamic, s_dev, z_dev, out, (float2*)ws, (hipStream_t)stream);
}

extern "C" int cham_quantize_act_lut(const float* X, const cham_lut* lut, const uint8_t* F_host, int32_t layer,
                                     int32_t t, int32_t dynamic, cham_aq* out, void* ws, size_t ws_bytes,
                                     void* stream) {
    if (!lut || !F_host || !lut->S || !lut->Z) return CHAM_EINVAL;
    if (layer < 0 || layer >= lut->L) return CHAM_EINVAL;
    const int32_t b = cham_bucket(t, lut->T, lut->B);
    if (b < 0) return CHAM_EINVAL;
    const int64_t i = (int64_t)layer * lut->B + b;
    const int fmt = F_host[i];
    return cham_quantize_act(X, fmt, dynamic, lut->S + i, lut->Z + i, out, ws, ws_bytes, stream);
}
