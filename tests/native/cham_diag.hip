// Diagnostic kernels for the test-suite only (built into tests/native/_build, never into the
// library): the library's correctly rounded reciprocal, rcp_rn, checked against the IEEE
// binary32 quotient 1/a over every input it can receive, and evaluated on given inputs so
// the host can compare it with an independent CPU reciprocal.
#include "../../paper_2609_33496_amd/csrc/cham_device.h"

namespace {

// Every binary32 bit pattern in [lo, hi): count the inputs where rcp_rn(a) and 1.0f / a
// (correctly rounded division) differ in any bit; out[1] keeps the smallest such pattern.
__global__ __launch_bounds__(256) void rcp_sweep_kernel(uint32_t lo, uint32_t hi, uint32_t* out) {
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    uint32_t bad = 0, first = 0xFFFFFFFFu;
    for (uint64_t b = (uint64_t)lo + (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; b < hi; b += stride) {
        const float a = __uint_as_float((uint32_t)b);
        const float r = cham::rcp_rn(a), q = 1.0f / a;
        if (__float_as_uint(r) != __float_as_uint(q)) {
            ++bad;
            first = min(first, (uint32_t)b);
        }
    }
    if (bad) {
        atomicAdd(&out[0], bad);
        atomicMin(&out[1], first);
    }
}

__global__ __launch_bounds__(256) void rcp_values_kernel(const float* a, float* r, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) r[i] = cham::rcp_rn(a[i]);
}

}  // namespace

// out: device [2] u32, set by the caller to {0, 0xFFFFFFFF} before the call.
extern "C" int cham_diag_rcp_sweep(uint32_t lo_bits, uint32_t hi_bits, uint32_t* out, void* stream) {
    if (!out || lo_bits >= hi_bits || hi_bits > 0x7F800000u || lo_bits < 0x00800000u) return CHAM_EINVAL;
    hipLaunchKernelGGL(rcp_sweep_kernel, dim3(4096), dim3(256), 0, (hipStream_t)stream, lo_bits, hi_bits, out);
    return hipGetLastError() == hipSuccess ? CHAM_OK : CHAM_EHIP;
}

// r[i] = rcp_rn(a[i]) for n inputs a[i] >= FLT_MIN (device arrays).
extern "C" int cham_diag_rcp_values(const float* a, float* r, int64_t n, void* stream) {
    if (!a || !r || n < 1) return CHAM_EINVAL;
    const int64_t blocks = (n + 255) / 256 < 8192 ? (n + 255) / 256 : 8192;
    hipLaunchKernelGGL(rcp_values_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, a, r, n);
    return hipGetLastError() == hipSuccess ? CHAM_OK : CHAM_EHIP;
}
