// Host-side parts of the C ABI that are not tied to one kernel: status strings, version,
// workspace sizes.
#include "cham_device.h"

size_t cham_stats_workspace_bytes(int64_t numel);
size_t cham_quant_workspace_bytes(int64_t n);
size_t cham_linear_workspace_bytes(int64_t M, int64_t N, int64_t K);
size_t cham_gselect_workspace_bytes(int64_t N);
size_t cham_colsq_workspace_bytes(int64_t K);

extern "C" const char* cham_status_string(int status) {
    switch (status) {
    case CHAM_OK: return "ok";
    case CHAM_EINVAL: return "invalid argument (NULL pointer, size or index out of range, misaligned buffer)";
    case CHAM_ESHAPE: return "unsupported shape (K must be a multiple of 32; of 64 when NF4 is enabled and for mixed_linear; for the weight search at most 32768, beyond 8192 a multiple of 64; at most 8192 for the group search)";
    case CHAM_EFORMAT: return "unknown format id or bad palette mask";
    case CHAM_EHIP: return "HIP launch or runtime error";
    case CHAM_EWORKSPACE: return "workspace missing or too small";
    default: return "unknown status";
    }
}

extern "C" int cham_version(void) { return (0 << 16) | (1 << 8) | 0; }

extern "C" size_t cham_workspace_bytes(int32_t op, int64_t M, int64_t N, int64_t K) {
    (void)N;
    switch (op) {
    case CHAM_OP_SELECT: return 0;
    case CHAM_OP_STATS: return M > 0 ? cham_stats_workspace_bytes(M) : 0;
    case CHAM_OP_QUANT_ACT: return (M > 0 && K > 0) ? cham_quant_workspace_bytes(M * K) : 0;
    case CHAM_OP_LINEAR: return (M > 0 && N > 0 && K > 0) ? cham_linear_workspace_bytes(M, N, K) : 0;
    case CHAM_OP_GSELECT: return cham_gselect_workspace_bytes(N);
    case CHAM_OP_COLSQ: return cham_colsq_workspace_bytes(K);
    default: return 0;
    }
}
