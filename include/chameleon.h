/*
 * chameleon.h -- C ABI of the MI355X (gfx950) hot path of Chameleon's per-tensor,
 * format-adaptive post-training quantization (arXiv 2609.33496, "Chameleon: Dynamic Format
 * Adapter for Efficient Diffusion"): the quantized linear layer of a denoiser.
 *
 *   cham_select_weight_formats  offline per-output-channel weight-format search + packing
 *                               (Sec. 4.5, Eq. weight-argmax; palettes of Sec. 4.2)
 *   cham_act_stats_accumulate   calibration power sums and range per (layer, bucket)
 *                               (Sec. 4.4; App. A.7, Alg. 1 first loop)
 *   cham_build_act_lut          kurtosis + SNR routing + ScaleZP -> format/scale/zero LUT
 *                               (Sec. 4.3; App. A.7, Alg. 1 second loop)
 *   cham_quantize_act           activation quantization to the LUT's format, static
 *                               (UNet path, Alg. 2) or dynamic per-tensor (DiT path, Alg. 3)
 *   cham_mixed_linear           Y = dequant(X codes) . dequant(W codes)^T with per-channel
 *                               weight formats (Sec. 6: same-format sub-GEMMs / weights
 *                               dequantized in registers)
 *
 * Conventions shared by every call:
 *   - Every pointer inside a descriptor or passed as a buffer is DEVICE memory unless its
 *     comment says "host".  The caller owns every buffer; the library allocates nothing and
 *     keeps no mutable global state beyond a per-device cache of the CU count (filled once,
 *     atomically) and, for cham_quantize_act_noalloc only, an 8 KB device array per GPU
 *     with its address (see there).  Calls are thread-safe, except that calls of
 *     cham_quantize_act_noalloc that overlap on one GPU share that array.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Every call only enqueues work
 *     on that stream and returns without synchronizing.
 *   - Argument errors are detected on the host and returned synchronously before anything is
 *     enqueued; launch errors are returned as CHAM_EHIP.  No exception crosses the ABI.
 *   - Layouts are row-major.  W is [N][K] (C_out x C_in, as nn.Linear stores it), X is [M][K],
 *     Y is [M][N].  MX blocks are 32 contiguous elements along K; NF4 blocks 64.
 *   - Workspace: calls that take (ws, ws_bytes) need at least cham_workspace_bytes(op, ...)
 *     bytes of device memory aligned to 256 bytes; its contents need not be initialized.
 */
#ifndef CHAMELEON_H_
#define CHAMELEON_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------------------------------
 * status codes
 * ------------------------------------------------------------------------------------- */
#define CHAM_OK 0
#define CHAM_EINVAL (-1)     /* NULL pointer, negative or zero size, bad layer/bucket index  */
#define CHAM_ESHAPE (-2)     /* K not a multiple of 32 (every call) or of 64 (NF4 enabled;
                                mixed_linear), or beyond a call's size limit               */
#define CHAM_EFORMAT (-3)    /* unknown format id, empty or out-of-range palette mask        */
#define CHAM_EHIP (-4)       /* a HIP launch or runtime call failed                          */
#define CHAM_EWORKSPACE (-5) /* ws NULL or smaller than cham_workspace_bytes()               */

/* Human-readable message for a status code (static storage, never NULL). */
const char* cham_status_string(int status);

/* Library version as (major << 16) | (minor << 8) | patch. */
int cham_version(void);

/* ---------------------------------------------------------------------------------------
 * number formats (Sec. 4.2)
 * ------------------------------------------------------------------------------------- */
/* Weight formats, in the paper's palette order F_w^(8) then F_w^(4).  palette_mask bit f
 * enables format f. */
#define CHAM_W_INT8_SYM 0
#define CHAM_W_INT8_ASYM 1
#define CHAM_W_MXINT8 2
#define CHAM_W_INT4_SYM 3
#define CHAM_W_INT4_ASYM 4
#define CHAM_W_NF4 5
#define CHAM_W_FP4 6
#define CHAM_W_MXINT4 7
#define CHAM_W_MXFP4 8
#define CHAM_W_NFMT 9
/* The few-step 4-bit search set {INT4-asym, NF4, FP4, MXINT4, MXFP4} and F_w^(8). */
#define CHAM_MASK_W4 0x1F0u
#define CHAM_MASK_W8 0x007u

/* Activation formats = the runtime LUT codes 0..4. */
#define CHAM_A_INT8_ASYM 0
#define CHAM_A_FP8_E4M3 1
#define CHAM_A_FP8_E5M2 2
#define CHAM_A_MXFP8_E4M3 3
#define CHAM_A_MXINT8 4
#define CHAM_A_NFMT 5

/* ---------------------------------------------------------------------------------------
 * 1. per-output-channel weight-format search (Sec. 4.5, Eq. weight-argmax)
 *
 * For each output channel n, W[n][:] is round-tripped through every enabled format and the
 * format with the smallest sum of squared reconstruction errors (= the largest SQNR; ties go
 * to the lowest id) is kept, with its codes and metadata.  Quantizers (App. A.11, App. A.12):
 *   INT-sym   s = amax/Q (Q = 127, 7), q = clamp(round(w/s), -Q, Q), w^ = q s
 *   INT-asym  App. A.7 ScaleZP on the channel's own [lo, hi]: s = (hi-lo)/L (L = 255, 15),
 *             z = round(-lo/s), not clamped (a one-sided row has z outside [0, L]);
 *             q = clamp(round(w/s) + z, 0, L), w^ = (q - z) s; a constant row (hi == lo)
 *             takes s = |lo| (1 if lo == 0), so z = -sign(lo) and w^ = w
 *   FP4 E2M1  per channel s = amax/6, e = E2M1(clamp(w/s, +-6)), w^ = e s
 *   NF4       per 64-block a = absmax, c = nearest NF4 level to w/a, w^ = v_c a
 *   MXINT8/4  per 32-block E = floor(log2 amax), k = clamp(round(w 2^(F-E)), +-Q),
 *             F = 6 / 2, Q = 127 / 7, w^ = k 2^(E-F)
 *   MXFP4     per 32-block E = floor(log2 amax) - 2 (OCP MX v1.0), e = E2M1(clamp(w/2^E, +-6))
 * "round" is half-to-even, w/s is computed as w * (1/s) in binary32, and every floating
 * scale is floored at FLT_MIN; E8M0 exponents are clamped to [-127, 127] (all-zero block
 * -> -127) and stored biased (E + 127).
 * ------------------------------------------------------------------------------------- */
typedef struct cham_wq {
    int64_t N, K;           /* W is [N][K]; K > 0, even; K % 64 == 0 if NF4 enabled,
                               K % 32 == 0 if any MX format enabled                          */
    uint32_t palette_mask;  /* bit f enables format f; nonzero, bits >= 9 must be clear        */
    int32_t code_bits;      /* 4 if every enabled format is 4-bit, else 8; filled in by
                               cham_select_weight_formats (the caller may leave it 0)        */
    uint8_t* fmt;           /* [N]      chosen format id per channel                          */
    uint8_t* codes;         /* [N][K/2] two 4-bit codes per byte, even k in the low nibble
                               (code_bits 4), or [N][K] one code per byte (code_bits 8).
                               Codes: INT-sym, MXINT two's complement; INT-asym unsigned q;
                               NF4 level index 0..15 (ascending); E2M1 sign|exp(2)|mantissa */
    float* scale;           /* [N]      s of INT-sym/INT-asym/FP4 channels, 0 otherwise       */
    float* zero;            /* [N]      z of INT-asym channels (an integral binary32, any
                               magnitude), 0 otherwise                                        */
    float* nf4_absmax;      /* [N][K/64] block absmax of NF4 channels, 0 otherwise;
                               may be NULL iff NF4 is not enabled                             */
    uint8_t* e8m0;          /* [N][K/32] biased block exponent of MX channels, 0 otherwise;
                               may be NULL iff no MX format is enabled                        */
    int32_t* perm;          /* [N]      channels stably sorted by chosen format; NULL = skip   */
    int32_t* group_off;     /* [10]     start of each format's group in perm, [9] = N;
                               NULL = skip                                                    */
    double* err;            /* [N][9]   per-format error sums (diagnostic, relative accuracy
                               1e-5; -1 for disabled formats); NULL = skip                    */
    void* packed;           /* cham_packed_bytes(N, K) bytes, 256-byte aligned: the weights in
                               the layout cham_mixed_linear consumes (per channel its format
                               parameters; per (64-wide k-step, channel, half) its codes and a
                               16-entry decode table).  Written by the search when non-NULL
                               (K must then be a multiple of 64); cham_mixed_linear reads it
                               instead of deriving it from the codes on every call.  It must
                               come from the search that wrote these codes.  NULL = skip.      */
} cham_wq;

/* Search the formats of W [N][K] (device, binary32, finite) and fill *wq's buffers.
 * Ownership: the caller owns W and every buffer in *wq.  Errors: CHAM_EINVAL (NULL W/wq/
 * required buffer, N < 1), CHAM_EFORMAT (mask), CHAM_ESHAPE (K not a multiple of 32, or of
 * 64 with NF4 enabled, a packed layout requested or K > 8192; K > 32768: a row is held in
 * the registers of one workgroup), CHAM_EHIP. */
int cham_select_weight_formats(const float* W, cham_wq* wq, void* stream);

/* Bytes of the packed GEMM layout of an N x K weight (see cham_wq.packed). */
size_t cham_packed_bytes(int64_t N, int64_t K);

/* The same search for nlayers independent weight matrices (Sec. 4.5 applies per layer):
 * W is a host array of nlayers device pointers, wq a host array of nlayers descriptors,
 * each with its own buffers.  Results are those of nlayers separate calls; layers that
 * share a kernel variant share launches (fewer, fuller launches for a model's layers).
 * Every layer is checked before anything is launched; the first error is returned.
 * Errors: as cham_select_weight_formats, CHAM_EINVAL also for NULL arrays or nlayers < 1. */
int cham_select_weight_formats_batch(const float* const* W, cham_wq* wq, int32_t nlayers, void* stream);

/* The packing step of the search on its own: writes wq[i].packed for n weights whose
 * fmt, codes, scale, zero, NF4 absmax and E8M0 a search (with packed = NULL) has already
 * filled, with code_bits as that search set it; perm, group_off and err are not touched.
 * The layout is the bits the search writes when it packs.  It lets a caller pack one group
 * of layers on another stream while the search of the next group runs.  wq: host array of
 * n descriptors.  Every descriptor is checked before anything is launched.  Errors:
 * CHAM_EINVAL (NULL arrays or buffers, n < 1, packed not 256-byte aligned, code_bits not
 * that of the palette), CHAM_EFORMAT (mask), CHAM_ESHAPE (K not a multiple of 64, or
 * K > 2^20), CHAM_EHIP. */
int cham_pack_weights_batch(const cham_wq* wq, int32_t n, void* stream);

/* ---------------------------------------------------------------------------------------
 * 1b. DiT joint (group size, format) weight search (Sec. 4.6 (i))
 *
 * For one linear layer W [N][K], every tuple (g, f) of the enabled group sizes g (groups of
 * g consecutive input channels along K; the last group holds K mod g when g does not divide
 * K) and enabled formats f is evaluated: each group is quantized with its own parameters as
 * the format's per-channel quantizer above defines them (INT-sym / INT-asym on the group's
 * range, FP4 amax/6, NF4 the group absmax), and the layer's input-aware error
 * sum_n sum_k energy[k] (w - w^)^2 (energy[k] = E[x_k^2], the activation energy of input
 * channel k) is formed in binary64.  The tuple with the smallest error (= the largest
 * input-aware SQNR) is chosen, ties to the lowest index t = group index * 9 + format; MX
 * formats use their own 32-blocks and are evaluated at g = 32 only.  The choice stays on
 * the device (choice[]), so no synchronization is needed before the GEMM.
 * ------------------------------------------------------------------------------------- */
#define CHAM_NGROUPS 5          /* group sizes 32, 64, 128, 192, 288 (bit i of group_mask)  */
#define CHAM_GMASK_ALL 0x1Fu
/* The DiT fork's 4-bit search set {INT4-asym, NF4, FP4}; at 8 bits F_w^(8). */
#define CHAM_MASK_DIT_W4 0x070u

typedef struct cham_gwq {
    int64_t N, K;           /* W is [N][K]; K % 32 == 0, K <= 8192                           */
    uint32_t palette_mask;  /* formats searched (bit f = format f)                            */
    uint32_t group_mask;    /* group sizes searched (bit i = the i-th size); nonzero          */
    int32_t code_bits;      /* 4 if every enabled format is 4-bit, else 8 (set by the search) */
    int32_t* choice;        /* [2] device: the chosen group size and format id                */
    uint8_t* fmt;           /* [N]      the chosen format id in every entry                   */
    uint8_t* codes;         /* [N][K/2] (4-bit) or [N][K] (8-bit), as in cham_wq              */
    float* gscale;          /* [N][K/32] per group j (at index j): INT scale, FP4 scale or NF4
                               absmax; 0 past the last group and for MX formats               */
    float* gzero;           /* [N][K/32] per group: INT-asym zero point (integral), else 0    */
    uint8_t* e8m0;          /* [N][K/32] MX block exponents (0 unless an MX format is chosen);
                               may be NULL iff no MX format is enabled                        */
    double* err;            /* [45]     layer error of tuple t (-1 if not evaluated); NULL = skip */
    void* packed;           /* cham_packed_bytes(N, K) bytes, 256-byte aligned: the GEMM
                               layout, written by the search when non-NULL (4-bit palettes and
                               K % 64 == 0 only); NULL = skip                                  */
} cham_gwq;

/* Search W [N][K] (device, binary32, finite, 16-byte aligned) with error weights energy[K]
 * (device, binary32, 16-byte aligned) and fill *gq.  ws: CHAM_OP_GSELECT bytes (the
 * per-channel errors).  Errors: CHAM_EINVAL (NULL or misaligned buffer, N < 1), CHAM_EFORMAT
 * (masks; only MX formats without g = 32), CHAM_ESHAPE (K, or packing with 8-bit codes),
 * CHAM_EWORKSPACE, CHAM_EHIP. */
int cham_select_group_formats(const float* W, const float* energy, cham_gwq* gq, void* ws, size_t ws_bytes,
                              void* stream);

/* Calibration pre-pass of the search's weights: colsq[k] += sum_m X[m][k]^2 over X [M][K]
 * (device binary32; colsq device binary64 [K]), summed in a fixed order (bitwise
 * reproducible); E[x_k^2] = colsq[k] / rows.  ws: CHAM_OP_COLSQ bytes.
 * Errors: CHAM_EINVAL, CHAM_EWORKSPACE, CHAM_EHIP. */
int cham_act_colsq_accumulate(const float* X, int64_t M, int64_t K, double* colsq, void* ws, size_t ws_bytes,
                              void* stream);

/* ---------------------------------------------------------------------------------------
 * 2. calibration statistics (Sec. 4.4; Alg. 1) and the LUT (Sec. 4.3; Alg. 1)
 * ------------------------------------------------------------------------------------- */
typedef struct cham_act_stats {
    int32_t L, B;  /* layers, timestep buckets                                            */
    double* nS;    /* [L*B][5] n, sum x, sum x^2, sum x^3, sum x^4 (binary64)               */
    float* lohi;   /* [L*B][2] running min, max (binary32)                                 */
} cham_act_stats;

/* Set every accumulator to n = S_k = 0, lo = +inf, hi = -inf. */
int cham_act_stats_reset(cham_act_stats* st, void* stream);

/* Add one activation tensor X (numel binary32 values, device, 16-byte aligned) of `layer` at a timestep of
 * `bucket` into the accumulator: n += numel, S_k += sum x^k, lo/hi = min/max.  The sums are
 * reduced in a fixed order (bitwise reproducible run to run).  ws: CHAM_OP_STATS bytes.
 * Errors: CHAM_EINVAL (NULL, numel < 1, layer/bucket out of range), CHAM_EWORKSPACE, CHAM_EHIP. */
int cham_act_stats_accumulate(const float* X, int64_t numel, int32_t layer, int32_t bucket,
                              cham_act_stats* st, void* ws, size_t ws_bytes, void* stream);

/* The same for n tensors X[i] (host array of device pointers) of (layer[i], bucket[i]),
 * e.g. every instrumented layer's input of one calibration forward pass: the result is
 * bitwise that of n calls in array order (tensors of the same (layer, bucket) are added in
 * that order), in fewer launches.  numel, layer, bucket: host arrays of n.  ws: the sum of
 * cham_workspace_bytes(CHAM_OP_STATS, numel[i], 0, 0) over i.  Every argument is checked
 * before anything is launched.  Errors: as cham_act_stats_accumulate. */
int cham_act_stats_accumulate_batch(const float* const* X, const int64_t* numel, const int32_t* layer,
                                    const int32_t* bucket, int32_t n, cham_act_stats* st, void* ws,
                                    size_t ws_bytes, void* stream);

#define CHAM_SCHED_SCALED_LINEAR 0
#define CHAM_SCHED_LINEAR 1
typedef struct cham_schedule {
    int32_t T;                   /* diffusion steps (betas indexed 0..T-1)                    */
    double beta0, beta1;         /* first and last beta                                        */
    int32_t kind;                /* CHAM_SCHED_SCALED_LINEAR: (sqrt(b0)+(sqrt(b1)-sqrt(b0))s/(T-1))^2
                                    CHAM_SCHED_LINEAR:        b0 + (b1-b0) s/(T-1)             */
    double kappa_lo, kappa_hi;   /* kurtosis gates (3, 5)                                      */
    double snr_lo, snr_hi;       /* SNR gates (0.2, 2.0)                                       */
    int32_t snr_gate_on;         /* 0 routes by kurtosis alone                                 */
} cham_schedule;

/* SDXL's scaled-linear schedule 0.00085 -> 0.012, T = 1000, gates (3, 5, 0.2, 2.0), on. */
void cham_schedule_default(cham_schedule* s);

typedef struct cham_lut {
    int32_t L, B, T;  /* layers, buckets, schedule length                                  */
    uint8_t* F;       /* [L*B] format code 0..4                                             */
    float* S;         /* [L*B] scale                                                        */
    float* Z;         /* [L*B] zero point (integral, binary32)                              */
} cham_lut;

/* For every (l, b): kappa = m4/m2^2 from the power sums; SNR at the bucket midpoint
 * t_b = floor(b T/B + T/(2B)) with alpha_bar_t = prod_{s<=t} (1 - beta_s) and
 * SNR = alpha_bar/(1 - alpha_bar) (Sec. 3.1, Eq. snr); Route (Sec. 4.3): shortcut -> 3,
 * kappa > hi or SNR < lo -> 2, kappa <= lo and SNR > hi -> 0, else 1; ScaleZP (App. A.7) on
 * the bucket's [lo, hi] (an empty bucket gets S = 1, Z = 0).  is_shortcut: device [L] or
 * NULL.  kappa: device [L*B] binary64 or NULL.  lut->L, B must equal st's (B <= 1024); lut->T
 * is set to sch->T.  The SNR product is evaluated as a tree of binary64 products.
 * Errors: CHAM_EINVAL, CHAM_EHIP. */
int cham_build_act_lut(const cham_act_stats* st, const cham_schedule* sch,
                       const uint8_t* is_shortcut, cham_lut* lut, double* kappa, void* stream);

/* Bucket of timestep t (Alg. 2): min(floor(t B / T), B - 1); -1 if t < 0 or T, B < 1. */
int32_t cham_bucket(int32_t t, int32_t T, int32_t B);

/* ---------------------------------------------------------------------------------------
 * 3. activation quantization (Alg. 2 static / Alg. 3 dynamic)
 * ------------------------------------------------------------------------------------- */
typedef struct cham_aq {
    int64_t M, K;      /* X is [M][K]                                                        */
    int32_t fmt;       /* activation format used (filled in by the quantize call)             */
    int32_t nsamples;  /* S >= 1 samples of M/S consecutive rows each (M % S == 0), e.g. the
                          two halves of a CFG-doubled batch; each has its own (s, z)          */
    uint8_t* codes;    /* [M][K] INT8-asym unsigned q, FP8 / MXFP8 codes, MXINT8 two's compl. */
    uint8_t* e8m0;     /* [M][K/32] biased block exponents (MX formats; may be NULL otherwise)*/
    float* scale;      /* [S] the scale s of each sample (1 for MX formats)                   */
    float* zero;       /* [S] the zero point z of each sample (0 unless INT8-asym)            */
} cham_aq;

/* Quantize X [M][K] (device, finite binary32, 16-byte aligned; out->codes 4-byte aligned)
 * to activation format `fmt`:
 *   INT8-asym  q = clamp(round(x/s) + z, 0, 255); dynamic (s, z) by ScaleZP on this X's own
 *              [lo, hi] (App. A.7: s = (hi-lo)/255, z = round(-lo/s), z not clamped)
 *   FP8        e = E4M3 / E5M2(clamp(x/s, +-448 / +-57344)), round to nearest even
 *   MXFP8      per 32-block E = floor(log2 amax) (the paper's exponent: values in (-2, 2)),
 *              e = E4M3(x / 2^E)
 *   MXINT8     per 32-block E = floor(log2 amax), k = clamp(round(x 2^(6-E)), +-127)
 * Static (dynamic = 0): s = *s_dev, z = *z_dev (device pointers, e.g. LUT entries), the same
 * for every sample.  Dynamic (dynamic = 1, Alg. 3's per-sample, per-forward micro-scaling):
 * each of the out->nsamples samples takes (s, z) = ScaleZP(fmt, min, max) of its own rows
 * (one sample = per-tensor); s_dev/z_dev are ignored.  The (s, z) used are written to
 * out->scale[S] / out->zero[S].  1 <= nsamples <= 1024.  ws: CHAM_OP_QUANT_ACT
 * bytes.  Errors: CHAM_EINVAL, CHAM_EFORMAT, CHAM_ESHAPE (K % 32 for MX), CHAM_EWORKSPACE,
 * CHAM_EHIP. */
int cham_quantize_act(const float* X, int32_t fmt, int32_t dynamic, const float* s_dev,
                      const float* z_dev, cham_aq* out, void* ws, size_t ws_bytes, void* stream);

/* cham_quantize_act without a workspace argument, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, results and errors as cham_quantize_act; it calls no
 * allocating routine.  The dynamic min/max partials live in an 8 KB array of device memory
 * that the library holds on each GPU it runs on until the process ends; it is large enough
 * for every size this call accepts (the launch caps its partials at 1024).  All calls on one
 * GPU share that array: calls that overlap on one GPU (different streams, other threads)
 * race and must be ordered by the caller.  Errors: as cham_quantize_act (without
 * CHAM_EWORKSPACE); CHAM_EHIP also if the array's address cannot be obtained. */
int cham_quantize_act_noalloc(const float* X, int32_t fmt, int32_t dynamic, const float* s_dev,
                              const float* z_dev, cham_aq* out, void* stream);

/* The per-step runtime lookup of Alg. 2 / Alg. 3: b = cham_bucket(t, lut->T, lut->B), the
 * format is F_host[layer*B + b] (a host mirror of lut->F, copied once after calibration, so
 * no device synchronization is needed per step), and the scale/zero are read on the device
 * from lut->S/Z[layer*B + b] (static) or computed from X (dynamic). */
int cham_quantize_act_lut(const float* X, const cham_lut* lut, const uint8_t* F_host,
                          int32_t layer, int32_t t, int32_t dynamic, cham_aq* out, void* ws,
                          size_t ws_bytes, void* stream);

/* Alg. 2's runtime quantization and Alg. 1's moment gathering in one pass over each input,
 * for a model that keeps calibrating while it runs: tensor X[i] (out[i].M x out[i].K
 * binary32, device, 16-byte aligned) of layer[i] at timestep t is quantized as
 * cham_quantize_act_lut(X[i], lut, F_host, layer[i], t, 0, &out[i], ...) would do it
 * (static scales: the LUT's S/Z of (layer[i], b), b = cham_bucket(t, lut->T, lut->B), as
 * the device holds them when the kernel runs), and its moments are added into st at
 * (layer[i], b) as cham_act_stats_accumulate_batch adds them.  Codes, E8M0 bytes, scales,
 * zero points and accumulators are the bits those two calls give, in that order, on the
 * same inputs.  A LUT built afterwards from st sees this call's moments; the codes of this
 * call do not depend on them.  out: host array of n descriptors (fmt is filled in from
 * F_host).  layer: host array of n.  st->L, B must equal lut's.  ws: the sum of
 * cham_workspace_bytes(CHAM_OP_STATS, out[i].M * out[i].K, 0, 0) over i.  Every argument is
 * checked before anything is launched.  Errors: CHAM_EINVAL, CHAM_EFORMAT, CHAM_ESHAPE
 * (K % 32), CHAM_EWORKSPACE, CHAM_EHIP. */
int cham_quantize_act_lut_accumulate_batch(const float* const* X, const int32_t* layer, int32_t n, int32_t t,
                                           const cham_lut* lut, const uint8_t* F_host, cham_aq* out,
                                           cham_act_stats* st, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------------------
 * 4. the mixed-format linear layer
 *
 * Y[m][n] = sum_k x^[m][k] w^[n][k], with x^ = DQ(xq) and w^ = DQ(wq) exactly as the
 * quantizers above define them, accumulated in binary32 on the matrix cores.  Accuracy:
 * |Y - Y_exact| <= 1e-3 * sum_k |x^ w^| per element.  Operands are decoded to half
 * precision: NF4 levels times their block absmax, and INT-asym weight levels q - z beyond
 * 2^11 in magnitude, carry one rounding (relative 2^-11; INT8-asym channels with |z| beyond
 * 2^22, whose values agree to 6e-5, up to 2^-10); INT8-asym activations are decoded
 * exactly, a zero point beyond +-1024 through a per-channel correction (the channel's sum of
 * dequantized weights, binary64, times (z - z') s in the epilogue).  Block-scaled operands
 * (NF4 and MX weights, MX activations) are held relative to the largest block of their
 * channel or row: blocks within 2^28 of it are exact (NF4: one rounding), blocks further
 * below fall into half precision's subnormal range and lose bits.  xq->K must equal wq->K and be a multiple of
 * 64; the kernels address operands with 32-bit offsets, so K <= 2^20, N < 2^21 and the
 * weights' decode layout (cham_packed_bytes) stays below 2^31 bytes (CHAM_ESHAPE otherwise);
 * xq->codes, wq->codes and Y must be 16-byte aligned.  Y [M][N] is written in the
 * original channel order.  When the output has too few tiles to fill the GPU, K is split
 * across workgroups whose partial outputs a second kernel adds in split order; no atomics
 * are used, so Y is bitwise reproducible run to run.  If wq->packed is set it supplies the
 * weights' decode layout; otherwise a pre-pass derives it from the codes and metadata into
 * the workspace.  ws: what cham_mixed_linear_workspace_query reports for these operands
 * (a half-precision copy of MX activations and their row scales, the weights' decode layout
 * when wq->packed is NULL, the k-split partial outputs when the plan splits; possibly 0,
 * then ws may be NULL), 256-byte aligned; CHAM_OP_LINEAR bytes always suffice.
 * Errors: CHAM_EINVAL, CHAM_EFORMAT, CHAM_ESHAPE, CHAM_EWORKSPACE, CHAM_EHIP.
 * ------------------------------------------------------------------------------------- */
int cham_mixed_linear(const cham_aq* xq, const cham_wq* wq, float* Y, void* ws, size_t ws_bytes,
                      void* stream);

/* Exact workspace bytes of cham_mixed_linear for these operands (host only: reads the
 * descriptors, launches nothing, dereferences no device pointer) into *bytes (host).
 * Errors: those of cham_mixed_linear's argument checks (CHAM_EINVAL, CHAM_EFORMAT,
 * CHAM_ESHAPE), and CHAM_EINVAL for a NULL bytes. */
int cham_mixed_linear_workspace_query(const cham_aq* xq, const cham_wq* wq, size_t* bytes);

/* The same linear layer with group-scaled weights from cham_select_group_formats (the DiT
 * path, Sec. 4.6 (i)): each 32-element half of a 64-wide k-step lies in one group (every
 * group size is a multiple of 32), whose scale and zero point build its decode table;
 * accuracy as above.  4-bit palettes only (gq->code_bits == 4; the 8-bit group-scaled
 * decode is not built: CHAM_EFORMAT).  ws: as cham_mixed_linear (exact bytes from
 * cham_mixed_linear_grouped_workspace_query; CHAM_OP_LINEAR bytes always suffice). */
int cham_mixed_linear_grouped(const cham_aq* xq, const cham_gwq* gq, float* Y, void* ws, size_t ws_bytes,
                              void* stream);

/* Exact workspace bytes of cham_mixed_linear_grouped (as cham_mixed_linear_workspace_query). */
int cham_mixed_linear_grouped_workspace_query(const cham_aq* xq, const cham_gwq* gq, size_t* bytes);

/* The UNet path's 3x3 convolution (stride 1, zero padding 1) on quantized activations, as
 * an implicit GEMM on the same kernels: the layers downstream of a shortcut concatenation
 * (up-block resnet conv1) whose inputs Sec. 4.6 routes to MXFP8 whatever the LUT's gates
 * say (cham_build_act_lut's is_shortcut).  xq: the activation codes of B images of H x W
 * pixels with C channels, channels last (xq->M = B H W rows, xq->K = C, C % 64 == 0; its
 * samples are 1 or B images).  wq: the weights as a linear layer [Co][9 C] with
 * k = (ky * 3 + kx) * C + c (searched like any linear weight).  Y [B H W][Co] (device,
 * binary32): Y[b,y,x][o] = sum over ky, kx, c of x^[b, y+ky-1, x+kx-1, c] w^[o, k],
 * out-of-image pixels zero.  A pre-pass writes the zero-padded activation in half
 * precision (MX formats relative to the tensor's largest block exponent: exact for blocks
 * within 2^28 of it; INT8-asym q - z rounded once when beyond 2^11) that the GEMM gathers
 * per output pixel and tap; accuracy as cham_mixed_linear.  ws: cham_conv3x3_workspace_bytes.
 * Errors: CHAM_EINVAL (sizes, pointers, samples), CHAM_EFORMAT, CHAM_ESHAPE (C % 64, the
 * padded copy beyond 2^31 bytes), CHAM_EWORKSPACE, CHAM_EHIP. */
int cham_conv3x3_mixed(const cham_aq* xq, int32_t B, int32_t H, int32_t W, const cham_wq* wq, float* Y,
                       void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes of cham_conv3x3_mixed for B images of H x W x C and Co output channels
 * (0 for sizes out of range). */
size_t cham_conv3x3_workspace_bytes(int64_t B, int64_t H, int64_t W, int64_t C, int64_t Co);

/* The launch plan cham_mixed_linear takes for M x N x K with 4- or 8-bit weight codes
 * (diagnostics; host only, launches nothing).  out (host, out_len >= 10 int32) receives
 * {launches (1 or 2), k-splits, then per launch: first row, end row, tile rows, tile
 * channels}; entries of an absent second launch are 0.  The plan depends on the current
 * device's CU count (256 when no device is visible).  Errors: CHAM_EINVAL (NULL out,
 * out_len < 10, sizes < 1, code_bits not 4 or 8). */
int cham_linear_plan(int64_t M, int64_t N, int64_t K, int32_t code_bits, int32_t* out, int32_t out_len);

/* ---------------------------------------------------------------------------------------
 * workspace sizes
 * ------------------------------------------------------------------------------------- */
#define CHAM_OP_SELECT 0
#define CHAM_OP_STATS 1
#define CHAM_OP_QUANT_ACT 2
#define CHAM_OP_LINEAR 3
#define CHAM_OP_GSELECT 4   /* cham_select_group_formats: N output channels              */
#define CHAM_OP_COLSQ 5     /* cham_act_colsq_accumulate: K input channels               */
/* Bytes of workspace op needs at these sizes (M rows of X -- numel for CHAM_OP_STATS --,
 * N output channels, K inner size).  0 means no workspace. */
size_t cham_workspace_bytes(int32_t op, int64_t M, int64_t N, int64_t K);

#ifdef __cplusplus
}
#endif
#endif /* CHAMELEON_H_ */
