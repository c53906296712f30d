/*
 * logbq.h -- C ABI of liblogbq, LogbQuant weight-only inference (4-bit and 8-bit codes) on AMD
 * MI355X (gfx950).
 *
 * LogbQuant (Bohn et al., arXiv 2607.01127) quantizes each weight matrix with its own
 * logarithmic codebook of base b and shift s (Sec. 3.1): a weight x maps to the integer
 * q = sign(x) * round(log_b|x| + s) with |q| <= q_max = 2^(n-1) - 1 (Eq. 1), and q decodes to
 * sign(q) * b^(|q| - s), or 0 for q = 0 (Eq. 2). b and s come from the effective weight range
 * [w_min, w_max] (Eq. 3, Eq. 4); w_min discards a fraction eps of the signal energy (Eq. 5).
 * Inference dequantizes through a lookup table instead of evaluating b^x (Sec. 3.3).
 *
 * Conventions shared by every call
 *   - Every call validates all of its arguments before it touches the GPU, and returns a
 *     logbq_status. No device memory is allocated inside a call. Device calls are enqueued on
 *     the given stream and return at once, so they can be captured in a HIP graph; the one
 *     exception is logbq_fit_device, which waits for each of its passes because the host
 *     chooses the next pass's bin. Faults of an enqueued kernel surface at the caller's next
 *     synchronisation.
 *   - `stream` is a hipStream_t passed as void*; NULL is the default stream.
 *   - The caller owns every buffer. "device" pointers are HIP device memory of the current
 *     device; "host" pointers are ordinary host memory.
 *   - Weights are row-major [N][K] (N out features, K in features, as a PyTorch Linear).
 *   - 4-bit codes: row-major [N][K/2] bytes; element (n, k) is the nibble at byte
 *     n*K/2 + k/2, the low nibble when k is even. A nibble is sign<<3 | magnitude: bit 3 set
 *     means negative, magnitude 0..7 is |q|. Code 8 ("-0") is never written and decodes to +0.
 *   - 8-bit codes: row-major [N][K] bytes, one code per weight: sign<<7 | magnitude (0..127).
 *     Code 128 ("-0") is never written and decodes to +0.
 *   - Shapes: K must be a multiple of 32 (every packed row is then 16-byte aligned);
 *     device pointers must be 16-byte aligned. N = 0 or M = 0 is a valid empty call.
 */
#ifndef LOGBQ_H
#define LOGBQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LOGBQ_ABI_VERSION 2

typedef enum logbq_status {
  LOGBQ_OK = 0,
  LOGBQ_ERR_INVALID_ARG = 1,   /* null pointer, negative size, eps outside (0,1), ... */
  LOGBQ_ERR_NONFINITE = 2,     /* fit: a weight is NaN or Inf                           */
  LOGBQ_ERR_DEGENERATE = 3,    /* fit: all weights zero, or w_min == w_max (b = 1)      */
  LOGBQ_ERR_UNSUPPORTED = 4,   /* bits not 4 or 8, K % 32 != 0, misaligned, too large    */
  LOGBQ_ERR_HIP = 5,           /* a HIP call failed (no device, launch failure, ...)    */
  LOGBQ_ERR_HOST_RESOURCE = 6  /* host scratch memory could not be allocated              */
} logbq_status;

/* Per-tensor codebook parameters (Sec. 3.1, Sec. 3.2). Plain data; copy freely.
 * ABI version 2 widened codebook and thresholds for 8-bit codes (version 1 had 16 and 8). */
typedef struct logbq_params {
  int32_t bits;            /* codebook bit width n: 4 or 8                                 */
  int32_t qmax;            /* q_max = 2^(n-1) - 1                                          */
  double eps;              /* pruned energy fraction of Eq. 5                               */
  double wmin;             /* w_min of Eq. 5                                                */
  double wmax;             /* w_max = max |w| (Sec. 3.2)                                    */
  double base;             /* b of Eq. 3                                                    */
  int32_t shift;           /* s of Eq. 4 (an integer)                                       */
  int32_t reserved;
  int64_t wmin_index;      /* position of w_min in |w| sorted ascending                     */
  float codebook[256];     /* Dequant (Eq. 2) of every n-bit code, float32; entries from
                              2^n on are 0                                                  */
  float thresholds[128];   /* [k] = smallest float32 whose magnitude index exceeds k,
                              k = 0..qmax-1; entries from qmax on are +inf                  */
} logbq_params;

/* Per-tensor parameters of the comparison baseline: asymmetric linear quantization,
 * Quant(s, z, x) = round(x / s) - z (Sec. 2), at tensor granularity (Sec. 4). Plain data.
 * s = (max w - min w) / (2^n - 1) and z = round(min w / s), ties rounded up; code q in
 * 0 .. 2^n - 1 stands for s (q + z). Only n = 4 is provided. */
typedef struct logbq_uniform {
  int32_t bits;            /* 4                                                            */
  int32_t zero;            /* z                                                            */
  double wmin;             /* min w (signed)                                               */
  double wmax;             /* max w (signed)                                               */
  double scale;            /* s                                                            */
  float codebook[16];      /* s (q + z) rounded to float32: the codebook logbq_linear and
                              logbq_dequantize take for these codes                        */
  float thresholds[15];    /* [j - 1] = smallest float32 x whose code is at least j (+inf
                              if none), j = 1 .. 15                                          */
  float reserved;
} logbq_uniform;

/* ABI version of the loaded library (LOGBQ_ABI_VERSION it was built with). */
int32_t logbq_abi_version(void);

/* Static English name of a status code; never NULL. */
const char* logbq_status_str(int32_t status);

/*
 * logbq_fit -- per-tensor codebook parameters (Sec. 3.1 Eq. 3-4, Sec. 3.2 Eq. 5). Host only.
 *   w_host : host, numel float32 weights, read only.
 *   bits   : codebook width n, 4 or 8.
 *   eps    : pruned energy fraction, 0 < eps < 1 (the paper uses 4e-3 at 4 bits, 1e-6 at 8).
 *   out    : host, filled on success; untouched on error.
 * w_max = max|w|. w_min is the smallest |w_i| at which the ascending float64 prefix sum of
 * w^2, divided by the total, reaches eps (sequential summation in ascending |w| order).
 * b = (w_max / w_min)^(1/q_max); s = q_max - J with J the largest integer such that
 * b^J <= w_max. codebook[k] = float32(b^(k-s)), codebook[h+k] = -codebook[k] (h = 2^(n-1),
 * k = 1..q_max), codebook[0] = codebook[h] = +0. thresholds[k] is exact: the smallest float32
 * t with t >= b^(k + 1/2 - s).
 * Errors: INVALID_ARG (null, numel < 2, eps outside (0,1)), UNSUPPORTED (bits not 4 or 8),
 * NONFINITE (NaN/Inf weight), DEGENERATE (w_max == 0, or w_min == w_max), HOST_RESOURCE (the
 * host scratch could not be allocated).
 * Reentrant; allocates host scratch of 8*numel bytes internally for the sort, which runs on up
 * to 16 threads (LOGBQ_HOST_THREADS = 1..16 in the environment sets the count; the result does
 * not depend on it; if no thread can be started the sort runs on the calling thread).
 */
int32_t logbq_fit(const float* w_host, int64_t numel, int32_t bits, double eps,
                  logbq_params* out);

/* Bytes of device workspace logbq_fit_device needs. */
#define LOGBQ_FIT_WORKSPACE_BYTES 110600

/*
 * logbq_fit_device -- the per-tensor fit on device-resident weights (Sec. 3.1 Eq. 3-4,
 * Sec. 3.2 Eq. 5), with the energy sums of Eq. 5 taken exactly.
 *   w_dev        : device, numel float32 weights, 16-byte aligned, read only.
 *   numel        : 2 <= numel < 2^40.
 *   bits, eps    : as logbq_fit.
 *   workspace_dev: device, LOGBQ_FIT_WORKSPACE_BYTES bytes, 8-byte aligned, owned by the
 *                  caller; overwritten.
 *   out          : host, filled on success; untouched on error.
 *   stream       : hipStream_t the passes run on.
 * w_max = max|w|. w_min = |w| at the smallest position i of |w| sorted ascending (ties in any
 * order) with sum_{j <= i} w_j^2 >= eps * sum_j w_j^2, both sums exact (squares of float32
 * values are exact rationals); wmin_index = i. b, s, codebook and thresholds then follow
 * exactly as in logbq_fit. logbq_fit sums in float64, in sequence; the two agree unless the
 * exact ratio lies within float64 rounding of eps.
 * Three radix-selection passes over the weights (bits 30..20, 19..11, 10..0 of the float32
 * pattern of |w|) accumulate per-bin counts and exact integer energy sums on the device; the
 * host picks each pass's bin with exact integer arithmetic. Blocks the calling thread until
 * the stream has run the passes (not capturable in a HIP graph).
 * Errors: INVALID_ARG (null, numel < 2, eps outside (0,1)), UNSUPPORTED (bits not 4 or 8,
 * numel too large, misaligned), NONFINITE (NaN/Inf weight), DEGENERATE (w_max == 0 or
 * w_min == w_max), HIP (a HIP call failed), HOST_RESOURCE (host copies of the bins could not
 * be allocated).
 */
int32_t logbq_fit_device(const float* w_dev, int64_t numel, int32_t bits, double eps,
                         void* workspace_dev, logbq_params* out, void* stream);

/*
 * logbq_fit_exact -- logbq_fit_device's fit on host weights: the same three radix-selection
 * passes, run on the host, and the same exact selection, so the parameters equal
 * logbq_fit_device's bit for bit (Sec. 3.2 Eq. 5 with exact sums, Sec. 3.1 Eq. 3-4).
 *   w_host, numel, bits, eps, out: as logbq_fit (2 <= numel < 2^40).
 * Errors: as logbq_fit (HOST_RESOURCE included). Reentrant; allocates at most 48 KiB of host
 * scratch.
 */
int32_t logbq_fit_exact(const float* w_host, int64_t numel, int32_t bits, double eps,
                        logbq_params* out);

/*
 * logbq_encode -- Quant (Eq. 1) of a weight matrix into 4-bit or 8-bit codes (Sec. 3.3 packing).
 *   w_dev        : device, [n][k] float32 weights.
 *   n, k         : shape; k % 32 == 0.
 *   p            : host, parameters from logbq_fit (bits 4 or 8).
 *   codes_dev    : device, written: [n][k/2] bytes for 4 bits, [n][k] for 8 bits.
 *   codebook_out : host, 2^bits floats, receives p->codebook[0 .. 2^bits) (may be NULL).
 *   stream       : hipStream_t or NULL.
 * The magnitude index of x is the number of thresholds t with |x| >= t, which equals
 * clamp(round-half-up(log_b|x| + s), 0, q_max); the sign bit (bit n-1) is set for negative x
 * with a nonzero magnitude. NaN and +-0 encode to 0, +-Inf to the largest magnitude with its
 * sign.
 * Errors: INVALID_ARG (null, negative size, qmax not 2^(bits-1) - 1, thresholds[0..qmax)
 * not positive and ascending), UNSUPPORTED (bits, k % 32, alignment), HIP (launch failure).
 */
int32_t logbq_encode(const float* w_dev, int64_t n, int64_t k, const logbq_params* p,
                     uint8_t* codes_dev, float* codebook_out, void* stream);

/*
 * logbq_linear -- y = x . W_hat^T on packed codes: weight-only inference with the codebook
 * lookup fused into the product (Sec. 3.3).
 *   x_dev     : device, [m][k] IEEE float16 activations (bit patterns as uint16).
 *   m, k      : batch rows and in features; k % 32 == 0, m <= 4194240 (65535 * 64).
 *   codes_dev : device, [n][k/2] packed codes.
 *   n         : out features.
 *   codebook  : host, 16 floats (logbq_params.codebook); copied into the kernel arguments,
 *               so the call is capturable in a HIP graph. Entries are rounded to float16 after
 *               a common power-of-two scaling, exact in the result up to float16 rounding.
 *   y_dev     : device, [m][n] float32, written.
 * Accumulation is float32. Four kernels, chosen from (m, k, n) alone: for 2 <= m <= 32 and
 * k in {1024, 2048, 4096, 8192} (and m <= 16 at k = 14336; there, as above m = 16, only for
 * sign-symmetric codebooks), a split-K
 * dequantize-into-MFMA kernel takes 5 <= m <= 16,
 * m = 4 unless n <= 1024 at k = 8192, m = 3 at n >= 4096, and 17 <= m <= 32 unless m > 20 at
 * k = 8192 and n > 16384 (above m = 16 only for sign-symmetric codebooks; at k = 8192 above
 * m = 16, and for sign-symmetric codebooks on narrow layers -- k = 8192 with n <= 2048 up to
 * m = 8 and n <= 8192 above, k = 4096 with n <= 2048 above m = 12 -- it first zeroes y and two
 * workgroups add their halves of K into each output); otherwise the wavefront-reduced GEMV
 * runs for m <= 8 unless m >= 3 and m * n > 65536; everything else (and shapes whose
 * activations do not fit the GEMV's registers) runs the stepped dequantize-into-MFMA skinny
 * GEMM, except m > 96 at n >= 4096, which runs a K-quartered MFMA GEMM for sign-symmetric
 * codebooks unless ceil(n / 64) * ceil(m / 128) <= 256. The stepped kernel runs in the launch
 * shape a cost model rates cheapest among those whose grid is on the chip at once (at most 256
 * workgroups): 64- or 128-row workgroups, batch blocks of 16 to 128 rows (to 64 for 8-bit codes
 * and codebooks that are not sign-symmetric), and K in one part or (from k = 4096) in two,
 * where y is zeroed first and each part adds into it; with none that fits, 128-row workgroups
 * with the largest batch blocks. logbq_linear_path reports the path, and logbq_linear_kernel
 * the kernel. Results are deterministic for every path.
 * k == 0 writes zeros. Errors: INVALID_ARG, UNSUPPORTED (k % 32, alignment, or k >= 2^24 on
 * the stepped or K-quartered MFMA kernel), HIP.
 */
int32_t logbq_linear(const uint16_t* x_dev, int64_t m, int64_t k, const uint8_t* codes_dev,
                     int64_t n, const float* codebook, float* y_dev, void* stream);

/*
 * logbq_linear_multi -- y_i = x . W_hat_i^T for 1 <= count <= 4 linears that share the same
 * activations (the query / key / value projections of a decoder layer, or its gate and up
 * projections), with one launch for the linears that take the GEMV in the same configuration
 * (wavefronts per row and chunks per lane, chosen from m, k and the linear's n) and one for
 * those that take the split-K kernel in the same configuration (chosen from m, k and the
 * linear's n, when their codebooks are sign-symmetric) (Sec. 3.3 lookup + product).
 *   x_dev, m, k : as logbq_linear; every W_i has k in features.
 *   count       : number of linears, 1..4.
 *   codes_dev   : host array of count device pointers, [n[i]][k/2] packed codes each.
 *   n           : host array of count out-feature counts (0 allowed).
 *   codebooks   : host array of count host pointers to 16 floats each.
 *   y_dev       : host array of count device pointers, [m][n[i]] float32 each.
 * Each y_i equals, bit for bit, what logbq_linear would write for the same operands.
 * Errors: INVALID_ARG (count outside 1..4, null arrays or entries), UNSUPPORTED, HIP.
 */
int32_t logbq_linear_multi(const uint16_t* x_dev, int64_t m, int64_t k, int32_t count,
                           const uint8_t* const* codes_dev, const int64_t* n,
                           const float* const* codebooks, float* const* y_dev, void* stream);

/*
 * logbq_dequantize -- Dequant (Eq. 2) of packed codes into float32 weights, by lookup.
 *   codes_dev : device, [n][k/2]; codebook: host, 16 floats; w_dev: device, [n][k] float32.
 * Bit-exact: w[n][k] = codebook[code(n, k)]. Errors: INVALID_ARG, UNSUPPORTED, HIP.
 */
int32_t logbq_dequantize(const uint8_t* codes_dev, int64_t n, int64_t k, const float* codebook,
                         float* w_dev, void* stream);

/*
 * logbq_linear8 -- y = x . W_hat^T on 8-bit codes (Sec. 3.1 at n = 8, Sec. 3.3 lookup).
 *   x_dev     : device, [m][k] IEEE float16 activations.
 *   m, k      : batch rows and in features; k % 32 == 0, m <= 4194240.
 *   codes_dev : device, [n][k] 8-bit codes.
 *   n         : out features.
 *   codebook  : host, 256 floats (logbq_params.codebook of an 8-bit fit); rounded to float16
 *               after a common power-of-two scaling, as for logbq_linear.
 *   y_dev     : device, [m][n] float32, written.
 * Float32 accumulation. For k in {2048, 4096, 8192} a split-K dequantize-into-MFMA kernel
 * takes 5 <= m <= 8 unless n <= 1024 at k >= 4096, m = 3, 4 at n >= 8192, and 9 <= m <= 16
 * unless n > 16384 at k = 8192; otherwise the GEMV runs for m <= 8 unless m >= 5 and
 * m * n > 65536, a K-quartered MFMA GEMM for m > 64 at n >= 16384, and the stepped
 * dequantize-into-MFMA skinny GEMM for the rest, in its cost-model launch shape (as for
 * logbq_linear; with K in two parts y is zeroed first). Results are deterministic.
 * Errors: as logbq_linear.
 */
int32_t logbq_linear8(const uint16_t* x_dev, int64_t m, int64_t k, const uint8_t* codes_dev,
                      int64_t n, const float* codebook, float* y_dev, void* stream);

/*
 * logbq_fit_uniform -- s, z, codebook and encoding thresholds of the asymmetric linear
 * baseline (Sec. 2, Quant(s, z, x)) for one tensor, from its full value range. Host only.
 *   w_host : host, numel float32 weights (any layout).
 *   bits   : 4.
 *   out    : host, filled on success.
 * Codes are decided in float64 as round(x / s) - z (ties up), clamped to 0 .. 15; the
 * thresholds reproduce that decision exactly with float32 comparisons.
 * Errors: INVALID_ARG (null, numel < 2), UNSUPPORTED (bits != 4), NONFINITE (NaN / Inf),
 * DEGENERATE (all weights equal).
 */
int32_t logbq_fit_uniform(const float* w_host, int64_t numel, int32_t bits, logbq_uniform* out);

/*
 * logbq_encode_uniform -- 4-bit asymmetric linear codes of float32 weights on the GPU:
 * code(x) = number of thresholds at or below x (NaN gives 0). Packing and layout as
 * logbq_encode ([n][k/2] bytes, low nibble = even k), but a nibble is the unsigned code q.
 * The codes run through logbq_linear / logbq_dequantize with u->codebook.
 *   w_dev     : device, [n][k] float32.   codes_dev : device, [n][k/2] bytes, written.
 *   u         : host, from logbq_fit_uniform (bits 4, thresholds non-decreasing).
 * Errors: INVALID_ARG, UNSUPPORTED (k % 32, alignment, bits), HIP.
 */
int32_t logbq_encode_uniform(const float* w_dev, int64_t n, int64_t k, const logbq_uniform* u,
                             uint8_t* codes_dev, void* stream);

/*
 * logbq_gptq -- GPTQ post-training calibration (the calibration used for every model in Sec. 4)
 * of one weight matrix with a fixed 4-bit codebook in its inner loop: LogbQuant (Eq. 1-2, from
 * `p`) or the asymmetric linear baseline (Sec. 2, from `uniform`). Columns are quantized in
 * order in blocks of 128; after column i, err = (w_i - q_i) / U_ii is subtracted, times U_ij,
 * from every later column j of its block, and after the block sum_i err_i U_ij from every
 * later column. All arithmetic is float32 in a fixed order, with no fused multiply-add:
 * err = (w - q) / U_ii; in the block w_j = w_j - err * U_ij; after it acc = acc + err_i * U_ij
 * over the block's columns in increasing i from 0, then w_j = w_j - acc.
 *   w_dev     : device, [n][k] float32, in/out. On return column i holds the value it had
 *               when it was quantized (the error-compensated weights).
 *   u_dev     : device, [k][k] float32 row-major: the upper Cholesky factor U of the damped
 *               inverse Hessian, H^-1 = U^T U (only j >= i is read; U_ii > 0).
 *   p, uniform: host; exactly one is non-NULL (bits 4). Its codebook is fixed for the whole
 *               loop (fit it on the original weights).
 *   err_dev   : device, [n][128] float32 workspace owned by the caller (overwritten).
 *   codes_dev : device, [n][k/2] packed codes, written (layout as logbq_encode; nibbles are
 *               sign + magnitude for LogbQuant, the unsigned code for the baseline).
 * Enqueues 2 * ceil(k / 128) kernels on `stream`. Errors: INVALID_ARG (null pointers, both or
 * neither of p / uniform, bad thresholds), UNSUPPORTED (bits, k % 32, alignment,
 * n > 1048560), HIP.
 */
int32_t logbq_gptq(float* w_dev, int64_t n, int64_t k, const float* u_dev, const logbq_params* p,
                   const logbq_uniform* uniform, float* err_dev, uint8_t* codes_dev,
                   void* stream);

/*
 * logbq_gptq_noalloc -- logbq_gptq without a caller-provided workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc). Same arguments, results (bit for bit) and kernels as logbq_gptq, except
 * err_dev: the [n][128] float32 error workspace is a fixed array in the library's code object,
 * 8 MiB per device, held by every GPU the library runs on until the process ends.
 *   w_dev, n, k, u_dev, p, uniform, codes_dev, stream: as logbq_gptq; n <= 16384.
 * Allocates nothing (no hipMalloc, hipFree or allocating library call); the first call on a
 * device looks up the array's device address once. Every call on a GPU uses that GPU's one
 * array: calls that overlap on one GPU (e.g. on two streams) race and must be serialised by
 * the caller. Each call writes every workspace entry it reads, so no clearing is needed.
 * Errors: as logbq_gptq, and UNSUPPORTED for n > 16384.
 */
int32_t logbq_gptq_noalloc(float* w_dev, int64_t n, int64_t k, const float* u_dev,
                           const logbq_params* p, const logbq_uniform* uniform,
                           uint8_t* codes_dev, void* stream);

/* Kernel that logbq_linear (bits 4) or logbq_linear8 (bits 8) runs for a call of a shape. */
typedef enum logbq_path {
  LOGBQ_PATH_NONE = 0,     /* m or n is 0 (nothing written) or k is 0 (zeros written)        */
  LOGBQ_PATH_GEMV = 1,     /* wavefront-reduced GEMV with the LDS pair table                  */
  LOGBQ_PATH_MFMA = 2,     /* stepped dequantize-into-MFMA skinny GEMM                        */
  LOGBQ_PATH_SPLITK = 3,   /* split-K dequantize-into-MFMA kernel (4-bit, 2 <= m <= 32; 8-bit,
                              3 <= m <= 16); above m = 16 a 4-bit codebook that is not
                              sign-symmetric runs the stepped kernel instead                  */
  LOGBQ_PATH_MFMA_KQ = 4   /* K-quartered dequantize-into-MFMA GEMM (4-bit, m > 96, n >= 4096;
                              8-bit, m > 64, n >= 16384); a 4-bit codebook that is not
                              sign-symmetric (never a fitted one) runs the stepped kernel     */
} logbq_path;

/*
 * logbq_linear_path -- the kernel a logbq_linear / logbq_linear8 call of shape (m, k, n)
 * runs (Sec. 3.3 product; the choice is this library's, not the method's). Host only: needs
 * no device and touches none. The choice depends on (bits, m, k, n) alone, so it is the same
 * for every linear of a logbq_linear_multi call.
 *   bits     : 4 or 8.
 *   m, k, n  : as logbq_linear; k % 32 == 0.
 *   path_out : host, one int32, written with a logbq_path on success.
 * Errors: INVALID_ARG (null path_out, negative size), UNSUPPORTED (bits, k % 32, m too large).
 */
int32_t logbq_linear_path(int32_t bits, int64_t m, int64_t k, int64_t n, int32_t* path_out);

/*
 * logbq_linear_kernel -- name of the kernel instance (with its template arguments, as a
 * profiler lists it) that reads the codes in a logbq_linear / logbq_linear8 call of shape
 * (m, k, n), e.g. "k_gemv<4, 1, 4, false, 2>" (Sec. 3.3 product; the choice is this
 * library's); a split-K call over workgroup pairs launches k_fill_zero before it, and one
 * that runs its batch in 16-row launches (k = 14336 above m = 16) is named by its first.
 * Host only: needs no device and touches none.
 *   bits, m, k, n : as logbq_linear_path; n fits in int32.
 *   codebook      : host, 2^bits floats, or NULL for a fitted (sign-symmetric) codebook; the
 *                   4-bit MFMA kernels dequantize in registers only for sign-symmetric ones.
 *   name_out      : host, name_len bytes, receives a NUL-terminated name ("none" for an empty
 *                   call, "k_fill_zero" for k = 0).
 * Errors: INVALID_ARG (null name_out, buffer too short, negative size, non-finite codebook
 * entry), UNSUPPORTED (bits, k % 32, m or n too large).
 */
int32_t logbq_linear_kernel(int32_t bits, int64_t m, int64_t k, int64_t n, const float* codebook,
                            char* name_out, int64_t name_len);

/*
 * logbq_dequantize8 -- Dequant (Eq. 2) of 8-bit codes: w[n][k] = codebook[codes[n][k]].
 *   codes_dev : device, [n][k]; codebook: host, 256 floats; w_dev: device, [n][k] float32.
 * Bit-exact. Errors: INVALID_ARG, UNSUPPORTED, HIP.
 */
int32_t logbq_dequantize8(const uint8_t* codes_dev, int64_t n, int64_t k, const float* codebook,
                          float* w_dev, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LOGBQ_H */
