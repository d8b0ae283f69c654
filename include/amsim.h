/*
 * amsim.h -- C ABI of the MI355X (gfx950) approximate-multiplier GEMM / convolution library.
 *
 * The library simulates an approximate floating-point multiplier the way AMSim does in
 * ApproxTrain (arXiv 2209.04161): every FP32 product a*b is replaced by
 *   sign(a) XOR sign(b), exponent Ea + Eb - 127 (+ carry), mantissa from a lookup table
 *   indexed by the concatenated top-M mantissa bits of a and b (Algorithm 2),
 * and products are accumulated in FP32 (Sec. "Experiment Setup", Datatype paragraph).
 * The table comes from a C functional model of the multiplier (Algorithm 1).
 *
 * Conventions for every entry point:
 *   - Return value: AMSIM_OK (0) or a negative AMSIM_ERR_* code.  Nothing throws across the
 *     ABI and nothing prints.
 *   - "device" pointers are HIP device allocations owned by the caller (e.g. torch tensors);
 *     "host" pointers are ordinary host memory owned by the caller.  Device pointers must be
 *     4-byte aligned; the library allocates nothing and frees nothing.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Device entry
 *     points only enqueue work on that stream: they do not synchronise and return before the
 *     work completes.  A HIP launch error is reported as AMSIM_ERR_HIP.
 *   - `lut` is a device copy of the table built by lut_build: uint32[2^(2*m_bits)], entry
 *     k * 2^M + j holds carry << 23 | mantissa(23 bits) for first-operand mantissa k and
 *     second-operand mantissa j.  Only its low 24 bits are read.
 *   - m_bits (the paper's M) must be in [1, 11].  The library stages the table rows that each
 *     step needs into LDS: rows of 128 entries for M <= 7, of 2^M entries for M = 8..11.
 *   - Products: zero/denormal operands give a signed zero, NaN operands NaN, Inf times a
 *     zero/denormal operand NaN, Inf times anything else a signed Inf; otherwise zero if
 *     Ea + Eb - 127 <= 0 (checked before the carry), Inf if it is >= 255 or the carry lifts
 *     it to 255, else sign | (Ea + Eb - 127 + carry) << 23 | mantissa.
 *   - Sums start from -0.0 and are FP32 with denormal results flushed to zero; summation
 *     order is unspecified (the results of one call are deterministic run to run).
 *   - Errors in the arguments (AMSIM_ERR_INVALID_ARG, _UNSUPPORTED, _WORKSPACE) are found before
 *     anything is launched.  AMSIM_ERR_HIP reports a failed launch; kernels the call enqueued
 *     before it may still run, and the output is then unspecified.
 */
#ifndef AMSIM_H
#define AMSIM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define AMSIM_OK 0
#define AMSIM_ERR_INVALID_ARG (-1) /* null pointer, bad size/stride/shape */
#define AMSIM_ERR_UNSUPPORTED (-2) /* m_bits outside [1, 11] or a shape beyond the limits */
#define AMSIM_ERR_MODEL (-3)       /* the model cannot be represented by a mantissa table */
#define AMSIM_ERR_WORKSPACE (-4)   /* workspace missing or smaller than the size query says */
#define AMSIM_ERR_HIP (-5)         /* a HIP runtime call or kernel launch failed */
#define AMSIM_ERR_IO (-6)          /* file could not be read/written or has a bad header */
#define AMSIM_ERR_SCRATCH (-7)     /* approx_gemm_noalloc: the call needs more than the fixed buffer */

/* Human-readable name of a status code (static string, never NULL). */
const char *amsim_status_string(int status);

/* Library version, major * 10000 + minor * 100 + patch. */
int amsim_version(void);

/* ----------------------------------------------------------------- functional models ----
 * A designer's approximate multiplier (Algorithm 1's input approx_mul): takes two FP32 values,
 * returns their approximate FP32 product.  lut_build calls it only with positive, normal
 * operands whose exponent fields keep the product's exponent in range.  `ctx` is passed through.
 */
typedef float (*amsim_model_fn)(float a, float b, void *ctx);

/* Built-in models; ctx points to an int holding M (1..11).
 * Mitchell's logarithmic multiplier (the paper's MIT16 at M = 7): log2(1 + x) ~= x on both
 * operands truncated to M mantissa bits, antilog 2^(c + f) ~= 2^c (1 + f). */
float amsim_model_mitchell(float a, float b, void *ctx);
/* Exact product of the operands truncated to M mantissa bits (bfloat16 truncation at M = 7,
 * Sec. "Experiment Setup": format conversion is bit truncation). */
float amsim_model_exact_trunc(float a, float b, void *ctx);

/* ----------------------------------------------------------------- table generation -----
 * lut_build: Algorithm 1.  Fills out[k * 2^M + j] = carry << 23 | mantissa(C) for
 * C = model(A, B, ctx), A = +1.k and B = +1.j (exponent field 127, k and j in the top M
 * mantissa bits), carry = 1 iff Exp(C) > Exp(A) + Exp(B) - 127.
 *   m_bits  M in [1, 11]                           (else AMSIM_ERR_UNSUPPORTED)
 *   model   host function pointer, non-NULL        (else AMSIM_ERR_INVALID_ARG)
 *   out     host uint32 array of out_len entries, out_len >= 2^(2M) (else INVALID_ARG)
 * Returns AMSIM_ERR_MODEL if the model's product is not positive and finite, its exponent is
 * neither Exp(A)+Exp(B)-127 nor one more, or a rebuild of a sample of entries at other legal
 * exponents and all four sign combinations disagrees (the model must depend on the
 * mantissas only, Sec. "Lookup Table Generation").  Runs on the calling thread. */
int lut_build(int m_bits, amsim_model_fn model, void *ctx, uint32_t *out, size_t out_len);

/* Table file (Sec. "Lookup Table Generation": tables are generated once and loaded at run
 * time).  Format: 16-byte header {"AMLT", uint32 version = 1, uint32 M, uint32 0}, then
 * 2^(2M) little-endian uint32 entries.
 * lut_save writes `lut` (host, len >= 2^(2M) entries) to `path`.
 * lut_load reads `path` into `out` (host, out_len entries); *m_bits receives M.  Passing
 * out = NULL only reads the header.  Errors: AMSIM_ERR_IO, AMSIM_ERR_INVALID_ARG. */
int lut_save(const char *path, int m_bits, const uint32_t *lut, size_t len);
int lut_load(const char *path, int *m_bits, uint32_t *out, size_t out_len);

/* ----------------------------------------------------------------- GEMM -----------------
 * approx_gemm: C = op(A) * op(B) with every product approximate (the paper's GEMM kernel with
 * AMSim, Sec. "Other Custom CUDA Kernels"; dense layers map onto it, Sec. "AMDENSE").
 * Row-major storage.  op(A) is m x k: A is m x k (lda >= k) or, with trans_a, k x m
 * (lda >= m).  op(B) is k x n: B is k x n (ldb >= n) or, with trans_b, n x k (ldb >= k).
 * C is m x n (ldc >= n) and is overwritten (no alpha/beta).  The product of element (i, kk)
 * of op(A) with element (kk, j) of op(B) takes op(A)'s element as the first operand (the
 * table's high index).  m or n == 0: nothing is done.  k == 0: C is filled with -0.0.
 * All matrix pointers and `lut` are device memory; `workspace` is device memory of at least
 * the size amsim_gemm_workspace_size reports (may be NULL when that size is 0). */
int amsim_gemm_workspace_size(int trans_a, int trans_b, int64_t m, int64_t n, int64_t k, int m_bits,
                              size_t *bytes);
int approx_gemm(int trans_a, int trans_b, int64_t m, int64_t n, int64_t k, const float *A, int64_t lda,
                const float *B, int64_t ldb, float *C, int64_t ldc, const uint32_t *lut, int m_bits,
                void *workspace, size_t workspace_bytes, void *stream);

/* approx_gemm_noalloc: approx_gemm without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, results and errors as approx_gemm (bit for bit the same C), but the
 * workspace is a fixed buffer of AMSIM_NOALLOC_SCRATCH_BYTES bytes inside the library, one per GPU,
 * held from the library's load until the process ends; the call allocates and frees nothing.
 *   - Returns AMSIM_ERR_SCRATCH, before anything is launched, when the call's workspace
 *     (amsim_gemm_workspace_size without options: the table path) exceeds the buffer.
 *   - The buffer used is the current device's; `stream` must belong to that device.  The first
 *     call on a device looks up its buffer's address (no allocation).
 *   - Every call on one GPU shares that GPU's buffer and leaves its contents behind (nothing in
 *     it has to start at zero).  Calls whose work overlaps on one GPU (other streams, other host
 *     threads without ordering) race on it and give unspecified results: order them on one
 *     stream or synchronise between them. */
#define AMSIM_NOALLOC_SCRATCH_BYTES (64u << 20)
int approx_gemm_noalloc(int trans_a, int trans_b, int64_t m, int64_t n, int64_t k, const float *A, int64_t lda,
                        const float *B, int64_t ldb, float *C, int64_t ldc, const uint32_t *lut, int m_bits,
                        void *stream);

/* Direct evaluation: the GEMM with no table, for the comparison the paper draws for AMSim
 * (Sec. "AMSim", its figure of GEMM run time with AMSim, with a direct simulation of the
 * multiplier and with the native multiply).
 *   AMSIM_DIRECT_NATIVE    C = A B with the native FP32 multiply (each product rounded, then
 *                          added); m_bits is ignored.
 *   AMSIM_DIRECT_MITCHELL  every product Mitchell's multiplier on the top m_bits mantissa bits,
 *                          computed from the operands' bits in the kernel -- the same products as
 *                          approx_gemm with a Mitchell table (same zero / denormal / Inf / NaN /
 *                          overflow rules), bit for bit.
 * Row-major A [m][k] (lda >= k) and B [k][n] (ldb >= n), C [m][n] (ldc >= n) overwritten; device
 * memory; sums start from -0.0 (k == 0 fills C with -0.0).  No workspace.  Returns
 * AMSIM_ERR_INVALID_ARG for an unknown mode, AMSIM_ERR_UNSUPPORTED for m_bits outside [1, 11]
 * (Mitchell) or sizes from 2^31 on. */
#define AMSIM_DIRECT_NATIVE 0
#define AMSIM_DIRECT_MITCHELL 1
int approx_gemm_direct(int mode, int m_bits, int64_t m, int64_t n, int64_t k, const float *A, int64_t lda,
                       const float *B, int64_t ldb, float *C, int64_t ldc, void *stream);

/* ----------------------------------------------------------------- 2-D convolution ------
 * NHWC activations, HWIO weights ([kh][kw][c_in][c_out]), explicit four-sided zero padding
 * (TF "SAME" is an asymmetric pad), stride >= 1, no dilation or groups (none in the paper).
 * OH = (h + pad_top + pad_bottom - kh) / stride_h + 1, OW likewise; both must be >= 1.
 * All sizes must be >= 1 (pads >= 0).  AMSIM_ERR_UNSUPPORTED when a (padded) tensor reaches
 * 2^29 elements, the zero-padded x or dy stored as 12 bytes per pixel and channel pair reaches
 * 2^31 bytes, a pad or kernel side reaches 65536, stride_h * stride_w exceeds 32, a channel
 * count exceeds 1048560, or w or OW reaches 4096. */
typedef struct amsim_conv2d {
    int n, h, w, c_in, c_out, kh, kw, stride_h, stride_w, pad_top, pad_bottom, pad_left, pad_right;
} amsim_conv2d;

#define AMSIM_CONV_FWD 0
#define AMSIM_CONV_BWD_DATA 1
#define AMSIM_CONV_BWD_WEIGHT 2

/* Device workspace bytes a pass needs for this shape and M (0 allowed for NULL workspace).  A 1 x 1
 * pass with stride 1 and no padding runs as its GEMM over the pixels (its im2col matrix is the
 * input itself) and needs that GEMM's workspace.  A stride-1 backward-data pass with every pad at
 * most the kernel extent minus one and c_out >= 16 runs as the forward pass over dy (padded by the
 * kernel extent minus one minus each pad) with the weights reversed in both kernel axes and c_in,
 * c_out exchanged -- the same products -- and needs that forward pass's workspace. */
int amsim_conv2d_workspace_size(const amsim_conv2d *desc, int pass, int m_bits, size_t *bytes);

/* Forward propagation (Algorithm 3): y[n,oh,ow,co] = sum_{kh,kw,ci}
 * amul(x[n, oh*sh+kh-pt, ow*sw+kw-pl, ci], w[kh,kw,ci,co]), where x outside the image is the
 * zero border, +0, which is multiplied like any operand (a signed zero, or NaN against an Inf or
 * NaN weight, as Algorithm 3's column matrix holds it).
 * x: device [n][h][w][c_in], w: device HWIO, y: device [n][OH][OW][c_out] (overwritten). */
int approx_conv2d_fwd(const amsim_conv2d *desc, const float *x, const float *w, float *y, const uint32_t *lut,
                      int m_bits, void *workspace, size_t workspace_bytes, void *stream);

/* Preceding-layer gradient (Algorithm 4, second half): dx[n,h,w,ci] = sum over every (kh,kw,co)
 * of amul(e, w[kh,kw,ci,co]), where e = dy[n,oh,ow,co] for the output position (oh,ow) with
 * oh*sh+kh-pt == h and ow*sw+kw-pl == w when it exists, else +0 -- the padded, dilated error
 * against the transposed and reversed weights, without materialising either; its zeros are
 * multiplied like any operand (a signed zero, or NaN against an Inf or NaN weight).
 * dy: device [n][OH][OW][c_out], w: device HWIO, dx: device [n][h][w][c_in] (overwritten). */
int approx_conv2d_bwd_data(const amsim_conv2d *desc, const float *dy, const float *w, float *dx,
                           const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes, void *stream);

/* Weights gradient (Algorithm 4, first half): dw[kh,kw,ci,co] = sum over (n,oh,ow) of
 * amul(x[n, oh*sh+kh-pt, ow*sw+kw-pl, ci], dy[n,oh,ow,co]), x outside the image being the zero
 * border (+0, multiplied like any operand) -- the stride dilation of the error is implicit.
 * x: device NHWC, dy: device [n][OH][OW][c_out], dw: device HWIO (overwritten). */
int approx_conv2d_bwd_weight(const amsim_conv2d *desc, const float *x, const float *dy, float *dw,
                             const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes,
                             void *stream);

/* ----------------------------------------------------------------- options --------------
 * The _ex variants of the GEMM, convolution and element-wise calls take the multiplier to
 * simulate (NULL = the defaults, which are what the plain calls do):
 *   multiply  AMSIM_MULTIPLY_TABLE: every product approximate, from the table (AMSim, the default);
 *             AMSIM_MULTIPLY_NATIVE: the native FP32 multiply in the same kernels (the paper's
 *             "AT with native multiply" configuration, Tables of training / inference time):
 *             products are IEEE FP32 (denormal operands and results flushed to zero), each fused
 *             into the sum; lut and m_bits are then ignored (lut may be NULL) and e_bits must be 8.
 *   e_bits    exponent bits e of the simulated (1, e, m) format, 2..8 (Sec. "AMSim": e can range up
 *             to 8 given an exponent-casting function; 8 = FP32's exponent, the default).  With
 *             e < 8, bias beta = 2^(e-1) - 1, every operand is first cast to the format (below;
 *             values in its range are unchanged), and Algorithm 2 runs in the format's constants:
 *             zero if Ea + Eb - beta <= 0 (before the carry), Inf if Ea + Eb - beta (+ carry)
 *             reaches 2^e - 1, else the product, returned as an FP32 value and summed in FP32.
 *             e = 1 (no finite non-zero value once the top field is reserved for Inf/NaN) is
 *             AMSIM_ERR_UNSUPPORTED.
 *   exp_cast  the exponent-casting function: a finite value whose unbiased exponent exceeds beta
 *             becomes a signed Inf (AMSIM_CAST_INF, the default) or the format's largest finite
 *             value (2 - 2^-M) * 2^beta (AMSIM_CAST_SATURATE); one below 1 - beta (the format's
 *             denormals included) a signed zero.
 * Unknown values give AMSIM_ERR_INVALID_ARG. */
typedef struct amsim_options {
    int multiply;
    int e_bits;
    int exp_cast;
} amsim_options;

#define AMSIM_MULTIPLY_TABLE 0
#define AMSIM_MULTIPLY_NATIVE 1
#define AMSIM_CAST_INF 0
#define AMSIM_CAST_SATURATE 1

/* The calls above with options (same arguments, same workspace sizes). */
int approx_gemm_ex(const amsim_options *opt, int trans_a, int trans_b, int64_t m, int64_t n, int64_t k,
                   const float *A, int64_t lda, const float *B, int64_t ldb, float *C, int64_t ldc, const uint32_t *lut,
                   int m_bits, void *workspace, size_t workspace_bytes, void *stream);
int approx_conv2d_fwd_ex(const amsim_options *opt, const amsim_conv2d *desc, const float *x, const float *w, float *y,
                         const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes, void *stream);
int approx_conv2d_bwd_data_ex(const amsim_options *opt, const amsim_conv2d *desc, const float *dy, const float *w,
                              float *dx, const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes,
                              void *stream);
int approx_conv2d_bwd_weight_ex(const amsim_options *opt, const amsim_conv2d *desc, const float *x, const float *dy,
                                float *dw, const uint32_t *lut, int m_bits, void *workspace, size_t workspace_bytes,
                                void *stream);

/* amsim_cast_exponent: the exponent-casting function on its own, y[i] = x[i] cast to the
 * (1, e_bits, m_bits) format as described above, as an FP32 value (device x, y; y may alias x;
 * n == 0: nothing is done).  Errors as for the options, plus m_bits outside [1, 11]. */
int amsim_cast_exponent(int e_bits, int exp_cast, int m_bits, int64_t n, const float *x, float *y, void *stream);

/* ----------------------------------------------------------------- element-wise --------
 * approx_mul_ew: c[i] = amul(a[i], b[i]) for i < n -- Algorithm 2 exactly as the GEMM and
 * convolution kernels evaluate it, exposed so that single products can be checked bit for
 * bit.  a, b, c, lut: device memory (c may alias neither input).  n == 0: nothing is done. */
int approx_mul_ew(int64_t n, const float *a, const float *b, float *c, const uint32_t *lut, int m_bits,
                  void *stream);
/* The same with options (multiply must be AMSIM_MULTIPLY_TABLE, else AMSIM_ERR_UNSUPPORTED). */
int approx_mul_ew_ex(const amsim_options *opt, int64_t n, const float *a, const float *b, float *c,
                     const uint32_t *lut, int m_bits, void *stream);

/* ----------------------------------------------------------------- kernel timing -------
 * Measurement support (no paper counterpart; the paper reports per-batch wall time only).
 * Between amsim_profile_start and amsim_profile_stop, every launch of a main kernel -- the
 * GEMM kernel of approx_gemm and the three convolution kernels, not their decode pre-passes
 * -- is bracketed by two HIP events recorded on the stream it is launched on.  The events are
 * timing-only (created without the system-scope fence on completion), so they add no cache
 * writeback around the kernels they time; they order nothing for the host.
 *   amsim_profile_start(max_launches): creates that many event pairs (host-side HIP calls; do
 *     it outside any timed region) and starts recording; AMSIM_ERR_INVALID_ARG if
 *     max_launches < 1, AMSIM_ERR_HIP on event creation failure.  Launches beyond the
 *     capacity are not timed.  Calling it again discards the previous records.
 *   amsim_profile_stop(): stops recording and waits for the recorded events.
 *   amsim_profile_read(kind, &launches, &total_ms): launches and summed durations (ms) of one
 *     kernel kind (AMSIM_KERNEL_*) since the last start; valid after amsim_profile_stop.
 * The timer state is process-wide and guarded by a lock. */
#define AMSIM_KERNEL_GEMM 0
#define AMSIM_KERNEL_CONV_FWD 1
#define AMSIM_KERNEL_CONV_BWD_DATA 2
#define AMSIM_KERNEL_CONV_BWD_WEIGHT 3
/* the same kernels with the native multiply (AMSIM_MULTIPLY_NATIVE) */
#define AMSIM_KERNEL_GEMM_NATIVE 4
#define AMSIM_KERNEL_CONV_FWD_NATIVE 5
#define AMSIM_KERNEL_CONV_BWD_DATA_NATIVE 6
#define AMSIM_KERNEL_CONV_BWD_WEIGHT_NATIVE 7
int amsim_profile_start(int max_launches);
/* amsim_profile_start, timing only the kernel kinds whose bit (1u << AMSIM_KERNEL_*) is set in
 * kinds: every other launch gets no events, so it runs as it would unprofiled.
 * AMSIM_ERR_INVALID_ARG for max_launches < 1, kinds == 0 or a bit above the last kind. */
int amsim_profile_start_kinds(int max_launches, unsigned kinds);
int amsim_profile_stop(void);
int amsim_profile_read(int kind, int *launches, double *total_ms);

#ifdef __cplusplus
}
#endif

#endif /* AMSIM_H */
