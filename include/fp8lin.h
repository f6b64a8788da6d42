/*
 * fp8lin.h -- C ABI of libfp8lin.so: the FP8 linear layer with dynamically
 * computed per-tensor power-of-two scaling biases, for AMD MI355X (gfx950).
 *
 * Method: Perez et al., "Training and inference of large language models
 * using 8-bit floating point" (arXiv 2309.17224).
 *   Sec. 2.3 Eq. 3   amax = max|T|, scaling bias b = floor(log2(max_num / amax))
 *   Sec. 2.1 Eq. 1   scaling = adding b to the exponent = multiplying by 2^b
 *                    before the cast to FP8
 *   Sec. 2.1 Eq. 2   after the FP8 matmul the output is unscaled by
 *                    -(b_w + b_x)
 *   Sec. 2.2         gradients use FP8 E5, weights and activations FP8 E4;
 *                    the backward pass has two FP8 matmuls (grad-input and
 *                    grad-weight), each unscaled by its inputs' biases
 *   Sec. 3           FP8-AMAX: one bias per tensor per call; Sec. 3.2 margin
 *   Sec. 3.1         post-training quantisation: weight bias computed once
 *
 * FP8 formats.  The matrix cores of gfx950 consume the OCP formats E4M3 and
 * E5M2, which are the "(b)" rows of Table 7 (App. A): E4M3 bias 7, max 448,
 * NaN = S.1111.111, no infinity; E5M2 bias 15, max 57344, IEEE infinities
 * and NaNs.  The paper's default "(a)" formats (bias 8 / 16, NaN = 0x80) are
 * accepted by the bias and cast calls only (FP8_E4_A, FP8_E5_A below).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every data pointer is a DEVICE pointer owned by the caller.  The library
 *    never allocates, frees or keeps memory, and never synchronises.
 *  - Every call is asynchronous on `stream` (a hipStream_t passed as void*;
 *    NULL is the null stream).
 *  - Arguments are checked on the host before anything is launched.  A call
 *    that returns an error has launched nothing.
 *  - Scaling biases are int32 in device memory, so amax -> bias -> cast ->
 *    matmul needs no copy to the host.
 *  - Numerical conditions are never errors.  *flags (optional, uint32 in
 *    device memory) is overwritten by fp8_scale_bias / ptq_quantise_weights
 *    with FP8_FLAG_NONFINITE when the amax is NaN or infinite and with
 *    FP8_FLAG_ZERO when it is zero; the bias is then 0.
 *  - Layouts are dense row-major unless a leading dimension (ld*, in
 *    elements) is given.
 *  - Rounding of the cast is to nearest, ties to even; values beyond the
 *    largest finite FP8 value, infinities included, clip to it with their
 *    sign (App. A); NaN becomes 0x7F with the input's sign bit.
 *  - Matmul accumulation is fp32 (MFMA); the unscale 2^-(b_a + b_b) is applied
 *    to the fp32 sum, which is then rounded once to the output type (to
 *    nearest, ties to even).  An output is NaN only when an operand holds a
 *    NaN code; its NaN encoding is unspecified.
 *  - Thread safety: calls hold no state and may be issued from any thread.
 */
#ifndef FP8LIN_H
#define FP8LIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define FP8_OK 0       /* launched (or nothing to do) */
#define FP8_EINVAL 1   /* bad argument: null pointer, negative or too large size,
                          leading dimension below the row length, misaligned
                          pointer, unknown format or dtype, workspace too small */
#define FP8_ENOTSUP 2  /* valid but unsupported combination */
#define FP8_EHIP 3     /* the HIP runtime reported a launch error */

/* FP8 formats.  OCP (Table 7 rows "(b)"), the formats of the matrix cores: */
#define FP8_E4M3 0
#define FP8_E5M2 1
/* The paper's own formats (Table 7 rows "(a)"): E4 bias 8, largest finite 240;
 * E5 bias 16, largest finite 57344; code 0x80 is the only NaN, no infinity,
 * no -0.  Accepted by the bias and cast calls (fp8_scale_bias,
 * fp8_bias_from_amax, fp8_cast, fp8_quantise), not by the matmuls.  Every code
 * finite in both families decodes in (a) to half its OCP value. */
#define FP8_E4_A 2
#define FP8_E5_A 3

/* Higher-precision element types of inputs and outputs. */
#define FP8_DT_BF16 0
#define FP8_DT_F32 1

/* Bits of *flags. */
#define FP8_FLAG_NONFINITE 1u
#define FP8_FLAG_ZERO 2u
#define FP8_FLAG_SATURATED 4u  /* fp8_quantise_delayed: the codes of this call clipped */

/* Largest accepted |margin|. */
#define FP8_MAX_MARGIN 65536

/* Text for a status code (static storage, never NULL). */
const char *fp8_status_string(int32_t status);

/* Version of this ABI (incremented on any incompatible change). */
int32_t fp8_abi_version(void);

/* Workspace bytes fp8_scale_bias needs for n elements (0 when n == 0). */
size_t fp8_scale_bias_ws_bytes(int64_t n);

/*
 * fp8_scale_bias -- the compute_bias step of FP8-AMAX (Sec. 2.3 Eq. 3, Sec. 3).
 *   amax = max_i |x_i| over all n elements (one tensor, one call), then
 *   *bias = floor(log2(max_num(fmt) / amax)) - margin,
 *   evaluated exactly: *bias is the largest integer b with amax * 2^b <= max_num,
 *   minus the margin.  max_num is 448 (E4M3) or 57344 (E5M2).
 * x:         n elements of type dt (FP8_DT_BF16 or FP8_DT_F32), aligned to the
 *            element size.  -0 counts as 0; a NaN makes the amax NaN.
 * margin:    subtracted from the bias (Sec. 3.2: 3 was used with FP16
 *            accumulation; 0 with fp32 accumulation).  |margin| <= FP8_MAX_MARGIN.
 * bias:      out, one int32 (device).
 * amax_bits: out, optional: the fp32 bit pattern of the amax (device); a
 *            tensor holding a NaN has amax 0x7FC00000, whatever the NaN
 *            payloads.
 * flags:     out, optional: see the conventions above (device).
 * ws:        device workspace of at least fp8_scale_bias_ws_bytes(n) bytes,
 *            4-byte aligned; its contents are scratch.  Concurrent calls need
 *            distinct workspaces.
 * n == 0 gives amax 0, bias 0 and FP8_FLAG_ZERO; n above 2^46 is FP8_EINVAL.
 */
int32_t fp8_scale_bias(const void *x, int32_t dt, int64_t n, int32_t fmt, int32_t margin,
                       int32_t *bias, uint32_t *amax_bits, uint32_t *flags,
                       void *ws, size_t ws_bytes, void *stream);

/*
 * fp8_bias_from_amax -- Eq. 3 from an amax already in device memory (for
 * example one produced by a matmul epilogue, see fp8_linear_fwd).
 * amax_bits: in, fp32 bit pattern (sign ignored).  Outputs as fp8_scale_bias.
 */
int32_t fp8_bias_from_amax(const uint32_t *amax_bits, int32_t fmt, int32_t margin,
                           int32_t *bias, uint32_t *flags, void *stream);

/*
 * fp8_cast_e4 / fp8_cast_e5 -- scale and cast (Sec. 2.1 Eq. 1; E4 for weights
 * and activations, E5 for gradients, Sec. 2.2):
 *   q[r, c] = RNE_saturate_fmt(x[r, c] * 2^(*bias))
 * The product is exact (a power-of-two scale of a bf16/fp32 value), so the
 * cast is the only rounding.
 * x:    [rows, cols] of type dt, row stride ldx >= cols elements.
 * bias: in, one int32 (device), e.g. written by fp8_scale_bias.
 * q:    out, [rows, cols] uint8 codes, row stride ldq >= cols; may be NULL
 *       if qT is given.
 * qT:   out, optional, the same codes transposed: [cols, rows], row stride
 *       ldqT >= rows.  The matmuls below take this copy where they contract
 *       over the rows of a tensor.
 * rows == 0 or cols == 0 is a no-op.  A tensor of more than INT32_MAX tiles
 * of 128 x 128 (one workgroup each) returns FP8_ENOTSUP.
 */
int32_t fp8_cast_e4(const void *x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx,
                    const int32_t *bias, uint8_t *q, int64_t ldq, uint8_t *qT, int64_t ldqT,
                    void *stream);
int32_t fp8_cast_e5(const void *x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx,
                    const int32_t *bias, uint8_t *q, int64_t ldq, uint8_t *qT, int64_t ldqT,
                    void *stream);

/*
 * fp8_cast -- fp8_cast_e4 / fp8_cast_e5 with the format as an argument: any of
 * FP8_E4M3, FP8_E5M2, FP8_E4_A, FP8_E5_A.  In the (a) formats, NaN becomes 0x80
 * and values that round to zero become 0x00 whatever their sign.
 */
int32_t fp8_cast(const void *x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx,
                 int32_t fmt, const int32_t *bias, uint8_t *q, int64_t ldq, uint8_t *qT,
                 int64_t ldqT, void *stream);

/*
 * fp8_quantise -- amax, Eq. 3 bias and scale+cast of one whole tensor in one
 * call (Sec. 2.3 Eq. 3, Sec. 2.1 Eq. 1): the same outputs, bit for bit, as
 * fp8_scale_bias over the rows x cols elements followed by fp8_cast_e4 (fmt
 * FP8_E4M3) or fp8_cast_e5 (FP8_E5M2).
 * Computing the bias needs the amax of the whole tensor before any element
 * can be cast, which costs a second pass over the tensor (Sec. 3).  A
 * predicted bias removes that pass when the prediction is right: the tensor
 * is read once, cast with the prediction while its amax is taken, and only if
 * the exact bias differs from the prediction are the codes written again
 * with the exact bias.  Biases of the same tensor change little from one step
 * to the next (Sec. 3), so the previous step's bias is a good prediction.
 * x, dt, rows, cols, ldx, q, ldq, qT, ldqT: as fp8_cast_e4 (strides allowed).
 * fmt, margin: as fp8_scale_bias.
 * bias_pred: in, optional, one int32 (device): the predicted bias; may be the
 *            same word as bias.  NULL: two passes (amax, then the cast).
 * bias, amax_bits, flags: out, as fp8_scale_bias (amax_bits, flags optional).
 * ws:        device workspace of at least fp8_quantise_ws_bytes(rows, cols)
 *            bytes, 4-byte aligned; scratch, distinct for concurrent calls.
 *            (fp8_quantise_ws_bytes is SIZE_MAX for a tensor of more than
 *            INT32_MAX tiles of 128 x 128, which fp8_quantise rejects with
 *            FP8_ENOTSUP.)
 * rows == 0 or cols == 0 gives amax 0, bias 0 and FP8_FLAG_ZERO, no codes.
 */
size_t fp8_quantise_ws_bytes(int64_t rows, int64_t cols);
int32_t fp8_quantise(const void *x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx,
                     int32_t fmt, int32_t margin, const int32_t *bias_pred, int32_t *bias,
                     uint32_t *amax_bits, uint32_t *flags, uint8_t *q, int64_t ldq,
                     uint8_t *qT, int64_t ldqT, void *ws, size_t ws_bytes, void *stream);

/*
 * fp8_quantise_noalloc -- fp8_quantise with no workspace argument, for callers
 * that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation.  Same arguments as
 * fp8_quantise without ws / ws_bytes, and the same outputs, bit for bit.
 * Its scratch words sit in a static device array of FP8_NOALLOC_SCRATCH_BYTES
 * bytes that each GPU the library runs on holds until the process ends; the
 * call allocates and frees nothing.
 * Limit: a tensor of at most FP8_NOALLOC_MAX_TILES tiles of 128 x 128
 * elements, ceil(rows / 128) * ceil(cols / 128) (about 4.29e9 elements);
 * FP8_EINVAL beyond.
 * Sharing: every call on one GPU uses that GPU's one array.  Calls that may
 * run at the same time on one GPU (other streams, other threads) race and give
 * wrong results: order them on one stream.
 * The stream must belong to the current device (FP8_EINVAL otherwise).  The
 * first call on each device looks up the array's address there
 * (hipGetSymbolAddress, no allocation); FP8_EHIP if that fails.
 */
#define FP8_NOALLOC_SCRATCH_BYTES 1048576
#define FP8_NOALLOC_MAX_TILES 262143
int32_t fp8_quantise_noalloc(const void *x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx,
                             int32_t fmt, int32_t margin, const int32_t *bias_pred, int32_t *bias,
                             uint32_t *amax_bits, uint32_t *flags, uint8_t *q, int64_t ldq,
                             uint8_t *qT, int64_t ldqT, void *stream);

/*
 * fp8_quantise_delayed -- delayed scaling: the remedy Sec. 3 cites for the
 * second pass over a tensor that computing its bias just in time costs.  The
 * bias comes from the amax of earlier calls, so the tensor is read once and
 * its codes are never recast; a tensor that outgrows the bias clips (App. A).
 *   codes  = cast(x * 2^(*bias))                (the bias on entry)
 *   a      = amax(x)  (Eq. 3's amax of this tensor; NaN gives 0x7FC00000)
 *   history[*count % history_len] = a;  *count += 1
 *   *bias  = floor(log2(max_num / max(history))) - margin   (Eq. 3; the bias
 *            of the next call; 0 when that maximum is zero or not finite)
 * x, dt, rows, cols, ldx, fmt, q, ldq, qT, ldqT, ws, ws_bytes: as fp8_quantise.
 * bias:        in/out, one int32 (device): the bias to cast with; replaced by
 *              the next call's bias.
 * history:     device uint32 [history_len], 1 <= history_len <= 65536: amax bit
 *              patterns of earlier calls as this call writes them; zeros before
 *              the first call.
 * count:       device uint32: calls so far (the next slot is count % history_len).
 * amax_bits:   out, optional: a.
 * flags:       out, optional: FP8_FLAG_NONFINITE / FP8_FLAG_ZERO for a, else
 *              FP8_FLAG_SATURATED when a * 2^bias > max_num (some codes clipped).
 * rows == 0 or cols == 0: a = 0 is recorded, FP8_FLAG_ZERO, no codes.
 * Calls that share a history must be ordered (one stream).
 */
int32_t fp8_quantise_delayed(const void *x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx,
                             int32_t fmt, int32_t margin, int32_t *bias, uint32_t *history,
                             int64_t history_len, uint32_t *count, uint32_t *amax_bits,
                             uint32_t *flags, uint8_t *q, int64_t ldq, uint8_t *qT, int64_t ldqT,
                             void *ws, size_t ws_bytes, void *stream);

/*
 * fp8_quantise_batch -- fp8_quantise of n tensors (1 <= n <=
 * FP8_QUANTISE_BATCH_MAX) of one element type dt and format fmt, with one
 * margin, in two launches instead of 2 n: the same outputs, bit for bit, as n
 * separate fp8_quantise calls in order.  Meant for tensors that are ready at
 * the same time (a linear's weight and input before its forward matmul).
 * t[i]: the arguments of call i (host array, read before returning; every
 * pointer in it is a device pointer).  Either every non-empty tensor has a
 * bias_pred or none has.  Workspaces must be distinct, and no output may
 * alias another tensor's input or outputs.  n == 0 does nothing.
 * Errors: those fp8_quantise would return for any t[i], FP8_EINVAL for n out
 * of range, a null t or mixed predictions; nothing is launched then.
 */
#define FP8_QUANTISE_BATCH_MAX 4
typedef struct fp8_quantise_args {
    const void *x;
    int64_t rows, cols, ldx;
    const int32_t *bias_pred;
    int32_t *bias;
    uint32_t *amax_bits, *flags;
    uint8_t *q;
    int64_t ldq;
    uint8_t *qT;
    int64_t ldqT;
    void *ws;
    size_t ws_bytes;
} fp8_quantise_args;
int32_t fp8_quantise_batch(int32_t n, const fp8_quantise_args *t, int32_t dt, int32_t fmt,
                           int32_t margin, void *stream);

/*
 * fp8_quantise_segments -- FP8-AMAX for every row segment of one tensor in one
 * call: the paper takes a bias per micro-batch and per data or tensor replica
 * (Sec. 4), and per data sample at inference (the per-sample activation biases
 * whose mode App. D and F plot).  Rows offsets[s] <= r < offsets[s+1] form
 * segment s; each segment gets its own amax, Eq. 3 bias (format fmt, margin)
 * and flags, and its rows are cast with its bias.
 * x:         [rows, cols] of type dt, row stride ldx >= cols.
 * offsets:   device int32 [nseg + 1], nondecreasing from 0 to rows (read on
 *            the device; other contents give unspecified biases and codes but
 *            never an access out of bounds).  nseg >= 1.
 * bias, amax_bits: out, device [nseg]; flags: out, optional, [nseg].
 * row_bias:  out, device int32 [rows]: the bias of each row's segment (the
 *            per-row bias of fp8_linear_fwd_rows).
 * q, qT:     out, optional: codes [rows, cols] (row stride ldq) and
 *            transposed codes [cols, rows] (row stride ldqT).
 * An empty segment has amax 0, bias 0 and FP8_FLAG_ZERO.
 */
int32_t fp8_quantise_segments(const void *x, int32_t dt, int64_t rows, int64_t cols, int64_t ldx, int32_t fmt,
                              int32_t margin, const int32_t *offsets, int64_t nseg, int32_t *bias,
                              uint32_t *amax_bits, uint32_t *flags, int32_t *row_bias, uint8_t *q, int64_t ldq,
                              uint8_t *qT, int64_t ldqT, void *stream);

/*
 * fp8_linear_fwd_rows -- the forward matmul of fp8_linear_fwd with one
 * activation bias per row (per data sample, Sec. 3.1 inference with the
 * activation bias of each sample):
 *   Y[m, n] = 2^-(bx_rows[m] + bw) * sum_k X8[m, k] * W8[k, n]
 * bx_rows: device int32 [M] (row_bias of fp8_quantise_segments).  The other
 * arguments are those of fp8_linear_fwd.
 */
int32_t fp8_linear_fwd_rows(const uint8_t *x8, const int32_t *bx_rows, const uint8_t *w8t, const int32_t *bw,
                            void *y, int32_t y_dt, int64_t M, int64_t N, int64_t K, uint32_t *y_amax_bits,
                            void *stream);

/*
 * fp8_bias_mode -- bias telemetry (App. D and F plot the statistical mode of
 * the per-sample biases of a batch, step by step): the mode of bias[0..n)
 * (the most frequent value; the smallest of equally frequent ones; a bias
 * below -1024 counts as -1024, one above 1023 as 1023) is written to
 * ring[*count % capacity], then *count is incremented, all on the device, so
 * a captured graph keeps appending.  n == 0 is a no-op.
 * ring: device int32 [capacity], capacity >= 1.  count: device uint32.
 */
int32_t fp8_bias_mode(const int32_t *bias, int64_t n, int32_t *ring, int64_t capacity, uint32_t *count,
                      void *stream);

/*
 * fp8_linear_fwd -- forward FP8 matmul with unscale (Sec. 2, Eq. 2):
 *   Y[m, n] = 2^-(bx + bw) * sum_k X8[m, k] * W8[k, n]
 * x8:  [M, K] E4M3 codes (dense), bias *bx.
 * w8t: [N, K] E4M3 codes: the weight [K, N] stored transposed (qT of its cast),
 *      bias *bw.
 * y:   out, [M, N] dense, y_dt = FP8_DT_BF16 or FP8_DT_F32.
 * y_amax_bits: optional out: if given, the fp32 bit pattern of max|Y| (of
 *      the rounded outputs) is written there, so that the next layer can take
 *      its bias with fp8_bias_from_amax instead of reading Y again.  A NaN
 *      output gives 0x7FC00000.
 * M == 0 or N == 0: nothing is computed and *y_amax_bits (if given) is set to
 * 0, the amax of an empty output; K == 0 writes zeros.
 * Alignment: x8 and w8t must start on 16-byte boundaries whatever K is, y on
 * its element size; FP8_EINVAL otherwise.
 * Kernels: K a multiple of 128 runs the matrix-core kernels that stage whole
 * 128-byte rows of both operands through LDS; any other K runs a 64 x 64 tile
 * kernel with bounds checks and zero fill, the same results: with K a
 * multiple of 16 it loads 16-byte chunks and takes about 4x the time of the
 * staged kernels (measured 4096 x 4096 x 4032: 225 us against 63 us for
 * K = 4096; 4096 x 11008 x 4032: 640 us against 147 us); with any other K
 * it loads single bytes, about 40x.
 * The same rules hold for every matmul entry point below.
 */
int32_t fp8_linear_fwd(const uint8_t *x8, const int32_t *bx, const uint8_t *w8t, const int32_t *bw,
                       void *y, int32_t y_dt, int64_t M, int64_t N, int64_t K,
                       uint32_t *y_amax_bits, void *stream);

/*
 * fp8_linear_bwd_dx -- grad-input FP8 matmul (Sec. 2.2):
 *   dX[m, k] = 2^-(bg + bw) * sum_n dY8[m, n] * W8[k, n]
 * dy8: [M, N] E5M2 codes, bias *bg.   w8: [K, N] E4M3 codes, bias *bw.
 * dx:  out, [M, K], dx_dt.   dx_amax_bits: optional, as in fp8_linear_fwd.
 */
int32_t fp8_linear_bwd_dx(const uint8_t *dy8, const int32_t *bg, const uint8_t *w8,
                          const int32_t *bw, void *dx, int32_t dx_dt, int64_t M, int64_t N,
                          int64_t K, uint32_t *dx_amax_bits, void *stream);

/*
 * fp8_linear_fwd_bias / fp8_linear_bwd_dx_bias -- fp8_linear_fwd /
 * fp8_linear_bwd_dx with the amax of the output turned into the Eq. 3 bias
 * (Sec. 3) for the layer that consumes it, in the same launch: the same
 * y / dx, bias, amax and flags as the matmul with y_amax_bits followed by
 * fp8_bias_from_amax, without the separate zeroing and bias launches (the
 * last workgroup of the matmul to finish computes the bias).
 * y / dx:  out, as fp8_linear_fwd / fp8_linear_bwd_dx (bf16 or fp32).
 * *_fmt, margin: format and margin of the bias (as fp8_scale_bias).
 * *_bias:  out, the bias.  *_amax_bits, *_flags: out, optional (NULL).
 * ws:      workspace of fp8_linear_bias_ws_bytes() bytes, 4-byte aligned,
 *          which must hold zeros before the first call; every call that
 *          returns FP8_OK and runs to completion leaves it zero again.
 *          Calls that may run at the same time need separate workspaces.
 * M == 0 or N == 0 (no output): bias 0, amax 0, flags FP8_FLAG_ZERO.
 */
size_t fp8_linear_bias_ws_bytes(void);
int32_t fp8_linear_fwd_bias(const uint8_t *x8, const int32_t *bx, const uint8_t *w8t, const int32_t *bw,
                            void *y, int32_t y_dt, int64_t M, int64_t N, int64_t K, int32_t y_fmt,
                            int32_t margin, int32_t *y_bias, uint32_t *y_amax_bits, uint32_t *y_flags,
                            void *ws, size_t ws_bytes, void *stream);
int32_t fp8_linear_bwd_dx_bias(const uint8_t *dy8, const int32_t *bg, const uint8_t *w8, const int32_t *bw,
                               void *dx, int32_t dx_dt, int64_t M, int64_t N, int64_t K, int32_t dx_fmt,
                               int32_t margin, int32_t *dx_bias, uint32_t *dx_amax_bits, uint32_t *dx_flags,
                               void *ws, size_t ws_bytes, void *stream);

/*
 * fp8_linear_fwd_quantise / fp8_linear_bwd_dx_quantise -- the matmul of
 * fp8_linear_fwd / fp8_linear_bwd_dx (bf16 output) with the amax, Eq. 3 bias
 * and cast of its output fused into the epilogue, for the next layer that
 * consumes it (Sec. 3: the bias of a tensor needs its amax before the cast, a
 * second pass over the output).  Same bits as the matmul followed by
 * fp8_quantise on its output: the epilogue casts with the predicted bias
 * while it takes the output's amax; if the exact bias differs, a second kernel
 * re-casts from the bf16 output it has just written.
 * y / dx:       out, the bf16 product [M, N] (fwd) / [M, K] (dx), dense.
 * *_fmt, margin, *_bias_pred, *_bias, *_amax_bits, *_flags: as fp8_quantise
 *               (bias_pred NULL: the matmul, then a two-pass quantise).
 * y8 / dx8:     out, codes of the output, row stride ld >= its columns.
 * y8t / dx8t:   out, optional, the transposed codes, row stride >= its rows.
 * ws:           workspace of fp8_linear_quantise_ws_bytes(rows, cols) bytes of
 *               the output, 4-byte aligned; scratch.
 */
size_t fp8_linear_quantise_ws_bytes(int64_t rows, int64_t cols);
int32_t fp8_linear_fwd_quantise(const uint8_t *x8, const int32_t *bx, const uint8_t *w8t,
                                const int32_t *bw, void *y, int64_t M, int64_t N, int64_t K,
                                int32_t y_fmt, int32_t margin, const int32_t *y_bias_pred,
                                int32_t *y_bias, uint32_t *y_amax_bits, uint32_t *y_flags,
                                uint8_t *y8, int64_t ldy8, uint8_t *y8t, int64_t ldy8t, void *ws,
                                size_t ws_bytes, void *stream);
int32_t fp8_linear_bwd_dx_quantise(const uint8_t *dy8, const int32_t *bg, const uint8_t *w8,
                                   const int32_t *bw, void *dx, int64_t M, int64_t N, int64_t K,
                                   int32_t dx_fmt, int32_t margin, const int32_t *dx_bias_pred,
                                   int32_t *dx_bias, uint32_t *dx_amax_bits, uint32_t *dx_flags,
                                   uint8_t *dx8, int64_t lddx8, uint8_t *dx8t, int64_t lddx8t,
                                   void *ws, size_t ws_bytes, void *stream);

/*
 * fp8_linear_bwd_dw -- grad-weight FP8 matmul (Sec. 2.2):
 *   dW[k, n] = 2^-(bx + bg) * sum_m X8[m, k] * dY8[m, n]
 * x8t:  [K, M] E4M3 codes: X8 transposed (qT of the activation cast), bias *bx.
 * dy8t: [N, M] E5M2 codes: dY8 transposed (qT of the gradient cast), bias *bg.
 * dw:   out, [K, N], dw_dt (fp32 recommended: it feeds the weight update).
 */
int32_t fp8_linear_bwd_dw(const uint8_t *x8t, const int32_t *bx, const uint8_t *dy8t,
                          const int32_t *bg, void *dw, int32_t dw_dt, int64_t M, int64_t N,
                          int64_t K, void *stream);

/*
 * ptq_quantise_weights -- post-training quantisation of one weight tensor
 * (Sec. 3.1): the bias is computed once from the whole tensor, then the
 * weight is scaled and cast to E4M3.
 * w:   [K, N] of type dt (dense).
 * w8:  out, optional, [K, N] E4M3 codes (operand of fp8_linear_bwd_dx).
 * w8t: out, optional, [N, K] E4M3 codes (operand of fp8_linear_fwd).
 *      At least one of w8 / w8t must be given.
 * bw:  out, the weight's bias (device).  flags: optional, as fp8_scale_bias.
 * ws:  workspace of fp8_scale_bias_ws_bytes(K * N) bytes.
 * K * N above the element count fp8_scale_bias accepts (2^46) is FP8_EINVAL.
 */
int32_t ptq_quantise_weights(const void *w, int32_t dt, int64_t K, int64_t N, uint8_t *w8,
                             uint8_t *w8t, int32_t *bw, uint32_t *flags, void *ws,
                             size_t ws_bytes, void *stream);

/*
 * ---- Llama 2 decoder layer: the higher-precision layers (App. E) ---------
 * The paper quantises the four linear layers of each decoder layer to FP8
 * (QKV projection, attention output projection, the two feed-forward
 * layers) and keeps the rest in higher precision; the Llama 2 decoder has
 * RMSNorm pre-normalisation, SwiGLU, rotary position embeddings and, in the
 * 70B model, grouped-query attention (Sec. 4.3, Table 1).  These calls are
 * that rest, in bf16 with fp32 arithmetic; every output is rounded once to
 * bf16 (nearest even).  All tensors are bf16, row-major, 16-byte aligned,
 * with row strides (ld*, in elements) that are multiples of 8.
 *
 * Fused quantise.  Where an FP8 linear consumes the output (RMSNorm, attention,
 * SwiGLU), the call can also produce its FP8-AMAX codes (Sec. 2.3 Eq. 3,
 * Sec. 2.1 Eq. 1): pass q (codes [rows, cols], 8-byte aligned, row stride ldq
 * a multiple of 8) and the arguments of fp8_quantise (fmt, margin,
 * bias_pred, bias, amax_bits, flags) with a workspace of the op's *_ws_bytes.
 * The bf16 output, bias, amax, flags and codes are bit for bit those of the
 * op followed by fp8_quantise of its output: the kernel casts with the
 * prediction while it takes the amax, and only a wrong prediction costs a
 * re-cast from the bf16 output.  q == NULL: no quantise (fmt, margin,
 * bias_pred, bias, amax_bits, flags and ws are then ignored).  An empty
 * output with q gives amax 0, bias 0 and FP8_FLAG_ZERO.
 * The workspace is scratch; concurrent calls need distinct workspaces.
 * Outputs must not overlap inputs unless stated.
 */

/*
 * llama_rmsnorm_quantise -- RMSNorm of each row, optionally of a residual sum:
 *   h = x (res == NULL) or round(x + res);
 *   y = round(h / sqrt(mean_j h_j^2 + eps) * g)
 * x, res: [rows, cols] (row strides ldx, ldr); g: the gain [cols].
 * h: out, optional, [rows, cols] (the new residual stream).
 * y: out, [rows, cols].  cols a multiple of 8; eps >= 0 (Llama 2: 1e-5).
 * The mean square is accumulated in fp32 in a fixed order.
 */
size_t llama_rmsnorm_ws_bytes(int64_t rows);
int32_t llama_rmsnorm_quantise(const void *x, int64_t ldx, const void *res, int64_t ldr, const void *g,
                               int64_t rows, int64_t cols, float eps, void *h, int64_t ldh, void *y,
                               int64_t ldy, int32_t fmt, int32_t margin, const int32_t *bias_pred,
                               int32_t *bias, uint32_t *amax_bits, uint32_t *flags, uint8_t *q, int64_t ldq,
                               void *ws, size_t ws_bytes, void *stream);

/*
 * llama_rope_table -- (cos, sin) of pos * theta^(-2i/d_head) for positions
 * 0 .. seq_len-1 and i < d_head/2, evaluated in fp64 and rounded to fp32:
 * table[2 * (pos * d_head/2 + i) + {0, 1}] (device, 8-byte aligned,
 * seq_len * d_head floats).  d_head a multiple of 16; theta > 0 (Llama 2: 10000).
 *
 * llama_rope -- rotary embedding, in place, of n_heads consecutive heads of
 * d_head columns starting at x: element i < d_head/2 of a head pairs with
 * element i + d_head/2 ("rotate half"), row r sits at position r mod seq_len:
 *   (a, b) -> round(a cos - b sin), round(b cos + a sin).
 * x: [rows, ld] with ld >= n_heads * d_head; table from llama_rope_table with
 * the same seq_len and d_head.
 */
int32_t llama_rope_table(int64_t seq_len, int32_t d_head, double theta, float *table, void *stream);
int32_t llama_rope(void *x, int64_t rows, int64_t ld, int32_t n_heads, int32_t d_head, int64_t seq_len,
                   const float *table, void *stream);

/*
 * llama_attention -- causal softmax attention with grouped-query heads:
 *   o_i = sum_{j <= i} softmax_j(q_i . k_j / sqrt(d_head)) v_j
 * within each sequence of seq_len consecutive rows (the last may be shorter).
 * qkv: [rows, ld], the QKV projection's output (after llama_rope on the Q and
 *      K heads): n_heads query heads, then n_kv_heads key heads, then
 *      n_kv_heads value heads, d_head columns each; query head h reads
 *      key/value head h / (n_heads / n_kv_heads).
 * o:   out, [rows, n_heads * d_head], row stride ldo.
 * d_head must be 128 (FP8_ENOTSUP otherwise); n_kv_heads divides n_heads.
 * Softmax in fp32; the probabilities are rounded to bf16 for the product
 * with V (accumulated in fp32).
 */
size_t llama_attention_ws_bytes(int64_t rows, int64_t seq_len, int32_t n_heads);
int32_t llama_attention(const void *qkv, int64_t rows, int64_t ld, int64_t seq_len, int32_t n_heads,
                        int32_t n_kv_heads, int32_t d_head, void *o, int64_t ldo, int32_t fmt, int32_t margin,
                        const int32_t *bias_pred, int32_t *bias, uint32_t *amax_bits, uint32_t *flags,
                        uint8_t *q, int64_t ldq, void *ws, size_t ws_bytes, void *stream);

/*
 * llama_swiglu_quantise -- SwiGLU on the fused gate+up projection output:
 *   a = round(g * sigmoid(g) * u),  g = gu[:, 0 .. ffn), u = gu[:, ffn .. 2 ffn)
 * gu: [rows, ldgu >= 2 ffn]; a: out, [rows, ffn] (row stride lda).
 * ffn a multiple of 8.
 */
size_t llama_swiglu_ws_bytes(void);
int32_t llama_swiglu_quantise(const void *gu, int64_t ldgu, int64_t rows, int64_t ffn, void *a, int64_t lda,
                              int32_t fmt, int32_t margin, const int32_t *bias_pred, int32_t *bias,
                              uint32_t *amax_bits, uint32_t *flags, uint8_t *q, int64_t ldq, void *ws,
                              size_t ws_bytes, void *stream);

/*
 * llama_residual_add -- out = round(a + b) over n elements (dense, n a
 * multiple of 8); out may be a or b.  Exact rounding of the sum.
 */
int32_t llama_residual_add(const void *a, const void *b, void *out, int64_t n, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* FP8LIN_H */
