/*
 * tbn.h -- C ABI of the Two-Bit Networks hot path on MI355X (gfx950).
 *
 * Method: Meng, Gu, Zhang, Wu, "Two-Bit Networks for Deep Learning on Resource-
 * Constrained Embedded Devices", arXiv 1701.00485.  Each real-valued filter W (n = c*w*h
 * elements) is approximated by alpha * W~ with W~_i in {-2,-1,1,2} (Sec. 2, Eq. 1-2),
 * W~ from the deterministic rule of Eq. (3) and alpha from Eq. (5).  Training follows
 * Algorithm 1 (Sec. 3): quantise every filter, run the forward and backward passes with
 * the approximate filters, and update the real weights with the gradient taken with
 * respect to the approximate filters.
 *
 * Conventions shared by every call
 *   - Activations are NHWC, dense, element (n,h,w,c) at ((n*H + h)*W + w)*C + c.
 *   - Real weights are [K][R][S][C] fp32 (filter k is row k of a [K][n] matrix with
 *     n = R*S*C, element i = (r*S + s)*C + c).
 *   - Convolution is cross-correlation with zero padding, dilation 1, one group;
 *     P = (H + 2*pad_h - R)/stride_h + 1 (floor), Q likewise.  A fully-connected layer is
 *     the 1x1 convolution over a 1x1 map (or the R x S "valid" convolution over the last
 *     map), as the paper's Sec. 3 allows.
 *   - Every pointer is a device pointer owned by the caller, 16-byte aligned, and must
 *     stay valid until the work queued on `stream` has finished.  The library allocates
 *     no memory and keeps no mutable global state; calls may come from any host thread.
 *   - Every call validates its arguments before queuing anything and returns a status;
 *     on an error nothing has been queued.  TBN_ERR_HIP reports a failed launch.  Faults
 *     during execution surface at the caller's next synchronisation of `stream`.
 *   - All work is queued asynchronously on `stream` (0 = the null stream).
 *
 * Two-bit packed codes ("TBN2" layout, this library's storage format; the paper fixes
 * only that the four values fit in two bits):
 *   filters are grouped in blocks of 64 and filter elements in blocks of 64.  With
 *   NB = ceil(n/64), KB = ceil(K/64) the array holds KB*NB*256 uint32 words and
 *   element (k, i) lives in word ((k/64*NB + i/64)*64 + k%64)*4 + (i%64)/16.  Inside a
 *   word, element e = i%16 uses j = e/2, h = e%2: bit 16h+j is set iff |W~| = 2 and bit
 *   16h+8+j is set iff W~ < 0.  Bits of padding filters and padding elements are zero.
 *   A 64-filter x 64-element block is 1 KiB and contiguous, so one wave reads it with
 *   one 16-byte load per lane, and the bf16 pair of elements (2j, 2j+1) of a word is
 *   ((word >> j) & 0x01010101) << 7 plus 0x3F803F80 -- two integer operations.
 */
#ifndef TBN_H
#define TBN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum tbn_status {
    TBN_OK = 0,
    TBN_ERR_NULL = 1,        /* a required pointer is NULL */
    TBN_ERR_SHAPE = 2,       /* a size or geometry is invalid (<= 0, empty output, overflow) */
    TBN_ERR_UNSUPPORTED = 3, /* valid request the library does not implement */
    TBN_ERR_ALIGN = 4,       /* a pointer is not 16-byte aligned */
    TBN_ERR_WORKSPACE = 5,   /* workspace missing or smaller than tbn_workspace_size() */
    TBN_ERR_HIP = 6          /* a HIP launch failed; see tbn_last_error() */
} tbn_status;

typedef enum tbn_dtype { TBN_BF16 = 0, TBN_F32 = 1 } tbn_dtype;

typedef enum tbn_op { TBN_OP_FWD = 0, TBN_OP_BWD_DATA = 1, TBN_OP_BWD_WEIGHT = 2 } tbn_op;

/* Geometry of one layer: input N x H x W x C, K filters of R x S x C. */
typedef struct tbn_conv_desc {
    int32_t n, h, w, c, k, r, s, stride_h, stride_w, pad_h, pad_w;
} tbn_conv_desc;

/* Optional fused output transform of the forward pass, applied per output element
 * (n,p,q,k) after the scale alpha_k:  y = act(alpha_k * scale[k] * acc + bias[k]
 * + residual[n,p,q,k]).  Any pointer may be NULL (scale 1, bias 0, no residual);
 * `residual` is NHWC [N][P][Q][K] with the output's dtype.  relu != 0 applies
 * max(., 0).  Used for inference-mode batch normalisation folded into scale and bias,
 * the residual add of a basic block, and ReLU. */
typedef struct tbn_epilogue {
    const float* scale;
    const float* bias;
    const void* residual;
    int32_t relu;
} tbn_epilogue;

/* Human-readable name of a status. Never NULL. */
const char* tbn_status_str(tbn_status status);

/* Detail of the last error raised on the calling thread ("" if none). */
const char* tbn_last_error(void);

/* Output spatial size of a geometry (see conventions). TBN_ERR_SHAPE if invalid. */
tbn_status tbn_conv_out_dims(const tbn_conv_desc* desc, int32_t* p, int32_t* q);

/* Number of uint32 words of the packed codes of K filters of n elements
 * (ceil(K/64) * ceil(n/64) * 256), or -1 if K or n <= 0. */
int64_t tbn_packed_words(int64_t k, int64_t n);

/* uint32 words that one filter row of n elements occupies in the TBN2 layout: the row is
 * padded to whole 64-code groups of 4 words, 4 * ceil(n/64); -1 if n <= 0. */
int64_t tbn_packed_row_words(int64_t n);

/* Bytes of the packed codes of K filters of n elements (4 * tbn_packed_words(k, n) =
 * 1024 * ceil(K/64) * ceil(n/64)), or -1 if K or n <= 0. */
int64_t tbn_packed_bytes(int64_t k, int64_t n);

/* Bytes of caller-provided workspace `op` needs for `desc` (0 = none needed).
 * Pass the same op and geometry to the corresponding call.  TBN_OP_FWD: fp32 partial sums
 * of a split reduction, or, for inputs with fewer than 8 channels and at least 2^20
 * elements, a zero-bordered bf16 copy of the input with the channels padded to a power of
 * two (the forward call writes it first); the size covers either input dtype. */
tbn_status tbn_workspace_size(tbn_op op, const tbn_conv_desc* desc, size_t* bytes);

/*
 * Quantise K real-valued filters (Sec. 2 Eq. 3 and Eq. 5; Algorithm 1, quantisation).
 *   w      [K][n] fp32, one filter per row.
 *   codes  out, tbn_packed_words(K, n) words in the TBN2 layout; every padding bit is
 *          written as zero.  W~_i = -2 if W_i < -1; -1 if -1 <= W_i <= 0 (both signed
 *          zeros); 1 if 0 < W_i <= 1; 2 if W_i > 1.  A NaN weight gets code -1.
 *   alpha  out, [K] fp32: (sum_{|W_i|<=1} |W_i| + 2 sum_{|W_i|>1} |W_i|) /
 *          (|B1| + 4|B2|) accumulated in fp64 and rounded once to fp32.  An all-zero
 *          filter gets alpha = 0 (the infimum of the paper's alpha > 0).
 *   counts out, optional (NULL to skip), [K][2] int32: |B1| = #{|W_i| <= 1} and
 *          |B2| = #{|W_i| > 1} (the index sets of Eq. 4).
 */
tbn_status tbn_quantize(const float* w, int64_t k, int64_t n, uint32_t* codes, float* alpha,
                        int32_t* counts, hipStream_t stream);

/*
 * Variants of the discretisation step (Sec. 2 chooses the deterministic rule of Eq. 3 "for
 * simplicity"; the scale is then the optimum of Eq. 4 for the chosen codes).
 *   threshold  t > 0 (finite): the magnitude-2 boundary of Eq. 3 moved from 1 to t,
 *              W~_i = -2 if W_i < -t; -1 if -t <= W_i <= 0; 1 if 0 < W_i <= t; 2 if W_i > t.
 *              t = 1 with uniform == NULL is exactly tbn_quantize.
 *   uniform    optional [K][n] fp32 numbers in [0, 1) (NULL = deterministic): stochastic
 *              discretisation.  a = clamp(W_i, -2, 2); if a > 1: 2 when u < a - 1, else 1;
 *              if a < -1: -2 when u < -1 - a, else -1; otherwise 1 when 2u < a + 1, else
 *              -1 (all fp32), so that E[W~_i] = clamp(W_i, -2, 2).  Requires t = 1
 *              (TBN_ERR_UNSUPPORTED otherwise).
 *   alpha      sum_i W_i W~_i / sum_i W~_i^2 (fp64 sums, one rounding to fp32): Eq. 5 for the
 *              deterministic rules.  codes, counts: as tbn_quantize (counts by |W~_i|).
 */
tbn_status tbn_quantize_variant(const float* w, int64_t k, int64_t n, float threshold, const float* uniform,
                                uint32_t* codes, float* alpha, int32_t* counts, hipStream_t stream);

/*
 * Forward pass of a two-bit layer (Sec. 2 Eq. 1, I * (alpha W~) = (alpha I) (+) W~;
 * Algorithm 1, forward step):  y[n,p,q,k] = alpha_k * sum_{r,s,c} x[n, p*sh-ph+r,
 * q*sw-pw+s, c] * W~[k,r,s,c], then the optional epilogue.  The products with the codes
 * are exact; accumulation is fp32 on bf16 operands; alpha is applied in fp32.
 *   x      NHWC [N][H][W][C], dtype xt (TBN_F32 input is rounded to bf16, nearest-even).
 *   codes  TBN2 packed codes of the K filters (n = R*S*C); alpha [K] fp32.
 *   ep     optional epilogue (NULL = none).
 *   y      NHWC [N][P][Q][K], dtype yt.
 *   ws     workspace of tbn_workspace_size(TBN_OP_FWD) bytes: fp32 partial sums when
 *          the layer has too few output tiles to fill the GPU and its reduction is split
 *          (may be NULL when that size is 0).  TBN_ERR_WORKSPACE if smaller.
 */
tbn_status tbn_conv2d_fwd(const tbn_conv_desc* desc, const void* x, tbn_dtype xt,
                          const uint32_t* codes, const float* alpha, const tbn_epilogue* ep,
                          void* y, tbn_dtype yt, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * The forward pass without caller workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid allocation).
 * Same arguments and results as tbn_conv2d_fwd (the same kernels run), except that the
 * workspace is a static device array of TBN_NOALLOC_SCRATCH_BYTES owned by the library:
 * one per device, held until the process ends, its address looked up on the first call on
 * each device.  The call allocates nothing.  A layer whose tbn_workspace_size(TBN_OP_FWD)
 * exceeds TBN_NOALLOC_SCRATCH_BYTES gets TBN_ERR_WORKSPACE (nothing queued); every batch-1
 * layer of the workloads fits.  All calls on one device share its array: calls whose work
 * overlaps in time on that device (other streams, other host threads) race on it and must
 * be serialised by the caller; calls on one stream are ordered and safe.
 */
#define TBN_NOALLOC_SCRATCH_BYTES (8u << 20)
tbn_status tbn_conv2d_fwd_noalloc(const tbn_conv_desc* desc, const void* x, tbn_dtype xt, const uint32_t* codes,
                                  const float* alpha, const tbn_epilogue* ep, void* y, tbn_dtype yt,
                                  hipStream_t stream);

/*
 * Integer-activation variant of the forward pass (an extension of Sec. 2 Eq. 1: the paper
 * keeps activations in full precision; its Sec. 1 motivates the two-bit filters by
 * arithmetic without multipliers).  The input I is represented as s * q, q int8, and the
 * layer runs on the int8 matrix cores, where the products q * W~ and their int32 sums are
 * exact.
 *
 * tbn_quantize_act_i8: activation codes q = clamp(round-half-even(x * inv_scale), -127, 127)
 *   with the product rounded to fp32 first; a NaN input gets 0.  x: `count` elements of
 *   dtype xt (any layout: elementwise); q: `count` int8.  inv_scale finite and > 0
 *   (typically 127 / max|x| over a calibration set), else TBN_ERR_SHAPE.
 *
 * tbn_conv2d_fwd_i8: y[n,p,q,k] = act(float(acc) * float(alpha_k * x_scale)) with
 *   acc = sum_{r,s,c} q[n, p*sh-ph+r, q*sw-pw+s, c] * W~[k,r,s,c] exact (zero padding),
 *   the scale product rounded to fp32 first; relu != 0 applies max(., 0).
 *   x      NHWC [N][H][W][C] int8 codes (for example from tbn_quantize_act_i8); x_scale =
 *          the s with x ~ s * q (1 / inv_scale), finite.
 *   codes  TBN2 packed codes of the K filters (n = R*S*C); alpha [K] fp32.
 *   y      NHWC [N][P][Q][K], dtype yt (bf16 rounded to nearest even, or fp32).
 *   Needs C % 16 == 0, R*S <= 63, 254 * R*S*C < 2^31 (int32 sums) and x and the codes
 *   below 2 GiB; TBN_ERR_UNSUPPORTED otherwise.  No workspace.
 */
tbn_status tbn_quantize_act_i8(const void* x, tbn_dtype xt, int64_t count, float inv_scale, int8_t* q,
                               hipStream_t stream);
tbn_status tbn_conv2d_fwd_i8(const tbn_conv_desc* desc, const int8_t* x, const uint32_t* codes, const float* alpha,
                             float x_scale, int32_t relu, void* y, tbn_dtype yt, hipStream_t stream);

/*
 * Eight-bit floating-point activation variant of the forward pass (an extension of Sec. 2
 * Eq. 1 of the same kind as the int8 one): the input I is represented as s * f with f an
 * E4M3 value, and the layer runs on the scaled fp8 x fp4 matrix cores, where the filter
 * values +-1 and +-2 are exact 4-bit E2M1 values and every product f * W~ is exact.
 *
 * tbn_quantize_act_fp8: activation codes f = E4M3(x * inv_scale), the product rounded to
 *   fp32 first, then the nearest finite E4M3 value (ties to the even code), |value| > 448
 *   saturating to +-448; the sign bit is kept for -0 and for values that round to zero; a
 *   NaN input gets code 0.  E4M3: bit 7 sign, bits 6-3 exponent (bias 7, 0 = subnormal),
 *   bits 2-0 fraction, no infinities, 0x7F and 0xFF NaN.  x: `count` elements of dtype xt
 *   (elementwise); q: `count` bytes.  inv_scale finite and > 0 (typically 448 / max|x|),
 *   else TBN_ERR_SHAPE.
 *
 * tbn_repack_codes_fp4: rewrites TBN2 packed codes (`words` 32-bit words, any number of
 *   filters) into the E2M1 operand layout that tbn_conv2d_fwd_fp8 reads: the same 16 bytes
 *   per filter and 64-element chunk, but word q of a chunk holds its elements 16 q + 8 r + j
 *   (r = 0, 1; j = 0..7) as magnitude bit 4 j + 1 - r and sign bit 4 j + 3 - r.  Done once
 *   per set of filters (after each quantisation); codes and out must not overlap.
 *
 * tbn_conv2d_fwd_fp8: y[n,p,q,k] = act(acc * fp32(alpha_k * x_scale)) with
 *   acc = sum_{r,s,c} f[n, p*sh-ph+r, q*sw-pw+s, c] * W~[k,r,s,c] (zero padding), each
 *   product exact and the sum in fp32 (order unspecified); relu != 0 applies max(., 0).
 *   x      NHWC [N][H][W][C] E4M3 codes (for example from tbn_quantize_act_fp8); x_scale =
 *          the s with x ~ s * f (1 / inv_scale), finite.
 *   codes  the K filters' codes (n = R*S*C) in the E2M1 layout of tbn_repack_codes_fp4;
 *          alpha [K] fp32.
 *   y      NHWC [N][P][Q][K], dtype yt (bf16 rounded to nearest even, or fp32).
 *   Needs C % 16 == 0, R*S <= 63 and x and the codes below 2 GiB; TBN_ERR_UNSUPPORTED
 *   otherwise.  No workspace.
 */
tbn_status tbn_quantize_act_fp8(const void* x, tbn_dtype xt, int64_t count, float inv_scale, uint8_t* q,
                                hipStream_t stream);
tbn_status tbn_repack_codes_fp4(const uint32_t* codes, int64_t words, uint32_t* out, hipStream_t stream);
tbn_status tbn_conv2d_fwd_fp8(const tbn_conv_desc* desc, const uint8_t* x, const uint32_t* codes, const float* alpha,
                              float x_scale, int32_t relu, void* y, tbn_dtype yt, hipStream_t stream);

/*
 * Forward pass of a layer kept in full precision (Eq. 1 with the real filters; the first
 * convolution of the CIFAR-shaped network stays unquantised):
 *   y[n,p,q,k] = sum_{r,s,c} x[n, p*sh-ph+r, q*sw-pw+s, c] * bf16(w[k,r,s,c]),
 * then the optional epilogue.  Filters are rounded to bf16 (nearest even) on load, as are
 * TBN_F32 activations; products and sums are fp32.  Meant for thin layers (few input
 * channels): it runs on the vector ALUs, not the matrix cores.
 *   x   NHWC [N][H][W][C], dtype xt.   w  [K][R][S][C] fp32.   y  NHWC [N][P][Q][K], dtype yt.
 */
tbn_status tbn_conv2d_fwd_dense(const tbn_conv_desc* desc, const void* x, tbn_dtype xt, const float* w,
                                const tbn_epilogue* ep, void* y, tbn_dtype yt, hipStream_t stream);

/*
 * Backward pass to the layer input through the approximate filters W^ = alpha W~
 * (Sec. 3: both passes use the approximate filters; Algorithm 1, backward step):
 *   dx[n,h,w,c] = sum over (p,q,k,r,s) with p*sh-ph+r = h, q*sw-pw+s = w of
 *                 alpha_k W~[k,r,s,c] dy[n,p,q,k].
 * alpha_k W~ is formed exactly from bf16(alpha_k) (the codes only flip the sign and add
 * one to the exponent), so the only rounding beyond fp32 accumulation is alpha to bf16.
 *   dy     NHWC [N][P][Q][K] bf16.   dx  NHWC [N][H][W][C], dtype dxt (overwritten).
 *   ws     tbn_workspace_size(TBN_OP_BWD_DATA) bytes: the codes re-packed for the
 *          transposed, flipped filter and the bf16 scales.
 * Requires stride 1 in both directions (TBN_ERR_UNSUPPORTED otherwise).
 */
tbn_status tbn_conv2d_bwd_data(const tbn_conv_desc* desc, const void* dy, const uint32_t* codes,
                               const float* alpha, void* dx, tbn_dtype dxt, void* ws,
                               size_t ws_bytes, hipStream_t stream);

/*
 * Gradient with respect to the approximate filter (Algorithm 1, backward step), which
 * Sec. 3 applies unchanged to the real-valued filter (straight-through):
 *   dw[k,r,s,c] (+)= sum_{n,p,q} dy[n,p,q,k] * x[n, p*sh-ph+r, q*sw-pw+s, c].
 *   x   NHWC [N][H][W][C] bf16.   dy  NHWC [N][P][Q][K] bf16.
 *   dw  [K][R][S][C] fp32; overwritten, or added to when accumulate != 0.
 *   ws  tbn_workspace_size(TBN_OP_BWD_WEIGHT) bytes of fp32 split-reduction partials.
 * The result is deterministic: partial sums are combined in a fixed order.
 */
tbn_status tbn_conv2d_bwd_weight(const tbn_conv_desc* desc, const void* x, const void* dy,
                                 float* dw, int32_t accumulate, void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/*
 * Update of the real weights (Algorithm 1, update step) with the optimiser of Sec. 4,
 * SGD with momentum and weight decay, no dampening, no Nesterov term:
 *   v = momentum * v + (g + weight_decay * w);   w = w - lr * v        (fp32, in place)
 *   w, v, g  [count] fp32.
 */
tbn_status tbn_sgd_step(float* w, float* v, const float* g, int64_t count, float lr,
                        float momentum, float weight_decay, hipStream_t stream);

/*
 * The update step of Algorithm 1 fused with the quantisation that opens the next
 * iteration (Sec. 2 Eq. 3 and Eq. 5 applied to the updated filters), in one pass over
 * the real weights:
 *   v = momentum * v + (g + weight_decay * w);   w = w - lr * v   (fp32, in place, the same
 *   rounding as tbn_sgd_step), then codes / alpha / counts of the updated w exactly as
 *   tbn_quantize would produce them.
 *   w, v, g  [K][n] fp32, one filter per row.   codes, alpha, counts: as tbn_quantize.
 * Reads 12 bytes and writes 8.25 bytes per weight, against 16 + 8.25 for tbn_sgd_step
 * followed by tbn_quantize.
 */
tbn_status tbn_sgd_step_quantize(float* w, float* v, const float* g, int64_t k, int64_t n, float lr,
                                 float momentum, float weight_decay, uint32_t* codes, float* alpha,
                                 int32_t* counts, hipStream_t stream);

/* ------------------------------------------------------------------------------------ */
/* Layers around the two-bit convolutions in the workloads (Sec. 4 names ResNet-18 with   */
/* batch normalisation; the smaller workloads add max pooling, ReLU and a softmax         */
/* cross-entropy loss).  Activations are NHWC bf16 unless stated; same conventions as    */
/* above (device pointers, 16-byte alignment, asynchronous on `stream`).                  */
/* ------------------------------------------------------------------------------------ */

/* Pooling geometry: input N x H x W x C, square window k, stride, zero-size padding
 * (padded positions never win a maximum).  P = (H + 2*pad - k)/stride + 1 (floor).
 * TBN_ERR_SHAPE if H*W, H + 2*pad + stride or W + 2*pad + stride exceeds 2^31 - 1 (positions
 * and argmax are 32-bit) or the input or output has more than 2^40 elements. */
typedef struct tbn_pool_desc {
    int32_t n, h, w, c, k, stride, pad;
} tbn_pool_desc;

tbn_status tbn_pool_out_dims(const tbn_pool_desc* desc, int32_t* p, int32_t* q);

/* y[n,p,q,c] = max over the window; argmax (optional, int32 [N][P][Q][C]) receives the
 * input position h*W + w of the maximum, ties going to the first in row-major window
 * order (-1 for an empty window, whose output is 0). */
tbn_status tbn_maxpool2d_fwd(const tbn_pool_desc* desc, const void* x, void* y, int32_t* argmax,
                             hipStream_t stream);

/* dx[n,h,w,c] = sum of dy[n,p,q,c] over the windows whose argmax is (h, w).  dx has dtype
 * dxt and is overwritten (deterministic gather, no atomics). */
tbn_status tbn_maxpool2d_bwd(const tbn_pool_desc* desc, const void* dy, const int32_t* argmax, void* dx,
                             tbn_dtype dxt, hipStream_t stream);

/* y[n][c] = mean over (h, w) of x[n][h][w][c] (fp32 sum); y has dtype yt.  TBN_ERR_SHAPE
 * if h*w > 2^31 - 1 or x has more than 2^40 elements. */
tbn_status tbn_avgpool_global(int32_t n, int32_t h, int32_t w, int32_t c, const void* x, void* y, tbn_dtype yt,
                              hipStream_t stream);

/* Bytes of fp32 workspace the two batch-normalisation calls need for rows x c (per-chunk
 * partial sums of the per-channel reductions). */
tbn_status tbn_batchnorm_workspace_size(int64_t rows, int32_t c, size_t* bytes);

/* Batch normalisation with batch statistics over rows = N*H*W positions per channel:
 * y = act(gamma (x - mean) inv_std + beta), inv_std = 1/sqrt(biased var + eps);
 * relu != 0 fuses max(., 0).  mean and inv_std [c] are written for the backward pass.
 * The mean and the centred sum of squares are two passes of fixed-order fp32 sums
 * (deterministic).  ws: tbn_batchnorm_workspace_size bytes (TBN_ERR_WORKSPACE if less). */
tbn_status tbn_batchnorm_train_fwd(const void* x, int64_t rows, int32_t c, const float* gamma, const float* beta,
                                   float eps, int32_t relu, void* y, float* mean, float* inv_std, void* ws,
                                   size_t ws_bytes, hipStream_t stream);

/* Backward of the above (through the batch statistics; with relu, g = dy * [y > 0]):
 * dx = gamma inv_std (g - mean(g) - xhat mean(g xhat)), dgamma = sum g xhat,
 * dbeta = sum g.  Sums are taken in a fixed order.  ws as for the forward call. */
tbn_status tbn_batchnorm_train_bwd(const void* x, const void* y, const void* dy, int64_t rows, int32_t c,
                                   int32_t relu, const float* mean, const float* inv_std, const float* gamma,
                                   float* dgamma, float* dbeta, void* dx, void* ws, size_t ws_bytes, hipStream_t stream);

/* dx = dy where y > 0, else 0 (ReLU'(0) = 0). */
tbn_status tbn_relu_bwd(const void* y, const void* dy, int64_t count, void* dx, hipStream_t stream);

/* Softmax cross-entropy over fp32 logits [n][classes] with int32 labels: loss[0] = mean
 * over the batch of logsumexp(z) - z[label]; dlogits (bf16) = (softmax(z) - onehot)/n.
 * loss_per_sample is caller workspace of n floats.  Labels live in device memory and are
 * not checked before the launch: a label outside [0, classes) gives that sample a NaN loss
 * (so loss[0] is NaN) and the gradient softmax(z)/n with no one-hot term; nothing is read
 * out of bounds. */
tbn_status tbn_softmax_xent(const float* logits, const int32_t* labels, int32_t n, int32_t classes, float* loss,
                            float* loss_per_sample, void* dlogits, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* TBN_H */
