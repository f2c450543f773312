/*
 * libquan -- the QUAN hot path on AMD Instinct MI355X (gfx950).
 *
 * Paper: "Quaternion Approximate Networks for Enhanced Image Classification
 * and Oriented Object Detection" (arXiv 2509.05512).
 *
 * Two operations, each a plain C entry point over device pointers:
 *   - the quaternion 2-D convolution as a Hamilton product (Section III-B,
 *     eqs. 5 and 6), and
 *   - Independent Quaternion Batch Normalization (Section III-C, eqs. 11, 12).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Quaternion components are ordered q = r, i, j, k (0..3).  A quaternion
 * feature map of C channels has the logical shape [N, 4, C, H, W]; in memory
 * it is channels-last by component, i.e. the dense array [N][H][W][4][C]: for
 * each pixel the 4*C reals are contiguous, component-major.  The same tensor
 * seen by PyTorch is x.permute(0, 3, 4, 1, 2) of a contiguous [N, H, W, 4, C].
 *
 * All tensor pointers are device pointers owned by the caller; the library
 * never frees or retains them.  Activation and output pointers must be 16-byte
 * aligned; every other pointer must be aligned to its element size.  No tensor
 * may hold 2^31 or more elements, and for the convolution one input image
 * (H*W*4*C elements) times (256 / (H_out*W_out) + 2) must stay below 2^31
 * bytes (the kernels address a tile's activations with 32-bit offsets).
 *
 * dtype is QUAN_F32 or QUAN_BF16 and applies to activations, weights, bias and
 * outputs of the convolution and to the IQBN input/output; accumulation is
 * always fp32, and IQBN's gamma, beta, mean and var are always fp32.
 *
 * Every call validates its arguments on the host before it touches the device
 * and returns QUAN_OK (0) or a negative QUAN_ERR_* code; quan_last_error()
 * then describes the failure (per thread).  A successful call has only
 * enqueued its kernels on `stream` (a hipStream_t; NULL is the default
 * stream): errors raised while they run surface at the next synchronisation.
 *
 * The library keeps a small per-(device, stream) workspace (the packed
 * convolution weights and IQBN partial statistics), allocated with hipMalloc
 * on first use and grown on demand; quan_release() frees it.  Calls issued to
 * different streams never share a workspace.
 */
#ifndef QUAN_H
#define QUAN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define QUAN_API __attribute__((visibility("default")))

enum quan_dtype { QUAN_F32 = 0, QUAN_BF16 = 1 };

enum quan_status {
    QUAN_OK = 0,
    QUAN_ERR_NULL = -1,        /* a required pointer is NULL */
    QUAN_ERR_SHAPE = -2,       /* a size is <= 0, or the output would be empty */
    QUAN_ERR_DTYPE = -3,       /* dtype is not QUAN_F32 / QUAN_BF16 */
    QUAN_ERR_ALIGN = -4,       /* a pointer violates its alignment requirement */
    QUAN_ERR_ALIAS = -5,       /* an output overlaps an input it may not overlap */
    QUAN_ERR_UNSUPPORTED = -6, /* a size exceeds the library's limits */
    QUAN_ERR_HIP = -7,         /* the HIP runtime reported an error */
    QUAN_ERR_NOMEM = -8,       /* the workspace could not be allocated */
    QUAN_ERR_LAYOUT = -9       /* a descriptor's strides are not the layout required */
};

/*
 * Quaternion convolution Y = W (x) X + b  (Section III-B, eq. 5; the signed
 * 4x4 block of eq. 6 at every tap).
 *
 * With W = W_r + W_i i + W_j j + W_k k and (x) the Hamilton product of eq. 3
 * with the kernel on the left, for every image n, output channel o and output
 * pixel (y, x):
 *
 *   Y[n,o,y,x] = b[o] + sum_{c, ky, kx} W[o,c,ky,kx] (x) X[n,c,iy,ix],
 *   iy = y*stride_h - pad_h + ky*dilation_h,  ix = x*stride_w - pad_w + kx*dilation_w,
 *
 * a cross-correlation (no kernel flip) in which taps outside the image read
 * zero.  Ho = (h + 2*pad_h - dilation_h*(k_h-1) - 1)/stride_h + 1, likewise Wo.
 *
 *   x       [n, 4, c_in, h, w] channels-last by component (see above)
 *   w_r..w_k  the four real kernels, each dense [c_out, c_in, k_h, k_w] (OIHW)
 *   bias    [4, c_out] (component-major), or NULL for no bias
 *   out     [n, 4, c_out, Ho, Wo] channels-last by component; written in full.
 *           It must not overlap x, a kernel or the bias.
 *   stride, dilation >= 1; pad >= 0; all sizes >= 1.
 *
 * bf16 outputs are the fp32 accumulator rounded to nearest even.
 * Returns QUAN_ERR_SHAPE when Ho or Wo would be < 1.
 */
QUAN_API int quan_qconv2d_forward(const void *x,
                                  const void *w_r, const void *w_i,
                                  const void *w_j, const void *w_k,
                                  const void *bias,
                                  int32_t stride_h, int32_t stride_w,
                                  int32_t pad_h, int32_t pad_w,
                                  int32_t dilation_h, int32_t dilation_w,
                                  void *out,
                                  int32_t n, int32_t c_in, int32_t h, int32_t w,
                                  int32_t c_out, int32_t k_h, int32_t k_w,
                                  int32_t dtype, void *stream);

/*
 * The same convolution split in two, for callers whose kernels stay fixed
 * across calls (inference): pack W_r..W_k once, then run the convolution on
 * the packed weights.  quan_qconv2d_forward is exactly
 * quan_qconv2d_pack_weights into a library workspace followed by
 * quan_qconv2d_forward_packed.
 *
 * quan_qconv2d_packed_bytes returns the size in bytes of the packed weights
 * for (c_in, c_out, k_h, k_w, dtype), or a negative QUAN_ERR_* code
 * (QUAN_ERR_UNSUPPORTED when they would reach 2^31 bytes).  The packed
 * layout is private to the library but depends only on these five values:
 * weights packed once serve every later call with the same ones.
 *
 * quan_qconv2d_pack_weights reads w_r..w_k (as in quan_qconv2d_forward) and
 * writes `packed`, a caller-owned, 16-byte-aligned device buffer of at least
 * quan_qconv2d_packed_bytes(...) bytes (`packed_bytes` states its size) that
 * must not overlap the kernels.
 *
 * quan_qconv2d_forward_packed takes the packed buffer in place of the four
 * kernels; every other argument is as in quan_qconv2d_forward, and out must
 * not overlap `packed` either.
 */
QUAN_API int64_t quan_qconv2d_packed_bytes(int32_t c_in, int32_t c_out, int32_t k_h, int32_t k_w,
                                           int32_t dtype);

QUAN_API int quan_qconv2d_pack_weights(const void *w_r, const void *w_i,
                                       const void *w_j, const void *w_k,
                                       int32_t c_in, int32_t c_out, int32_t k_h, int32_t k_w,
                                       int32_t dtype, void *packed, int64_t packed_bytes,
                                       void *stream);

QUAN_API int quan_qconv2d_forward_packed(const void *x, const void *packed, const void *bias,
                                         int32_t stride_h, int32_t stride_w,
                                         int32_t pad_h, int32_t pad_w,
                                         int32_t dilation_h, int32_t dilation_w,
                                         void *out,
                                         int32_t n, int32_t c_in, int32_t h, int32_t w,
                                         int32_t c_out, int32_t k_h, int32_t k_w,
                                         int32_t dtype, void *stream);

/*
 * The separable QUAN convolution of Section III-B, eq. 7, with the same
 * arguments, layouts, packed weights and limits as quan_qconv2d_forward and
 * quan_qconv2d_forward_packed: each output component is a signed sum of the
 * four real convolutions W_q (*) x_q only,
 *
 *   y_r = W_r*x_r - W_i*x_i - W_j*x_j - W_k*x_k
 *   y_i = W_r*x_r + W_i*x_i + W_j*x_j - W_k*x_k
 *   y_j = W_r*x_r - W_i*x_i + W_j*x_j + W_k*x_k
 *   y_k = W_r*x_r + W_i*x_i - W_j*x_j + W_k*x_k      (+ bias per component)
 *
 * a quarter of the Hamilton product's multiply-adds.  It is not a Hamilton
 * product (the identity kernel maps x to (x_r, x_r, x_r, x_r)); its sign
 * matrix is the transpose of the mixing matrix printed for the backward
 * pass (eq. 9).  The four sums are formed in fp32 and rounded once.
 */
QUAN_API int quan_qconv2d_separable_forward(const void *x, const void *w_r, const void *w_i,
                                            const void *w_j, const void *w_k, const void *bias,
                                            int32_t stride_h, int32_t stride_w,
                                            int32_t pad_h, int32_t pad_w,
                                            int32_t dilation_h, int32_t dilation_w,
                                            void *out, int32_t n, int32_t c_in, int32_t h,
                                            int32_t w, int32_t c_out, int32_t k_h, int32_t k_w,
                                            int32_t dtype, void *stream);

QUAN_API int quan_qconv2d_separable_forward_packed(const void *x, const void *packed,
                                                   const void *bias, int32_t stride_h,
                                                   int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                                   int32_t dilation_h, int32_t dilation_w,
                                                   void *out, int32_t n, int32_t c_in, int32_t h,
                                                   int32_t w, int32_t c_out, int32_t k_h,
                                                   int32_t k_w, int32_t dtype, void *stream);

/*
 * Independent Quaternion Batch Normalization (Section III-C, eqs. 11, 12).
 *
 * For every component q and channel ch separately, over the P = n*h*w values
 * x[:, q, ch, :, :]:
 *
 *   mean[q,ch] = (1/P) sum x
 *   var[q,ch]  = (1/P) sum (x - mean)^2          (biased, as in eq. 11)
 *   out = (x - mean) / sqrt(var + eps) * gamma[q,ch] + beta[q,ch]
 *
 *   x, out        [n, 4, c, h, w] channels-last by component; out may equal x
 *                 (in place) but may not otherwise overlap it.
 *   gamma, beta   [4, c] fp32 device arrays.
 *   mean, var     [4, c] fp32 device arrays receiving the batch statistics used
 *                 for normalisation.  Running statistics are the caller's.
 *   eps           > 0.
 *
 * Tensors of 16 MiB or more whose rows fit the registers and LDS of one
 * work-group per compute unit (about 100 MB on MI355X) are normalised in
 * one launch that reads x once; its work-groups exchange partial sums
 * through device memory and wait for each other, so the launch needs every
 * compute unit of the device at once.  If other work holds compute units
 * for more than about a second meanwhile, the waits give up and the rows
 * and statistics of the work-groups that gave up come back as NaN (never a
 * hang).  Smaller or larger tensors run in three launches with no such
 * wait.
 */
QUAN_API int quan_iqbn_forward(const void *x, const float *gamma, const float *beta,
                               float eps, void *out, float *mean, float *var,
                               int32_t n, int32_t c, int32_t h, int32_t w,
                               int32_t dtype, void *stream);

/*
 * quan_iqbn_forward for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, result and validation as quan_iqbn_forward;
 * the partial statistics live in a fixed 8 MiB array of device memory per
 * GPU (held until the process ends) instead of a library workspace, so the
 * call performs no allocation.  It returns QUAN_ERR_UNSUPPORTED, before any
 * device work, when the tensor needs more scratch than that ((2 * blocks +
 * 3) * 4c floats, at most 512 blocks: up to 510 channels at any size,
 * more for small batches).  Every call on one GPU shares that GPU's array:
 * calls that may overlap in time (other streams, other threads) race, and
 * must be serialised by the caller.
 */
QUAN_API int quan_iqbn_forward_noalloc(const void *x, const float *gamma, const float *beta,
                                       float eps, void *out, float *mean, float *var,
                                       int32_t n, int32_t c, int32_t h, int32_t w,
                                       int32_t dtype, void *stream);

/* As quan_iqbn_forward, followed by a component-wise max(0, .) on out (the
 * IQBN + ReLU pairing of the quaternion networks of Section IV). */
QUAN_API int quan_iqbn_relu_forward(const void *x, const float *gamma, const float *beta,
                                    float eps, void *out, float *mean, float *var,
                                    int32_t n, int32_t c, int32_t h, int32_t w,
                                    int32_t dtype, void *stream);

/*
 * Tensor descriptors
 * ------------------
 * The same convolution and IQBN (Section III-B eqs. 5/6, Section III-C eqs.
 * 11/12) for callers that hold tensors as (pointer, shape, strides) and want
 * the library, not themselves, to check the memory layout.  A descriptor
 * names a device buffer owned by the caller, its element type, and per axis
 * the logical extent and the distance in ELEMENTS between neighbours along
 * that axis.  An axis of extent 1 is never stepped, so its stride is not
 * checked (as in PyTorch's contiguity rule).
 *
 *   activation   ndim 5, logical [N, 4, C, H, W], strides (H*W*4*C, C, 1,
 *                W*4*C, 4*C): channels-last by component, the dense
 *                [N][H][W][4][C] array of every entry point above
 *   conv weight  ndim 4, [C_out, C_in, k_h, k_w], dense OIHW strides
 *                (C_in*k_h*k_w, k_h*k_w, k_w, 1)
 *   conv bias    ndim 2, [4, C_out], strides (C_out, 1)
 *   IQBN gamma, beta, mean, var   ndim 2, [4, C], strides (C, 1), QUAN_F32
 *
 * Any other strides (e.g. NCHW-ordered [N, 4, C, H, W] memory) return
 * QUAN_ERR_LAYOUT; a wrong ndim or extent returns QUAN_ERR_SHAPE; a dtype
 * that differs from x's (or is not QUAN_F32 for the IQBN parameters and
 * statistics) returns QUAN_ERR_DTYPE; a NULL descriptor or data pointer
 * returns QUAN_ERR_NULL (bias: a NULL descriptor means no bias).  An extent
 * of 2^31 or more returns QUAN_ERR_UNSUPPORTED.  All of this is checked on
 * the host before any HIP call; the call then behaves exactly like the
 * plain-pointer entry point named below, including its alignment and
 * overlap checks and its asynchronous completion on `stream`.
 */
typedef struct quan_tensor {
    void *data;
    int32_t dtype;
    int32_t ndim;
    int64_t shape[5];
    int64_t strides[5];
} quan_tensor;

/* quan_qconv2d_forward on descriptors: x [N, 4, C_in, H, W], w_r..w_k
 * [C_out, C_in, k_h, k_w], bias [4, C_out] or NULL, out [N, 4, C_out, Ho,
 * Wo]; stride, pad and dilation are (h, w) pairs. */
QUAN_API int quan_qconv2d_forward_desc(const quan_tensor *x,
                                       const quan_tensor *w_r, const quan_tensor *w_i,
                                       const quan_tensor *w_j, const quan_tensor *w_k,
                                       const quan_tensor *bias,
                                       const int32_t stride[2], const int32_t pad[2],
                                       const int32_t dilation[2],
                                       quan_tensor *out, void *stream);

/* quan_iqbn_forward and quan_iqbn_relu_forward on descriptors: x and out
 * [N, 4, C, H, W] (out may be x), gamma, beta, mean, var [4, C] fp32. */
QUAN_API int quan_iqbn_forward_desc(const quan_tensor *x, const quan_tensor *gamma,
                                    const quan_tensor *beta, float eps, quan_tensor *out,
                                    quan_tensor *mean, quan_tensor *var, void *stream);
QUAN_API int quan_iqbn_relu_forward_desc(const quan_tensor *x, const quan_tensor *gamma,
                                         const quan_tensor *beta, float eps, quan_tensor *out,
                                         quan_tensor *mean, quan_tensor *var, void *stream);

/* Where quan_qconv2d_iqbn_forward gathers the batch statistics. */
enum quan_stats_mode {
    QUAN_STATS_AUTO = 0,     /* the library's choice (see quan_qconv2d_iqbn_forward) */
    QUAN_STATS_EPILOGUE = 1, /* per-tile statistics in the convolution's epilogue */
    QUAN_STATS_PASS = 2      /* a separate statistics pass over out */
};

/*
 * The convolution followed by IQBN (+ ReLU when relu = 1) of its output, in
 * place: out receives IQBN(quan_qconv2d_forward_packed(x, packed, bias, ...)),
 * and mean, var ([4, c_out] fp32) the batch statistics of the convolution's
 * output (eqs. 11 and 12), as quan_iqbn_forward / quan_iqbn_relu_forward
 * would give up to rounding.  Every argument is as in
 * quan_qconv2d_forward_packed and quan_iqbn_forward; gamma, beta, mean and
 * var may not overlap each other, x or out.
 *
 *   stats   a quan_stats_mode.  QUAN_STATS_EPILOGUE has every output tile's
 *           mean and squared deviations computed in the convolution's
 *           epilogue and merged exactly in fp64 afterwards (normalising then
 *           costs one read and one write of out); tiles that cannot gather
 *           them (fewer than 32 output channels, or c_out not a multiple of
 *           8 for bf16 / 4 for fp32) use the separate pass instead.
 *           QUAN_STATS_PASS runs the plain convolution and then
 *           quan_iqbn_forward's normalisation on out: on tensors of up to
 *           32 MiB whose rows hold at least 193 reals (4 c_out), two
 *           launches (statistics, then the normalisation with the finalize
 *           merged in); on other tensors of 16 MiB or more that one
 *           work-group per compute unit can hold (about 100 MB on MI355X),
 *           one launch that reads out once and writes it once; otherwise
 *           three launches that read it twice.
 *           QUAN_STATS_AUTO picks the pass where it takes two launches, or
 *           one launch on a tensor of at least 64 MiB (measured on MI355X:
 *           133.0 against 137.3 us for the 32 x 14 x 14, 256-channel
 *           layer's 12.8 MB; 262.7 against 267.5 us for the 64 x 56 x 56,
 *           64-channel layer's 103 MB; 52 MB layers are faster with the
 *           epilogue), and the epilogue elsewhere.  All modes are
 *           deterministic.
 */
QUAN_API int quan_qconv2d_iqbn_forward(const void *x, const void *packed, const void *bias,
                                       int32_t stride_h, int32_t stride_w,
                                       int32_t pad_h, int32_t pad_w,
                                       int32_t dilation_h, int32_t dilation_w,
                                       const float *gamma, const float *beta, float eps,
                                       int32_t relu, int32_t stats, void *out, float *mean,
                                       float *var, int32_t n, int32_t c_in, int32_t h, int32_t w,
                                       int32_t c_out, int32_t k_h, int32_t k_w,
                                       int32_t dtype, void *stream);

/*
 * Inference-mode convolution + IQBN (+ ReLU when relu = 1): eq. 12 with
 * stored statistics in place of the batch statistics, folded into the
 * convolution's epilogue (no pass over out after the convolution):
 *
 *   out = (conv(x) + bias - running_mean) / sqrt(running_var + eps)
 *         * gamma + beta
 *
 * per output component and channel, computed as conv(x) * scale + shift in
 * fp32 before the single rounding to dtype, with scale = gamma / sqrt(var +
 * eps) and shift = (bias - mean) * scale + beta formed in fp64 on the
 * device.  running_mean, running_var, gamma, beta are [4, c_out] fp32 device
 * arrays (4-byte aligned) that out may not overlap; every other argument is
 * as in quan_qconv2d_forward_packed.  Uses a small library workspace per
 * (device, stream) for scale and shift.
 */
QUAN_API int quan_qconv2d_iqbn_inference(const void *x, const void *packed, const void *bias,
                                         int32_t stride_h, int32_t stride_w,
                                         int32_t pad_h, int32_t pad_w,
                                         int32_t dilation_h, int32_t dilation_w,
                                         const float *running_mean, const float *running_var,
                                         const float *gamma, const float *beta, float eps,
                                         int32_t relu, void *out,
                                         int32_t n, int32_t c_in, int32_t h, int32_t w,
                                         int32_t c_out, int32_t k_h, int32_t k_w,
                                         int32_t dtype, void *stream);

/*
 * Poincare mapping of RGB images into quaternions (Section III-A, eq. 4):
 * per pixel, with n2 = r^2 + g^2 + b^2,
 *
 *   q = ((1 - n2), 2r, 2g, 2b) / (1 + n2),
 *
 * a unit quaternion.  rgb: [n, 3, h, w] colour planes (dtype, aligned to
 * its element); out: the one-channel quaternion map [n, 4, 1, h, w] in the
 * activation layout of quan_qconv2d_forward, i.e. [n][h][w][4] (aligned to
 * four elements), which may not overlap rgb.  Computed in fp32 and rounded
 * once to dtype.
 */
QUAN_API int quan_poincare_map(const void *rgb, void *out, int32_t n, int32_t h, int32_t w,
                               int32_t dtype, void *stream);

/*
 * The first convolution of a network on RGB input with the Poincare mapping
 * of eq. 4 fused into its loads: out = quan_qconv2d_forward_packed(
 * quan_poincare_map(rgb), packed, bias, ...) of a one-channel (c_in = 1)
 * layer, without the quaternion map ever reaching memory.  The kernel
 * forms each tap's input quaternion from the three colour samples in fp32
 * and rounds it once to dtype, as quan_poincare_map does.
 *
 *   rgb     [n, 3, h, w] colour planes (dtype, aligned to its element).
 *   packed  quan_qconv2d_pack_weights of the four [c_out, 1, k_h, k_w]
 *           kernels (c_in = 1).
 *   out     [n, 4, c_out, Ho, Wo] channels-last by component, 16-byte
 *           aligned, overlapping neither rgb, packed nor bias.
 * Every other argument, rule and error is quan_qconv2d_forward_packed's.
 */
QUAN_API int quan_qconv2d_poincare_forward(const void *rgb, const void *packed, const void *bias,
                                           int32_t stride_h, int32_t stride_w,
                                           int32_t pad_h, int32_t pad_w,
                                           int32_t dilation_h, int32_t dilation_w, void *out,
                                           int32_t n, int32_t h, int32_t w, int32_t c_out,
                                           int32_t k_h, int32_t k_w, int32_t dtype, void *stream);

/*
 * Input gradient of the Hamilton convolution (the backward pass of
 * quan_qconv2d_forward with respect to x): for dL/dY = dy,
 *
 *   dx[n,c,iy,ix] = sum over (o, ky, kx, oy, ox) with iy = oy*stride_h -
 *                   pad_h + ky*dilation_h (ix likewise) of
 *                   conj(W[o,c,ky,kx]) (x) dy[n,o,oy,ox],
 *
 * since the Hamilton matrix of the conjugate quaternion is the transpose of
 * W's (eq. 6).  Computed as the forward convolution of dy (strided layers:
 * dy with stride-1 zero rows and columns inserted, staged in a library
 * workspace) with the transposed, spatially flipped, conjugated kernel,
 * stride 1, padding dilation*(k-1) - pad.
 *
 *   dy   [n, 4, c_out, h_out, w_out] (the forward's output shape), device
 *        layout, 16-byte aligned.
 *   w_*  the forward's four kernels [c_out, c_in, k_h, k_w].
 *   dx   [n, 4, c_in, h, w] output, device layout, 16-byte aligned, not
 *        overlapping dy or the kernels.
 * Sizes, strides, pads and dilations are the forward layer's; a pad larger
 * than dilation*(k-1) returns QUAN_ERR_UNSUPPORTED.
 */
QUAN_API int quan_qconv2d_backward_data(const void *dy, const void *w_r, const void *w_i,
                                        const void *w_j, const void *w_k,
                                        int32_t stride_h, int32_t stride_w,
                                        int32_t pad_h, int32_t pad_w,
                                        int32_t dilation_h, int32_t dilation_w, void *dx,
                                        int32_t n, int32_t c_in, int32_t h, int32_t w,
                                        int32_t c_out, int32_t k_h, int32_t k_w,
                                        int32_t dtype, void *stream);

/*
 * Weight and bias gradients of the Hamilton convolution for dL/dY = dy.
 * With Y_p = sum_q s(p, q) W_{p xor q} (x) X_q at every tap (eq. 6: s the
 * sign of entry (p, q), p xor q the kernel component it holds),
 *
 *   dW_m[o,c,ky,kx] = sum_p s(p, p xor m) sum over (n, oy, ox) of
 *                     dy[n,p,o,oy,ox] * x[n, p xor m, c, iy, ix]
 *   db[p,o]         = sum over (n, oy, ox) of dy[n,p,o,oy,ox]
 *
 * (iy = oy*stride_h - pad_h + ky*dilation_h, ix likewise; taps outside the
 * image contribute nothing).  A GEMM over the output pixels per tap, in
 * slices whose fp32 partial sums are added in a fixed order in fp64:
 * deterministic.
 *
 *   x          the forward input [n, 4, c_in, h, w], device layout.
 *   dy         [n, 4, c_out, h_out, w_out], device layout.
 *   dw_r..dw_k fp32 outputs [c_out, c_in, k_h, k_w] (4-byte aligned).
 *   db         fp32 output [4, c_out], or NULL.
 * Gradients may overlap neither each other nor x or dy.  Uses a library
 * workspace per (device, stream).
 */
QUAN_API int quan_qconv2d_backward_weight(const void *x, const void *dy,
                                          int32_t stride_h, int32_t stride_w,
                                          int32_t pad_h, int32_t pad_w,
                                          int32_t dilation_h, int32_t dilation_w,
                                          float *dw_r, float *dw_i, float *dw_j, float *dw_k,
                                          float *db, int32_t n, int32_t c_in, int32_t h,
                                          int32_t w, int32_t c_out, int32_t k_h, int32_t k_w,
                                          int32_t dtype, void *stream);

/*
 * Gradients of the separable convolution (quan_qconv2d_separable_forward,
 * eq. 7) by Section III-B's eqs. 8-10: the output gradients are mixed by the
 * backward matrix M printed with eq. 9 (M = S^T for eq. 7's sign matrix S),
 * and each mixed component meets only its own kernel and input,
 *
 *   z_q = sum_p M[q][p] dy_p                      (per pixel and channel)
 *   dx_q[n,c,iy,ix] = sum over (o, ky, kx, oy, ox) with iy = oy*stride_h -
 *                     pad_h + ky*dilation_h (ix likewise) of
 *                     W_q[o,c,ky,kx] * z_q[n,o,oy,ox]
 *   dW_q[o,c,ky,kx] = sum over (n, oy, ox) of z_q[n,o,oy,ox] * x_q[n,c,iy,ix]
 *   db_p[o]         = sum over (n, oy, ox) of dy_p[n,o,oy,ox]
 *
 * with every argument, layout, limit and error as in
 * quan_qconv2d_backward_data / quan_qconv2d_backward_weight.  The input
 * gradient runs as one convolution of dy (for strides above 1, staged with
 * zeros inserted) whose 4x4 block weight holds M[p][q] W'_p in block
 * (p, q), W'_p the transposed, spatially flipped real kernel: the mixing is
 * accumulated in fp32 with the products and rounded once.  Weight gradients
 * are fp32, deterministic.
 */
QUAN_API int quan_qconv2d_separable_backward_data(const void *dy, const void *w_r, const void *w_i,
                                                  const void *w_j, const void *w_k,
                                                  int32_t stride_h, int32_t stride_w,
                                                  int32_t pad_h, int32_t pad_w,
                                                  int32_t dilation_h, int32_t dilation_w, void *dx,
                                                  int32_t n, int32_t c_in, int32_t h, int32_t w,
                                                  int32_t c_out, int32_t k_h, int32_t k_w,
                                                  int32_t dtype, void *stream);

QUAN_API int quan_qconv2d_separable_backward_weight(const void *x, const void *dy,
                                                    int32_t stride_h, int32_t stride_w,
                                                    int32_t pad_h, int32_t pad_w,
                                                    int32_t dilation_h, int32_t dilation_w,
                                                    float *dw_r, float *dw_i, float *dw_j,
                                                    float *dw_k, float *db, int32_t n, int32_t c_in,
                                                    int32_t h, int32_t w, int32_t c_out, int32_t k_h,
                                                    int32_t k_w, int32_t dtype, void *stream);

/*
 * Gradient of training-mode IQBN (eqs. 11 and 12) with respect to its
 * input, gamma and beta, given the batch statistics the forward call
 * returned.  Per component and channel, over the P = n*h*w values, with
 * s = sqrt(var + eps), xhat = (x - mean) / s and g = dout (zero where the
 * forward's ReLU output y is <= 0, when y is given):
 *
 *   dbeta  = sum g
 *   dgamma = sum g xhat
 *   dx     = (gamma / s) (g - dbeta / P - xhat dgamma / P)
 *
 *   x, dout, y, dx  [n, 4, c, h, w] channels-last by component (dtype,
 *                   16-byte aligned); y may be NULL (IQBN without ReLU); dx
 *                   may equal dout (in place) but may not otherwise overlap
 *                   x, y or dout.
 *   mean, var       the forward's batch mean and biased variance, [4, c] fp32.
 *   gamma           [4, c] fp32.
 *   dgamma, dbeta   [4, c] fp32 outputs, overlapping nothing else.
 * Partial sums are added in fp64 in a fixed order: deterministic.
 */
QUAN_API int quan_iqbn_backward(const void *x, const void *dout, const void *y,
                                const float *mean, const float *var, const float *gamma,
                                float eps, void *dx, float *dgamma, float *dbeta,
                                int32_t n, int32_t c, int32_t h, int32_t w,
                                int32_t dtype, void *stream);

/* Message describing the last failure of a quan_* call on this thread
 * ("" if none).  The pointer stays valid until the next call on the thread. */
QUAN_API const char *quan_last_error(void);

/* Synchronise every device the library has used and free its workspaces.
 * Returns QUAN_OK or QUAN_ERR_HIP.  Later calls allocate afresh. */
QUAN_API int quan_release(void);

/* Library version string. */
QUAN_API const char *quan_version(void);

#ifdef __cplusplus
}
#endif

#endif /* QUAN_H */
