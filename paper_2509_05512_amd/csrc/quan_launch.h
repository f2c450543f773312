// Internal launch interface between the C ABI (quan_api.cpp) and the HIP
// kernels.  Host-only declarations; every argument has been validated by the
// caller before one of these runs.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace quan {

enum class DType : int { F32 = 0, BF16 = 1 };

// Bit 4*p + q is set when entry (p, q) of the Hamilton matrix (eq. 6) is
// negative.  Row r: + - - -, row i: + + - +, row j: + + + -, row k: + - + +.
constexpr unsigned kHamiltonNeg =
    (1u << 1) | (1u << 2) | (1u << 3) | (1u << 6) | (1u << 11) | (1u << 13);

// Geometry of one quaternion convolution (quaternion channel counts).
struct ConvGeom {
    int n, c_in, h, w, c_out, k_h, k_w;
    int s_h, s_w, p_h, p_w, d_h, d_w;
    int h_out, w_out;
    int64_t m() const { return int64_t(n) * h_out * w_out; }
};

// Layout of the packed weights: [tap][cblk][kernel r,i,j,k][cout_pad][pk]
// with pk input channels per block (one 128-byte stage row holds pk channels
// of all four components).  It depends only on (dtype, c_in, c_out, k_h,
// k_w), never on the tile configuration, so weights packed once serve every
// later call.
struct PackGeom {
    int pk;        // input channels per block: 128 bytes / (4 components x element size)
    int n_cblk;    // ceil(c_in / pk)
    int cout_pad;  // c_out rounded up to kPackCoutAlign
    size_t bytes;  // bytes of packed weights
};
constexpr int kPackCoutAlign = 64;
PackGeom qconv2d_pack_geom(int c_in, int c_out, int k_h, int k_w, DType dt);

// Tile configuration chosen for a convolution.
struct ConvPlan {
    int id;              // index into the kernel table
    int bm, bnc;         // output pixels, output channels per component
    int m_tiles, n_tiles;
    int stat_rows;       // output pixels per IQBN statistics partial
    int stat_tiles;      // statistics partials per column: ceil(m / stat_rows)
    const char *name;
    // the pointwise streaming kernel (qconv2d_pointwise_run) instead of the
    // implicit-GEMM kernel table: group_stages 32-pixel stages per work-group
    bool pointwise;
    int group_stages;
};

// What a convolution launch computes: the Hamilton product (eq. 5), the
// separable form (eq. 7), or the separable form's input gradient (eqs.
// 8-10: block (p, q) of the 4x4 block weight is M[p][q] W'_p).
enum class ConvForm : int { Hamilton = 0, Separable = 1, SeparableGradData = 2 };

// Pick a tile configuration for the convolution.
ConvPlan qconv2d_plan(const ConvGeom &g, DType dt, ConvForm form);

// Pack W_r..W_k (OIHW) into the PackGeom layout, zero padded.
hipError_t qconv2d_pack_weights(const PackGeom &pg, int c_in, int c_out, int k_h, int k_w, DType dt,
                                const void *w_r, const void *w_i, const void *w_j,
                                const void *w_k, void *wpack, hipStream_t stream);

// The implicit-GEMM Hamilton convolution.  With `stats` non-NULL (only where
// qconv2d_writes_stats holds) it also writes IQBN statistics of its output
// per run of plan.stat_rows consecutive output pixels: stats[0][col][t] =
// the run's mean, stats[1][col][t] = sum of squared deviations from it,
// col = p * c_out + o, t < plan.stat_tiles; run t covers pixels
// [t * stat_rows, min((t + 1) * stat_rows, m)).
//
// With `fold` non-NULL the epilogue applies out = scale[col] * acc +
// shift[col] (fp32, [4][c_out] each, col = p * c_out + o) and max(0, .) when
// relu is set, instead of adding the bias (inference IQBN folded in).
struct ConvFold {
    const float *scale;
    const float *shift;
    bool relu;
};
//
// With `poincare` (a stem layer: g.c_in == 1, bias epilogue) x is the colour
// planes [n][3][h][w] of the input images, mapped to quaternions by eq. 4
// as the convolution loads them.
bool qconv2d_writes_stats(const ConvPlan &plan, const ConvGeom &g, DType dt);
//
// `claim` (optional): buf, qconv2d_claim_bytes() of device memory, zero
// before the first launch that uses it, which every launch leaves zero
// again (the launches that use one buffer must not overlap: one buffer per
// stream); epoch, the tag of the next launch on the buffer, which each
// launch advances.  With it a layer whose last round of tiles would leave
// work-groups idle ends in 32-pixel tail blocks that the work-groups claim
// as they finish; NULL: whole tiles only.
struct ConvClaim {
    unsigned *buf;
    unsigned epoch;
};
hipError_t qconv2d_run(const ConvPlan &plan, const PackGeom &pg, const ConvGeom &g, DType dt,
                       const void *x, const void *wpack, const void *bias, void *out,
                       float *stats, const ConvFold *fold, hipStream_t stream, bool poincare = false,
                       ConvClaim *claim = nullptr);
size_t qconv2d_claim_bytes();

// The pointwise streaming kernel (1x1 kernel, no padding, any stride; bf16,
// 32 or 64 input and output channels, input under 2 GiB): whether it takes
// the layer; its stages per work-group on `cus` compute units; the launch
// (stats with stat_tiles == the number of work-groups, one partial per
// work-group run of 32 * group_stages pixels; or fold; or neither).
bool qconv2d_pointwise_takes(const ConvGeom &g, DType dt);
int qconv2d_pointwise_group_stages(int64_t m, int cus);
int qconv2d_pointwise_stage_pixels();
hipError_t qconv2d_pointwise_run(const ConvGeom &g, const PackGeom &pg, int group_stages, const void *x,
                                 const void *wpack, const void *bias, void *out, float *stats, int stat_tiles,
                                 const ConvFold *fold, hipStream_t stream);

// The stem layer (g.c_in == 1, bf16) as its own kernel: rgb is the colour
// planes [n][3][h][w], mapped to quaternions by eq. 4 as they are loaded;
// wpack the packed weights (qconv2d_pack_weights); out as qconv2d_run.
// Returns hipErrorNotSupported, before any launch, where the layer is not
// one it takes: fp32, more than 64 output channels, or more than 32 MFMA
// weight fragments (B * ceil(taps / 4), B = ceil(4 c_out / 32) rounded up
// to a power of two).
hipError_t qconv2d_stem_run(const PackGeom &pg, const ConvGeom &g, DType dt, const void *rgb, const void *wpack,
                            const void *bias, void *out, hipStream_t stream);

// Input gradient of the Hamilton convolution: dX = conv(Z, W'), Z = dY (stride
// 1) or dY scattered with s-1 zeros between rows/columns (staged in `stage`,
// qconv2d_grad_data_stage_bytes bytes), W' the conjugated, transposed,
// flipped kernel (packed into `wpack`: qconv2d_pack_geom of the gradient
// geometry), stride 1, pad d(k-1) - p (must be >= 0).  g is the forward
// layer's geometry; dy [n][h_out][w_out][4][c_out], dx [n][h][w][4][c_in].
// With sep, the separable form's input gradient (eqs. 8-10) instead:
// dX_p = sum_q M[p][q] (W'_p (*) Z_q), W'_p the transposed, flipped real
// kernel and M the backward mixing matrix, accumulated in fp32.
ConvGeom qconv2d_grad_data_geom(const ConvGeom &g);
size_t qconv2d_grad_data_stage_bytes(const ConvGeom &g, DType dt);
hipError_t qconv2d_backward_data_run(const ConvGeom &g, DType dt, const void *dy, const void *w_r, const void *w_i,
                                     const void *w_j, const void *w_k, void *dx, void *wpack, void *stage,
                                     hipStream_t stream, bool sep = false, ConvClaim *claim = nullptr);

// Weight and bias gradients of the Hamilton convolution for dL/dY = dy:
// dw_r..dw_k [c_out][c_in][k_h][k_w] and db [4][c_out] (NULL: skipped), all
// fp32; x [n][h][w][4][c_in], dy [n][h_out][w_out][4][c_out].  `work` must
// hold qconv2d_wgrad_work_bytes(g) bytes.
// With sep, the gradients of the separable form instead (eqs. 8-10):
// dW_q = sum_p S[p][q] sum_pix dY_p X_q (S the sign matrix of eq. 7).
size_t qconv2d_wgrad_work_bytes(const ConvGeom &g);
hipError_t qconv2d_backward_weight_run(const ConvGeom &g, DType dt, const void *x, const void *dy, float *dw_r,
                                       float *dw_i, float *dw_j, float *dw_k, float *db, void *work,
                                       hipStream_t stream, bool sep = false);

// Error reporting shared by the entry points of every source file: report()
// stores the thread's last-error message and returns `code`.
void clear_error();
int report(int code, const char *fmt, ...);

// Argument checks of quan_iqbn_forward (QUAN_OK, or a QUAN_ERR_* code with
// the message set); they touch no device state.
int iqbn_validate(const void *x, const float *gamma, const float *beta, float eps, const void *out,
                  const float *mean, const float *var, int32_t n, int32_t c, int32_t h, int32_t w, int32_t dtype);

// IQBN.  `work` must hold iqbn_workspace_bytes(...) bytes.  `flags` holds the
// grid-barrier flags of the one-launch form: iqbn_barrier_bytes() of device
// memory, zero when first allocated, used by no other code and by one stream
// at a time (NULL: always the three-launch form).
size_t iqbn_workspace_bytes(int64_t pixels, int c);
size_t iqbn_barrier_bytes();
// Whether iqbn_run (given flags) normalises this tensor in one launch that
// reads it once, on the current device.
bool iqbn_one_launch(int64_t pixels, int c, DType dt);
// Whether iqbn_run takes two launches with the finalize merged into the
// normalization (small tensors with wide rows).
bool iqbn_merged(int64_t pixels, int c, DType dt);
hipError_t iqbn_run(const void *x, const float *gamma, const float *beta, float eps, bool relu,
                    void *out, float *mean, float *var, int64_t pixels, int c, DType dt,
                    void *work, unsigned *flags, hipStream_t stream);

// Gradient of training-mode IQBN given the forward's saved mean and biased
// variance ([4][c] fp32): dx (dtype dt, x's layout), dgamma, dbeta ([4][c]
// fp32).  y (the forward output after ReLU) masks the gradient where y <= 0;
// NULL: no ReLU.  `work` must hold iqbn_workspace_bytes(...) bytes.
hipError_t iqbn_backward_run(const void *x, const void *dout, const void *y, const float *mean, const float *var,
                             const float *gamma, float eps, void *dx, float *dgamma, float *dbeta, int64_t pixels,
                             int c, DType dt, void *work, hipStream_t stream);

// IQBN of a convolution output whose per-tile statistics the convolution
// wrote (qconv2d_run with stats): `part` holds iqbn_tile_stats_bytes(m_tiles,
// c) bytes, the statistics first; the normalization runs in place on `io`.
size_t iqbn_tile_stats_bytes(int m_tiles, int c);
hipError_t iqbn_from_tiles_run(const float *part, int m_tiles, int tile_rows, const float *gamma,
                               const float *beta, float eps, bool relu, void *io, float *mean, float *var,
                               int64_t pixels, int c, DType dt, hipStream_t stream);

// Inference IQBN folded into a convolution: per column col of [4][c],
// scale = gamma / sqrt(var + eps) and shift = (bias - mean) * scale + beta
// (computed in fp64, stored fp32); bias (dtype dt) may be NULL.
hipError_t iqbn_fold_run(const float *mean, const float *var, const float *gamma, const float *beta,
                         const void *bias, float eps, int c, DType dt, float *scale, float *shift,
                         hipStream_t stream);

// Poincare mapping (eq. 4): rgb [n][3][h][w] -> out [n][h][w][4].
hipError_t poincare_run(const void *rgb, void *out, int64_t n, int64_t h, int64_t w, DType dt,
                        hipStream_t stream);

}  // namespace quan
