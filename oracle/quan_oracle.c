/*
 * CPU oracle for the QUAN hot path -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct fp64 reference for what the GPU library
 * computes.  Only the test suite, the smoke check and the benchmark's CPU
 * baseline leg load this file; the product path never calls it and shares no
 * code with it (no headers, tables or helpers in common).
 *
 * Paper: "Quaternion Approximate Networks for Enhanced Image Classification
 * and Oriented Object Detection" (arXiv 2509.05512).
 *
 * Logical layouts used here (all row-major, fp64):
 *   activations  x[n][q][c][h][w]      q in {r=0, i=1, j=2, k=3}
 *   conv weights w[q][o][c][kh][kw]    the four real kernels W_r, W_i, W_j, W_k
 *   conv bias    b[q][o]               one quaternion bias per output channel
 *   IQBN params  gamma[q][c], beta[q][c], mean[q][c], var[q][c]
 *
 * Readings of the paper taken here (the paper does not spell these out):
 *   - the convolution symbol inside eq. 5 is a deep-learning cross-correlation
 *     (no kernel flip) with zero padding, summed over input channels;
 *   - the kernel multiplies from the left (W (x) X), as eqs. 5 and 6 write it;
 *   - IQBN normalises with the biased (population) variance of eq. 11 over the
 *     batch and both spatial axes, separately for each (component, channel).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>

/* Hamilton product p (x) q, written out term by term as in Section III-A,
 * eq. 3.  out must not alias p or q. */
void quan_oracle_hamilton(const double p[4], const double q[4], double out[4])
{
    const double pr = p[0], pi = p[1], pj = p[2], pk = p[3];
    const double qr = q[0], qi = q[1], qj = q[2], qk = q[3];
    out[0] = pr * qr - pi * qi - pj * qj - pk * qk;
    out[1] = pr * qi + pi * qr + pj * qk - pk * qj;
    out[2] = pr * qj - pi * qk + pj * qr + pk * qi;
    out[3] = pr * qk + pi * qj - pj * qi + pk * qr;
}

/* Output extent of one spatial axis of a strided, padded, dilated window. */
int64_t quan_oracle_out_size(int64_t in, int64_t k, int64_t stride, int64_t pad, int64_t dil)
{
    return (in + 2 * pad - dil * (k - 1) - 1) / stride + 1;
}

/* Full quaternion convolution of Section III-B, eq. 5 (equivalently the
 * Hamilton matrix of eq. 6 applied at every tap):
 *
 *   Y[n,o,y,x] = bias[o] + sum_{c,ky,kx} W[o,c,ky,kx] (x) X[n,c,iy,ix]
 *   iy = y*sh - ph + ky*dh,  ix = x*sw - pw + kx*dw,
 *
 * with quaternion-valued W, X, Y and (x) the Hamilton product; taps that fall
 * outside the image contribute nothing (zero padding).  bias may be NULL. */
void quan_oracle_qconv2d(const double *x, const double *w, const double *bias, double *y,
                         int64_t N, int64_t Cin, int64_t H, int64_t W,
                         int64_t Cout, int64_t KH, int64_t KW,
                         int64_t sh, int64_t sw, int64_t ph, int64_t pw,
                         int64_t dh, int64_t dw)
{
    const int64_t Ho = quan_oracle_out_size(H, KH, sh, ph, dh);
    const int64_t Wo = quan_oracle_out_size(W, KW, sw, pw, dw);
    if (Ho <= 0 || Wo <= 0)
        return;
    const int64_t wq = Cout * Cin * KH * KW; /* stride between W_r, W_i, ... */
    const int64_t xq = Cin * H * W;          /* stride between X_r, X_i, ... */

#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t o = 0; o < Cout; ++o) {
            for (int64_t oy = 0; oy < Ho; ++oy) {
                for (int64_t ox = 0; ox < Wo; ++ox) {
                    double acc[4] = {0.0, 0.0, 0.0, 0.0};
                    if (bias) {
                        for (int q = 0; q < 4; ++q)
                            acc[q] = bias[q * Cout + o];
                    }
                    for (int64_t c = 0; c < Cin; ++c) {
                        for (int64_t ky = 0; ky < KH; ++ky) {
                            const int64_t iy = oy * sh - ph + ky * dh;
                            if (iy < 0 || iy >= H)
                                continue;
                            for (int64_t kx = 0; kx < KW; ++kx) {
                                const int64_t ix = ox * sw - pw + kx * dw;
                                if (ix < 0 || ix >= W)
                                    continue;
                                const int64_t widx = ((o * Cin + c) * KH + ky) * KW + kx;
                                const int64_t xidx = ((n * 4 * Cin + c) * H + iy) * W + ix;
                                double wv[4], xv[4], prod[4];
                                for (int q = 0; q < 4; ++q) {
                                    wv[q] = w[q * wq + widx];
                                    xv[q] = x[q * xq + xidx];
                                }
                                quan_oracle_hamilton(wv, xv, prod);
                                for (int q = 0; q < 4; ++q)
                                    acc[q] += prod[q];
                            }
                        }
                    }
                    for (int q = 0; q < 4; ++q)
                        y[((n * 4 * Cout + q * Cout + o) * Ho + oy) * Wo + ox] = acc[q];
                }
            }
        }
    }
}

/* Independent Quaternion Batch Normalization, Section III-C, eqs. 11 and 12:
 * for every component q and channel c separately, over the n = N*H*W values
 * X[:, q, c, :, :],
 *
 *   mu     = (1/n) sum x
 *   sigma2 = (1/n) sum (x - mu)^2                (two passes, biased)
 *   out    = (x - mu) / sqrt(sigma2 + eps) * gamma[q,c] + beta[q,c]
 *
 * followed by a component-wise max(0, .) when relu is non-zero.  mean and var
 * receive mu and sigma2 (either may be NULL). */
void quan_oracle_iqbn(const double *x, const double *gamma, const double *beta, double eps,
                      int relu, double *out, double *mean, double *var,
                      int64_t N, int64_t C, int64_t H, int64_t W)
{
    const int64_t hw = H * W;
    const double cnt = (double)(N * hw);

#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t q = 0; q < 4; ++q) {
        for (int64_t c = 0; c < C; ++c) {
            double s = 0.0;
            for (int64_t n = 0; n < N; ++n) {
                const double *xs = x + (n * 4 * C + q * C + c) * hw;
                for (int64_t t = 0; t < hw; ++t)
                    s += xs[t];
            }
            const double mu = s / cnt;
            double ss = 0.0;
            for (int64_t n = 0; n < N; ++n) {
                const double *xs = x + (n * 4 * C + q * C + c) * hw;
                for (int64_t t = 0; t < hw; ++t) {
                    const double d = xs[t] - mu;
                    ss += d * d;
                }
            }
            const double sigma2 = ss / cnt;
            const double inv = 1.0 / sqrt(sigma2 + eps);
            const double g = gamma[q * C + c], b = beta[q * C + c];
            for (int64_t n = 0; n < N; ++n) {
                const double *xs = x + (n * 4 * C + q * C + c) * hw;
                double *os = out + (n * 4 * C + q * C + c) * hw;
                for (int64_t t = 0; t < hw; ++t) {
                    double v = (xs[t] - mu) * inv * g + b;
                    if (relu && v < 0.0)
                        v = 0.0;
                    os[t] = v;
                }
            }
            if (mean)
                mean[q * C + c] = mu;
            if (var)
                var[q * C + c] = sigma2;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Separable QUAN convolution, Section III-B, eq. 7: each output component p
 * is a signed sum of the four real convolutions W_q (*) x_q only (no cross
 * terms W_a (*) x_b with a != b):
 *
 *   y_p = bias[p] + sum_q S[p][q] (W_q (*) x_q),
 *
 * S being the sign pattern eq. 7 prints, rows y_r, y_i, y_j, y_k.  The real
 * convolution is the same cross-correlation as in quan_oracle_qconv2d. */
static const double kSeparableSign[4][4] = {
    {1.0, -1.0, -1.0, -1.0}, /* y_r = W_r x_r - W_i x_i - W_j x_j - W_k x_k */
    {1.0, 1.0, 1.0, -1.0},   /* y_i = W_r x_r + W_i x_i + W_j x_j - W_k x_k */
    {1.0, -1.0, 1.0, 1.0},   /* y_j = W_r x_r - W_i x_i + W_j x_j + W_k x_k */
    {1.0, 1.0, -1.0, 1.0},   /* y_k = W_r x_r + W_i x_i - W_j x_j + W_k x_k */
};

void quan_oracle_qconv2d_separable(const double *x, const double *w, const double *bias, double *y,
                                   int64_t N, int64_t Cin, int64_t H, int64_t W,
                                   int64_t Cout, int64_t KH, int64_t KW,
                                   int64_t sh, int64_t sw, int64_t ph, int64_t pw,
                                   int64_t dh, int64_t dw)
{
    const int64_t Ho = quan_oracle_out_size(H, KH, sh, ph, dh);
    const int64_t Wo = quan_oracle_out_size(W, KW, sw, pw, dw);
    if (Ho <= 0 || Wo <= 0)
        return;
    const int64_t wq = Cout * Cin * KH * KW;
    const int64_t xq = Cin * H * W;

#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t o = 0; o < Cout; ++o) {
            for (int64_t oy = 0; oy < Ho; ++oy) {
                for (int64_t ox = 0; ox < Wo; ++ox) {
                    double conv[4] = {0.0, 0.0, 0.0, 0.0}; /* W_q (*) x_q */
                    for (int q = 0; q < 4; ++q) {
                        for (int64_t c = 0; c < Cin; ++c) {
                            for (int64_t ky = 0; ky < KH; ++ky) {
                                const int64_t iy = oy * sh - ph + ky * dh;
                                if (iy < 0 || iy >= H)
                                    continue;
                                for (int64_t kx = 0; kx < KW; ++kx) {
                                    const int64_t ix = ox * sw - pw + kx * dw;
                                    if (ix < 0 || ix >= W)
                                        continue;
                                    conv[q] += w[q * wq + ((o * Cin + c) * KH + ky) * KW + kx] *
                                               x[q * xq + ((n * 4 * Cin + c) * H + iy) * W + ix];
                                }
                            }
                        }
                    }
                    for (int p = 0; p < 4; ++p) {
                        double v = bias ? bias[p * Cout + o] : 0.0;
                        for (int q = 0; q < 4; ++q)
                            v += kSeparableSign[p][q] * conv[q];
                        y[((n * 4 * Cout + p * Cout + o) * Ho + oy) * Wo + ox] = v;
                    }
                }
            }
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Backward pass of the separable convolution, Section III-B, eqs. 8-10.  The
 * gradients keep eq. 7's separable structure: the output gradients are
 * mixed by the matrix M printed with eq. 9, and each mixed component z_q
 * then meets only its own kernel W_q and input x_q:
 *
 *   z_q[n,o,oy,ox] = sum_p M[q][p] dy_p[n,o,oy,ox]
 *   dx_q[n,c,iy,ix] += W_q[o,c,ky,kx] z_q[n,o,oy,ox]     (a transposed conv)
 *   dW_q[o,c,ky,kx] += x_q[n,c,iy,ix] z_q[n,o,oy,ox]      (a correlation)
 *   db_p[o]         += dy_p[n,o,oy,ox]
 *
 * over every (n, o, oy, ox, c, ky, kx) whose tap lies inside the image.  The
 * printed equations index M_q^T ambiguously; read as M[q][p] = S[p][q]
 * (M is eq. 7's sign matrix transposed), this is the exact adjoint of
 * quan_oracle_qconv2d_separable.  dx, dw and db are overwritten; any may be
 * NULL (not computed). */
static const double kMixing[4][4] = {
    {1.0, 1.0, 1.0, 1.0},
    {-1.0, 1.0, -1.0, 1.0},
    {-1.0, 1.0, 1.0, -1.0},
    {-1.0, -1.0, 1.0, 1.0},
};

void quan_oracle_qconv2d_separable_backward(const double *x, const double *w, const double *dy,
                                            double *dx, double *dwt, double *db,
                                            int64_t N, int64_t Cin, int64_t H, int64_t W,
                                            int64_t Cout, int64_t KH, int64_t KW,
                                            int64_t sh, int64_t sw, int64_t ph, int64_t pw,
                                            int64_t dh, int64_t dw)
{
    const int64_t Ho = quan_oracle_out_size(H, KH, sh, ph, dh);
    const int64_t Wo = quan_oracle_out_size(W, KW, sw, pw, dw);
    const int64_t wq = Cout * Cin * KH * KW;
    const int64_t xq = Cin * H * W;
    const int64_t yq = Cout * Ho * Wo;

    if (dx) {
        for (int64_t i = 0; i < N * 4 * xq; ++i)
            dx[i] = 0.0;
        /* each image's input gradient is written by one thread */
#pragma omp parallel for schedule(dynamic)
        for (int64_t n = 0; n < N; ++n) {
            for (int64_t o = 0; o < Cout; ++o)
                for (int64_t oy = 0; oy < Ho; ++oy)
                    for (int64_t ox = 0; ox < Wo; ++ox) {
                        double z[4];
                        for (int q = 0; q < 4; ++q) {
                            z[q] = 0.0;
                            for (int p = 0; p < 4; ++p)
                                z[q] += kMixing[q][p] * dy[n * 4 * yq + p * yq + (o * Ho + oy) * Wo + ox];
                        }
                        for (int q = 0; q < 4; ++q)
                            for (int64_t c = 0; c < Cin; ++c)
                                for (int64_t ky = 0; ky < KH; ++ky) {
                                    const int64_t iy = oy * sh - ph + ky * dh;
                                    if (iy < 0 || iy >= H)
                                        continue;
                                    for (int64_t kx = 0; kx < KW; ++kx) {
                                        const int64_t ix = ox * sw - pw + kx * dw;
                                        if (ix < 0 || ix >= W)
                                            continue;
                                        dx[n * 4 * xq + q * xq + (c * H + iy) * W + ix] +=
                                            w[q * wq + ((o * Cin + c) * KH + ky) * KW + kx] * z[q];
                                    }
                                }
                    }
        }
    }
    if (dwt) {
        /* each output channel's weight gradient is written by one thread */
#pragma omp parallel for schedule(dynamic)
        for (int64_t o = 0; o < Cout; ++o) {
            for (int q = 0; q < 4; ++q)
                for (int64_t t = 0; t < Cin * KH * KW; ++t)
                    dwt[q * wq + o * Cin * KH * KW + t] = 0.0;
            for (int64_t n = 0; n < N; ++n)
                for (int64_t oy = 0; oy < Ho; ++oy)
                    for (int64_t ox = 0; ox < Wo; ++ox) {
                        double z[4];
                        for (int q = 0; q < 4; ++q) {
                            z[q] = 0.0;
                            for (int p = 0; p < 4; ++p)
                                z[q] += kMixing[q][p] * dy[n * 4 * yq + p * yq + (o * Ho + oy) * Wo + ox];
                        }
                        for (int q = 0; q < 4; ++q)
                            for (int64_t c = 0; c < Cin; ++c)
                                for (int64_t ky = 0; ky < KH; ++ky) {
                                    const int64_t iy = oy * sh - ph + ky * dh;
                                    if (iy < 0 || iy >= H)
                                        continue;
                                    for (int64_t kx = 0; kx < KW; ++kx) {
                                        const int64_t ix = ox * sw - pw + kx * dw;
                                        if (ix < 0 || ix >= W)
                                            continue;
                                        dwt[q * wq + ((o * Cin + c) * KH + ky) * KW + kx] +=
                                            x[n * 4 * xq + q * xq + (c * H + iy) * W + ix] * z[q];
                                    }
                                }
                    }
        }
    }
    if (db) {
        for (int p = 0; p < 4; ++p)
            for (int64_t o = 0; o < Cout; ++o) {
                double s = 0.0;
                for (int64_t n = 0; n < N; ++n)
                    for (int64_t t = 0; t < Ho * Wo; ++t)
                        s += dy[n * 4 * yq + p * yq + o * Ho * Wo + t];
                db[p * Cout + o] = s;
            }
    }
}

/* ------------------------------------------------------------------------ */
/* IQBN with given statistics (inference: eq. 12 with stored running mean and
 * variance in place of the batch statistics of eq. 11):
 *
 *   out = (x - mean[q,c]) / sqrt(var[q,c] + eps) * gamma[q,c] + beta[q,c]
 *
 * followed by a component-wise max(0, .) when relu is non-zero. */
void quan_oracle_iqbn_inference(const double *x, const double *mean, const double *var,
                                const double *gamma, const double *beta, double eps, int relu,
                                double *out, int64_t N, int64_t C, int64_t H, int64_t W)
{
    const int64_t hw = H * W;
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t q = 0; q < 4; ++q) {
            for (int64_t c = 0; c < C; ++c) {
                const double inv = 1.0 / sqrt(var[q * C + c] + eps);
                const double mu = mean[q * C + c], g = gamma[q * C + c], b = beta[q * C + c];
                const double *xs = x + (n * 4 * C + q * C + c) * hw;
                double *os = out + (n * 4 * C + q * C + c) * hw;
                for (int64_t t = 0; t < hw; ++t) {
                    double v = (xs[t] - mu) * inv * g + b;
                    if (relu && v < 0.0)
                        v = 0.0;
                    os[t] = v;
                }
            }
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Poincare mapping of an RGB image into quaternions, Section III-A, eq. 4:
 * with n2 = r^2 + g^2 + b^2 at every pixel,
 *
 *   q = ((1 - n2), 2r, 2g, 2b) / (1 + n2),
 *
 * rgb [N][3][H][W] -> q [N][4][1][H][W] (one quaternion channel). */
void quan_oracle_poincare(const double *rgb, double *q, int64_t N, int64_t H, int64_t W)
{
    const int64_t hw = H * W;
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t t = 0; t < hw; ++t) {
            const double r = rgb[(n * 3 + 0) * hw + t];
            const double g = rgb[(n * 3 + 1) * hw + t];
            const double b = rgb[(n * 3 + 2) * hw + t];
            const double n2 = r * r + g * g + b * b;
            const double den = 1.0 + n2;
            q[(n * 4 + 0) * hw + t] = (1.0 - n2) / den;
            q[(n * 4 + 1) * hw + t] = 2.0 * r / den;
            q[(n * 4 + 2) * hw + t] = 2.0 * g / den;
            q[(n * 4 + 3) * hw + t] = 2.0 * b / den;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Backward pass of the full quaternion convolution (the gradient of
 * quan_oracle_qconv2d).  The Hamilton product p (x) q is linear in q with
 * matrix L(p) and linear in p with matrix R(q); both are read off the product
 * itself, column j being the product with the j-th unit quaternion. */
static void left_matrix(const double p[4], double L[4][4])
{
    for (int j = 0; j < 4; ++j) {
        double e[4] = {0.0, 0.0, 0.0, 0.0}, col[4];
        e[j] = 1.0;
        quan_oracle_hamilton(p, e, col);
        for (int i = 0; i < 4; ++i)
            L[i][j] = col[i];
    }
}

static void right_matrix(const double q[4], double R[4][4])
{
    for (int j = 0; j < 4; ++j) {
        double e[4] = {0.0, 0.0, 0.0, 0.0}, col[4];
        e[j] = 1.0;
        quan_oracle_hamilton(e, q, col);
        for (int i = 0; i < 4; ++i)
            R[i][j] = col[i];
    }
}

/* Given dy = dL/dY [N][4][Cout][Ho][Wo] for Y = qconv2d(x, w, bias), every
 * (n, o, oy, ox, c, ky, kx) whose tap lies inside the image contributes
 *
 *   dx[n,c,iy,ix] += L(W[o,c,ky,kx])^T dy[n,o,oy,ox]
 *   dw[o,c,ky,kx] += R(X[n,c,iy,ix])^T dy[n,o,oy,ox]
 *
 * and db[o] = sum over (n, oy, ox) of dy[n,o,oy,ox].  dx, dw and db are
 * overwritten; any of them may be NULL (not computed). */
void quan_oracle_qconv2d_backward(const double *x, const double *w, const double *dy,
                                  double *dx, double *dwt, double *db,
                                  int64_t N, int64_t Cin, int64_t H, int64_t W,
                                  int64_t Cout, int64_t KH, int64_t KW,
                                  int64_t sh, int64_t sw, int64_t ph, int64_t pw,
                                  int64_t dh, int64_t dw)
{
    const int64_t Ho = quan_oracle_out_size(H, KH, sh, ph, dh);
    const int64_t Wo = quan_oracle_out_size(W, KW, sw, pw, dw);
    const int64_t wq = Cout * Cin * KH * KW;
    const int64_t xq = Cin * H * W;
    const int64_t yq = Cout * Ho * Wo;

    if (dx) {
        for (int64_t i = 0; i < N * 4 * xq; ++i)
            dx[i] = 0.0;
        /* each image's input gradient is written by one thread */
#pragma omp parallel for schedule(dynamic)
        for (int64_t n = 0; n < N; ++n) {
            for (int64_t o = 0; o < Cout; ++o)
                for (int64_t oy = 0; oy < Ho; ++oy)
                    for (int64_t ox = 0; ox < Wo; ++ox) {
                        double g[4];
                        for (int q = 0; q < 4; ++q)
                            g[q] = dy[n * 4 * yq + q * yq + (o * Ho + oy) * Wo + ox];
                        for (int64_t c = 0; c < Cin; ++c)
                            for (int64_t ky = 0; ky < KH; ++ky) {
                                const int64_t iy = oy * sh - ph + ky * dh;
                                if (iy < 0 || iy >= H)
                                    continue;
                                for (int64_t kx = 0; kx < KW; ++kx) {
                                    const int64_t ix = ox * sw - pw + kx * dw;
                                    if (ix < 0 || ix >= W)
                                        continue;
                                    double wv[4], L[4][4];
                                    for (int q = 0; q < 4; ++q)
                                        wv[q] = w[q * wq + ((o * Cin + c) * KH + ky) * KW + kx];
                                    left_matrix(wv, L);
                                    for (int q = 0; q < 4; ++q) {
                                        double s = 0.0;
                                        for (int p = 0; p < 4; ++p)
                                            s += L[p][q] * g[p];
                                        dx[n * 4 * xq + q * xq + (c * H + iy) * W + ix] += s;
                                    }
                                }
                            }
                    }
        }
    }
    if (dwt) {
        /* each output channel's weight gradient is written by one thread */
#pragma omp parallel for schedule(dynamic)
        for (int64_t o = 0; o < Cout; ++o) {
            for (int q = 0; q < 4; ++q)
                for (int64_t t = 0; t < Cin * KH * KW; ++t)
                    dwt[q * wq + o * Cin * KH * KW + t] = 0.0;
            for (int64_t n = 0; n < N; ++n)
                for (int64_t oy = 0; oy < Ho; ++oy)
                    for (int64_t ox = 0; ox < Wo; ++ox) {
                        double g[4];
                        for (int q = 0; q < 4; ++q)
                            g[q] = dy[n * 4 * yq + q * yq + (o * Ho + oy) * Wo + ox];
                        for (int64_t c = 0; c < Cin; ++c)
                            for (int64_t ky = 0; ky < KH; ++ky) {
                                const int64_t iy = oy * sh - ph + ky * dh;
                                if (iy < 0 || iy >= H)
                                    continue;
                                for (int64_t kx = 0; kx < KW; ++kx) {
                                    const int64_t ix = ox * sw - pw + kx * dw;
                                    if (ix < 0 || ix >= W)
                                        continue;
                                    double xv[4], R[4][4];
                                    for (int q = 0; q < 4; ++q)
                                        xv[q] = x[n * 4 * xq + q * xq + (c * H + iy) * W + ix];
                                    right_matrix(xv, R);
                                    for (int q = 0; q < 4; ++q) {
                                        double s = 0.0;
                                        for (int p = 0; p < 4; ++p)
                                            s += R[p][q] * g[p];
                                        dwt[q * wq + ((o * Cin + c) * KH + ky) * KW + kx] += s;
                                    }
                                }
                            }
                    }
        }
    }
    if (db) {
        for (int64_t q = 0; q < 4; ++q)
            for (int64_t o = 0; o < Cout; ++o) {
                double s = 0.0;
                for (int64_t n = 0; n < N; ++n)
                    for (int64_t t = 0; t < Ho * Wo; ++t)
                        s += dy[n * 4 * yq + q * yq + o * Ho * Wo + t];
                db[q * Cout + o] = s;
            }
    }
}

/* ------------------------------------------------------------------------ */
/* Backward pass of training-mode IQBN (eqs. 11 and 12) for one layer, from
 * the chain rule through the batch mean and biased variance.  Per component
 * q and channel c, over the n = N*H*W values, with s = sqrt(sigma2 + eps),
 * xhat = (x - mu) / s and g = dout (times [gamma xhat + beta > 0] when relu
 * is non-zero):
 *
 *   dbeta  = sum g
 *   dgamma = sum g xhat
 *   dx     = (gamma / s) (g - dbeta / n - xhat dgamma / n)
 *
 * dx, dgamma, dbeta are overwritten; dgamma and dbeta may be NULL. */
void quan_oracle_iqbn_backward(const double *x, const double *gamma, const double *beta, double eps,
                               int relu, const double *dout, double *dx, double *dgamma,
                               double *dbeta, int64_t N, int64_t C, int64_t H, int64_t W)
{
    const int64_t hw = H * W;
    const double cnt = (double)(N * hw);
    for (int64_t q = 0; q < 4; ++q) {
        for (int64_t c = 0; c < C; ++c) {
            double s1 = 0.0;
            for (int64_t n = 0; n < N; ++n)
                for (int64_t t = 0; t < hw; ++t)
                    s1 += x[(n * 4 * C + q * C + c) * hw + t];
            const double mu = s1 / cnt;
            double s2 = 0.0;
            for (int64_t n = 0; n < N; ++n)
                for (int64_t t = 0; t < hw; ++t) {
                    const double d = x[(n * 4 * C + q * C + c) * hw + t] - mu;
                    s2 += d * d;
                }
            const double sd = sqrt(s2 / cnt + eps);
            const double ga = gamma[q * C + c], be = beta[q * C + c];
            double sg = 0.0, sgx = 0.0;
            for (int64_t n = 0; n < N; ++n)
                for (int64_t t = 0; t < hw; ++t) {
                    const int64_t idx = (n * 4 * C + q * C + c) * hw + t;
                    const double xhat = (x[idx] - mu) / sd;
                    double g = dout[idx];
                    if (relu && !(ga * xhat + be > 0.0))
                        g = 0.0;
                    sg += g;
                    sgx += g * xhat;
                }
            for (int64_t n = 0; n < N; ++n)
                for (int64_t t = 0; t < hw; ++t) {
                    const int64_t idx = (n * 4 * C + q * C + c) * hw + t;
                    const double xhat = (x[idx] - mu) / sd;
                    double g = dout[idx];
                    if (relu && !(ga * xhat + be > 0.0))
                        g = 0.0;
                    dx[idx] = ga / sd * (g - sg / cnt - xhat * sgx / cnt);
                }
            if (dbeta)
                dbeta[q * C + c] = sg;
            if (dgamma)
                dgamma[q * C + c] = sgx;
        }
    }
}
