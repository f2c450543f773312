// Independent Quaternion Batch Normalization (Section III-C, eqs. 11 and 12)
// for gfx950.
//
// The tensor is channels-last by component: P = N*H*W rows of L = 4*C reals,
// and every one of the L columns (component q, channel c) is normalised on
// its own with its batch mean and biased variance.  Three launches on the
// caller's stream, no host synchronisation:
//
//   1. iqbn_stats     streams x once.  Each thread owns one 16-byte column
//                     chunk and a strided set of rows and accumulates shifted
//                     sums  s1 = sum(x - K), s2 = sum((x - K)^2)  in fp32, with
//                     K the column's value in row 0 (so the variance does not
//                     cancel when |mean| >> std).  A fixed-order LDS reduction
//                     gives one (s1, s2) per column per block.
//   2. iqbn_finalize  merges the per-block partials in fp64, in block order
//                     (deterministic: no atomics), and writes mean, var and the
//                     per-column scale = gamma / sqrt(var + eps).
//   3. iqbn_affine    streams x again: out = (x - mean) * scale + beta, optional
//                     ReLU.  Subtracting the mean first keeps a near-constant
//                     column exact (a folded x * scale + shift would cancel
//                     two terms of size |mean| * scale).
//
// After a convolution that wrote per-tile statistics of its output (fused
// into its epilogue), iqbn_finalize_tiles replaces passes 1 and 2: the
// normalization then costs one read and one write of the tensor.
#include <hip/hip_runtime.h>

#include "quan_launch.h"

namespace quan {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxBlocks = 512;  // partial-statistics blocks per column group (grid.x)
// blocks per column group of the element-wise passes (normalization and the
// input gradient), which keep no partials: four work-groups per compute unit
constexpr int kStreamBlocks = 1024;
constexpr int kMinRowsPerThread = 24;

template <typename T, int VW>
struct alignas(sizeof(T) * VW) Vec {
    T v[VW];
};


// A 16-byte store the element-wise passes will not read back soon (their
// output goes to the next layer or to the caller): non-temporal, so it does
// not displace lines the pass is still reading.  Measured: the input-gradient
// pass 52 -> 48 us on a 206 MB + 103 MB stream.
typedef unsigned int nt_u32x4 __attribute__((ext_vector_type(4)));
template <typename V>
__device__ __forceinline__ void store_stream(V *p, const V &v)
{
    if constexpr (sizeof(V) == 16)
        __builtin_nontemporal_store(__builtin_bit_cast(nt_u32x4, v), reinterpret_cast<nt_u32x4 *>(p));
    else
        *p = v;
}

// Thread layout shared by the stats and affine passes.
struct Layout {
    int64_t pixels;          // rows
    int row_len;             // L = 4*C
    int vw;                  // elements per column chunk
    int chunks;              // L / vw
    int cg;                  // chunk columns per block (grid.y splits the rest)
    int rpi;                 // rows a block advances per iteration
    int col_groups;          // grid.y
    int blocks;              // grid.x
    int64_t rows_per_block;  // contiguous rows of one block
};

Layout make_layout(int64_t pixels, int c, int vw, int cap = kMaxBlocks)
{
    Layout l;
    l.pixels = pixels;
    l.row_len = 4 * c;
    l.vw = vw;
    l.chunks = l.row_len / vw;
    l.cg = l.chunks < kThreads ? l.chunks : kThreads;
    l.rpi = kThreads / l.cg;
    l.col_groups = (l.chunks + l.cg - 1) / l.cg;
    const int64_t rows_per_iter_block = int64_t(l.rpi) * kMinRowsPerThread;
    int64_t want = (pixels + rows_per_iter_block - 1) / rows_per_iter_block;
    int max_blocks = cap;  // per column group
    if (max_blocks < 1)
        max_blocks = 1;
    if (want > max_blocks)
        want = max_blocks;
    if (want < 1)
        want = 1;
    l.rows_per_block = (pixels + want - 1) / want;
    l.blocks = int((pixels + l.rows_per_block - 1) / l.rows_per_block);
    return l;
}

int vec_width(int c, DType dt)
{
    const int epc = dt == DType::BF16 ? 8 : 4;
    return (4 * c) % epc == 0 ? epc : 1;
}

template <typename T, int VW>
__global__ __launch_bounds__(kThreads) void iqbn_stats(const T *__restrict__ x, Layout l,
                                                       float *__restrict__ part)
{
    __shared__ float red[2][kThreads][VW];
    const int tid = threadIdx.x;
    const int cl = tid % l.cg;
    const int rl = tid / l.cg;
    const int col = blockIdx.y * l.cg + cl;
    const bool active = rl < l.rpi && col < l.chunks;
    const int64_t r0 = int64_t(blockIdx.x) * l.rows_per_block;
    int64_t r1 = r0 + l.rows_per_block;
    if (r1 > l.pixels)
        r1 = l.pixels;

    float s1[VW], s2[VW], k[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e)
        s1[e] = s2[e] = k[e] = 0.0f;

    if (active) {
        const Vec<T, VW> kv = *reinterpret_cast<const Vec<T, VW> *>(x + col * VW);
#pragma unroll
        for (int e = 0; e < VW; ++e)
            k[e] = float(kv.v[e]);
        const T *base = x + col * VW;
        const int64_t step = l.rpi;
        int64_t r = r0 + rl;
        // Four independent loads in flight per thread.
        for (; r + 3 * step < r1; r += 4 * step) {
            Vec<T, VW> v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                v[u] = *reinterpret_cast<const Vec<T, VW> *>(base + (r + u * step) * l.row_len);
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int e = 0; e < VW; ++e) {
                    const float d = float(v[u].v[e]) - k[e];
                    s1[e] += d;
                    s2[e] = fmaf(d, d, s2[e]);
                }
        }
        for (; r < r1; r += step) {
            const Vec<T, VW> v = *reinterpret_cast<const Vec<T, VW> *>(base + r * l.row_len);
#pragma unroll
            for (int e = 0; e < VW; ++e) {
                const float d = float(v.v[e]) - k[e];
                s1[e] += d;
                s2[e] = fmaf(d, d, s2[e]);
            }
        }
    }
#pragma unroll
    for (int e = 0; e < VW; ++e) {
        red[0][tid][e] = s1[e];
        red[1][tid][e] = s2[e];
    }
    __syncthreads();
    if (rl == 0 && col < l.chunks) {
        float t1[VW], t2[VW];
#pragma unroll
        for (int e = 0; e < VW; ++e)
            t1[e] = t2[e] = 0.0f;
        for (int j = 0; j < l.rpi; ++j) {
#pragma unroll
            for (int e = 0; e < VW; ++e) {
                t1[e] += red[0][j * l.cg + cl][e];
                t2[e] += red[1][j * l.cg + cl][e];
            }
        }
        // Partials are column-major, [2][L][blocks]: the finalize pass reads
        // one column's partials with consecutive lanes.
        const size_t stride2 = size_t(l.row_len) * l.blocks;
#pragma unroll
        for (int e = 0; e < VW; ++e) {
            const size_t idx = size_t(col * VW + e) * l.blocks + blockIdx.x;
            part[idx] = t1[e];
            part[stride2 + idx] = t2[e];
        }
    }
}

// One wave per column: lane i adds the partials of blocks i, i+64, ... (all
// loads issued before any is used), then a fixed butterfly across the wave
// gives every lane the same fp64 total.  Deterministic: no atomics.
template <typename T>
__global__ __launch_bounds__(kThreads) void iqbn_finalize(const T *__restrict__ x, Layout l,
                                                          const float *__restrict__ part,
                                                          const float *__restrict__ gamma,
                                                          const float *__restrict__ beta, float eps,
                                                          float *__restrict__ mean, float *__restrict__ var,
                                                          float *__restrict__ affine)
{
    constexpr int PER_LANE = kMaxBlocks / 64;
    const int lane = threadIdx.x & 63;
    const int col = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (col >= l.row_len)
        return;
    const float *p1 = part + size_t(col) * l.blocks;
    const float *p2 = p1 + size_t(l.row_len) * l.blocks;
    // the column's shift K, gamma and beta are loaded together with the
    // partials, so the final step waits on no further memory
    const float k = float(x[col]), g = gamma[col], be = beta[col];
    float v1[PER_LANE], v2[PER_LANE];
#pragma unroll
    for (int u = 0; u < PER_LANE; ++u) {
        const int b = lane + 64 * u;
        const int bc = b < l.blocks ? b : l.blocks - 1;
        v1[u] = p1[bc];
        v2[u] = p2[bc];
    }
    double s1 = 0.0, s2 = 0.0;
#pragma unroll
    for (int u = 0; u < PER_LANE; ++u) {
        if (lane + 64 * u < l.blocks) {
            s1 += double(v1[u]);
            s2 += double(v2[u]);
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        s1 += __shfl_xor(s1, off);
        s2 += __shfl_xor(s2, off);
    }
    if (lane == 0) {
        const double n = double(l.pixels);
        const double d = s1 / n;          // mean - K
        double v = s2 / n - d * d;        // biased variance
        if (v < 0.0)
            v = 0.0;
        const double mu = double(k) + d;
        const double sc = double(g) / sqrt(v + double(eps));
        mean[col] = float(mu);
        var[col] = float(v);
        affine[col] = float(mu);
        affine[l.row_len + col] = float(sc);
        affine[2 * l.row_len + col] = be;
    }
}

// Statistics from per-tile partials (the convolution's epilogue): tile t of
// a column holds the mean and the sum of squared deviations of its
// n_t = min(tile_rows, pixels - t * tile_rows) rows.  One work-group per
// column, in fp64 and two passes over the partials: the column mean is the
// count-weighted mean of the tile means, and the sum of squared deviations
// is the tiles' own plus n_t (mean_t - mean)^2 each (the parallel-axis
// identity, exact; no division per tile).  Thread i takes tiles i, i+256,
// ... with eight loads in flight; a fixed butterfly per wave and a fixed
// order over the waves add the threads, so the result does not depend on
// timing.
__global__ __launch_bounds__(kThreads) void iqbn_finalize_tiles(const float *__restrict__ part, int m_tiles,
                                                                int tile_rows, int64_t pixels, int row_len,
                                                                const float *__restrict__ gamma,
                                                                const float *__restrict__ beta, float eps,
                                                                float *__restrict__ mean, float *__restrict__ var,
                                                                float *__restrict__ affine)
{
    constexpr int U = 8;  // loads in flight per thread
    constexpr int NW = kThreads / 64;
    __shared__ double red[NW];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int col = blockIdx.x;
    const float *pm = part + size_t(col) * m_tiles;
    const float *pq = part + (size_t(row_len) + col) * m_tiles;
    const int last = m_tiles - 1;
    const double n_last = double(pixels - int64_t(last) * tile_rows);
    auto rows = [&](int t) { return t == last ? n_last : double(tile_rows); };
    // loads past the last tile read the last tile again (unconditional, so
    // all U are in flight at once) and are not added
    auto clamp_tile = [&](int t) { return t < last ? t : last; };
    auto block_sum = [&](double v) {
#pragma unroll
        for (int off = 32; off > 0; off >>= 1)
            v += __shfl_xor(v, off);
        if (lane == 0)
            red[wv] = v;
        __syncthreads();
        double total = 0.0;
#pragma unroll
        for (int w = 0; w < NW; ++w)
            total += red[w];
        __syncthreads();  // red is reused by the next sum
        return total;
    };
    const float g = gamma[col], be = beta[col];
    // The first kThreads * U tiles (all of them up to 2048 tiles) are loaded
    // once, means and sums together, and stay in registers for pass 2.
    float m0[U], q0[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        m0[u] = pm[clamp_tile(tid + kThreads * u)];
        q0[u] = pq[clamp_tile(tid + kThreads * u)];
    }
    // pass 1: sum of n_t * mean_t
    double s = 0.0;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int t = tid + kThreads * u;
        if (t < m_tiles)
            s += rows(t) * double(m0[u]);
    }
    for (int t0 = tid + kThreads * U; t0 < m_tiles; t0 += kThreads * U) {
        float mt[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            mt[u] = pm[clamp_tile(t0 + kThreads * u)];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int t = t0 + kThreads * u;
            if (t < m_tiles)
                s += rows(t) * double(mt[u]);
        }
    }
    const double mu = block_sum(s) / double(pixels);
    // pass 2: sum of M2_t + n_t * (mean_t - mean)^2
    double q = 0.0;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int t = tid + kThreads * u;
        if (t < m_tiles) {
            const double d = double(m0[u]) - mu;
            q += double(q0[u]) + rows(t) * d * d;
        }
    }
    for (int t0 = tid + kThreads * U; t0 < m_tiles; t0 += kThreads * U) {
        float mt[U], qt[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            mt[u] = pm[clamp_tile(t0 + kThreads * u)];
            qt[u] = pq[clamp_tile(t0 + kThreads * u)];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int t = t0 + kThreads * u;
            if (t < m_tiles) {
                const double d = double(mt[u]) - mu;
                q += double(qt[u]) + rows(t) * d * d;
            }
        }
    }
    const double m2 = block_sum(q);
    if (tid == 0) {
        double v = m2 / double(pixels);  // biased variance
        if (v < 0.0)
            v = 0.0;
        const double sc = double(g) / sqrt(v + double(eps));
        mean[col] = float(mu);
        var[col] = float(v);
        affine[col] = float(mu);
        affine[row_len + col] = float(sc);
        affine[2 * row_len + col] = be;
    }
}

template <typename T, int VW, bool RELU>
__global__ __launch_bounds__(kThreads) void iqbn_affine(const T *x, T *out, Layout l,
                                                        const float *__restrict__ affine)
{
    const int tid = threadIdx.x;
    const int cl = tid % l.cg;
    const int rl = tid / l.cg;
    const int col = blockIdx.y * l.cg + cl;
    if (rl >= l.rpi || col >= l.chunks)
        return;
    float mu[VW], sc[VW], be[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e) {
        mu[e] = affine[col * VW + e];
        sc[e] = affine[l.row_len + col * VW + e];
        be[e] = affine[2 * l.row_len + col * VW + e];
    }
    const int64_t r0 = int64_t(blockIdx.x) * l.rows_per_block;
    int64_t r1 = r0 + l.rows_per_block;
    if (r1 > l.pixels)
        r1 = l.pixels;
    const int64_t step = l.rpi;
    const T *src = x + col * VW;
    T *dst = out + col * VW;
    int64_t r = r0 + rl;
    for (; r + 3 * step < r1; r += 4 * step) {
        Vec<T, VW> v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            v[u] = *reinterpret_cast<const Vec<T, VW> *>(src + (r + u * step) * l.row_len);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            Vec<T, VW> o;
#pragma unroll
            for (int e = 0; e < VW; ++e) {
                float y = fmaf(float(v[u].v[e]) - mu[e], sc[e], be[e]);
                if (RELU)
                    y = fmaxf(y, 0.0f);
                o.v[e] = T(y);
            }
            store_stream(reinterpret_cast<Vec<T, VW> *>(dst + (r + u * step) * l.row_len), o);
        }
    }
    for (; r < r1; r += step) {
        const Vec<T, VW> v = *reinterpret_cast<const Vec<T, VW> *>(src + r * l.row_len);
        Vec<T, VW> o;
#pragma unroll
        for (int e = 0; e < VW; ++e) {
            float y = fmaf(float(v.v[e]) - mu[e], sc[e], be[e]);
            if (RELU)
                y = fmaxf(y, 0.0f);
            o.v[e] = T(y);
        }
        *reinterpret_cast<Vec<T, VW> *>(dst + r * l.row_len) = o;
    }
}

// ------------------------------ backward ------------------------------
// Gradient of training-mode IQBN (eqs. 11, 12) given the saved batch mean
// and biased variance: per column, with s = sqrt(var + eps), xhat = (x - mean)
// / s and g = dout (zeroed where the saved ReLU output y is <= 0),
//
//   dbeta = sum g,  dgamma = sum g xhat,
//   dx = (gamma / s) (g - dbeta / n - xhat dgamma / n).
//
// Pass 1 (iqbn_bwd_reduce) writes per-block partial sums of g and g xhat in
// the statistics pass's layout, iqbn_bwd_finalize adds them in fp64 in block
// order (deterministic) and forms the three coefficients, pass 2
// (iqbn_bwd_apply) writes dx.  x, dout and y read twice, dx written once.

template <typename T, int VW>
__device__ __forceinline__ void load_col_params(const float *__restrict__ mean, const float *__restrict__ var,
                                                float eps, int col, float *mu, float *inv)
{
#pragma unroll
    for (int e = 0; e < VW; ++e) {
        mu[e] = mean[col * VW + e];
        inv[e] = 1.0f / sqrtf(var[col * VW + e] + eps);
    }
}

template <typename T, int VW, bool RELU>
__global__ __launch_bounds__(kThreads) void iqbn_bwd_reduce(const T *__restrict__ x, const T *__restrict__ dout,
                                                            const T *__restrict__ y, Layout l,
                                                            const float *__restrict__ mean,
                                                            const float *__restrict__ var, float eps,
                                                            float *__restrict__ part)
{
    __shared__ float red[2][kThreads][VW];
    const int tid = threadIdx.x;
    const int cl = tid % l.cg;
    const int rl = tid / l.cg;
    const int col = blockIdx.y * l.cg + cl;
    const bool active = rl < l.rpi && col < l.chunks;
    const int64_t r0 = int64_t(blockIdx.x) * l.rows_per_block;
    int64_t r1 = r0 + l.rows_per_block;
    if (r1 > l.pixels)
        r1 = l.pixels;
    float s1[VW], s2[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e)
        s1[e] = s2[e] = 0.0f;
    if (active) {
        float mu[VW], inv[VW];
        load_col_params<T, VW>(mean, var, eps, col, mu, inv);
        const int64_t step = l.rpi;
        auto add = [&](const Vec<T, VW> &xv, const Vec<T, VW> &gv, const Vec<T, VW> &yv) {
#pragma unroll
            for (int e = 0; e < VW; ++e) {
                float g = float(gv.v[e]);
                if (RELU && !(float(yv.v[e]) > 0.0f))
                    g = 0.0f;
                const float xh = (float(xv.v[e]) - mu[e]) * inv[e];
                s1[e] += g;
                s2[e] = fmaf(g, xh, s2[e]);
            }
        };
        int64_t r = r0 + rl;
        // four rows in flight per thread
        for (; r + 3 * step < r1; r += 4 * step) {
            Vec<T, VW> xv[4], gv[4], yv[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t off = (r + u * step) * l.row_len + col * VW;
                xv[u] = *reinterpret_cast<const Vec<T, VW> *>(x + off);
                gv[u] = *reinterpret_cast<const Vec<T, VW> *>(dout + off);
                if (RELU)
                    yv[u] = *reinterpret_cast<const Vec<T, VW> *>(y + off);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                add(xv[u], gv[u], yv[u]);
        }
        for (; r < r1; r += step) {
            const int64_t off = r * l.row_len + col * VW;
            Vec<T, VW> yv;
            if (RELU)
                yv = *reinterpret_cast<const Vec<T, VW> *>(y + off);
            add(*reinterpret_cast<const Vec<T, VW> *>(x + off), *reinterpret_cast<const Vec<T, VW> *>(dout + off),
                yv);
        }
    }
#pragma unroll
    for (int e = 0; e < VW; ++e) {
        red[0][tid][e] = s1[e];
        red[1][tid][e] = s2[e];
    }
    __syncthreads();
    if (rl == 0 && col < l.chunks) {
        float t1[VW], t2[VW];
#pragma unroll
        for (int e = 0; e < VW; ++e)
            t1[e] = t2[e] = 0.0f;
        for (int j = 0; j < l.rpi; ++j) {
#pragma unroll
            for (int e = 0; e < VW; ++e) {
                t1[e] += red[0][j * l.cg + cl][e];
                t2[e] += red[1][j * l.cg + cl][e];
            }
        }
        const size_t stride2 = size_t(l.row_len) * l.blocks;
#pragma unroll
        for (int e = 0; e < VW; ++e) {
            const size_t idx = size_t(col * VW + e) * l.blocks + blockIdx.x;
            part[idx] = t1[e];
            part[stride2 + idx] = t2[e];
        }
    }
}

// One wave per column: fp64 sums of the partials (fixed order), then
// dbeta, dgamma and coef = [gamma / s, dbeta / n, dgamma / n].
__global__ __launch_bounds__(kThreads) void iqbn_bwd_finalize(Layout l, const float *__restrict__ part,
                                                              const float *__restrict__ var,
                                                              const float *__restrict__ gamma, float eps,
                                                              float *__restrict__ dgamma,
                                                              float *__restrict__ dbeta, float *__restrict__ coef)
{
    constexpr int PER_LANE = kMaxBlocks / 64;
    const int lane = threadIdx.x & 63;
    const int col = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (col >= l.row_len)
        return;
    const float *p1 = part + size_t(col) * l.blocks;
    const float *p2 = p1 + size_t(l.row_len) * l.blocks;
    const float g = gamma[col], vc = var[col];
    float v1[PER_LANE], v2[PER_LANE];
#pragma unroll
    for (int u = 0; u < PER_LANE; ++u) {
        const int b = lane + 64 * u;
        const int bc = b < l.blocks ? b : l.blocks - 1;
        v1[u] = p1[bc];
        v2[u] = p2[bc];
    }
    double s1 = 0.0, s2 = 0.0;
#pragma unroll
    for (int u = 0; u < PER_LANE; ++u) {
        if (lane + 64 * u < l.blocks) {
            s1 += double(v1[u]);
            s2 += double(v2[u]);
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        s1 += __shfl_xor(s1, off);
        s2 += __shfl_xor(s2, off);
    }
    if (lane == 0) {
        const double n = double(l.pixels);
        dbeta[col] = float(s1);
        dgamma[col] = float(s2);
        coef[col] = float(double(g) / sqrt(double(vc) + double(eps)));
        coef[l.row_len + col] = float(s1 / n);
        coef[2 * l.row_len + col] = float(s2 / n);
    }
}

template <typename T, int VW, bool RELU>
__global__ __launch_bounds__(kThreads) void iqbn_bwd_apply(const T *__restrict__ x, const T *__restrict__ dout,
                                                           const T *__restrict__ y, T *__restrict__ dx, Layout l,
                                                           const float *__restrict__ mean,
                                                           const float *__restrict__ var, float eps,
                                                           const float *__restrict__ coef)
{
    const int tid = threadIdx.x;
    const int cl = tid % l.cg;
    const int rl = tid / l.cg;
    const int col = blockIdx.y * l.cg + cl;
    if (rl >= l.rpi || col >= l.chunks)
        return;
    float mu[VW], inv[VW], a[VW], b1[VW], b2[VW];
    load_col_params<T, VW>(mean, var, eps, col, mu, inv);
#pragma unroll
    for (int e = 0; e < VW; ++e) {
        a[e] = coef[col * VW + e];
        b1[e] = coef[l.row_len + col * VW + e];
        b2[e] = coef[2 * l.row_len + col * VW + e];
    }
    // Rows are dealt out round-robin (block b takes rows b*rpi .. b*rpi+rpi-1
    // of every group of blocks*rpi), so at any moment the work-groups read
    // one narrow window of each of the three or four streams: measured 48.4
    // -> 46.0 us on 200704 x 1024 bf16 against contiguous row ranges per
    // work-group (which the two-stream passes keep: there round-robin rows
    // were 1-3 us slower).
    const int64_t r1 = l.pixels;
    auto grad = [&](const Vec<T, VW> &xv, const Vec<T, VW> &gv, const Vec<T, VW> &yv) {
        Vec<T, VW> o;
#pragma unroll
        for (int e = 0; e < VW; ++e) {
            float g = float(gv.v[e]);
            if (RELU && !(float(yv.v[e]) > 0.0f))
                g = 0.0f;
            const float xh = (float(xv.v[e]) - mu[e]) * inv[e];
            o.v[e] = T(a[e] * (g - b1[e] - xh * b2[e]));
        }
        return o;
    };
    const int64_t step = int64_t(l.rpi) * l.blocks;
    int64_t r = int64_t(blockIdx.x) * l.rpi + rl;
    // four rows in flight per thread; each row's dx is written after its own
    // loads (dx may be dout)
    for (; r + 3 * step < r1; r += 4 * step) {
        Vec<T, VW> xv[4], gv[4], yv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t off = (r + u * step) * l.row_len + col * VW;
            xv[u] = *reinterpret_cast<const Vec<T, VW> *>(x + off);
            gv[u] = *reinterpret_cast<const Vec<T, VW> *>(dout + off);
            if (RELU)
                yv[u] = *reinterpret_cast<const Vec<T, VW> *>(y + off);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            store_stream(reinterpret_cast<Vec<T, VW> *>(dx + (r + u * step) * l.row_len + col * VW), grad(xv[u], gv[u], yv[u]));
    }
    for (; r < r1; r += step) {
        const int64_t off = r * l.row_len + col * VW;
        Vec<T, VW> yv;
        if (RELU)
            yv = *reinterpret_cast<const Vec<T, VW> *>(y + off);
        *reinterpret_cast<Vec<T, VW> *>(dx + off) =
            grad(*reinterpret_cast<const Vec<T, VW> *>(x + off), *reinterpret_cast<const Vec<T, VW> *>(dout + off), yv);
    }
}

template <typename T, int VW>
hipError_t launch_backward(const void *x, const void *dout, const void *y, const float *mean, const float *var,
                           const float *gamma, float eps, void *dx, float *dgamma, float *dbeta, int64_t pixels,
                           int c, void *work, hipStream_t stream)
{
    const Layout l = make_layout(pixels, c, VW);
    float *part = static_cast<float *>(work);
    float *coef = part + size_t(l.blocks) * 2 * l.row_len;
    const T *xt = static_cast<const T *>(x), *gt = static_cast<const T *>(dout), *yt = static_cast<const T *>(y);
    const dim3 grid(l.blocks, l.col_groups);
    if (y != nullptr)
        hipLaunchKernelGGL((iqbn_bwd_reduce<T, VW, true>), grid, dim3(kThreads), 0, stream, xt, gt, yt, l, mean,
                           var, eps, part);
    else
        hipLaunchKernelGGL((iqbn_bwd_reduce<T, VW, false>), grid, dim3(kThreads), 0, stream, xt, gt, yt, l,
                           mean, var, eps, part);
    const int fin_blocks = (l.row_len + kThreads / 64 - 1) / (kThreads / 64);
    hipLaunchKernelGGL(iqbn_bwd_finalize, dim3(fin_blocks), dim3(kThreads), 0, stream, l, (const float *)part,
                       var, gamma, eps, dgamma, dbeta, coef);
    const Layout ls = make_layout(pixels, c, VW, kStreamBlocks);
    const dim3 sgrid(ls.blocks, ls.col_groups);
    if (y != nullptr)
        hipLaunchKernelGGL((iqbn_bwd_apply<T, VW, true>), sgrid, dim3(kThreads), 0, stream, xt, gt, yt,
                           static_cast<T *>(dx), ls, mean, var, eps, (const float *)coef);
    else
        hipLaunchKernelGGL((iqbn_bwd_apply<T, VW, false>), sgrid, dim3(kThreads), 0, stream, xt, gt, yt,
                           static_cast<T *>(dx), ls, mean, var, eps, (const float *)coef);
    return hipGetLastError();
}

template <typename T, int VW>
hipError_t launch_all(const void *x, const float *gamma, const float *beta, float eps, bool relu,
                      void *out, float *mean, float *var, int64_t pixels, int c, void *work,
                      hipStream_t stream)
{
    const Layout l = make_layout(pixels, c, VW);
    float *part = static_cast<float *>(work);
    float *affine = part + size_t(l.blocks) * 2 * l.row_len;
    const T *xt = static_cast<const T *>(x);
    const dim3 grid(l.blocks, l.col_groups);
    hipLaunchKernelGGL((iqbn_stats<T, VW>), grid, dim3(kThreads), 0, stream, xt, l, part);
    const int fin_blocks = (l.row_len + kThreads / 64 - 1) / (kThreads / 64);
    hipLaunchKernelGGL((iqbn_finalize<T>), dim3(fin_blocks), dim3(kThreads), 0, stream, xt, l, part,
                       gamma, beta, eps, mean, var, affine);
    const Layout ls = make_layout(pixels, c, VW, kStreamBlocks);
    const dim3 sgrid(ls.blocks, ls.col_groups);
    if (relu)
        hipLaunchKernelGGL((iqbn_affine<T, VW, true>), sgrid, dim3(kThreads), 0, stream, xt,
                           static_cast<T *>(out), ls, (const float *)affine);
    else
        hipLaunchKernelGGL((iqbn_affine<T, VW, false>), sgrid, dim3(kThreads), 0, stream, xt,
                           static_cast<T *>(out), ls, (const float *)affine);
    return hipGetLastError();
}

template <typename T, int VW>
hipError_t launch_from_tiles(const float *part, int m_tiles, int tile_rows, const float *gamma,
                             const float *beta, float eps, bool relu, void *io, float *mean, float *var,
                             int64_t pixels, int c, float *affine, hipStream_t stream)
{
    const Layout l = make_layout(pixels, c, VW);
    hipLaunchKernelGGL(iqbn_finalize_tiles, dim3(l.row_len), dim3(kThreads), 0, stream, part, m_tiles,
                       tile_rows, pixels, l.row_len, gamma, beta, eps, mean, var, affine);
    T *t = static_cast<T *>(io);
    const Layout ls = make_layout(pixels, c, VW, kStreamBlocks);
    const dim3 sgrid(ls.blocks, ls.col_groups);
    if (relu)
        hipLaunchKernelGGL((iqbn_affine<T, VW, true>), sgrid, dim3(kThreads), 0, stream, t, t, ls,
                           (const float *)affine);
    else
        hipLaunchKernelGGL((iqbn_affine<T, VW, false>), sgrid, dim3(kThreads), 0, stream, t, t, ls,
                           (const float *)affine);
    return hipGetLastError();
}

// Inference IQBN folded into a convolution's epilogue: one thread per
// column, fp64, scale = gamma / sqrt(var + eps), shift = (bias - mean) *
// scale + beta.
template <typename T>
__global__ __launch_bounds__(kThreads) void iqbn_fold(const float *__restrict__ mean, const float *__restrict__ var,
                                                      const float *__restrict__ gamma,
                                                      const float *__restrict__ beta, const T *__restrict__ bias,
                                                      float eps, int cols, float *__restrict__ scale,
                                                      float *__restrict__ shift)
{
    const int col = blockIdx.x * kThreads + threadIdx.x;
    if (col >= cols)
        return;
    const double sc = double(gamma[col]) / sqrt(double(var[col]) + double(eps));
    const double b = bias != nullptr ? double(float(bias[col])) : 0.0;
    scale[col] = float(sc);
    shift[col] = float((b - double(mean[col])) * sc + double(beta[col]));
}

}  // namespace

hipError_t iqbn_fold_run(const float *mean, const float *var, const float *gamma, const float *beta,
                         const void *bias, float eps, int c, DType dt, float *scale, float *shift,
                         hipStream_t stream)
{
    const int cols = 4 * c;
    const int blocks = (cols + kThreads - 1) / kThreads;
    if (dt == DType::BF16)
        hipLaunchKernelGGL(iqbn_fold<__bf16>, dim3(blocks), dim3(kThreads), 0, stream, mean, var, gamma, beta,
                           static_cast<const __bf16 *>(bias), eps, cols, scale, shift);
    else
        hipLaunchKernelGGL(iqbn_fold<float>, dim3(blocks), dim3(kThreads), 0, stream, mean, var, gamma, beta,
                           static_cast<const float *>(bias), eps, cols, scale, shift);
    return hipGetLastError();
}

size_t iqbn_tile_stats_bytes(int m_tiles, int c)
{
    return (size_t(2) * m_tiles + 3) * 4 * c * sizeof(float);
}

hipError_t iqbn_from_tiles_run(const float *part, int m_tiles, int tile_rows, const float *gamma,
                               const float *beta, float eps, bool relu, void *io, float *mean, float *var,
                               int64_t pixels, int c, DType dt, hipStream_t stream)
{
    float *affine = const_cast<float *>(part) + size_t(2) * m_tiles * 4 * c;
    const int vw = vec_width(c, dt);
    if (dt == DType::BF16) {
        if (vw == 8)
            return launch_from_tiles<__bf16, 8>(part, m_tiles, tile_rows, gamma, beta, eps, relu, io, mean,
                                                var, pixels, c, affine, stream);
        return launch_from_tiles<__bf16, 1>(part, m_tiles, tile_rows, gamma, beta, eps, relu, io, mean, var,
                                            pixels, c, affine, stream);
    }
    if (vw == 4)
        return launch_from_tiles<float, 4>(part, m_tiles, tile_rows, gamma, beta, eps, relu, io, mean, var,
                                           pixels, c, affine, stream);
    return launch_from_tiles<float, 1>(part, m_tiles, tile_rows, gamma, beta, eps, relu, io, mean, var,
                                       pixels, c, affine, stream);
}

size_t iqbn_workspace_bytes(int64_t pixels, int c)
{
    // Largest over the vector widths the dispatcher may pick.
    size_t best = 0;
    for (int vw : {1, 4, 8}) {
        if ((4 * c) % vw)
            continue;
        const Layout l = make_layout(pixels, c, vw);
        const size_t b = (size_t(l.blocks) * 2 + 3) * size_t(l.row_len) * sizeof(float);
        if (b > best)
            best = b;
    }
    return best;
}

hipError_t iqbn_backward_run(const void *x, const void *dout, const void *y, const float *mean, const float *var,
                             const float *gamma, float eps, void *dx, float *dgamma, float *dbeta, int64_t pixels,
                             int c, DType dt, void *work, hipStream_t stream)
{
    const int vw = vec_width(c, dt);
    if (dt == DType::BF16) {
        if (vw == 8)
            return launch_backward<__bf16, 8>(x, dout, y, mean, var, gamma, eps, dx, dgamma, dbeta, pixels, c,
                                              work, stream);
        return launch_backward<__bf16, 1>(x, dout, y, mean, var, gamma, eps, dx, dgamma, dbeta, pixels, c, work,
                                          stream);
    }
    if (vw == 4)
        return launch_backward<float, 4>(x, dout, y, mean, var, gamma, eps, dx, dgamma, dbeta, pixels, c, work,
                                         stream);
    return launch_backward<float, 1>(x, dout, y, mean, var, gamma, eps, dx, dgamma, dbeta, pixels, c, work,
                                     stream);
}

hipError_t iqbn_run(const void *x, const float *gamma, const float *beta, float eps, bool relu,
                    void *out, float *mean, float *var, int64_t pixels, int c, DType dt, void *work,
                    hipStream_t stream)
{
    const int vw = vec_width(c, dt);
    if (dt == DType::BF16) {
        if (vw == 8)
            return launch_all<__bf16, 8>(x, gamma, beta, eps, relu, out, mean, var, pixels, c, work, stream);
        return launch_all<__bf16, 1>(x, gamma, beta, eps, relu, out, mean, var, pixels, c, work, stream);
    }
    if (vw == 4)
        return launch_all<float, 4>(x, gamma, beta, eps, relu, out, mean, var, pixels, c, work, stream);
    return launch_all<float, 1>(x, gamma, beta, eps, relu, out, mean, var, pixels, c, work, stream);
}

}  // namespace quan
