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
// Tensors of up to 32 MiB whose rows span at least four 64-column groups
// take two launches instead: iqbn_stats over blocks of 64 columns (at most
// 64 partials per column), then iqbn_merge_affine, which merges the partials
// inside the normalization pass while its first loads of x are in flight.
// Larger tensors take the one-launch form below where it fits.
//
// After a convolution that wrote per-tile statistics of its output (fused
// into its epilogue), iqbn_finalize_tiles replaces passes 1 and 2: the
// normalization then costs one read and one write of the tensor.
#include <hip/hip_runtime.h>

#include <mutex>
#include <type_traits>

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

// Merged finalize and normalization, for tensors whose columns have few
// statistics partials: the finalize step runs inside the normalization pass
// instead of a launch of its own.  A block covers kMergeCols columns of a run
// of rows; it issues the loads of its first rows, merges its columns'
// partials in fp64 (a fixed order, the same in every block of the column
// group) while those loads are in flight, and then normalises its rows.
constexpr int kMergeCols = 64;
constexpr int kMergeMaxParts = 64;                   // statistics blocks per column
constexpr int kMergeSlices = kThreads / kMergeCols;  // merge threads per column
constexpr int kMergeBlocks = 256;                    // target blocks per launch
constexpr int64_t kMergeMaxBytes = int64_t(32) << 20;

// Column-group layout of the merged path: kMergeCols columns per block,
// blocks_x runs of rows per column group (grid (blocks, col_groups), so that
// consecutive blocks, which the XCDs take in turn, stream different rows).
Layout make_layout_narrow(int64_t pixels, int c, int vw, int blocks_x)
{
    Layout l;
    l.pixels = pixels;
    l.row_len = 4 * c;
    l.vw = vw;
    l.chunks = l.row_len / vw;
    const int want_cg = kMergeCols / vw;
    l.cg = l.chunks < want_cg ? l.chunks : want_cg;
    l.rpi = kThreads / l.cg;
    l.col_groups = (l.chunks + l.cg - 1) / l.cg;
    if (blocks_x < 1)
        blocks_x = 1;
    l.rows_per_block = (pixels + blocks_x - 1) / blocks_x;
    l.blocks = int((pixels + l.rows_per_block - 1) / l.rows_per_block);
    return l;
}

// Row blocks per column group of the merged path: about kMergeBlocks blocks
// in all, at most kMergeMaxParts, and at least one row per thread.
int merge_blocks_x(int64_t pixels, int c, int vw)
{
    const Layout l = make_layout_narrow(pixels, c, vw, 1);
    int64_t bx = (kMergeBlocks + l.col_groups - 1) / l.col_groups;
    const int64_t by_rows = (pixels + l.rpi - 1) / l.rpi;
    if (bx > by_rows)
        bx = by_rows;
    if (bx > kMergeMaxParts)
        bx = kMergeMaxParts;
    return bx < 1 ? 1 : int(bx);
}

// Whether IQBN takes the merged path: a tensor of at most kMergeMaxBytes
// whose rows span at least four column groups (so the launch has enough
// blocks).  Measured on MI355X, cold: 12.8 MB (6272 rows of 1024 columns)
// 16.4 us against 23.4 for three launches; 25.7 MB 21.7 us against 27.7 for
// the one-launch form; at 52 MB the one-launch form is ahead (35.0 against
// 38.4 us with up to 128 partials per column), and at 103 MB (54.6 against
// 63.0).
bool merge_takes(int64_t pixels, int c, int vw, int elem)
{
    const Layout l = make_layout_narrow(pixels, c, vw, 1);
    return pixels * l.row_len * elem <= kMergeMaxBytes && l.col_groups >= 4;
}

int vec_width(int c, DType dt)
{
    const int epc = dt == DType::BF16 ? 8 : 4;
    return (4 * c) % epc == 0 ? epc : 1;
}

template <typename T, int VW>
__global__ __launch_bounds__(kThreads) void iqbn_stats(const T *__restrict__ x, Layout l,
                                                       float *__restrict__ part, float *__restrict__ kout)
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
        // Partials are column-major, [2][L][blocks], for iqbn_finalize (it
        // reads one column's partials with consecutive lanes), or, with
        // kout given, block-major, [2][blocks][L], for iqbn_merge_affine
        // (consecutive lanes take consecutive columns).
        const size_t stride2 = size_t(l.row_len) * l.blocks;
#pragma unroll
        for (int e = 0; e < VW; ++e) {
            const size_t idx = kout != nullptr ? size_t(blockIdx.x) * l.row_len + col * VW + e
                                               : size_t(col * VW + e) * l.blocks + blockIdx.x;
            part[idx] = t1[e];
            part[stride2 + idx] = t2[e];
        }
        // the shifts K, for a finalize that cannot read x's row 0 (the
        // merged pass normalises in place)
        if (kout != nullptr && blockIdx.x == 0)
#pragma unroll
            for (int e = 0; e < VW; ++e)
                kout[col * VW + e] = k[e];
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

// The merged finalize + normalization (see kMergeCols), after iqbn_stats
// with block-major partials: part[b][col] = s1 of block b, part[n_part][...]
// the s2, then the shifts K (part + 2 L n_part).  Merge thread t takes
// column t % kMergeCols (so a wave's loads are 64 consecutive floats) and
// blocks t / kMergeCols + kMergeSlices i; the slices are added in slice
// order, in fp64, the same in every block.  The blocks of row block 0 also
// write mean and var.  In place (x == out) is allowed: a block reads and
// writes only its own rows, and K comes from the partials.
struct MergeArgs {
    const float *part;
    int n_part;
    const float *gamma;
    const float *beta;
    float eps;
    float *mean;
    float *var;
};

template <typename T, int VW, bool RELU>
__global__ __launch_bounds__(kThreads) void iqbn_merge_affine(const T *x, T *out, Layout l, MergeArgs a)
{
    constexpr int MP = kMergeMaxParts / kMergeSlices;
    __shared__ double red[2][kMergeSlices][kMergeCols];
    __shared__ float coef[3][kMergeCols];
    const int tid = threadIdx.x;
    const int cl = tid % l.cg, rl = tid / l.cg;
    const int chunk = blockIdx.y * l.cg + cl;
    const bool active = rl < l.rpi && chunk < l.chunks;
    const int64_t r0 = int64_t(blockIdx.x) * l.rows_per_block;
    int64_t r1 = r0 + l.rows_per_block;
    if (r1 > l.pixels)
        r1 = l.pixels;
    const int64_t step = l.rpi;
    const T *src = x + chunk * VW;
    T *dst = out + chunk * VW;

    // the block's first rows, in flight during the merge
    int64_t r = r0 + rl;
    Vec<T, VW> v[4];
    if (active) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (r + u * step < r1)
                v[u] = *reinterpret_cast<const Vec<T, VW> *>(src + (r + u * step) * l.row_len);
    }

    // merge: wave sl is slice sl (its branches are wave-uniform)
    const int j = tid % kMergeCols, sl = tid / kMergeCols;
    const int col0 = blockIdx.y * l.cg * VW;
    const int col = col0 + j;
    const bool mcol = j < l.cg * VW && col < l.row_len;
    const int cc = mcol ? col : col0;
    const size_t plane = size_t(a.n_part) * l.row_len;
    float pv[MP], qv[MP];
#pragma unroll
    for (int i = 0; i < MP; ++i) {
        const int b = sl + kMergeSlices * i;
        pv[i] = 0.0f;
        qv[i] = 0.0f;
        if (b < a.n_part) {
            pv[i] = a.part[size_t(b) * l.row_len + cc];
            qv[i] = a.part[plane + size_t(b) * l.row_len + cc];
        }
    }
    double s1 = 0.0, s2 = 0.0;
#pragma unroll
    for (int i = 0; i < MP; ++i) {
        if (sl + kMergeSlices * i < a.n_part) {
            s1 += double(pv[i]);
            s2 += double(qv[i]);
        }
    }
    red[0][sl][j] = s1;
    red[1][sl][j] = s2;
    __syncthreads();
    if (sl == 0 && mcol) {
        double t1 = 0.0, t2 = 0.0;
#pragma unroll
        for (int w = 0; w < kMergeSlices; ++w) {
            t1 += red[0][w][j];
            t2 += red[1][w][j];
        }
        const double n = double(l.pixels);
        const double d = t1 / n;  // mean - K
        double var = t2 / n - d * d;
        if (var < 0.0)
            var = 0.0;
        const double mu = double(a.part[2 * plane + col]) + d;
        const double sc = double(a.gamma[col]) / sqrt(var + double(a.eps));
        coef[0][j] = float(mu);
        coef[1][j] = float(sc);
        coef[2][j] = a.beta[col];
        if (blockIdx.x == 0) {
            a.mean[col] = float(mu);
            a.var[col] = float(var);
        }
    }
    __syncthreads();
    if (!active)
        return;
    float mu[VW], sc[VW], be[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e) {
        mu[e] = coef[0][cl * VW + e];
        sc[e] = coef[1][cl * VW + e];
        be[e] = coef[2][cl * VW + e];
    }
    auto norm = [&](const Vec<T, VW> &in) {
        Vec<T, VW> o;
#pragma unroll
        for (int e = 0; e < VW; ++e) {
            float y = fmaf(float(in.v[e]) - mu[e], sc[e], be[e]);
            if (RELU)
                y = fmaxf(y, 0.0f);
            o.v[e] = T(y);
        }
        return o;
    };
#pragma unroll
    for (int u = 0; u < 4; ++u)
        if (r + u * step < r1)
            store_stream(reinterpret_cast<Vec<T, VW> *>(dst + (r + u * step) * l.row_len), norm(v[u]));
    r += 4 * step;
    for (; r + 3 * step < r1; r += 4 * step) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
            v[u] = *reinterpret_cast<const Vec<T, VW> *>(src + (r + u * step) * l.row_len);
#pragma unroll
        for (int u = 0; u < 4; ++u)
            store_stream(reinterpret_cast<Vec<T, VW> *>(dst + (r + u * step) * l.row_len), norm(v[u]));
    }
    for (; r < r1; r += step)
        store_stream(reinterpret_cast<Vec<T, VW> *>(dst + r * l.row_len),
                     norm(*reinterpret_cast<const Vec<T, VW> *>(src + r * l.row_len)));
}

// ------------------------ one-launch resident IQBN ------------------------
// Where the tensor fits in the registers and LDS of one work-group per
// compute unit (up to about 100 MB on 256 CUs), IQBN runs as ONE launch that
// reads x from memory once:
//
//   phase 1  work-group w copies its contiguous rows [w * R, (w + 1) * R) into
//            VGPRs (the first kResRegChunks 16-byte chunks of each thread) and
//            LDS (the next kResLdsChunks, by direct global->LDS loads), and
//            reduces the shifted sums s1 = sum(x - K), s2 = sum((x - K)^2)
//            of every column over its rows (K = the column's value in row
//            0, as in iqbn_stats) in a fixed order: one (s1, s2) pair per
//            column per work-group.
//   barrier  every work-group has published its partials.
//   phase 2  work-group w merges its ceil(L / G) columns over the G partials
//            in fp64, in work-group order, and publishes mean and scale.
//   barrier  every column's mean and scale are published.
//   phase 3  every work-group normalises the rows it holds and writes them.
//
// The grid is one work-group per compute unit and each work-group needs a
// whole compute unit's LDS, so all G are resident together.  Partials,
// coefficients and barrier flags are read by other XCDs (each XCD has its own
// L2): they are written and read with system-scope atomic stores and loads,
// which go to memory, and every thread waits for its own stores to complete
// before its work-group raises its flag.  The barrier has no read-modify-
// write: work-group w raises only its own flag, flags[w], and waits until
// every flag has reached the same value; each launch raises every flag by
// exactly two, so a work-group takes its targets from its own flag at the
// start.  The wait is bounded (kSpinLimit polls, about a second): a work-group
// that gives up writes NaN where its results would be, so a launch that could
// not run all its work-groups at once shows as NaNs, never as a hang.
constexpr int kResThreads = 512;
constexpr int kResRegChunks = 36;  // 16-byte chunks per thread held in VGPRs
constexpr int kResLdsChunks = 15;  // ... and in LDS
constexpr int kResChunks = kResRegChunks + kResLdsChunks;
constexpr int kResMaxGroups = 512;
constexpr int kResMaxCols = 16;     // columns merged per work-group in phase 2
constexpr int kFlagStride = 32;     // unsigned ints between flags: one 128-byte line each
constexpr long kSpinLimit = 1L << 20;
// Below 16 MiB the three launches are as fast (measured on MI355X: 12.8 MB
// tensors take 21-24 us either way, 16.8 MB 22.1 against 23.7, 52 MB 34.4
// against 37.7, 103 MB 54.6 against 59.4, cold), so only larger tensors rely
// on all work-groups being resident together; up to 32 MiB the merged
// two-launch form (merge_takes) is ahead where it applies.
constexpr int64_t kResMinBytes = int64_t(16) << 20;

typedef unsigned int res_u32x4 __attribute__((ext_vector_type(4)));

struct ResArgs {
    const void *x;
    void *out;
    const float *gamma, *beta;
    float eps;
    float *mean, *var;
    float *part;      // [2][G][L] partial (s1, s2) per work-group
    float *coef;      // [2][L] mean, scale
    unsigned *flags;  // [kResMaxGroups][kFlagStride]
    int64_t pixels;
    int row_len;      // L = 4*C
    int cpr;          // 16-byte chunks per row
    int rpi;          // rows per pass of the work-group: kResThreads / cpr
    int rows_per_wg;  // R
    int chunks;       // chunks per thread: ceil(R / rpi) <= kResChunks
    int groups;       // G
    int cols_per_wg;  // ceil(L / G) <= kResMaxCols
    int tpc;          // phase-2 threads per column: kResThreads / next power of two >= cols_per_wg
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t res_rsrc(const void *base, unsigned bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

// 16 bytes per lane from byte offset voff of [base, base + bytes) straight
// into LDS at m0 + 16 * lane (offsets past the end land as zeros).  The
// issuing wave waits for it with s_waitcnt vmcnt(0) before it reads the LDS.
__device__ __forceinline__ void res_dma16(const void *base, unsigned bytes, unsigned voff, unsigned m0)
{
    const unsigned long long b = (unsigned long long)base;
    const unsigned lo = __builtin_amdgcn_readfirstlane(unsigned(b));
    const unsigned hi = __builtin_amdgcn_readfirstlane(unsigned(b >> 32));
    const __amdgpu_buffer_rsrc_t rsrc =
        res_rsrc((const void *)(((unsigned long long)hi << 32) | lo), __builtin_amdgcn_readfirstlane(bytes));
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voff), "s"(rsrc),
                 "s"(__builtin_amdgcn_readfirstlane(m0))
                 : "memory");
}

__device__ __forceinline__ void res_store(float *p, float v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__device__ __forceinline__ float res_load(const float *p)
{
    return __hip_atomic_load(const_cast<float *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__device__ __forceinline__ unsigned res_flag(const unsigned *p)
{
    return __hip_atomic_load(const_cast<unsigned *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// This work-group raises its flag to `target` and waits until all G flags
// have reached it.  False (in every thread) if the wait gave up.
__device__ __forceinline__ bool res_barrier(unsigned *flags, int groups, unsigned target)
{
    __builtin_amdgcn_s_waitcnt(0);  // this thread's stores have completed
    __syncthreads();
    if (threadIdx.x == 0)
        __hip_atomic_store(flags + blockIdx.x * kFlagStride, target, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    int late = 0;
    for (int b = threadIdx.x; b < groups; b += kResThreads) {
        long i = 0;
        while (int(res_flag(flags + b * kFlagStride) - target) < 0) {
            if (++i >= kSpinLimit) {
                late = 1;
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
    return __syncthreads_or(late) == 0;
}

template <typename T>
__device__ __forceinline__ void res_unpack(const res_u32x4 &v, float (&f)[16 / sizeof(T)])
{
    if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            f[2 * i] = __builtin_bit_cast(float, v[i] << 16);
            f[2 * i + 1] = __builtin_bit_cast(float, v[i] & 0xffff0000u);
        }
    } else {
        // (each element through a scalar first: a bit-cast of a vector
        // element read the vector's first element here)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const unsigned u = v[i];
            f[i] = __builtin_bit_cast(float, u);
        }
    }
}

template <typename T>
__device__ __forceinline__ res_u32x4 res_pack(const float (&f)[16 / sizeof(T)])
{
    Vec<T, 16 / sizeof(T)> o;
#pragma unroll
    for (int e = 0; e < 16 / int(sizeof(T)); ++e)
        o.v[e] = T(f[e]);
    return __builtin_bit_cast(res_u32x4, o);
}

template <typename T, bool RELU>
__global__ __launch_bounds__(kResThreads) void iqbn_resident(ResArgs a)
{
    constexpr int VW = 16 / sizeof(T);
    constexpr int NV = kResRegChunks, NL = kResLdsChunks;
    constexpr int NW = kResThreads / 64;
    __shared__ res_u32x4 held[NL][kResThreads];
    __shared__ float red[2 * VW][kResThreads + 1];  // +1: the pass over it reads eight rows at once
    __shared__ double wsum[2][NW];
    __shared__ unsigned base_flag;

    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int wg = blockIdx.x;
    const int L = a.row_len, G = a.groups;
    const int cc = t % a.cpr, rl = t / a.cpr;
    const bool active = rl < a.rpi;
    const int64_t r0 = int64_t(wg) * a.rows_per_wg;
    const int nrows = r0 < a.pixels ? int(min(int64_t(a.rows_per_wg), a.pixels - r0)) : 0;
    const T *xw = static_cast<const T *>(a.x) + (nrows > 0 ? r0 : 0) * L;
    const unsigned wbytes = unsigned(nrows) * unsigned(L) * unsigned(sizeof(T));
    const unsigned kOut = 0x80000000u;  // an offset past every work-group's rows: loads give zero
    auto chunk_off = [&](int k) {
        const int lr = rl + k * a.rpi;
        return active && lr < nrows ? unsigned(lr * L + cc * VW) * unsigned(sizeof(T)) : kOut;
    };
    auto chunk_valid = [&](int k) { return active && rl + k * a.rpi < nrows; };
    if (t == 0)
        base_flag = res_flag(a.flags + wg * kFlagStride);
    // phase 2's column of this thread, with its shift value and gamma loaded
    // now, off the path between the two barriers
    const int ci = t / a.tpc, j = t % a.tpc;
    const int col = wg * a.cols_per_wg + ci;
    const bool mine = ci < a.cols_per_wg && col < L;
    const float k0 = mine ? float(static_cast<const T *>(a.x)[col]) : 0.0f;
    const float g0 = mine ? a.gamma[col] : 0.0f;
    float beta0[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e)
        beta0[e] = a.beta[cc * VW + e];

    // ---- phase 1: rows into LDS (direct loads) and VGPRs; shifted sums
#pragma unroll
    for (int k = 0; k < NL; ++k)
        if (NV + k < a.chunks)
            res_dma16(xw, wbytes, chunk_off(NV + k),
                      unsigned((size_t)(const __attribute__((address_space(3))) void *)&held[k][wave * 64]));
    const __amdgpu_buffer_rsrc_t src = res_rsrc(xw, wbytes);
    res_u32x4 v[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k)
        v[k] = k < a.chunks ? __builtin_amdgcn_raw_buffer_load_b128(src, chunk_off(k), 0, 0) : res_u32x4{0, 0, 0, 0};
    float shift[VW];
    {
        const res_u32x4 kv = *reinterpret_cast<const res_u32x4 *>(static_cast<const T *>(a.x) + cc * VW);
        res_unpack<T>(kv, shift);
    }
    float s1[VW], s2[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e)
        s1[e] = s2[e] = 0.0f;
    auto accumulate = [&](const res_u32x4 &c) {
        float f[VW];
        res_unpack<T>(c, f);
#pragma unroll
        for (int e = 0; e < VW; ++e) {
            const float d = f[e] - shift[e];
            s1[e] += d;
            s2[e] = fmaf(d, d, s2[e]);
        }
    };
#pragma unroll
    for (int k = 0; k < NV; ++k)
        if (k < a.chunks && chunk_valid(k))
            accumulate(v[k]);
    __builtin_amdgcn_s_waitcnt(0);  // the direct-to-LDS loads have landed
    asm volatile("" ::: "memory");
#pragma unroll
    for (int k = 0; k < NL; ++k)
        if (NV + k < a.chunks && chunk_valid(NV + k))
            accumulate(held[k][t]);
    // one (s1, s2) per column of this work-group: the rpi threads of a
    // column chunk are added in row order, and the partials go out as
    // contiguous rows of L floats
#pragma unroll
    for (int e = 0; e < VW; ++e) {
        red[e][t] = s1[e];
        red[VW + e][t] = s2[e];
    }
    __syncthreads();
    const unsigned target1 = base_flag + 1, target2 = base_flag + 2;
    for (int p = t; p < 2 * L; p += kResThreads) {
        const int which = p / L, col = p % L;  // which: 0 = s1, 1 = s2
        const int pc = col / VW, pe = which * VW + col % VW;
        float sum = 0.0f;
        for (int j = 0; j < a.rpi; ++j)
            sum += red[pe][pc + j * a.cpr];
        res_store(a.part + (size_t(which) * G + wg) * L + col, sum);
    }
    bool ok = res_barrier(a.flags, G, target1);

    // ---- phase 2: this work-group's columns merged over the G partials (fp64)
    {
        // NU = ceil(G / tpc) partials per thread, all loads issued (at
        // in-range addresses) before any is added
        double d1 = 0.0, d2 = 0.0;
        auto gather = [&](auto nu) {
            constexpr int NU = decltype(nu)::value;
            const int cl = mine ? col : 0;
            float p1[NU], p2[NU];
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                const int b = min(j + u * a.tpc, G - 1);
                p1[u] = res_load(a.part + size_t(b) * L + cl);
                p2[u] = res_load(a.part + (size_t(G) + b) * L + cl);
            }
#pragma unroll
            for (int u = 0; u < NU; ++u)
                if (mine && j + u * a.tpc < G) {
                    d1 += double(p1[u]);
                    d2 += double(p2[u]);
                }
        };
        const int nu = (G + a.tpc - 1) / a.tpc;
        if (nu <= 1)
            gather(std::integral_constant<int, 1>{});
        else if (nu <= 2)
            gather(std::integral_constant<int, 2>{});
        else if (nu <= 4)
            gather(std::integral_constant<int, 4>{});
        else if (nu <= 8)
            gather(std::integral_constant<int, 8>{});
        else
            gather(std::integral_constant<int, 16>{});
        // the tpc threads of a column: a butterfly within the wave, then the
        // column's waves in order
        for (int off = (a.tpc < 64 ? a.tpc : 64) >> 1; off > 0; off >>= 1) {
            d1 += __shfl_xor(d1, off);
            d2 += __shfl_xor(d2, off);
        }
        if (lane == 0) {
            wsum[0][wave] = d1;
            wsum[1][wave] = d2;
        }
        __syncthreads();
        if (mine && j == 0) {
            double t1 = d1, t2 = d2;
            if (a.tpc > 64) {
                t1 = t2 = 0.0;
                for (int q = 0; q < a.tpc / 64; ++q) {
                    t1 += wsum[0][wave + q];
                    t2 += wsum[1][wave + q];
                }
            }
            const double n = double(a.pixels);
            const double d = t1 / n;      // mean - K
            double var = t2 / n - d * d;  // biased variance
            if (var < 0.0)
                var = 0.0;
            const double mu = double(k0) + d;
            const double sc = double(g0) / sqrt(var + double(a.eps));
            a.mean[col] = ok ? float(mu) : __builtin_nanf("");
            a.var[col] = ok ? float(var) : __builtin_nanf("");
            res_store(a.coef + col, float(mu));
            res_store(a.coef + L + col, float(sc));
        }
    }
    ok = res_barrier(a.flags, G, target2) && ok;
    if (!ok && mine && j == 0) {
        // a wait gave up: this work-group's statistics are marked too
        a.mean[col] = __builtin_nanf("");
        a.var[col] = __builtin_nanf("");
    }

    // ---- phase 3: normalise the held rows and write them
    if (!active)
        return;
    float mu[VW], sc[VW], be[VW];
    {
        // 16-byte loads with the cache policy of the system-scope loads
        // above (sc0 sc1: from memory, past the L2)
        constexpr int kSysCoherent = 17;
        const __amdgpu_buffer_rsrc_t crs = res_rsrc(a.coef, unsigned(2 * L) * unsigned(sizeof(float)));
#pragma unroll
        for (int h = 0; h < VW / 4; ++h) {
            const res_u32x4 m = __builtin_amdgcn_raw_buffer_load_b128(crs, unsigned(cc * VW + 4 * h) * 4u, 0, kSysCoherent);
            const res_u32x4 q =
                __builtin_amdgcn_raw_buffer_load_b128(crs, unsigned(L + cc * VW + 4 * h) * 4u, 0, kSysCoherent);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const unsigned mi = m[i], qi = q[i];
                mu[4 * h + i] = __builtin_bit_cast(float, mi);
                sc[4 * h + i] = __builtin_bit_cast(float, qi);
            }
        }
#pragma unroll
        for (int e = 0; e < VW; ++e)
            be[e] = beta0[e];
    }
    T *ow = static_cast<T *>(a.out) + (nrows > 0 ? r0 : 0) * L;
    auto emit = [&](int k, const res_u32x4 &c) {
        float f[VW];
        res_unpack<T>(c, f);
#pragma unroll
        for (int e = 0; e < VW; ++e) {
            float y = fmaf(f[e] - mu[e], sc[e], be[e]);
            if (RELU)
                y = fmaxf(y, 0.0f);
            f[e] = ok ? y : __builtin_nanf("");
        }
        const int lr = rl + k * a.rpi;
        __builtin_nontemporal_store(res_pack<T>(f),
                                    reinterpret_cast<res_u32x4 *>(ow + size_t(lr) * L + cc * VW));
    };
#pragma unroll
    for (int k = 0; k < NV; ++k)
        if (k < a.chunks && chunk_valid(k))
            emit(k, v[k]);
#pragma unroll
    for (int k = 0; k < NL; ++k)
        if (NV + k < a.chunks && chunk_valid(NV + k))
            emit(NV + k, held[k][t]);
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

// Geometry of the resident launch for this tensor on the current device, or
// false where it does not apply (chunks that are not 16 bytes, rows longer
// than kResThreads chunks, more rows per work-group than it can hold, more
// than kResMaxCols columns per work-group to merge).
struct ResPlan {
    int groups, cpr, rpi, rows_per_wg, chunks, cols_per_wg, tpc;
};

std::mutex g_res_mutex;
int g_res_groups[64];
bool g_res_known[64];

// Work-groups of the resident launch on the current device: one per compute
// unit, where a compute unit holds exactly one (0: not available).
int resident_groups()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return 0;
    std::lock_guard<std::mutex> lock(g_res_mutex);
    if (!g_res_known[dev]) {
        int cus = 0, per_cu = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            cus = 0;
        // every instantiation holds the same LDS and thread count
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, iqbn_resident<__bf16, false>, kResThreads, 0) !=
            hipSuccess)
            per_cu = 0;
        g_res_groups[dev] = per_cu == 1 && cus > 0 && cus <= kResMaxGroups ? cus : 0;
        g_res_known[dev] = true;
    }
    return g_res_groups[dev];
}

bool resident_plan(int64_t pixels, int c, DType dt, ResPlan *rp)
{
    const int es = dt == DType::BF16 ? 2 : 4;
    const int row_bytes = 4 * c * es;
    if (row_bytes % 16 != 0)
        return false;
    const int cpr = row_bytes / 16;
    if (cpr > kResThreads || pixels * row_bytes < kResMinBytes)
        return false;
    const int groups = resident_groups();
    if (groups <= 0)
        return false;
    const int rpi = kResThreads / cpr;
    const int64_t rows_per_wg = (pixels + groups - 1) / groups;
    const int64_t chunks = (rows_per_wg + rpi - 1) / rpi;
    const int cols_per_wg = (4 * c + groups - 1) / groups;
    if (chunks > kResChunks || cols_per_wg > kResMaxCols)
        return false;
    int pow2 = 1;
    while (pow2 < cols_per_wg)
        pow2 *= 2;
    rp->groups = groups;
    rp->cpr = cpr;
    rp->rpi = rpi;
    rp->rows_per_wg = int(rows_per_wg);
    rp->chunks = int(chunks);
    rp->cols_per_wg = cols_per_wg;
    rp->tpc = kResThreads / pow2;
    return true;
}

size_t resident_bytes(const ResPlan &rp, int c)
{
    return (size_t(2) * rp.groups + 2) * 4 * size_t(c) * sizeof(float);
}

template <typename T>
hipError_t launch_resident(const ResPlan &rp, const void *x, const float *gamma, const float *beta, float eps,
                           bool relu, void *out, float *mean, float *var, int64_t pixels, int c, void *work,
                           unsigned *flags, hipStream_t stream)
{
    ResArgs a;
    a.x = x;
    a.out = out;
    a.gamma = gamma;
    a.beta = beta;
    a.eps = eps;
    a.mean = mean;
    a.var = var;
    a.part = static_cast<float *>(work);
    a.coef = a.part + size_t(2) * 4 * c * rp.groups;
    a.flags = flags;
    a.pixels = pixels;
    a.row_len = 4 * c;
    a.cpr = rp.cpr;
    a.rpi = rp.rpi;
    a.rows_per_wg = rp.rows_per_wg;
    a.chunks = rp.chunks;
    a.groups = rp.groups;
    a.cols_per_wg = rp.cols_per_wg;
    a.tpc = rp.tpc;
    if (relu)
        hipLaunchKernelGGL((iqbn_resident<T, true>), dim3(rp.groups), dim3(kResThreads), 0, stream, a);
    else
        hipLaunchKernelGGL((iqbn_resident<T, false>), dim3(rp.groups), dim3(kResThreads), 0, stream, a);
    return hipGetLastError();
}

template <typename T, int VW>
hipError_t launch_all(const void *x, const float *gamma, const float *beta, float eps, bool relu,
                      void *out, float *mean, float *var, int64_t pixels, int c, void *work,
                      hipStream_t stream)
{
    const T *xt = static_cast<const T *>(x);
    float *part = static_cast<float *>(work);
    if (merge_takes(pixels, c, VW, int(sizeof(T)))) {
        // two launches: statistics, then the merged finalize + normalization
        const Layout l = make_layout_narrow(pixels, c, VW, merge_blocks_x(pixels, c, VW));
        const dim3 grid(l.blocks, l.col_groups);
        hipLaunchKernelGGL((iqbn_stats<T, VW>), grid, dim3(kThreads), 0, stream, xt, l, part,
                           part + size_t(l.blocks) * 2 * l.row_len);
        const MergeArgs a = {part, l.blocks, gamma, beta, eps, mean, var};
        if (relu)
            hipLaunchKernelGGL((iqbn_merge_affine<T, VW, true>), grid, dim3(kThreads), 0, stream, xt,
                               static_cast<T *>(out), l, a);
        else
            hipLaunchKernelGGL((iqbn_merge_affine<T, VW, false>), grid, dim3(kThreads), 0, stream, xt,
                               static_cast<T *>(out), l, a);
        return hipGetLastError();
    }
    const Layout l = make_layout(pixels, c, VW);
    float *affine = part + size_t(l.blocks) * 2 * l.row_len;
    const dim3 grid(l.blocks, l.col_groups);
    hipLaunchKernelGGL((iqbn_stats<T, VW>), grid, dim3(kThreads), 0, stream, xt, l, part, nullptr);
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

bool iqbn_merged(int64_t pixels, int c, DType dt)
{
    return merge_takes(pixels, c, vec_width(c, dt), dt == DType::BF16 ? 2 : 4);
}

bool iqbn_one_launch(int64_t pixels, int c, DType dt)
{
    ResPlan rp;
    return !merge_takes(pixels, c, vec_width(c, dt), dt == DType::BF16 ? 2 : 4) && resident_plan(pixels, c, dt, &rp);
}

size_t iqbn_barrier_bytes()
{
    return size_t(kResMaxGroups) * kFlagStride * sizeof(unsigned);
}

size_t iqbn_workspace_bytes(int64_t pixels, int c)
{
    // Largest over the vector widths the dispatcher may pick, and the
    // resident launch where it applies.
    size_t best = 0;
    ResPlan rp;
    for (DType dt : {DType::BF16, DType::F32})
        if (resident_plan(pixels, c, dt, &rp) && resident_bytes(rp, c) > best)
            best = resident_bytes(rp, c);
    for (int vw : {1, 4, 8}) {
        if ((4 * c) % vw)
            continue;
        const Layout l = make_layout(pixels, c, vw);
        const size_t b = (size_t(l.blocks) * 2 + 3) * size_t(l.row_len) * sizeof(float);
        if (b > best)
            best = b;
        // the merged path: partials and the shifts K
        const Layout ln = make_layout_narrow(pixels, c, vw, merge_blocks_x(pixels, c, vw));
        const size_t bn = (size_t(ln.blocks) * 2 + 1) * size_t(ln.row_len) * sizeof(float);
        if (bn > best)
            best = bn;
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
                    unsigned *flags, hipStream_t stream)
{
    ResPlan rp;
    const int vw = vec_width(c, dt);
    const bool merged = merge_takes(pixels, c, vw, dt == DType::BF16 ? 2 : 4);
    if (!merged && flags != nullptr && resident_plan(pixels, c, dt, &rp))
        return dt == DType::BF16 ? launch_resident<__bf16>(rp, x, gamma, beta, eps, relu, out, mean, var, pixels,
                                                           c, work, flags, stream)
                                 : launch_resident<float>(rp, x, gamma, beta, eps, relu, out, mean, var, pixels, c,
                                                          work, flags, stream);
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
