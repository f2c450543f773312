// The stem layer of a quaternion network on gfx950: the Poincare mapping of
// RGB pixels to quaternions (Section III-A, eq. 4) feeding the first
// quaternion convolution (Section III-B, eqs. 5/6), whose one input channel
// makes it a short contraction: K = 4 components x k_h*k_w taps (36 for a
// 3x3 stem) against a few dozen output reals per pixel.  The implicit-GEMM
// kernel would stage 16 input channels per step with 15 of them zero; this
// kernel builds each MFMA's K = 16 slice (two taps x four components) of
// one output pixel per lane straight from the colour planes, with the map
// of eq. 4 evaluated in fp32 (one division per tap) and rounded once to
// bf16.  The layer is bound
// by writing its output (4 * c_out reals per pixel against 3 inputs).
//
// Per wave: 32 consecutive output pixels at a time, D = W^T X^T with
//   A (32 output reals x 16 k): the signed Hamilton block weight of eq. 6,
//       row r = p * c_out + c (component p, channel c), k = 4 * tap + q,
//       entry sign(p, q) * W_{p xor q}[c][tap]; built once per work-group in
//       LDS as NBLK blocks of 32 rows x KM slices of 16 k (one 1 KB MFMA
//       fragment each);
//   B (16 k x 32 pixels): lane l holds pixel l % 32, k = 16m + 8(l/32) + e,
//       i.e. taps 4m + 2(l/32) and 4m + 2(l/32) + 1, all four components;
//   D: lane l holds rows 8j + 4(l/32) + i (i, j < 4) of its pixel, so each
//       group of four rows goes out as one 8-byte store of bf16.
#include <hip/hip_runtime.h>

#include "quan_launch.h"

namespace quan {
namespace {

typedef __bf16 stem_bf16x8 __attribute__((ext_vector_type(8)));
typedef float stem_f32x16 __attribute__((ext_vector_type(16)));

constexpr int kStemThreads = 256;
constexpr int kStemMaxFrags = 32;  // NBLK x KM weight fragments held in LDS (1 KB each)

struct StemArgs {
    const __bf16 *rgb;   // [n][3][h][w]
    const __bf16 *wpack; // packed weights: W_m[o][tap] at ((tap * 4 + m) * cout_pad + o) * pk
    const __bf16 *bias;  // [4][c_out] or NULL
    __bf16 *out;         // [n][h_out][w_out][4][c_out]
    int n, h, w, c_out, k_h, k_w, s_h, s_w, p_h, p_w, d_h, d_w, h_out, w_out;
    int cout_pad, pk;
    int km;              // K slices of 16: ceil(taps / 4)
    int64_t m;           // output pixels
    int64_t groups;      // ceil(m / 32)
};

template <int NBLK>
__global__ __launch_bounds__(kStemThreads) void qconv2d_stem(StemArgs a)
{
    // A fragments of the signed block weight, fragment (b, m) for lane l:
    // rows 32b + l%32, k = 16m + 8(l/32) .. +7; and the bias of every row
    __shared__ stem_bf16x8 wtab[kStemMaxFrags][64];
    __shared__ float btab[32 * NBLK];
    const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
    const int taps = a.k_h * a.k_w;
    const int rows = 4 * a.c_out;
    for (int idx = threadIdx.x; idx < NBLK * a.km * 64; idx += kStemThreads) {
        const int fl = idx & 63, fm = (idx >> 6) % a.km, fb = (idx >> 6) / a.km;
        const int r = 32 * fb + (fl & 31);
        const int p = r < rows ? r / a.c_out : 0, c = r < rows ? r - p * a.c_out : 0;
        stem_bf16x8 f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int k = 16 * fm + 8 * (fl >> 5) + e, tap = k >> 2, q = k & 3;
            float v = 0.0f;
            if (r < rows && tap < taps) {
                v = float(a.wpack[(size_t(tap * 4 + (p ^ q)) * a.cout_pad + c) * a.pk]);
                if ((kHamiltonNeg >> (4 * p + q)) & 1u)
                    v = -v;
            }
            f[e] = __bf16(v);
        }
        wtab[fb * a.km + fm][fl] = f;
    }
    for (int r = threadIdx.x; r < 32 * NBLK; r += kStemThreads)
        btab[r] = (a.bias != nullptr && r < rows) ? float(a.bias[r]) : 0.0f;
    __syncthreads();

    const int hw = a.h * a.w, hw_out = a.h_out * a.w_out;
    const int64_t waves = int64_t(gridDim.x) * (kStemThreads / 64);
    const int64_t wid = int64_t(blockIdx.x) * (kStemThreads / 64) + (threadIdx.x >> 6);
    for (int64_t grp = wid; grp < a.groups; grp += waves) {
        const int64_t pix = grp * 32 + l32;
        const bool live = pix < a.m;
        int img = 0, oy = 0, ox = 0;
        if (live) {
            img = int(pix / hw_out);
            const int rr = int(pix - int64_t(img) * hw_out);
            oy = rr / a.w_out;
            ox = rr - oy * a.w_out;
        }
        const __bf16 *plane = a.rgb + size_t(img) * 3 * hw;
        // accumulators start at the bias of the lane's rows 32b + 8j + 4*half + i
        stem_f32x16 acc[NBLK];
#pragma unroll
        for (int b = 0; b < NBLK; ++b)
#pragma unroll
            for (int i = 0; i < 16; ++i)
                acc[b][i] = btab[32 * b + 8 * (i >> 2) + 4 * half + (i & 3)];
        for (int m = 0; m < a.km; ++m) {
            // the pixel's quaternions (eq. 4) at taps 4m + 2*half and 4m + 2*half + 1
            stem_bf16x8 xq;
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int tap = 4 * m + 2 * half + u;
                float q0 = 0.0f, q1 = 0.0f, q2 = 0.0f, q3 = 0.0f;
                if (live && tap < taps) {
                    const int ky = tap / a.k_w, kx = tap - ky * a.k_w;
                    const int iy = oy * a.s_h - a.p_h + ky * a.d_h, ix = ox * a.s_w - a.p_w + kx * a.d_w;
                    if ((unsigned)iy < (unsigned)a.h && (unsigned)ix < (unsigned)a.w) {
                        const __bf16 *px = plane + iy * a.w + ix;
                        const float r = float(px[0]), g = float(px[hw]), bl = float(px[2 * hw]);
                        const float n2 = r * r + g * g + bl * bl;
                        const float inv = 1.0f / (1.0f + n2);
                        q0 = (1.0f - n2) * inv;
                        q1 = (2.0f * r) * inv;
                        q2 = (2.0f * g) * inv;
                        q3 = (2.0f * bl) * inv;
                    }
                }
                xq[4 * u + 0] = __bf16(q0);
                xq[4 * u + 1] = __bf16(q1);
                xq[4 * u + 2] = __bf16(q2);
                xq[4 * u + 3] = __bf16(q3);
            }
#pragma unroll
            for (int b = 0; b < NBLK; ++b)
                acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wtab[b * a.km + m][lane], xq, acc[b], 0, 0, 0);
        }
        if (!live)
            continue;
        __bf16 *orow = a.out + pix * rows;
#pragma unroll
        for (int b = 0; b < NBLK; ++b)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r0 = 32 * b + 8 * j + 4 * half;
                if (r0 < rows) {
                    __bf16 v[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        v[i] = __bf16(acc[b][4 * j + i]);
                    unsigned long long bits;
                    __builtin_memcpy(&bits, v, 8);
                    *reinterpret_cast<unsigned long long *>(orow + r0) = bits;
                }
            }
    }
}

template <int NBLK>
hipError_t launch_stem(const StemArgs &a, hipStream_t stream)
{
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const int64_t wgs_needed = (a.groups + kStemThreads / 64 - 1) / (kStemThreads / 64);
    const int64_t cap = int64_t(cus) * 8;
    const int wgs = int(wgs_needed < cap ? wgs_needed : cap);
    hipLaunchKernelGGL((qconv2d_stem<NBLK>), dim3(wgs), dim3(kStemThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t qconv2d_stem_run(const PackGeom &pg, const ConvGeom &g, DType dt, const void *rgb, const void *wpack,
                            const void *bias, void *out, hipStream_t stream)
{
    const int taps = g.k_h * g.k_w;
    const int km = (taps + 3) / 4;
    const int nblk = (4 * g.c_out + 31) / 32;
    // the kernel's block count (a power of two) sizes its weight table
    const int nblk_t = nblk <= 1 ? 1 : nblk <= 2 ? 2 : nblk <= 4 ? 4 : 8;
    if (dt != DType::BF16 || g.c_in != 1 || nblk > 8 || nblk_t * km > kStemMaxFrags)
        return hipErrorNotSupported;
    StemArgs a;
    a.rgb = static_cast<const __bf16 *>(rgb);
    a.wpack = static_cast<const __bf16 *>(wpack);
    a.bias = static_cast<const __bf16 *>(bias);
    a.out = static_cast<__bf16 *>(out);
    a.n = g.n;
    a.h = g.h;
    a.w = g.w;
    a.c_out = g.c_out;
    a.k_h = g.k_h;
    a.k_w = g.k_w;
    a.s_h = g.s_h;
    a.s_w = g.s_w;
    a.p_h = g.p_h;
    a.p_w = g.p_w;
    a.d_h = g.d_h;
    a.d_w = g.d_w;
    a.h_out = g.h_out;
    a.w_out = g.w_out;
    a.cout_pad = pg.cout_pad;
    a.pk = pg.pk;
    a.km = km;
    a.m = g.m();
    a.groups = (a.m + 31) / 32;
    if (nblk == 1)
        return launch_stem<1>(a, stream);
    if (nblk == 2)
        return launch_stem<2>(a, stream);
    if (nblk <= 4)
        return launch_stem<4>(a, stream);
    return launch_stem<8>(a, stream);
}

}  // namespace quan
