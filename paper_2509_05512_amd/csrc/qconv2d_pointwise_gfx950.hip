// Pointwise (1x1) quaternion convolution (Hamilton product, Section III-B,
// eqs. 5 and 6) as a streaming kernel for gfx950.
//
// With a 1x1 kernel the layer is a GEMM whose reduction is one pixel's 4*c_in
// reals: Y[m, (p, o)] = sum_{q, c} x[m][q][c] * sign(p, q) W_{p xor q}[o, c].
// At 64 -> 64 channels it does 128 FLOPs per byte of activation read and
// output written, under the 312 FLOPs per byte at which the MFMA peak meets
// the HBM bandwidth, so the layer runs at the pace of HBM and the kernel is
// built to stream.  A work-group is eight waves in three roles:
//   - four compute waves: wave p owns output component p and keeps the
//     signed fragments of its 4x4 block row (kernel p xor q with the eq. 6
//     sign, for every input component q) in registers for the whole launch,
//     so weights never move after the start.  The MFMA runs transposed,
//     D = W_p^T x^T: the 32 pixels of a stage are D's columns and output
//     channels its rows, so a wave reads each activation fragment once for
//     all of its channels; D's rows are a permutation of the channels chosen
//     so that every lane ends up holding 16 or 32 consecutive channels of
//     one pixel.  The epilogue adds the bias (or applies the folded
//     inference IQBN), rounds to bf16 and parks the stage in LDS;
//   - two producer waves move 32-pixel stages of activations from HBM into
//     a ring in LDS with buffer_load ... lds (1 KB per instruction, two to
//     eight whole pixel rows), six stages ahead of the compute waves (seven
//     slots of 16 KB at 64 input channels, fourteen of 8 KB at 32);
//   - two store waves write each parked stage to memory in 16-byte pieces
//     (whole 128-byte lines at 64 output channels) while the compute waves
//     run the next one, and reduce it for the IQBN statistics when asked:
//     per column the stage's exact mean, then the squared deviations from
//     it, merged into a running (mean, M2) by Chan et al.'s pairwise update;
//     a work-group writes one partial per column for its run of pixels.
// One barrier per stage orders the three.  Every work-group takes the same
// number of consecutive stages (the last one fewer), so the statistics
// partials are runs of equal length.
#include <hip/hip_runtime.h>

#include "gfx950_dma.h"
#include "quan_launch.h"

namespace quan {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kPwEpiBias = 0, kPwEpiStats = 1, kPwEpiFold = 2;
constexpr int kPwComputeWaves = 4, kPwProducerWaves = 2, kPwStoreWaves = 2;
constexpr int kPwThreads = 64 * (kPwComputeWaves + kPwProducerWaves + kPwStoreWaves);
constexpr int kPwStagePixels = 32;
constexpr int kPwRingBytes = 114688;  // 7 stages of 64 input channels, 14 of 32
// Output stores carry device scope (sc1): each line goes on to memory as it
// is written instead of waiting in the L2 for the kernel's closing release.
constexpr int kPwStorePolicy = 16;

struct PwArgs {
    const void *x;      // [n][h][w][4][c_in] bf16
    const void *wpack;  // packed kernels (PackGeom layout of a 1x1 layer)
    const void *bias;   // [4][c_out] bf16 or NULL
    void *out;          // [n][h_out][w_out][4][c_out] bf16
    int m;              // output pixels
    int h, w, h_out, w_out, s_h, s_w;
    int cout_pad;
    int stages;         // ceil(m / 32)
    int group_stages;   // stages per work-group
    unsigned x_bytes;
    float *stats;       // [2][4 c_out][stat_tiles] (EPI statistics)
    int stat_tiles;
    const float *scale;  // [4 c_out] (EPI fold)
    const float *shift;
    int relu;
};

// XOR swizzle of the 16-byte chunk index in an LDS row of CPR chunks, as a
// function of the row: a ds_read_b128 or ds_write_b128 whose 16-lane groups
// address one chunk of 16 consecutive rows then touches 16 distinct 16-byte
// bank slots (the full 256-byte bank width).
template <int CPR>
__device__ __forceinline__ int pw_swz(int row)
{
    static_assert(CPR == 4 || CPR == 8 || CPR == 16 || CPR == 32, "rows of 4 to 32 chunks");
    if constexpr (CPR >= 16)
        return row & 15;
    else
        return (row / (16 / CPR)) % CPR;
}

// Wait until at most c stages of NI loads each are still in flight (c
// wave-uniform, 0 <= c <= C).
template <int NI, int C>
__device__ __forceinline__ void wait_loads(int c)
{
    if constexpr (C == 0) {
        wait_vmcnt<0>();
    } else {
        if (c >= C)
            wait_vmcnt<C * NI>();
        else
            wait_loads<NI, C - 1>(c);
    }
}

__device__ __forceinline__ unsigned pack_bf16(float lo, float hi)
{
    const bf16x2 v = {__bf16(lo), __bf16(hi)};
    return __builtin_bit_cast(unsigned, v);
}

template <int CIN, int COUT, int EPI>
__global__ __launch_bounds__(kPwThreads) void qconv2d_pointwise(PwArgs a)
{
    constexpr int KS = CIN / 4;           // k-steps of 16 reals
    constexpr int NBW = COUT / 32;        // 32-row D blocks per compute wave
    constexpr int RB = 8 * CIN;           // bytes of one activation row (4 components x CIN bf16)
    constexpr int CPR = RB / 16;          // 16-byte chunks per activation row
    constexpr int STAGE = kPwStagePixels * RB;
    constexpr int NI = STAGE / 1024 / kPwProducerWaves;  // DMA instructions per producer and stage
    constexpr int RING = kPwRingBytes / STAGE;
    constexpr int LA = RING - 1;          // stages in flight ahead of the compute waves
    constexpr int PRB = 2 * COUT;         // bytes of one parked output row (one component)
    constexpr int PCPR = PRB / 16;
    constexpr int PARK = kPwStagePixels * PRB;  // one component's parked stage
    constexpr int DRAIN = PARK / 1024;    // 16-byte pieces per lane and component
    constexpr int CPS = 4 / kPwStoreWaves;  // components per store wave
    static_assert(CIN == 32 || CIN == 64, "32 or 64 input channels");
    static_assert(COUT == 32 || COUT == 64, "32 or 64 output channels");
    static_assert(NI >= 1 && LA * NI <= 63, "one producer's loads in flight fit vmcnt");
    static_assert(NI * kPwProducerWaves * 1024 == STAGE, "a stage splits into whole DMA instructions");
    static_assert(RING * STAGE == kPwRingBytes, "whole stages in the ring");

    __shared__ __attribute__((aligned(16))) unsigned char ring[RING * STAGE];
    __shared__ __attribute__((aligned(16))) unsigned char park[2][4 * PARK];  // [stage parity][component]
    __shared__ __attribute__((aligned(16))) float cmap[2 * 4 * COUT];  // bias, or (scale, shift)

    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    const int st0 = blockIdx.x * a.group_stages;
    const int n = a.stages - st0 < a.group_stages ? a.stages - st0 : a.group_stages;
    constexpr int kFirstProducer = kPwComputeWaves, kFirstStore = kPwComputeWaves + kPwProducerWaves;

    // Every wave passes n + 1 barriers: B_i (i < n) publishes stage i in
    // the ring and, for i > 0, stage i - 1's parked output; B_n the last
    // parked stage.
    if (wave >= kFirstProducer && wave < kFirstStore) {
        // Producer: this wave's NI instructions of a stage cover LDS bytes
        // [1024 j, 1024 j + 1024) of the slot, j = pw * NI + ii; lane l's
        // 16 bytes there are physical chunk pc of pixel row pp, which holds
        // logical chunk pc ^ swz(pp) of that pixel.
        const int pw = wave - kFirstProducer;
        int pp[NI], coff[NI];
#pragma unroll
        for (int ii = 0; ii < NI; ++ii) {
            const int byte = 1024 * (pw * NI + ii) + 16 * lane;
            pp[ii] = byte / RB;
            coff[ii] = 16 * (((byte % RB) / 16) ^ pw_swz<CPR>(pp[ii]));
        }
        const bool dense = a.s_h == 1 && a.s_w == 1 && a.h_out == a.h && a.w_out == a.w;
        const int hw_out = a.h_out * a.w_out;
        auto issue = [&](int i) {
            const int m0 = (st0 + i) * kPwStagePixels;
            const unsigned slot = lds_addr(ring + (i % RING) * STAGE);
#pragma unroll
            for (int ii = 0; ii < NI; ++ii) {
                const int m = m0 + pp[ii];
                unsigned off = 0x7ffffff0u;  // past the end: lands as zeros
                if (m < a.m) {
                    unsigned row;
                    if (dense) {
                        row = unsigned(m);
                    } else {
                        const int img = m / hw_out, rem = m - img * hw_out;
                        const int oh = rem / a.w_out, ow = rem - oh * a.w_out;
                        row = unsigned((img * a.h + oh * a.s_h) * a.w + ow * a.s_w);
                    }
                    off = row * unsigned(RB) + unsigned(coff[ii]);
                }
                dma16(a.x, a.x_bytes, off, 0u, slot + 1024u * unsigned(pw * NI + ii));
            }
        };
        const int pre = n < LA ? n : LA;
        for (int i = 0; i < pre; ++i)
            issue(i);
        wait_loads<NI, LA - 1>(pre - 1);  // stage 0 has landed
        for (int i = 0; i < n; ++i) {
            __syncthreads();  // B_i: stage i visible; slot (i - 1) % RING read
            if (i + LA < n)
                issue(i + LA);
            if (i + 1 < n) {
                const int last = i + LA < n - 1 ? i + LA : n - 1;
                wait_loads<NI, LA - 1>(last - (i + 1));  // stage i + 1 has landed
            }
        }
        __syncthreads();  // B_n
        return;
    }

    if (wave >= kFirstStore) {
        // Store wave: after B_i, the parked stage i - 1 of components
        // CPS * sw .. + CPS - 1 goes to memory in 16-byte pieces (piece it
        // of a component's region holds its bytes [1024 it, 1024 it +
        // 1024): lane l's 16 bytes are chunk cc of row jj), and its IQBN
        // statistics are merged into the running partials.
        const int sw = wave - kFirstStore;
        unsigned char *const outb = static_cast<unsigned char *>(a.out);
        constexpr size_t OUT_ROW = size_t(8) * COUT;  // bytes of one output pixel
        // statistics: lane l covers column pair cp = l % 32 (channels 2 cp,
        // 2 cp + 1) of the wave's component CPS * sw + l / 32 over all 32
        // pixels of a stage (with 32 output channels, lanes cp >= 16 idle)
        static_assert(CPS == 2, "two components per store wave: one per half-wave");
        const int cp = lane % 32, sc = lane / 32;
        const bool st_lane = cp < COUT / 2;
        float run_mean[2] = {0.0f, 0.0f}, run_m2[2] = {0.0f, 0.0f};
        float run_n = 0.0f;
        for (int i = 0; i <= n; ++i) {
            __syncthreads();  // B_i
            if (i == 0)
                continue;
            const int j = i - 1;
            const int m0 = (st0 + j) * kPwStagePixels;
            const unsigned char *const region = park[j % 2];
            u32x4 v[CPS][DRAIN];
#pragma unroll
            for (int c = 0; c < CPS; ++c) {
#pragma unroll
                for (int it = 0; it < DRAIN; ++it) {
                    const int byte = 1024 * it + 16 * lane;
                    const int jj = byte / PRB, cc = (byte % PRB) / 16;
                    v[c][it] = *reinterpret_cast<const u32x4 *>(region + (CPS * sw + c) * PARK + jj * PRB +
                                                                16 * (cc ^ pw_swz<PCPR>(jj)));
                }
            }
            // buffer stores over the stage's valid rows: rows past M fall
            // outside the range and are dropped
            const int rows = a.m - m0 < kPwStagePixels ? a.m - m0 : kPwStagePixels;
            const __amdgpu_buffer_rsrc_t dst =
                make_rsrc(outb + size_t(m0) * OUT_ROW, unsigned(rows) * unsigned(OUT_ROW));
#pragma unroll
            for (int c = 0; c < CPS; ++c) {
#pragma unroll
                for (int it = 0; it < DRAIN; ++it) {
                    const int byte = 1024 * it + 16 * lane;
                    const int jj = byte / PRB, cc = (byte % PRB) / 16;
                    __builtin_amdgcn_raw_buffer_store_b128(v[c][it], dst,
                                                           unsigned(jj * OUT_ROW + (CPS * sw + c) * PRB + 16 * cc),
                                                           0, kPwStorePolicy);
                }
            }
            if constexpr (EPI == kPwEpiStats) {
                // Exact mean of the stage's valid rows, then the squared
                // deviations from it (nothing cancels), then Chan et al.'s
                // pairwise merge into the running partial.  Rows past M
                // (the last stage only) are left out by selects.
                const unsigned char *const reg = region + (CPS * sw + sc) * PARK + 4 * (cp % 4);
                const int nv = a.m - m0 < kPwStagePixels ? a.m - m0 : kPwStagePixels;
                // y*[r] holds row r ^ sc: the two half-waves read rows of
                // opposite parity at once, on disjoint banks
                float y0[kPwStagePixels], y1[kPwStagePixels];
#pragma unroll
                for (int r = 0; r < kPwStagePixels; ++r) {
                    const int row = r ^ sc;
                    const unsigned u = st_lane ? *reinterpret_cast<const unsigned *>(
                                                     reg + row * PRB + 16 * ((cp / 4) ^ pw_swz<PCPR>(row)))
                                               : 0u;
                    y0[r] = __builtin_bit_cast(float, u << 16);
                    y1[r] = __builtin_bit_cast(float, u & 0xffff0000u);
                }
                float s0 = 0.0f, s1 = 0.0f, t0 = 0.0f, t1 = 0.0f;
                float mean0, mean1, q0 = 0.0f, q1 = 0.0f, qa = 0.0f, qb = 0.0f;
                if (nv == kPwStagePixels) {
#pragma unroll
                    for (int r = 0; r < kPwStagePixels; r += 2) {
                        s0 += y0[r];
                        t0 += y0[r + 1];
                        s1 += y1[r];
                        t1 += y1[r + 1];
                    }
                    mean0 = (s0 + t0) * (1.0f / kPwStagePixels);
                    mean1 = (s1 + t1) * (1.0f / kPwStagePixels);
#pragma unroll
                    for (int r = 0; r < kPwStagePixels; r += 2) {
                        const float e0 = y0[r] - mean0, f0 = y0[r + 1] - mean0;
                        const float e1 = y1[r] - mean1, f1 = y1[r + 1] - mean1;
                        q0 = fmaf(e0, e0, q0);
                        qa = fmaf(f0, f0, qa);
                        q1 = fmaf(e1, e1, q1);
                        qb = fmaf(f1, f1, qb);
                    }
                } else {
#pragma unroll
                    for (int r = 0; r < kPwStagePixels; ++r) {
                        s0 += (r ^ sc) < nv ? y0[r] : 0.0f;
                        s1 += (r ^ sc) < nv ? y1[r] : 0.0f;
                    }
                    mean0 = s0 / float(nv);
                    mean1 = s1 / float(nv);
#pragma unroll
                    for (int r = 0; r < kPwStagePixels; ++r) {
                        const float e0 = (r ^ sc) < nv ? y0[r] - mean0 : 0.0f;
                        const float e1 = (r ^ sc) < nv ? y1[r] - mean1 : 0.0f;
                        q0 = fmaf(e0, e0, q0);
                        q1 = fmaf(e1, e1, q1);
                    }
                }
                q0 += qa;
                q1 += qb;
                const float nb = float(nv), tot = run_n + nb;
                const float f = nb / tot, g = run_n * f;
                const float d0 = mean0 - run_mean[0], d1 = mean1 - run_mean[1];
                run_mean[0] = fmaf(d0, f, run_mean[0]);
                run_mean[1] = fmaf(d1, f, run_mean[1]);
                run_m2[0] = run_m2[0] + q0 + d0 * d0 * g;
                run_m2[1] = run_m2[1] + q1 + d1 * d1 * g;
                run_n = tot;
            }
        }
        if constexpr (EPI == kPwEpiStats) {
            if (st_lane) {
                const size_t cols = size_t(4) * COUT;
                const size_t t = blockIdx.x;
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const size_t col = size_t(CPS * sw + sc) * COUT + 2 * cp + e;
                    a.stats[col * a.stat_tiles + t] = run_mean[e];
                    a.stats[(cols + col) * a.stat_tiles + t] = run_m2[e];
                }
            }
        }
        return;
    }

    // Compute wave `wave` = output component p.
    const int p = wave;
    const int r = lane % 32, kh = lane / 32;
    // The epilogue's per-column map, [4][COUT] floats (a second [4][COUT]
    // for the shift of the folded map).
    {
        const int col = threadIdx.x;  // 0..255 covers 4 * COUT
        if (col < 4 * COUT) {
            if constexpr (EPI == kPwEpiFold) {
                cmap[col] = a.scale[col];
                cmap[4 * COUT + col] = a.shift[col];
            } else {
                cmap[col] = a.bias != nullptr ? float(static_cast<const __bf16 *>(a.bias)[col]) : 0.0f;
            }
        }
    }
    // Signed weight fragments of component p's block row, resident for the
    // launch.  Fragment (b, s) is the MFMA A operand for D rows 32b..32b+31
    // and k-step s: lane l holds row l % 32 and the 8 reals k = 16 s + 8 kh
    // .. + 7, i.e. input component q = k / CIN, channels c = k % CIN .. + 7.
    // D row (b, r) is output channel oc(b, r) = 16 NBW ((r / 4) % 2) + 16 b +
    // 4 (r / 8) + r % 4: then the 16 accumulator values of lane l in block b
    // are channels 16 NBW (l / 32) + 16 b + 0..15, consecutive.
    u32x4 wf[NBW][KS];
    {
        const __bf16 *wp = static_cast<const __bf16 *>(a.wpack);
#pragma unroll
        for (int b = 0; b < NBW; ++b) {
            const int oc = 16 * NBW * ((r >> 2) & 1) + 16 * b + 4 * (r >> 3) + (r & 3);
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                const int k = 16 * s + 8 * kh;
                const int q = k / CIN, c = k % CIN;
                const int km = p ^ q;
                const __bf16 *src = wp + ((size_t(c / 16) * 4 + km) * a.cout_pad + oc) * 16 + (c % 16);
                u32x4 v = *reinterpret_cast<const u32x4 *>(src);
                if ((kHamiltonNeg >> (4 * p + q)) & 1u)
                    v ^= 0x80008000u;
                wf[b][s] = v;
            }
        }
    }
    const unsigned char *arow_base = ring + r * RB;
    const int az = pw_swz<CPR>(r);
    const int pz = pw_swz<PCPR>(r);
    for (int i = 0; i < n; ++i) {
        __syncthreads();  // B_i: stage i has landed (and, at i = 0, cmap is written)
        const unsigned char *arow = arow_base + (i % RING) * STAGE;
        f32x16 acc[NBW];
#pragma unroll
        for (int b = 0; b < NBW; ++b)
            acc[b] = f32x16{};
        // B operand (activations): lane l holds pixel l % 32, reals k = 16 s
        // + 8 kh .. + 7 = logical chunk 2 s + kh of the pixel's row.
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            const u32x4 av = *reinterpret_cast<const u32x4 *>(arow + 16 * ((2 * s + kh) ^ az));
#pragma unroll
            for (int b = 0; b < NBW; ++b)
                acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, wf[b][s]),
                                                                 __builtin_bit_cast(bf16x8, av), acc[b], 0, 0, 0);
        }
        // Epilogue: lane l holds pixel r of the stage, channels ch0 + 0..15
        // of block b; map, round and park them as row r of component p's
        // region for the store waves.
        unsigned char *const mypark = park[i % 2] + p * PARK;
#pragma unroll
        for (int b = 0; b < NBW; ++b) {
            const int ch0 = 16 * NBW * kh + 16 * b;
            const float *mul = cmap + p * COUT + ch0;
            const float *add = EPI == kPwEpiFold ? cmap + 4 * COUT + p * COUT + ch0 : mul;
            float v[16];
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const float x = acc[b][e];
                if constexpr (EPI == kPwEpiFold) {
                    const float y = fmaf(mul[e], x, add[e]);
                    v[e] = a.relu ? fmaxf(y, 0.0f) : y;
                } else {
                    v[e] = x + add[e];
                }
            }
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                u32x4 pk;
                pk[0] = pack_bf16(v[8 * t + 0], v[8 * t + 1]);
                pk[1] = pack_bf16(v[8 * t + 2], v[8 * t + 3]);
                pk[2] = pack_bf16(v[8 * t + 4], v[8 * t + 5]);
                pk[3] = pack_bf16(v[8 * t + 6], v[8 * t + 7]);
                const int chunk = ch0 / 8 + t;
                *reinterpret_cast<u32x4 *>(mypark + r * PRB + 16 * (chunk ^ pz)) = pk;
            }
        }
    }
    __syncthreads();  // B_n: the last parked stage
}

template <int CIN, int COUT>
const void *pw_kernel(int epi)
{
    switch (epi) {
    case kPwEpiStats:
        return (const void *)&qconv2d_pointwise<CIN, COUT, kPwEpiStats>;
    case kPwEpiFold:
        return (const void *)&qconv2d_pointwise<CIN, COUT, kPwEpiFold>;
    default:
        return (const void *)&qconv2d_pointwise<CIN, COUT, kPwEpiBias>;
    }
}

}  // namespace

bool qconv2d_pointwise_takes(const ConvGeom &g, DType dt)
{
    if (dt != DType::BF16 || g.k_h != 1 || g.k_w != 1 || g.p_h != 0 || g.p_w != 0)
        return false;
    if ((g.c_in != 32 && g.c_in != 64) || (g.c_out != 32 && g.c_out != 64) || g.m() < 1)
        return false;
    const int64_t x_bytes = int64_t(g.n) * g.h * g.w * 8 * g.c_in;
    return x_bytes <= int64_t(0x7fffffef) && g.m() <= int64_t(0x7fffffff) - 64;
}

int qconv2d_pointwise_group_stages(int64_t m, int cus)
{
    const int64_t stages = (m + kPwStagePixels - 1) / kPwStagePixels;
    const int64_t per = (stages + cus - 1) / cus;
    return int(per < 1 ? 1 : per);
}

int qconv2d_pointwise_stage_pixels()
{
    return kPwStagePixels;
}

hipError_t qconv2d_pointwise_run(const ConvGeom &g, const PackGeom &pg, int group_stages, const void *x,
                                 const void *wpack, const void *bias, void *out, float *stats, int stat_tiles,
                                 const ConvFold *fold, hipStream_t stream)
{
    if (!qconv2d_pointwise_takes(g, DType::BF16) || group_stages < 1 || pg.pk != 16)
        return hipErrorInvalidValue;
    PwArgs a;
    a.x = x;
    a.wpack = wpack;
    a.bias = bias;
    a.out = out;
    a.m = int(g.m());
    a.h = g.h;
    a.w = g.w;
    a.h_out = g.h_out;
    a.w_out = g.w_out;
    a.s_h = g.s_h;
    a.s_w = g.s_w;
    a.cout_pad = pg.cout_pad;
    a.stages = (a.m + kPwStagePixels - 1) / kPwStagePixels;
    a.group_stages = group_stages;
    a.x_bytes = unsigned(int64_t(g.n) * g.h * g.w * 8 * g.c_in);
    a.stats = stats;
    a.stat_tiles = stat_tiles;
    a.scale = fold != nullptr ? fold->scale : nullptr;
    a.shift = fold != nullptr ? fold->shift : nullptr;
    a.relu = fold != nullptr && fold->relu ? 1 : 0;
    const int blocks = (a.stages + group_stages - 1) / group_stages;
    if (stats != nullptr && (fold != nullptr || stat_tiles != blocks))
        return hipErrorInvalidValue;
    if (fold != nullptr && (fold->scale == nullptr || fold->shift == nullptr))
        return hipErrorInvalidValue;
    const int epi = stats != nullptr ? kPwEpiStats : fold != nullptr ? kPwEpiFold : kPwEpiBias;
    const void *fn = g.c_in == 64 ? (g.c_out == 64 ? pw_kernel<64, 64>(epi) : pw_kernel<64, 32>(epi))
                                  : (g.c_out == 64 ? pw_kernel<32, 64>(epi) : pw_kernel<32, 32>(epi));
    void *args[] = {&a};
    return hipLaunchKernel(fn, dim3(blocks), dim3(kPwThreads), args, 0, stream);
}

}  // namespace quan
