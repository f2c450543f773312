// Weight and bias gradients of the Hamilton convolution (the backward pass of
// Section III-B's eq. 5/6 with respect to W and the bias) for gfx950.
//
// With Y_p = sum_q s(p, q) W_{p xor q} (x) X_q per tap (eq. 6's sign s and
// component index), the gradient of kernel component m at tap (ky, kx) is
//
//   dW_m[o][c] = sum_p s(p, p xor m) sum_pix dY[pix][p][o] X[pix + tap][p xor m][c],
//
// a GEMM whose reduction dimension is the output pixels (N * Ho * Wo), over
// both operands stored channels-last.  One work-group takes one tap, a
// 64 x 64 tile of (output, input) channels and a contiguous slice of the
// pixels; it stages 32-pixel chunks of dY (all four components) and of the
// tap-shifted X (zero outside the image) in LDS, bank-conflict free (see
// kRowBf16) and double-buffered, with the global loads (16-byte buffer loads
// at 32-bit offsets, zeros past the end, each thread's pixel coordinates
// advanced incrementally) issued two chunks ahead; its four waves each
// accumulate the four dW_m of one 32 x 32 (o, c) block, reading the next
// k-step's fragments while the MFMAs of the current one run, a sign flip
// being one XOR per fragment dword.  The taps of one (slice, tile) are placed
// on one XCD (work-group b runs on XCD b % 8), so the nine reads of a slice
// of dY and its shifted copies of X share that XCD's L2.  MFMA operands need
// eight consecutive pixels per lane: bf16 fragments come from the pixel-major
// rows with two transposing LDS reads (ds_read_b64_tr_b16), fp32 fragments
// (one pixel per lane) with plain reads.  Slices write fp32 partial sums; a
// second kernel adds them in slice order in fp64
// (deterministic) into dW.  Layers of at most 16 channels run the kernel on
// whole pixel rows (one component of 4*C channels) for the dense product of
// all sixteen component pairs, and the reduction forms dW from it.  The bias
// gradient is the column sum of dY.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "quan_launch.h"

namespace quan {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Bit 4*p + q is set when entry (p, q) of the Hamilton matrix (eq. 6) is
// negative.  Row r: + - - -, row i: + + - +, row j: + + + -, row k: + - + +.
constexpr unsigned kNeg = (1u << 1) | (1u << 2) | (1u << 3) | (1u << 6) | (1u << 11) | (1u << 13);
// Bit 4*p + q is set when the separable form (eq. 7) subtracts W_q (*) x_q
// from output component p: S[p][q] = -1.  Row r: + - - -, row i: + + + -,
// row j: + - + +, row k: + + - +.
constexpr unsigned kSepNeg = (1u << 1) | (1u << 2) | (1u << 3) | (1u << 7) | (1u << 9) | (1u << 14);

constexpr int kThreads = 256;
constexpr int kTileO = 64;   // output channels per work-group
constexpr int kTileC = 64;   // input channels per work-group
constexpr int kChunk = 32;   // pixels per staged chunk
// LDS rows of a staged chunk: bf16 rows are 64 elements (128 bytes) with the
// 16-byte chunks of rows 2..3 mod 4 XOR-swizzled by 4, so that neither the
// row-wise 16-byte stores nor the transposing 8-byte reads (four rows of
// one 64-byte column group per 16 lanes) meet in a bank; fp32 rows are
// padded to 80 elements.
constexpr int kRowBf16 = 64, kRowF32 = 80;
__device__ __forceinline__ int chunk_swz(int row) { return 4 * ((row >> 1) & 1); }

struct WArgs {
    const void *x, *dy;
    float *part;  // [splits][taps][4][c_out][c_in]
    int n, c_in, h, w, c_out, k_h, k_w, s_h, s_w, p_h, p_w, d_h, d_w, h_out, w_out;
    int64_t pixels;       // n * h_out * w_out
    int64_t per_split;    // pixels of one slice
    int o_tiles, c_tiles, taps;
    int groups;  // slices x tiles
};

template <typename T>
struct Frag;
template <>
struct Frag<__bf16> {
    typedef bf16x8 type;
};
template <>
struct Frag<float> {
    typedef float type;
};

// 16-byte chunk of one (component, pixel) row: channels ch0 .. ch0+EPC-1 of
// a row of `len` channels starting at src, zeros where `valid` is false or
// past len.  Branch-free: an invalid lane loads from `safe` (the tensor's
// first element) and selects zero, so every load of a chunk stays in flight
// together.  VEC: rows 16-byte aligned and len a multiple of EPC, so a chunk
// is wholly inside or outside; otherwise element by element.
template <typename T, bool VEC>
__device__ __forceinline__ u32x4 load_chunk(const T *src, bool valid, int ch0, int len, const T *safe)
{
    constexpr int EPC = 16 / int(sizeof(T));
    if constexpr (VEC) {
        const bool ok = valid && ch0 < len;
        const u32x4 v = *reinterpret_cast<const u32x4 *>(ok ? src + ch0 : safe);
        const unsigned keep = ok ? 0xffffffffu : 0u;
        return u32x4{v[0] & keep, v[1] & keep, v[2] & keep, v[3] & keep};
    } else {
        T e[EPC];
#pragma unroll
        for (int i = 0; i < EPC; ++i) {
            const bool ok = valid && ch0 + i < len;
            const T u = *(ok ? src + ch0 + i : safe);
            e[i] = ok ? u : T(0);
        }
        u32x4 v;
        __builtin_memcpy(&v, e, 16);
        return v;
    }
}

// 16 bytes at byte offset off of the buffer [base, base + bytes); offsets
// past the end read as zeros.
__device__ __forceinline__ u32x4 load16(const void *base, unsigned bytes, unsigned off)
{
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// NC: components per pixel row as the kernel sees it.  4: the Hamilton
// form above.  1 (layers of at most 16 channels): the whole pixel row is one
// component of 4*C channels (a.c_out, a.c_in are then 4*C), and the kernel
// computes the dense product G[(p,o)][(q,c)] = sum_pix dY[pix][p][o]
// X[pix+tap][q][c] of which the reduction forms every dW_m; on a 64 x 64
// tile this does the useful work once instead of sixteen times.
// SEP (NC = 4): the separable form's gradients (eqs. 8-10), dW_q = sum_p
// S[p][q] dY_p X_q: the same sixteen component pairs, each added into the
// accumulator of its input component q with eq. 7's sign.
template <typename T, bool VEC, int NC, bool SEP = false>
__global__ __launch_bounds__(kThreads) void qconv2d_wgrad(WArgs a)
{
    static_assert(NC == 4 || NC == 1, "four components or one dense row");
    constexpr int NM = NC == 4 ? 4 : 1;        // accumulator sets: dW_m, or G
    constexpr int ES = int(sizeof(T));
    constexpr int kRow = ES == 2 ? kRowBf16 : kRowF32;
    constexpr int EPC = 16 / ES;               // elements per 16-byte chunk
    constexpr int CPR = kTileO / EPC;          // chunks per (component, pixel) row of the tile
    constexpr int PXT = kThreads / CPR;        // pixels one pass of the threads covers
    constexpr int PASSES = kChunk / PXT;
    constexpr int COMP = kChunk * kRow;        // elements per component block of a tensor in LDS
    constexpr int TENSOR = NC * COMP;
    constexpr int BUF = 2 * TENSOR;            // dY then X
    static_assert(kTileO == kTileC && PXT * PASSES == kChunk, "tile geometry");
    __shared__ __attribute__((aligned(16))) T lds[2 * BUF];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // work-group b on XCD b % 8 takes tap (b / 8) % taps of group
    // b % 8 + 8 * (b / 8 / taps)
    const int xs = int(blockIdx.x) >> 3;
    const int tap = xs % a.taps;
    int b = (int(blockIdx.x) & 7) + 8 * (xs / a.taps);
    if (b >= a.groups)
        return;  // padding of the last round of groups: nothing to do
    const int ot = b % a.o_tiles;
    b /= a.o_tiles;
    const int ct = b % a.c_tiles;
    const int split = b / a.c_tiles;
    const int ky = tap / a.k_w, kx = tap - (tap / a.k_w) * a.k_w;
    const int o0 = ot * kTileO, c0 = ct * kTileC;
    const int64_t pix0 = int64_t(split) * a.per_split;
    int64_t pix1 = pix0 + a.per_split;
    if (pix1 > a.pixels)
        pix1 = a.pixels;
    const int chunks = pix0 < pix1 ? int((pix1 - pix0 + kChunk - 1) / kChunk) : 0;
    const T *dy = static_cast<const T *>(a.dy);
    const T *x = static_cast<const T *>(a.x);
    const int hw_out = a.h_out * a.w_out;

    // ---- staging: thread t moves chunk t % CPR of pixel rows t / CPR + PXT * i
    const int cc = tid % CPR, pr = tid / CPR;
    struct Staged {
        u32x4 v[2][PASSES][NC];  // [tensor][pass][component]
    };
    // VEC: 16-byte buffer loads at 32-bit offsets from the slice's first
    // pixel (dY) and first image (X), zeros past a buffer's end; each pass
    // keeps its pixel's (image, row, column), advanced by one chunk per
    // fetch, so chunks are fetched in order.
    const int span = int(pix1 - pix0 > 0 ? pix1 - pix0 : 0);
    const int64_t img0 = pix0 / hw_out;
    const T *const dy_s = dy + pix0 * NC * a.c_out;
    const T *const x_s = x + img0 * int64_t(a.h) * a.w * NC * a.c_in;
    const unsigned dy_bytes = unsigned(int64_t(span) * NC * a.c_out * ES);
    const int64_t x_left = (int64_t(a.n) - img0) * a.h * a.w * NC * a.c_in * ES;
    const unsigned x_bytes = unsigned(x_left < 0x7fffffffLL ? x_left : 0x7fffffffLL);
    const bool o_in = o0 + cc * EPC < a.c_out, c_in_ok = c0 + cc * EPC < a.c_in;
    int cur_img[PASSES], cur_oy[PASSES], cur_ox[PASSES];
#pragma unroll
    for (int i = 0; i < PASSES; ++i) {
        const int64_t pix = pix0 + pr + PXT * i;
        const int64_t img = pix / hw_out;
        const int rr = int(pix - img * hw_out);
        cur_img[i] = int(img - img0);
        cur_oy[i] = rr / a.w_out;
        cur_ox[i] = rr - cur_oy[i] * a.w_out;
    }
    auto fetch = [&](int k, Staged &st) {
#pragma unroll
        for (int i = 0; i < PASSES; ++i) {
            const int rel = k * kChunk + pr + PXT * i;  // pixel - pix0
            const bool yok = rel < span;
            const int iy = cur_oy[i] * a.s_h - a.p_h + ky * a.d_h, ix = cur_ox[i] * a.s_w - a.p_w + kx * a.d_w;
            if constexpr (VEC) {
                const bool xok = yok && c_in_ok && unsigned(iy) < unsigned(a.h) && unsigned(ix) < unsigned(a.w);
                const unsigned yoff = yok && o_in ? unsigned((rel * NC * a.c_out + o0 + cc * EPC) * ES) : 0x80000000u;
                const unsigned xoff =
                    xok ? unsigned((((cur_img[i] * a.h + iy) * a.w + ix) * NC * a.c_in + c0 + cc * EPC) * ES)
                        : 0x80000000u;
#pragma unroll
                for (int q = 0; q < NC; ++q) {
                    st.v[0][i][q] = load16(dy_s, dy_bytes, yoff + unsigned(q * a.c_out * ES));
                    st.v[1][i][q] = load16(x_s, x_bytes, xoff + unsigned(q * a.c_in * ES));
                }
            } else {
                const bool xok = yok && iy >= 0 && iy < a.h && ix >= 0 && ix < a.w;
                const T *yrow = dy_s + int64_t(yok ? rel : 0) * NC * a.c_out;
                const T *xrow = x_s + ((int64_t(cur_img[i]) * a.h + (xok ? iy : 0)) * a.w + (xok ? ix : 0)) * NC * a.c_in;
#pragma unroll
                for (int q = 0; q < NC; ++q) {
                    st.v[0][i][q] = load_chunk<T, VEC>(yrow + q * a.c_out + o0, yok, cc * EPC, a.c_out - o0, dy);
                    st.v[1][i][q] = load_chunk<T, VEC>(xrow + q * a.c_in + c0, xok, cc * EPC, a.c_in - c0, x);
                }
            }
            // next chunk: kChunk pixels on
            int ox = cur_ox[i] + kChunk, oy = cur_oy[i], im = cur_img[i];
            while (ox >= a.w_out) {
                ox -= a.w_out;
                if (++oy == a.h_out) {
                    oy = 0;
                    ++im;
                }
            }
            cur_ox[i] = ox;
            cur_oy[i] = oy;
            cur_img[i] = im;
        }
    };
    auto store = [&](int buf, const Staged &st) {
        T *base = lds + buf * BUF;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int i = 0; i < PASSES; ++i)
#pragma unroll
                for (int q = 0; q < NC; ++q)
                    *reinterpret_cast<u32x4 *>(base + t * TENSOR + q * COMP + (pr + PXT * i) * kRow +
                                               (ES == 2 ? (cc ^ chunk_swz(pr + PXT * i)) : cc) * EPC) =
                        st.v[t][i][q];
    };

    // ---- compute: wave w owns o-block w / 2 and c-block w % 2
    const int ob = (wave >> 1) * 32, cb = (wave & 1) * 32;
    f32x16 acc[NM];
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int e = 0; e < 16; ++e)
            acc[m][e] = 0.0f;

    // Fragment of component block `comp` of tensor t (0 dY, 1 X), channel
    // block col0, k-step ks: lane l gets channel col0 + l%32 at the pixels
    // the MFMA's operand layout assigns it.
    auto frag = [&](const T *base, int comp, int col0, int ks) {
        typename Frag<T>::type f;
        if constexpr (ES == 2) {
            // two transposing reads of rows 16ks + 8(g/2) + 4r + j, columns
            // col0 + 16(g%2) + 4a (g = l/16, a = l%4, j = (l%16)/4)
            const int g = lane >> 4, aa = lane & 3, j = (lane & 15) >> 2;
            const int row = 16 * ks + 8 * (g >> 1) + j, col = col0 + 16 * (g & 1) + 4 * aa;
            // rows row and row + 4 share the swizzle
            const T *p0 = base + comp * COMP + row * kRow + (((col >> 3) ^ chunk_swz(row)) << 3) + (col & 7);
            const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) s16x4 *)(p0));
            const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) s16x4 *)(p0 + 4 * kRow));
            s16x4 both[2] = {lo, hi};
            __builtin_memcpy(&f, both, 16);
        } else {
            // one pixel per lane: row 2ks + l/32, column col0 + l%32
            f = base[comp * COMP + (2 * ks + (lane >> 5)) * kRow + col0 + (lane & 31)];
        }
        return f;
    };
    constexpr int KSTEPS = ES == 2 ? kChunk / 16 : kChunk / 2;
    typedef typename Frag<T>::type F;
    struct KFrags {
        F fy[NC], fx[NC];
    };
    auto read_k = [&](int buf, int ks, KFrags &f) {
        const T *yb = lds + buf * BUF, *xb = yb + TENSOR;
#pragma unroll
        for (int q = 0; q < NC; ++q) {
            f.fy[q] = frag(yb, q, ob, ks);
            f.fx[q] = frag(xb, q, cb, ks);
        }
    };
    // sign flip of a fragment: the sign bit of every element
    auto negate = [&](F v) {
        if constexpr (ES == 2) {
            u32x4 u = __builtin_bit_cast(u32x4, v);
            u ^= 0x80008000u;
            return __builtin_bit_cast(F, u);
        } else {
            return __builtin_bit_cast(F, __builtin_bit_cast(unsigned, v) ^ 0x80000000u);
        }
    };
    auto mfmas = [&](const KFrags &f) {
        if constexpr (NC == 1) {
            if constexpr (ES == 2)
                acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.fy[0], f.fx[0], acc[0], 0, 0, 0);
            else
                acc[0] = __builtin_amdgcn_mfma_f32_32x32x2f32(f.fy[0], f.fx[0], acc[0], 0, 0, 0);
        } else {
#pragma unroll
            for (int p = 0; p < NC; ++p) {
                const F pos = f.fy[p], neg = negate(f.fy[p]);
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    const int q = p ^ m;
                    const int d = SEP ? q : m;  // the gradient this pair adds into
                    const bool minus = ((SEP ? kSepNeg : kNeg) >> (4 * p + q)) & 1u;
                    if constexpr (ES == 2)
                        acc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(minus ? neg : pos, f.fx[q], acc[d], 0, 0, 0);
                    else
                        acc[d] = __builtin_amdgcn_mfma_f32_32x32x2f32(minus ? neg : pos, f.fx[q], acc[d], 0, 0, 0);
                }
            }
        }
    };
    // The k-steps of one chunk, reading k-step ks + 1 while ks runs: the
    // sign flips first, then each MFMA followed by one fragment read.
    constexpr int NRD = ES == 2 ? 16 : 8;  // LDS reads of one k-step
    auto sched = [&]() {
        if constexpr (NC == 1)
            return;  // one MFMA per k-step: nothing to interleave
        __builtin_amdgcn_sched_group_barrier(0x002, ES == 2 ? 16 : 4, 0);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            if (i < NRD)
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
    };
    auto compute = [&](int buf) {
        KFrags fa, fb;
        read_k(buf, 0, fa);
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ks += 2) {
            __builtin_amdgcn_sched_barrier(0);
            if (ks + 1 < KSTEPS)
                read_k(buf, ks + 1, fb);
            mfmas(fa);
            if (ks + 1 < KSTEPS)
                sched();
            __builtin_amdgcn_sched_barrier(0);
            if (ks + 2 < KSTEPS)
                read_k(buf, ks + 2, fa);
            if (ks + 1 < KSTEPS)
                mfmas(fb);
            if (ks + 2 < KSTEPS)
                sched();
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // Chunk k is computed from LDS buffer k % 2 while chunk k + 1 waits in
    // registers (loaded an iteration earlier) and chunk k + 2 is loaded; after
    // the computation chunk k + 1 goes to the other buffer, which the previous
    // barrier freed.  Two register sets alternate, so the loop is unrolled by
    // two.
    Staged sa, sb;
    auto iteration = [&](int k, Staged &next, Staged &after) {
        if (k + 2 < chunks)
            fetch(k + 2, after);
        compute(k & 1);
        if (k + 1 < chunks)
            store((k + 1) & 1, next);
        __syncthreads();
    };
    if (chunks > 0) {
        fetch(0, sa);
        if (chunks > 1)
            fetch(1, sb);
        store(0, sa);
        __syncthreads();
        int k = 0;
        for (; k + 1 < chunks; k += 2) {
            iteration(k, sb, sa);
            iteration(k + 1, sa, sb);
        }
        if (k < chunks)
            iteration(k, sb, sa);
    }

    // ---- partial sums: register 4g + e of lane l is (o, c) = (ob + 8g +
    // 4(l/32) + e, cb + l%32) of the wave's block
    const int c = c0 + cb + (lane & 31);
#pragma unroll
    for (int m = 0; m < NM; ++m) {
        float *dst = a.part + ((int64_t(split) * a.taps + tap) * NM + m) * a.c_out * a.c_in;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int o = o0 + ob + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (o < a.c_out && c < a.c_in)
                dst[int64_t(o) * a.c_in + c] = acc[m][r];
        }
    }
}

// dW_m[o][c][ky][kx] = sum over slices of the partials, in slice order, fp64.
// Consecutive threads take consecutive (o, c) of one (m, tap), so every
// slice's partials are read contiguously.
__global__ __launch_bounds__(kThreads) void qconv2d_wgrad_reduce(const float *__restrict__ part, int splits, int taps,
                                                                 int c_out, int c_in, float *__restrict__ dw0,
                                                                 float *__restrict__ dw1, float *__restrict__ dw2,
                                                                 float *__restrict__ dw3)
{
    const int64_t oc_n = int64_t(c_out) * c_in;
    const int64_t idx = int64_t(blockIdx.x) * kThreads + threadIdx.x;  // over [m][tap][o][c]
    if (idx >= 4 * taps * oc_n)
        return;
    const int64_t oc = idx % oc_n;  // o * c_in + c
    const int mt = int(idx / oc_n);
    const int m = mt / taps, tap = mt - (mt / taps) * taps;
    double s = 0.0;
    for (int sp = 0; sp < splits; ++sp)
        s += double(part[((int64_t(sp) * taps + tap) * 4 + m) * c_out * c_in + oc]);
    float *dw = m == 0 ? dw0 : m == 1 ? dw1 : m == 2 ? dw2 : dw3;
    dw[oc * taps + tap] = float(s);
}

// Layers of at most 16 channels (the kernel's NC = 1 form): the partials
// are G[(p,o)][(q,c)] per slice and tap ([splits][taps][4*c_out][4*c_in]), and
// dW_m[o][c][tap] = sum over slices, then over p in order, of
// s(p, p xor m) G[(p,o)][(p xor m, c)] (eq. 6's signs), in fp64; with sep
// (the separable form) dW_m = sum of S[p][m] G[(p,o)][(m,c)] (eq. 7's signs).
__global__ __launch_bounds__(kThreads) void qconv2d_wgrad_reduce_dense(const float *__restrict__ part, int splits,
                                                                       int taps, int c_out, int c_in, int sep,
                                                                       float *__restrict__ dw0,
                                                                       float *__restrict__ dw1,
                                                                       float *__restrict__ dw2,
                                                                       float *__restrict__ dw3)
{
    const int64_t oc_n = int64_t(c_out) * c_in;
    const int64_t idx = int64_t(blockIdx.x) * kThreads + threadIdx.x;  // over [m][tap][o][c]
    if (idx >= 4 * taps * oc_n)
        return;
    const int64_t oc = idx % oc_n;
    const int o = int(oc / c_in), c = int(oc - int64_t(o) * c_in);
    const int mt = int(idx / oc_n);
    const int m = mt / taps, tap = mt - (mt / taps) * taps;
    const int64_t g_n = int64_t(4 * c_out) * (4 * c_in);  // one slice's G of one tap
    double s = 0.0;
    for (int sp = 0; sp < splits; ++sp) {
        const float *g = part + (int64_t(sp) * taps + tap) * g_n;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const int q = sep ? m : p ^ m;
            const double v = double(g[int64_t(p * c_out + o) * (4 * c_in) + q * c_in + c]);
            s += (((sep ? kSepNeg : kNeg) >> (4 * p + q)) & 1u) ? -v : v;
        }
    }
    float *dw = m == 0 ? dw0 : m == 1 ? dw1 : m == 2 ? dw2 : dw3;
    dw[oc * taps + tap] = float(s);
}

// Bias gradient: column sums of the [pixels][cols = 4 * c_out] rows of dY.
// Thread t of a block sums the VW-element column chunk t % CG over rows
// t / CG + RPI * i of the block's row range (four rows in flight), the
// threads sharing a chunk add in a fixed order through LDS, and each block
// writes one partial per column; colsum_final adds the blocks in order in
// fp64.
template <typename T, int VW>
__global__ __launch_bounds__(kThreads) void colsum_partial(const T *__restrict__ dy, int64_t pixels, int cols,
                                                           int64_t rows_per_block, float *__restrict__ part)
{
    __shared__ float red[kThreads][VW];
    const int chunks = cols / VW;
    const int cg = chunks < kThreads ? chunks : kThreads;
    const int rpi = kThreads / cg;
    const int tid = threadIdx.x, cl = tid % cg, rl = tid / cg;
    const int chunk = blockIdx.y * cg + cl;
    const bool active = rl < rpi && chunk < chunks;
    const int64_t r0 = int64_t(blockIdx.x) * rows_per_block;
    int64_t r1 = r0 + rows_per_block;
    if (r1 > pixels)
        r1 = pixels;
    struct alignas(sizeof(T) * VW) V {
        T e[VW];
    };
    float acc[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e)
        acc[e] = 0.0f;
    if (active) {
        const T *base = dy + chunk * VW;
        int64_t r = r0 + rl;
        for (; r + 3 * rpi < r1; r += 4 * rpi) {
            V v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                v[u] = *reinterpret_cast<const V *>(base + (r + u * rpi) * cols);
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int e = 0; e < VW; ++e)
                    acc[e] += float(v[u].e[e]);
        }
        for (; r < r1; r += rpi) {
            const V v = *reinterpret_cast<const V *>(base + r * cols);
#pragma unroll
            for (int e = 0; e < VW; ++e)
                acc[e] += float(v.e[e]);
        }
    }
#pragma unroll
    for (int e = 0; e < VW; ++e)
        red[tid][e] = acc[e];
    __syncthreads();
    if (rl == 0 && chunk < chunks) {
        float t[VW];
#pragma unroll
        for (int e = 0; e < VW; ++e)
            t[e] = 0.0f;
        for (int j = 0; j < rpi; ++j)
#pragma unroll
            for (int e = 0; e < VW; ++e)
                t[e] += red[j * cg + cl][e];
#pragma unroll
        for (int e = 0; e < VW; ++e)
            part[int64_t(blockIdx.x) * cols + chunk * VW + e] = t[e];
    }
}

// One wave per column: lane i adds blocks i, i+64, ... (eight loads in
// flight), then a fixed butterfly adds the lanes in fp64.
__global__ __launch_bounds__(kThreads) void colsum_final(const float *__restrict__ part, int blocks, int cols,
                                                         float *__restrict__ db)
{
    constexpr int U = 8;
    const int lane = threadIdx.x & 63;
    const int col = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (col >= cols)
        return;
    double s = 0.0;
    for (int b0 = lane; b0 < blocks; b0 += 64 * U) {
        float v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int b = b0 + 64 * u;
            v[u] = part[int64_t(b < blocks ? b : blocks - 1) * cols + col];
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (b0 + 64 * u < blocks)
                s += double(v[u]);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        s += __shfl_xor(s, off);
    if (lane == 0)
        db[col] = float(s);
}

constexpr int kBiasBlocks = 512;

struct WPlan {
    int o_tiles, c_tiles, taps, splits;
    int64_t per_split;
};

// Layers whose whole pixel rows (4 * C reals) fit one tile take the dense
// (NC = 1) form of the kernel.
bool wgrad_dense(const ConvGeom &g)
{
    return 4 * g.c_out <= kTileO && 4 * g.c_in <= kTileC;
}

WPlan wgrad_plan(const ConvGeom &g)
{
    WPlan p;
    const int nc = wgrad_dense(g) ? 4 : 1;  // channels per kernel-side row, in units of C
    p.o_tiles = (nc * g.c_out + kTileO - 1) / kTileO;
    p.c_tiles = (nc * g.c_in + kTileC - 1) / kTileC;
    p.taps = g.k_h * g.k_w;
    const int64_t pixels = g.m();
    const int64_t per_split_pass = int64_t(p.o_tiles) * p.c_tiles * p.taps;
    // about two work-groups per compute unit, each at least a few chunks long
    int64_t splits = (512 + per_split_pass - 1) / per_split_pass;
    const int64_t max_splits = (pixels + 8 * kChunk - 1) / (8 * kChunk);
    if (splits > max_splits)
        splits = max_splits;
    if (splits < 1)
        splits = 1;
    p.per_split = (pixels + splits - 1) / splits;
    p.per_split = (p.per_split + kChunk - 1) / kChunk * kChunk;
    p.splits = int((pixels + p.per_split - 1) / p.per_split);
    return p;
}

}  // namespace

size_t qconv2d_wgrad_work_bytes(const ConvGeom &g)
{
    const WPlan p = wgrad_plan(g);
    const size_t dw_part = size_t(p.splits) * p.taps * (wgrad_dense(g) ? 16 : 4) * g.c_out * g.c_in * sizeof(float);
    const size_t b_part = size_t(kBiasBlocks) * 4 * g.c_out * sizeof(float);
    return dw_part > b_part ? dw_part : b_part;
}

hipError_t qconv2d_backward_weight_run(const ConvGeom &g, DType dt, const void *x, const void *dy, float *dw_r,
                                       float *dw_i, float *dw_j, float *dw_k, float *db, void *work,
                                       hipStream_t stream, bool sep)
{
    const WPlan p = wgrad_plan(g);
    const bool dense = wgrad_dense(g);
    WArgs a;
    a.x = x;
    a.dy = dy;
    a.part = static_cast<float *>(work);
    a.n = g.n;
    a.c_in = dense ? 4 * g.c_in : g.c_in;  // channels of the kernel's one component
    a.h = g.h;
    a.w = g.w;
    a.c_out = dense ? 4 * g.c_out : g.c_out;
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
    a.pixels = g.m();
    a.per_split = p.per_split;
    a.o_tiles = p.o_tiles;
    a.c_tiles = p.c_tiles;
    a.taps = p.taps;
    a.groups = p.splits * p.c_tiles * p.o_tiles;
    const unsigned blocks = unsigned(int64_t(8) * p.taps * ((a.groups + 7) / 8));
    const int epc = dt == DType::BF16 ? 8 : 4, es = dt == DType::BF16 ? 2 : 4;
    // the 16-byte buffer loads take 32-bit offsets within a slice's pixels
    // of dY and the images of X it touches
    const int64_t hw_out = int64_t(g.h_out) * g.w_out;
    const int64_t dy_span = p.per_split * 4 * g.c_out * es;
    const int64_t x_span = ((p.per_split + hw_out - 1) / hw_out + 1) * g.h * g.w * 4 * g.c_in * es;
    const bool vec = a.c_in % epc == 0 && a.c_out % epc == 0 && dy_span < 0x7fffffffLL && x_span < 0x7fffffffLL;
    auto launch = [&](auto t, auto v, auto nc) {
        using T = decltype(t);
        constexpr int NC = decltype(nc)::value;
        if (sep && NC == 4)
            hipLaunchKernelGGL((qconv2d_wgrad<T, decltype(v)::value, NC, NC == 4>), dim3(blocks), dim3(kThreads), 0,
                               stream, a);
        else
            hipLaunchKernelGGL((qconv2d_wgrad<T, decltype(v)::value, NC>), dim3(blocks), dim3(kThreads), 0, stream,
                               a);
    };
    using VT = std::true_type;
    using VF = std::false_type;
    using N4 = std::integral_constant<int, 4>;
    using N1 = std::integral_constant<int, 1>;
    if (dt == DType::BF16) {
        if (dense)
            vec ? launch(__bf16{}, VT{}, N1{}) : launch(__bf16{}, VF{}, N1{});
        else
            vec ? launch(__bf16{}, VT{}, N4{}) : launch(__bf16{}, VF{}, N4{});
    } else {
        if (dense)
            vec ? launch(float{}, VT{}, N1{}) : launch(float{}, VF{}, N1{});
        else
            vec ? launch(float{}, VT{}, N4{}) : launch(float{}, VF{}, N4{});
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    const int64_t outs = int64_t(4) * g.c_out * g.c_in * p.taps;
    const dim3 rgrid(unsigned((outs + kThreads - 1) / kThreads));
    if (dense)
        hipLaunchKernelGGL(qconv2d_wgrad_reduce_dense, rgrid, dim3(kThreads), 0, stream, (const float *)a.part,
                           p.splits, p.taps, g.c_out, g.c_in, sep ? 1 : 0, dw_r, dw_i, dw_j, dw_k);
    else
        hipLaunchKernelGGL(qconv2d_wgrad_reduce, rgrid, dim3(kThreads), 0, stream, (const float *)a.part, p.splits,
                           p.taps, g.c_out, g.c_in, dw_r, dw_i, dw_j, dw_k);
    e = hipGetLastError();
    if (e != hipSuccess || db == nullptr)
        return e;
    // the partials of dW are consumed: reuse the workspace for the bias
    const int cols = 4 * g.c_out;
    const int64_t pixels = g.m();
    const int64_t rpb = (pixels + kBiasBlocks - 1) / kBiasBlocks;
    const int nb = int((pixels + rpb - 1) / rpb);
    const int vw = cols % (dt == DType::BF16 ? 8 : 4) == 0 ? (dt == DType::BF16 ? 8 : 4) : 1;
    const int chunks = cols / vw;
    const int cg = chunks < kThreads ? chunks : kThreads;
    const dim3 grid(nb, (chunks + cg - 1) / cg);
    if (dt == DType::BF16) {
        if (vw == 8)
            hipLaunchKernelGGL((colsum_partial<__bf16, 8>), grid, dim3(kThreads), 0, stream, (const __bf16 *)dy,
                               pixels, cols, rpb, a.part);
        else
            hipLaunchKernelGGL((colsum_partial<__bf16, 1>), grid, dim3(kThreads), 0, stream, (const __bf16 *)dy,
                               pixels, cols, rpb, a.part);
    } else {
        if (vw == 4)
            hipLaunchKernelGGL((colsum_partial<float, 4>), grid, dim3(kThreads), 0, stream, (const float *)dy,
                               pixels, cols, rpb, a.part);
        else
            hipLaunchKernelGGL((colsum_partial<float, 1>), grid, dim3(kThreads), 0, stream, (const float *)dy,
                               pixels, cols, rpb, a.part);
    }
    hipLaunchKernelGGL(colsum_final, dim3((cols + kThreads / 64 - 1) / (kThreads / 64)), dim3(kThreads), 0, stream,
                       (const float *)a.part, nb, cols, db);
    return hipGetLastError();
}

}  // namespace quan
