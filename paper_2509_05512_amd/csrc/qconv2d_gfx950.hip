// Quaternion 2-D convolution (Hamilton product) as an implicit-GEMM MFMA
// kernel for gfx950 (MI355X).
//
// The operation (Section III-B, eqs. 5 and 6): for every output pixel and
// output channel o, Y[o] = sum over input channels c and taps of the Hamilton
// product W[o,c,tap] (x) X[c, pixel + tap].  Over real numbers this is a GEMM
//
//   Y[m, (p, o)] = sum_{tap, q, c} A[m, (tap, q, c)] * B[(tap, q, c), (p, o)]
//   A[m, (tap, q, c)] = x[pixel m shifted by tap][component q][channel c]
//   B[(tap, q, c), (p, o)] = sign(p, q) * W_{p xor q}[o, c, tap]
//
// where (p, q) is the position in the 4x4 Hamilton matrix of eq. 6: with
// components ordered r, i, j, k = 0..3, the entry in row p, column q is the
// kernel component p xor q, negated at (r,i) (r,j) (r,k) (i,j) (j,k) (k,i).
//
// Data flow of one work-group tile (BM output pixels x 4*BNC output reals):
//   - the K loop runs over stages (tap, channel block of BKC channels); a
//     stage holds all four input components of those channels;
//   - activations are loaded channels-last (16-byte vectors along c) into an
//     LDS tile [BM][4*BKC], XOR-swizzled so the MFMA fragment reads are
//     bank-conflict free; taps outside the image load zeros;
//   - only the four shared real kernels are staged: LDS holds
//     W_0..W_3 [BNC][BKC] for the stage.  The signed 4x4 Hamilton block is
//     formed on the LDS->register read: the fragment for (output component p,
//     input component q) reads kernel p xor q and flips its sign bits with
//     one XOR when sign(p, q) < 0;
//   - v_mfma_f32_32x32x16_bf16 (bf16) / v_mfma_f32_32x32x2f32 (fp32) with fp32
//     accumulators; two LDS stages, register prefetch of the next stage while
//     the current one is multiplied;
//   - epilogue: bias, round to the output type (RNE), channels-last stores.
#include <hip/hip_runtime.h>

#include "quan_launch.h"

namespace quan {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Bit 4*p + q is set when entry (p, q) of the Hamilton matrix (eq. 6) is
// negative.  Row r: + - - -, row i: + + - +, row j: + + + -, row k: + - + +.
constexpr unsigned kHamiltonNeg =
    (1u << 1) | (1u << 2) | (1u << 3) | (1u << 6) | (1u << 11) | (1u << 13);

template <typename T>
struct Elem;
template <>
struct Elem<__bf16> {
    static constexpr int per_chunk = 8;            // elements per 16-byte chunk
    static constexpr unsigned sign = 0x80008000u;  // sign bits of a packed pair
};
template <>
struct Elem<float> {
    static constexpr int per_chunk = 4;
    static constexpr unsigned sign = 0x80000000u;
};

struct KArgs {
    const void *x;
    const void *wpack;
    const void *bias;
    void *out;
    int c_in, h, w, c_out, k_w;
    int s_h, s_w, p_h, p_w, d_h, d_w;
    int h_out, w_out;
    int m;       // n * h_out * w_out output pixels
    int stages;  // taps * n_cblk
    int n_cblk;
    int cout_pad;
    int n_tiles;
    int vec_in;  // c_in is a multiple of the 16-byte chunk
};

// XOR swizzle of the 16-byte chunk index within an LDS row of `cpr` chunks:
// rows that a group of 8 lanes reads together land in 8 different bank
// groups.
template <int CPR>
__device__ __forceinline__ int swz(int row)
{
    if constexpr (CPR >= 8)
        return row & 7;
    else
        return (row * CPR / 8) % CPR;
}

template <typename T>
__device__ __forceinline__ u32x4 load_chunk_masked(const T *p, int valid_elems)
{
    // Element-wise load of a partial chunk (input channels not a multiple of
    // the vector width); missing elements are zero.
    constexpr int E = Elem<T>::per_chunk;
    T v[E];
#pragma unroll
    for (int e = 0; e < E; ++e)
        v[e] = e < valid_elems ? p[e] : T(0);
    u32x4 r;
    __builtin_memcpy(&r, v, 16);
    return r;
}

template <typename T>
__device__ __forceinline__ void mfma_step(f32x16 &acc, u32x4 a, u32x4 b)
{
    if constexpr (sizeof(T) == 2) {
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                      __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
    } else {
        // Lane l holds k = l/32 of each 32x32x2 step; the four floats of the
        // chunk are four consecutive steps.  (Cast the whole vector: casting
        // single elements of a u32x4 let the compiler fold every step onto
        // element 0.)
        const f32x4 af = __builtin_bit_cast(f32x4, a);
        const f32x4 bf = __builtin_bit_cast(f32x4, b);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(af[e], bf[e], acc, 0, 0, 0);
    }
}

template <typename T, int BM, int BNC, int WAVES_M, int WAVES_N, int BKC>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) void qconv2d_igemm(KArgs a)
{
    constexpr int EPC = Elem<T>::per_chunk;
    constexpr int NT = 64 * WAVES_M * WAVES_N;
    constexpr int BN = 4 * BNC;
    constexpr int CPQ = BKC / EPC;  // chunks per component in a stage
    constexpr int CPR = 4 * CPQ;    // chunks per activation row in a stage
    constexpr int WTM = BM / WAVES_M;
    constexpr int WTN = BN / WAVES_N;
    constexpr int MB = WTM / 32;
    constexpr int NB = WTN / 32;
    constexpr int A_CHUNKS = BM * CPR;
    constexpr int B_CHUNKS = 4 * BNC * CPQ;
    constexpr int A_PER_T = A_CHUNKS / NT;
    constexpr int B_PER_T = (B_CHUNKS + NT - 1) / NT;
    constexpr int A_BYTES = A_CHUNKS * 16;
    constexpr int B_BYTES = B_CHUNKS * 16;
    constexpr int STAGE = A_BYTES + B_BYTES;
    constexpr int ROWS_PER_PASS = NT / CPR;
    static_assert(A_CHUNKS % NT == 0 && NT % CPR == 0, "activation tile must split evenly");
    static_assert(CPQ % 2 == 0, "a k-step takes two chunks of one component");
    static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must be whole 32x32 blocks");
    static_assert(BNC % 4 == 0, "epilogue stores groups of four channels");

    __shared__ __attribute__((aligned(16))) unsigned char smem[2 * STAGE];

    const T *__restrict__ xp = static_cast<const T *>(a.x);
    const T *__restrict__ wp = static_cast<const T *>(a.wpack);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WAVES_M;
    const int wn = wave / WAVES_M;
    const int khalf = lane >> 5;
    const int l32 = lane & 31;

    // Work-groups are dealt to the 8 XCDs round-robin; give each XCD a
    // contiguous run of tiles so neighbouring tiles share its L2.
    const int nblk = gridDim.x;
    const int bid = blockIdx.x;
    const int per = nblk >> 3, rem = nblk & 7, xcd = bid & 7;
    const int tile = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + (bid >> 3);
    const int n_tile = tile % a.n_tiles;
    const int m0 = (tile / a.n_tiles) * BM;
    const int o0 = n_tile * BNC;

    // ---- activation rows this thread loads (fixed for the whole K loop) ----
    const int cc = tid % CPR;  // chunk column within the stage row
    const int q_ld = cc / CPQ;
    const int piece = cc % CPQ;
    const int hw_out = a.h_out * a.w_out;
    int row_iy0[A_PER_T], row_ix0[A_PER_T], row_img[A_PER_T];
#pragma unroll
    for (int i = 0; i < A_PER_T; ++i) {
        const int m = m0 + i * ROWS_PER_PASS + tid / CPR;
        if (m < a.m) {
            const int img = m / hw_out;
            const int rr = m - img * hw_out;
            const int oy = rr / a.w_out;
            const int ox = rr - oy * a.w_out;
            row_img[i] = img * a.h * a.w;
            row_iy0[i] = oy * a.s_h - a.p_h;
            row_ix0[i] = ox * a.s_w - a.p_w;
        } else {
            row_img[i] = 0;
            row_iy0[i] = -0x20000000;  // never inside the image
            row_ix0[i] = 0;
        }
    }
    const int row_elems = 4 * a.c_in;

    u32x4 ra[A_PER_T], rb[B_PER_T];

    auto load_stage = [&](int s) {
        const int tap = s / a.n_cblk;
        const int cblk = s - tap * a.n_cblk;
        const int ky = tap / a.k_w;
        const int kx = tap - ky * a.k_w;
        const int dy = ky * a.d_h, dx = kx * a.d_w;
        const int c = cblk * BKC + piece * EPC;
        const int cvalid = a.c_in - c;  // elements of this chunk inside c_in
#pragma unroll
        for (int i = 0; i < A_PER_T; ++i) {
            const int iy = row_iy0[i] + dy;
            const int ix = row_ix0[i] + dx;
            const bool inside = (unsigned)iy < (unsigned)a.h && (unsigned)ix < (unsigned)a.w && cvalid > 0;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (inside) {
                const T *src = xp + ((row_img[i] + iy * a.w + ix) * row_elems + q_ld * a.c_in + c);
                if (a.vec_in)
                    v = *reinterpret_cast<const u32x4 *>(src);
                else
                    v = load_chunk_masked<T>(src, cvalid);
            }
            ra[i] = v;
        }
        const T *wsrc = wp + ((size_t)(tap * a.n_cblk + cblk) * 4 * a.cout_pad + o0) * BKC;
#pragma unroll
        for (int j = 0; j < B_PER_T; ++j) {
            const int id = j * NT + tid;
            if (B_CHUNKS % NT == 0 || id < B_CHUNKS) {
                const int ws = id / (BNC * CPQ);
                const int rest = id - ws * (BNC * CPQ);
                rb[j] = *reinterpret_cast<const u32x4 *>(wsrc + (size_t)ws * a.cout_pad * BKC +
                                                         rest * EPC);
            }
        }
    };

    auto store_stage = [&](int buf) {
        unsigned char *As = smem + buf * STAGE;
        unsigned char *Bs = As + A_BYTES;
#pragma unroll
        for (int i = 0; i < A_PER_T; ++i) {
            const int r = i * ROWS_PER_PASS + tid / CPR;
            *reinterpret_cast<u32x4 *>(As + (r * CPR + (cc ^ swz<CPR>(r))) * 16) = ra[i];
        }
#pragma unroll
        for (int j = 0; j < B_PER_T; ++j) {
            const int id = j * NT + tid;
            if (B_CHUNKS % NT == 0 || id < B_CHUNKS) {
                const int row = id / CPQ;  // kernel slice * BNC + o
                const int pc = id - row * CPQ;
                *reinterpret_cast<u32x4 *>(Bs + (row * CPQ + (pc ^ swz<CPQ>(row))) * 16) = rb[j];
            }
        }
    };

    // Per-lane output component and channel of the weight-fragment rows.
    int frag_p[NB], frag_o[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int tn = wn * WTN + nb * 32 + l32;
        frag_p[nb] = tn / BNC;
        frag_o[nb] = tn - frag_p[nb] * BNC;
    }

    f32x16 acc[NB][MB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                acc[nb][mb][e] = 0.0f;

    auto compute = [&](int buf) {
        const unsigned char *As = smem + buf * STAGE;
        const unsigned char *Bs = As + A_BYTES;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
            for (int kk = 0; kk < CPQ / 2; ++kk) {
                const int pc = kk * 2 + khalf;
                u32x4 wf[NB], pf[MB];
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    const int p = frag_p[nb];
                    const int row = (p ^ q) * BNC + frag_o[nb];
                    u32x4 v = *reinterpret_cast<const u32x4 *>(Bs + (row * CPQ + (pc ^ swz<CPQ>(row))) * 16);
                    const unsigned flip = ((kHamiltonNeg >> (4 * p + q)) & 1u) ? Elem<T>::sign : 0u;
                    v ^= flip;
                    wf[nb] = v;
                }
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) {
                    const int r = wm * WTM + mb * 32 + l32;
                    const int lc = q * CPQ + pc;
                    pf[mb] = *reinterpret_cast<const u32x4 *>(As + (r * CPR + (lc ^ swz<CPR>(r))) * 16);
                }
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb)
                        mfma_step<T>(acc[nb][mb], wf[nb], pf[mb]);
            }
        }
    };

    // ---- main loop: two LDS stages, next stage prefetched into registers ----
    load_stage(0);
    store_stage(0);
    __syncthreads();
    for (int s = 0; s < a.stages; ++s) {
        const int cur = s & 1;
        const bool more = s + 1 < a.stages;
        if (more)
            load_stage(s + 1);
        compute(cur);
        if (more)
            store_stage(cur ^ 1);
        __syncthreads();
    }

    // ---- epilogue: bias, round, channels-last store ----
    // Accumulator register 4*g + e of lane l holds output channel row
    // 8*g + 4*(l/32) + e of the 32x32 block and pixel column l%32.
    const T *__restrict__ bias = static_cast<const T *>(a.bias);
    T *__restrict__ out = static_cast<T *>(a.out);
    const bool vec_out = (a.c_out & 3) == 0;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int tn = wn * WTN + nb * 32 + 8 * g + 4 * khalf;
            const int p = tn / BNC;
            const int o = o0 + (tn - p * BNC);
            if (o >= a.c_out)
                continue;
            float bv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                bv[e] = (bias != nullptr && o + e < a.c_out) ? float(bias[p * a.c_out + o + e]) : 0.0f;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                const int m = m0 + wm * WTM + mb * 32 + l32;
                if (m >= a.m)
                    continue;
                T *dst = out + ((size_t)m * 4 * a.c_out + p * a.c_out + o);
                T v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    v[e] = T(acc[nb][mb][4 * g + e] + bv[e]);
                if (vec_out) {
                    if constexpr (sizeof(T) == 2) {
                        uint2 pk;
                        __builtin_memcpy(&pk, v, 8);
                        *reinterpret_cast<uint2 *>(dst) = pk;
                    } else {
                        float4 pk;
                        __builtin_memcpy(&pk, v, 16);
                        *reinterpret_cast<float4 *>(dst) = pk;
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (o + e < a.c_out)
                            dst[e] = v[e];
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Pipelined variant: global -> LDS direct loads into a ring of STAGES LDS
// buffers, so the loads of the next STAGES-1 stages are in flight while the
// current stage is multiplied.  Each global_load_lds_dwordx4 of a wave writes
// 64 consecutive 16-byte LDS slots (lane order); the swizzled layout is
// obtained by choosing which global chunk each lane fetches.  Taps outside
// the image, channels past c_in and rows past M fetch a zero chunk.
// Requires c_in to be a multiple of the 16-byte vector (vec_in).
// ---------------------------------------------------------------------------

__device__ __attribute__((aligned(64))) unsigned int g_qconv_zero16[16];

template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    // gfx9 s_waitcnt: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14]
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ void block_barrier()
{
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// One wave-wide 16-byte-per-lane global -> LDS load: lane l's 16 bytes land at
// LDS byte address lds_base + 16*l.  Issued as assembly so that the compiler
// does not track it as an LDS write (it would otherwise wait for every such
// load before each LDS read); completion is awaited explicitly with
// wait_vmcnt before the barrier that publishes the stage.  M0 is set here and
// is not used by any other instruction of these kernels; the s_nop is the
// wait state the ISA requires between writing M0 and an LDS DMA reading it.
__device__ __forceinline__ void dma16(const void *g, const unsigned char *lds_slot0)
{
    const unsigned base = __builtin_amdgcn_readfirstlane(
        (unsigned)(size_t)(const __attribute__((address_space(3))) void *)lds_slot0);
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(base)
                 : "memory");
}

template <typename T, int BM, int BNC, int WAVES_M, int WAVES_N, int BKC, int STAGES>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) void qconv2d_igemm_dma(KArgs a)
{
    constexpr int EPC = Elem<T>::per_chunk;
    constexpr int NWAVES = WAVES_M * WAVES_N;
    constexpr int BN = 4 * BNC;
    constexpr int CPQ = BKC / EPC;
    constexpr int CPR = 4 * CPQ;
    constexpr int WTM = BM / WAVES_M;
    constexpr int WTN = BN / WAVES_N;
    constexpr int MB = WTM / 32;
    constexpr int NB = WTN / 32;
    constexpr int A_BYTES = BM * CPR * 16;
    constexpr int B_BYTES = 4 * BNC * CPQ * 16;
    constexpr int STAGE = A_BYTES + B_BYTES;
    constexpr int A_INSTR = A_BYTES / 1024;  // 1 KB wave-loads per stage
    constexpr int B_INSTR = B_BYTES / 1024;
    constexpr int A_PER_WAVE = A_INSTR / NWAVES;
    // Weight loads are dealt round-robin: wave w issues loads w, w+NWAVES, ...
    constexpr int B_MAX = (B_INSTR + NWAVES - 1) / NWAVES;
    constexpr int LPS_HI = A_PER_WAVE + B_MAX;  // loads per stage, waves with B_MAX weight loads
    constexpr int LPS_LO = B_INSTR % NWAVES == 0 ? LPS_HI : LPS_HI - 1;
    constexpr int A_ROWS_PER_INSTR = 64 / CPR;
    constexpr int B_ROWS_PER_INSTR = 64 / CPQ;
    static_assert(A_BYTES % 1024 == 0 && A_INSTR % NWAVES == 0, "activation stage must split into wave loads");
    static_assert(B_BYTES % 1024 == 0, "weight stage must be whole 1 KB wave loads");
    static_assert(CPR <= 64 && CPQ % 2 == 0, "stage geometry");
    static_assert(WTM % 32 == 0 && WTN % 32 == 0 && BNC % 4 == 0, "tile geometry");
    static_assert(STAGES >= 2, "need at least two stages");

    __shared__ __attribute__((aligned(1024))) unsigned char smem[STAGES * STAGE];
    auto ring = [&](int b) -> unsigned char * { return smem + b * STAGE; };

    const T *__restrict__ xp = static_cast<const T *>(a.x);
    const T *__restrict__ wp = static_cast<const T *>(a.wpack);
    const void *zero = g_qconv_zero16;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WAVES_M;
    const int wn = wave / WAVES_M;
    const int khalf = lane >> 5;
    const int l32 = lane & 31;

    const int nblk = gridDim.x;
    const int bid = blockIdx.x;
    const int per = nblk >> 3, rem = nblk & 7, xcd = bid & 7;
    const int tile = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + (bid >> 3);
    const int n_tile = tile % a.n_tiles;
    const int m0 = (tile / a.n_tiles) * BM;
    const int o0 = n_tile * BNC;

    // ---- per-lane activation load plan: A_PER_WAVE rows, one chunk each ----
    const int hw_out = a.h_out * a.w_out;
    int a_img[A_PER_WAVE], a_iy0[A_PER_WAVE], a_ix0[A_PER_WAVE];
    int a_coff[A_PER_WAVE];  // component offset + channel offset of the chunk
    int a_cin[A_PER_WAVE];   // channel offset of the chunk inside its component
#pragma unroll
    for (int i = 0; i < A_PER_WAVE; ++i) {
        const int r = (wave * A_PER_WAVE + i) * A_ROWS_PER_INSTR + lane / CPR;
        const int lc = (lane % CPR) ^ swz<CPR>(r);  // logical chunk this slot holds
        const int q = lc / CPQ, piece = lc % CPQ;
        a_coff[i] = q * a.c_in + piece * EPC;  // + cblk * BKC at each stage
        a_cin[i] = piece * EPC;
        const int m = m0 + r;
        if (m < a.m) {
            const int img = m / hw_out;
            const int rr = m - img * hw_out;
            const int oy = rr / a.w_out;
            const int ox = rr - oy * a.w_out;
            a_img[i] = img * a.h * a.w;
            a_iy0[i] = oy * a.s_h - a.p_h;
            a_ix0[i] = ox * a.s_w - a.p_w;
        } else {
            a_img[i] = 0;
            a_iy0[i] = -0x20000000;
            a_ix0[i] = 0;
        }
    }
    // ---- per-lane weight load plan ----
    const bool b_full = B_INSTR % NWAVES == 0 || wave < B_INSTR % NWAVES;  // issues B_MAX loads
    int b_off[B_MAX];  // element offset inside one stage's packed block
#pragma unroll
    for (int j = 0; j < B_MAX; ++j) {
        const int row = (wave + j * NWAVES) * B_ROWS_PER_INSTR + lane / CPQ;  // ws * BNC + o
        const int lc = (lane % CPQ) ^ swz<CPQ>(row);
        const int ws = row / BNC, o = row - (row / BNC) * BNC;
        b_off[j] = ws * a.cout_pad * BKC + (o0 + o) * BKC + lc * EPC;
    }
    const int row_elems = 4 * a.c_in;

    auto issue = [&](int s, int buf) {
        const int tap = s / a.n_cblk;
        const int cblk = s - tap * a.n_cblk;
        const int ky = tap / a.k_w;
        const int kx = tap - ky * a.k_w;
        const int dy = ky * a.d_h, dx = kx * a.d_w;
        const int cbase = cblk * BKC;
        unsigned char *As = ring(buf);
        unsigned char *Bs = As + A_BYTES;
#pragma unroll
        for (int i = 0; i < A_PER_WAVE; ++i) {
            const int iy = a_iy0[i] + dy;
            const int ix = a_ix0[i] + dx;
            const int c = a_coff[i] + cbase;
            const bool inside = (unsigned)iy < (unsigned)a.h && (unsigned)ix < (unsigned)a.w &&
                                cbase + a_cin[i] < a.c_in;
            const void *src = zero;
            if (inside)
                src = xp + ((a_img[i] + iy * a.w + ix) * row_elems + c);
            dma16(src, As + (wave * A_PER_WAVE + i) * 1024);
        }
        const T *wsrc = wp + (size_t)(tap * a.n_cblk + cblk) * 4 * a.cout_pad * BKC;
#pragma unroll
        for (int j = 0; j < B_MAX; ++j)
            if (j < B_MAX - 1 || b_full)
                dma16(wsrc + b_off[j], Bs + (wave + j * NWAVES) * 1024);
    };

    int frag_p[NB], frag_o[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int tn = wn * WTN + nb * 32 + l32;
        frag_p[nb] = tn / BNC;
        frag_o[nb] = tn - frag_p[nb] * BNC;
    }

    f32x16 acc[NB][MB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                acc[nb][mb][e] = 0.0f;

    auto compute = [&](int buf) {
        const unsigned char *As = ring(buf);
        const unsigned char *Bs = As + A_BYTES;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
            for (int kk = 0; kk < CPQ / 2; ++kk) {
                const int pc = kk * 2 + khalf;
                u32x4 wf[NB], pf[MB];
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    const int p = frag_p[nb];
                    const int row = (p ^ q) * BNC + frag_o[nb];
                    u32x4 v = *reinterpret_cast<const u32x4 *>(Bs + (row * CPQ + (pc ^ swz<CPQ>(row))) * 16);
                    const unsigned flip = ((kHamiltonNeg >> (4 * p + q)) & 1u) ? Elem<T>::sign : 0u;
                    v ^= flip;
                    wf[nb] = v;
                }
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) {
                    const int r = wm * WTM + mb * 32 + l32;
                    const int lc = q * CPQ + pc;
                    pf[mb] = *reinterpret_cast<const u32x4 *>(As + (r * CPR + (lc ^ swz<CPR>(r))) * 16);
                }
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb)
                        mfma_step<T>(acc[nb][mb], wf[nb], pf[mb]);
            }
        }
    };

    // ---- main loop: STAGES-deep ring, one barrier per stage ----
    const int S = a.stages;
#pragma unroll
    for (int u = 0; u < STAGES - 1; ++u)
        if (u < S)
            issue(u, u);
    for (int s0 = 0; s0 < S; s0 += STAGES) {
#pragma unroll
        for (int u = 0; u < STAGES; ++u) {
            const int s = s0 + u;
            if (s < S) {
                // Loads of stages s .. s+STAGES-2 may be in flight; wait for s.
                if (s + STAGES - 2 >= S)
                    wait_vmcnt<0>();
                else if (b_full)
                    wait_vmcnt<LPS_HI * (STAGES - 2)>();
                else
                    wait_vmcnt<LPS_LO * (STAGES - 2)>();
                block_barrier();
                if (s + STAGES - 1 < S)
                    issue(s + STAGES - 1, (u + STAGES - 1) % STAGES);
                compute(u);
            }
        }
    }

    // ---- epilogue: bias, round, channels-last store ----
    const T *__restrict__ bias = static_cast<const T *>(a.bias);
    T *__restrict__ out = static_cast<T *>(a.out);
    const bool vec_out = (a.c_out & 3) == 0;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int tn = wn * WTN + nb * 32 + 8 * g + 4 * khalf;
            const int p = tn / BNC;
            const int o = o0 + (tn - p * BNC);
            if (o >= a.c_out)
                continue;
            float bv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                bv[e] = (bias != nullptr && o + e < a.c_out) ? float(bias[p * a.c_out + o + e]) : 0.0f;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                const int m = m0 + wm * WTM + mb * 32 + l32;
                if (m >= a.m)
                    continue;
                T *dst = out + ((size_t)m * 4 * a.c_out + p * a.c_out + o);
                T v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    v[e] = T(acc[nb][mb][4 * g + e] + bv[e]);
                if (vec_out) {
                    if constexpr (sizeof(T) == 2) {
                        uint2 pk;
                        __builtin_memcpy(&pk, v, 8);
                        *reinterpret_cast<uint2 *>(dst) = pk;
                    } else {
                        float4 pk;
                        __builtin_memcpy(&pk, v, 16);
                        *reinterpret_cast<float4 *>(dst) = pk;
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (o + e < a.c_out)
                            dst[e] = v[e];
                }
            }
        }
    }
}

// Packs W_r, W_i, W_j, W_k (each OIHW) into [tap][cblk][kernel][cout_pad][bkc]
// so that one stage of one N-tile is four contiguous runs; padding is zero.
template <typename T>
__global__ __launch_bounds__(256) void qconv2d_pack(const T *__restrict__ w0, const T *__restrict__ w1,
                                                    const T *__restrict__ w2, const T *__restrict__ w3,
                                                    T *__restrict__ wp, int c_in, int c_out, int k_h,
                                                    int k_w, int n_cblk, int bkc, int cout_pad, int total)
{
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    int t = idx;
    const int cc = t % bkc;
    t /= bkc;
    const int o = t % cout_pad;
    t /= cout_pad;
    const int ws = t & 3;
    t >>= 2;
    const int cblk = t % n_cblk;
    const int tap = t / n_cblk;
    const int c = cblk * bkc + cc;
    const int ky = tap / k_w, kx = tap - (tap / k_w) * k_w;
    const T *src = ws == 0 ? w0 : ws == 1 ? w1 : ws == 2 ? w2 : w3;
    T v = T(0);
    if (o < c_out && c < c_in)
        v = src[((o * c_in + c) * k_h + ky) * k_w + kx];
    wp[idx] = v;
}

// ----------------------------- kernel table -------------------------------

struct KernelEntry {
    int bm, bnc, bkc, threads;
    DType dt;
    bool dma;  // pipelined direct-to-LDS kernel (needs c_in % vector == 0)
    const void *fn;
    const char *name;
};

#define QCONV_REG(T, DT, BM, BNC, WM, WN, BKC)                                                  \
    KernelEntry                                                                                 \
    {                                                                                           \
        BM, BNC, BKC, 64 * WM * WN, DT, false, (const void *)&qconv2d_igemm<T, BM, BNC, WM, WN, BKC>, \
            "reg_" #T "_bm" #BM "_bnc" #BNC "_w" #WM "x" #WN "_bkc" #BKC                        \
    }
#define QCONV_DMA(T, DT, BM, BNC, WM, WN, BKC, ST)                                                  \
    KernelEntry                                                                                     \
    {                                                                                               \
        BM, BNC, BKC, 64 * WM * WN, DT, true,                                                       \
            (const void *)&qconv2d_igemm_dma<T, BM, BNC, WM, WN, BKC, ST>,                          \
            "dma_" #T "_bm" #BM "_bnc" #BNC "_w" #WM "x" #WN "_bkc" #BKC "_s" #ST                   \
    }

// Every entry's BKC equals the pack block (16 bf16, 8 fp32) and its BNC
// divides kPackCoutAlign.
enum KernelId {
    kRegBf16N64 = 0,
    kRegBf16N32,
    kRegBf16N16,
    kRegF32,
    kDmaBf16M256N64,
    kDmaBf16M128N64,
    kDmaBf16M128N32,
    kDmaBf16M128N16,
    kDmaF32,
};
const KernelEntry kKernels[] = {
    QCONV_REG(__bf16, DType::BF16, 128, 64, 2, 2, 16),
    QCONV_REG(__bf16, DType::BF16, 128, 32, 2, 2, 16),
    QCONV_REG(__bf16, DType::BF16, 128, 16, 2, 2, 16),
    QCONV_REG(float, DType::F32, 64, 16, 2, 2, 8),
    QCONV_DMA(__bf16, DType::BF16, 256, 64, 4, 2, 16, 3),
    QCONV_DMA(__bf16, DType::BF16, 128, 64, 2, 2, 16, 3),
    QCONV_DMA(__bf16, DType::BF16, 128, 32, 2, 2, 16, 3),
    QCONV_DMA(__bf16, DType::BF16, 128, 16, 2, 2, 16, 3),
    QCONV_DMA(float, DType::F32, 64, 16, 2, 2, 8, 3),
};

}  // namespace

PackGeom qconv2d_pack_geom(int c_in, int c_out, int k_h, int k_w, DType dt)
{
    PackGeom pg;
    pg.pk = dt == DType::BF16 ? 16 : 8;
    pg.n_cblk = (c_in + pg.pk - 1) / pg.pk;
    pg.cout_pad = (c_out + kPackCoutAlign - 1) / kPackCoutAlign * kPackCoutAlign;
    const size_t esz = dt == DType::BF16 ? 2 : 4;
    pg.bytes = size_t(k_h) * k_w * pg.n_cblk * 4 * pg.cout_pad * pg.pk * esz;
    return pg;
}

ConvPlan qconv2d_plan(const ConvGeom &g, DType dt)
{
    const int epc = dt == DType::BF16 ? 8 : 4;
    const bool vec = g.c_in % epc == 0;
    const int64_t m = g.m();
    int id;
    if (dt == DType::F32) {
        id = vec ? kDmaF32 : kRegF32;
    } else if (g.c_out >= 64) {
        // 256-pixel tiles when they still give the 256 CUs two rounds of work.
        const int64_t tiles256 = (m + 255) / 256 * ((g.c_out + 63) / 64);
        id = !vec ? kRegBf16N64 : (tiles256 >= 512 ? kDmaBf16M256N64 : kDmaBf16M128N64);
    } else if (g.c_out > 16) {
        id = vec ? kDmaBf16M128N32 : kRegBf16N32;
    } else {
        id = vec ? kDmaBf16M128N16 : kRegBf16N16;
    }
    const KernelEntry &k = kKernels[id];
    ConvPlan p;
    p.id = id;
    p.bm = k.bm;
    p.bnc = k.bnc;
    p.n_tiles = (g.c_out + k.bnc - 1) / k.bnc;
    p.m_tiles = int((m + k.bm - 1) / k.bm);
    p.name = k.name;
    return p;
}

hipError_t qconv2d_pack_weights(const PackGeom &pg, int c_in, int c_out, int k_h, int k_w, DType dt,
                                const void *w_r, const void *w_i, const void *w_j, const void *w_k,
                                void *wpack, hipStream_t stream)
{
    const int total = int(pg.bytes / (dt == DType::BF16 ? 2 : 4));
    const int blocks = (total + 255) / 256;
    if (dt == DType::BF16)
        hipLaunchKernelGGL(qconv2d_pack<__bf16>, dim3(blocks), dim3(256), 0, stream,
                           (const __bf16 *)w_r, (const __bf16 *)w_i, (const __bf16 *)w_j,
                           (const __bf16 *)w_k, (__bf16 *)wpack, c_in, c_out, k_h, k_w, pg.n_cblk,
                           pg.pk, pg.cout_pad, total);
    else
        hipLaunchKernelGGL(qconv2d_pack<float>, dim3(blocks), dim3(256), 0, stream,
                           (const float *)w_r, (const float *)w_i, (const float *)w_j,
                           (const float *)w_k, (float *)wpack, c_in, c_out, k_h, k_w, pg.n_cblk,
                           pg.pk, pg.cout_pad, total);
    return hipGetLastError();
}

hipError_t qconv2d_run(const ConvPlan &plan, const PackGeom &pg, const ConvGeom &g, DType dt,
                       const void *x, const void *wpack, const void *bias, void *out,
                       hipStream_t stream)
{
    const KernelEntry &k = kKernels[plan.id];
    const int epc = dt == DType::BF16 ? 8 : 4;
    if (k.bkc != pg.pk || kPackCoutAlign % k.bnc != 0 || k.dt != dt || (k.dma && g.c_in % epc != 0))
        return hipErrorInvalidValue;
    KArgs a;
    a.x = x;
    a.wpack = wpack;
    a.bias = bias;
    a.out = out;
    a.c_in = g.c_in;
    a.h = g.h;
    a.w = g.w;
    a.c_out = g.c_out;
    a.k_w = g.k_w;
    a.s_h = g.s_h;
    a.s_w = g.s_w;
    a.p_h = g.p_h;
    a.p_w = g.p_w;
    a.d_h = g.d_h;
    a.d_w = g.d_w;
    a.h_out = g.h_out;
    a.w_out = g.w_out;
    a.m = int(g.m());
    a.stages = g.k_h * g.k_w * pg.n_cblk;
    a.n_cblk = pg.n_cblk;
    a.cout_pad = pg.cout_pad;
    a.n_tiles = plan.n_tiles;
    a.vec_in = (g.c_in % epc) == 0;
    void *args[] = {&a};
    const unsigned blocks = unsigned(plan.m_tiles) * unsigned(plan.n_tiles);
    return hipLaunchKernel(k.fn, dim3(blocks), dim3(k.threads), args, 0, stream);
}

}  // namespace quan
