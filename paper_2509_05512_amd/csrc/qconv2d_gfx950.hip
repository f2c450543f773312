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
// One work-group computes a tile of BM output pixels x 4*BNC output reals
// (all four output components of BNC channels):
//   - K runs over stages.  A stage is QS input components x CS channels with
//     QS*CS*sizeof(T) = 128 bytes, so each activation row of a stage is one
//     contiguous 128-byte piece of the channels-last pixel (full cache lines);
//   - only the four shared real kernels are staged: an LDS weight block holds
//     W_0..W_3 [BNC][CS] for one (tap, channel block) and serves all 4/QS
//     stages of that block.  The signed 4x4 Hamilton block is formed on the
//     LDS->register read: the fragment for (output component p, input
//     component q) reads kernel p xor q and flips its sign bits with one XOR;
//   - global -> LDS direct loads (global_load_lds_dwordx4) fill a ring of three
//     activation stages and two weight blocks two stages ahead; the layout in
//     LDS is XOR-swizzled so the MFMA fragment reads are bank-conflict free.
//     Taps outside the image read a zero chunk;
//   - fragments of the next k-step are read from LDS while the current
//     k-step's MFMAs run; the next loads are issued after the stage's last LDS
//     read (an LDS DMA holds back later LDS reads of its wave until it lands);
//   - v_mfma_f32_32x32x16_bf16 (bf16) / v_mfma_f32_32x32x2f32 (fp32), fp32
//     accumulators; epilogue adds the bias, rounds to the output type (RNE)
//     and stores channels-last.
#include <hip/hip_runtime.h>

#include <cstdlib>

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

// XOR swizzle of the 16-byte chunk index within an LDS row of CPR chunks.
// A ds_read_b128 from a wave reads one chunk from each of 16 consecutive rows
// per group of 16 lanes (256 bytes, the full bank width) and from 8
// consecutive rows per group of 8 lanes (128 bytes); the swizzle puts every
// such group on distinct 16-byte bank slots in both views, so the MFMA
// fragment reads are conflict free.
template <int CPR>
__device__ __forceinline__ int swz(int row)
{
    static_assert(CPR == 2 || CPR == 4 || CPR == 8 || CPR == 16, "swizzle defined for 32..256-byte rows");
    if constexpr (CPR == 16)
        return row & 15;
    else if constexpr (CPR == 8)
        return (row & 7) ^ ((row >> 3) & 1);
    else if constexpr (CPR == 4)
        return ((row >> 1) ^ (row >> 3)) & 3;
    else
        return ((row >> 2) ^ (row >> 3)) & 1;
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

// Stage geometry of the pipelined kernel: a K stage is QS input components
// x CS channels, chosen so that one activation row of a stage is exactly one
// contiguous 128-byte segment of the channels-last pixel.  The weight block
// of a (tap, channel block) -- the four real kernels W_0..W_3 for BNC output
// channels x CS input channels -- serves all 4/QS stages of that block.
template <typename T, int QS>
struct StageGeom {
    static constexpr int EPC = Elem<T>::per_chunk;
    static constexpr int CS = 128 / (QS * int(sizeof(T)));  // channels per component
    static constexpr int CPQ = CS / EPC;                     // chunks per component
    static constexpr int NQG = 4 / QS;                       // stages per weight block
};

template <typename T, int BM, int BNC, int WAVES_M, int WAVES_N, int QS>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) void qconv2d_igemm_dma(KArgs a)
{
    using SG = StageGeom<T, QS>;
    constexpr int EPC = SG::EPC;
    constexpr int CS = SG::CS;
    constexpr int CPQ = SG::CPQ;
    constexpr int NQG = SG::NQG;
    constexpr int NWAVES = WAVES_M * WAVES_N;
    constexpr int BN = 4 * BNC;
    constexpr int CPR = 8;  // 128-byte activation rows
    constexpr int WTM = BM / WAVES_M;
    constexpr int WTN = BN / WAVES_N;
    constexpr int MB = WTM / 32;
    constexpr int NB = WTN / 32;
    constexpr int A_ST = 3;                   // activation ring
    constexpr int B_ST = NQG == 1 ? 3 : 2;    // weight-block ring
    constexpr int A_BYTES = BM * 128;
    constexpr int B_BYTES = 4 * BNC * CPQ * 16;
    constexpr int A_INSTR = A_BYTES / 1024;  // 1 KB wave loads per stage
    constexpr int B_INSTR = B_BYTES / 1024;  // 1 KB wave loads per weight block
    constexpr int A_PER_WAVE = A_INSTR / NWAVES;
    constexpr int B_MAX = (B_INSTR + NWAVES - 1) / NWAVES;  // round-robin over waves
    constexpr int LB_HI = B_MAX;
    constexpr int LB_LO = B_INSTR % NWAVES == 0 ? B_MAX : B_MAX - 1;
    constexpr int B_ROWS_PER_INSTR = 64 / CPQ;
    constexpr int KSTEPS = 4;  // 32x32 MFMA k-steps per stage (two chunks each)
    static_assert(A_INSTR % NWAVES == 0, "activation stage must split into wave loads");
    static_assert(B_BYTES % 1024 == 0, "weight block must be whole 1 KB wave loads");
    static_assert(WTM % 32 == 0 && WTN % 32 == 0 && BNC % 4 == 0, "tile geometry");
    static_assert(QS * CPQ == 8, "a stage row is eight chunks");

    __shared__ __attribute__((aligned(1024))) unsigned char smem[A_ST * A_BYTES + B_ST * B_BYTES];
    unsigned char *const a_ring = smem;
    unsigned char *const b_ring = smem + A_ST * A_BYTES;

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
    // a_off: element offset of the chunk at tap (0, 0), channel block 0,
    // component group 0 (only used when the tap lies inside the image).
    const int hw_out = a.h_out * a.w_out;
    const int row_elems = 4 * a.c_in;
    int a_off[A_PER_WAVE], a_iy0[A_PER_WAVE], a_ix0[A_PER_WAVE], a_cin[A_PER_WAVE];
#pragma unroll
    for (int i = 0; i < A_PER_WAVE; ++i) {
        const int r = (wave * A_PER_WAVE + i) * 8 + lane / 8;
        const int lc = (lane % 8) ^ swz<CPR>(r);  // logical chunk this slot holds
        const int qi = lc / CPQ, piece = lc % CPQ;
        a_cin[i] = piece * EPC;
        const int m = m0 + r;
        if (m < a.m) {
            const int img = m / hw_out;
            const int rr = m - img * hw_out;
            const int oy = rr / a.w_out;
            const int ox = rr - oy * a.w_out;
            a_iy0[i] = oy * a.s_h - a.p_h;
            a_ix0[i] = ox * a.s_w - a.p_w;
            a_off[i] = ((img * a.h + a_iy0[i]) * a.w + a_ix0[i]) * row_elems + qi * a.c_in + piece * EPC;
        } else {
            a_iy0[i] = -0x20000000;  // rows past M never load
            a_ix0[i] = 0;
            a_off[i] = 0;
        }
    }
    // ---- per-lane weight load plan ----
    const bool b_full = B_INSTR % NWAVES == 0 || wave < B_INSTR % NWAVES;  // issues B_MAX loads
    int b_off[B_MAX];
#pragma unroll
    for (int j = 0; j < B_MAX; ++j) {
        const int row = (wave + j * NWAVES) * B_ROWS_PER_INSTR + lane / CPQ;  // ws * BNC + o
        const int lc = (lane % CPQ) ^ swz<CPQ>(row);
        const int ws = row / BNC, o = row - (row / BNC) * BNC;
        b_off[j] = ws * a.cout_pad * CS + (o0 + o) * CS + lc * EPC;
    }

    // Loads of stage s: its weight block first when s opens a block, then the
    // activation tile.
    auto issue = [&](int s) {
        const int blk = s / NQG;
        const int qg = s - blk * NQG;
        if (qg == 0) {
            unsigned char *Bs = b_ring + (blk % B_ST) * B_BYTES;
            const T *wsrc = wp + (size_t)blk * 4 * a.cout_pad * CS;
#pragma unroll
            for (int j = 0; j < B_MAX; ++j)
                if (j < B_MAX - 1 || b_full)
                    dma16(wsrc + b_off[j], Bs + (wave + j * NWAVES) * 1024);
        }
        const int tap = blk / a.n_cblk;
        const int cblk = blk - tap * a.n_cblk;
        const int ky = tap / a.k_w;
        const int kx = tap - ky * a.k_w;
        const int dy = ky * a.d_h, dx = kx * a.d_w;
        const int cbase = cblk * CS;
        const int shift = (dy * a.w + dx) * row_elems + qg * QS * a.c_in + cbase;  // uniform
        unsigned char *As = a_ring + (s % A_ST) * A_BYTES;
#pragma unroll
        for (int i = 0; i < A_PER_WAVE; ++i) {
            const bool inside = (unsigned)(a_iy0[i] + dy) < (unsigned)a.h &&
                                (unsigned)(a_ix0[i] + dx) < (unsigned)a.w && cbase + a_cin[i] < a.c_in;
            const void *src = inside ? (const void *)(xp + (a_off[i] + shift)) : zero;
            dma16(src, As + (wave * A_PER_WAVE + i) * 1024);
        }
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

    // The eight chunks of a stage row form four 32x32 k-steps; k-step j uses
    // chunks 2*(j % (CPQ/2)) + {0, 1} of local component j / (CPQ/2), i.e.
    // input component q = qbase + j / (CPQ/2).
    auto read_frags = [&](const unsigned char *As, const unsigned char *Bs, int qbase, int j,
                          u32x4 (&wf)[NB], u32x4 (&pf)[MB]) {
        const int qi = j / (CPQ / 2);
        const int pc = 2 * (j % (CPQ / 2)) + khalf;
        const int q = qbase + qi;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const int row = (frag_p[nb] ^ q) * BNC + frag_o[nb];
            wf[nb] = *reinterpret_cast<const u32x4 *>(Bs + (row * CPQ + (pc ^ swz<CPQ>(row))) * 16);
        }
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const int r = wm * WTM + mb * 32 + l32;
            const int lc = qi * CPQ + pc;
            pf[mb] = *reinterpret_cast<const u32x4 *>(As + (r * CPR + (lc ^ swz<CPR>(r))) * 16);
        }
    };
    // Sign of block (p, q) applied to the weight fragment, then the MFMAs.
    auto mfmas = [&](int qbase, int j, u32x4 (&wf)[NB], const u32x4 (&pf)[MB]) {
        const int q = qbase + j / (CPQ / 2);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const unsigned flip = ((kHamiltonNeg >> (4 * frag_p[nb] + q)) & 1u) ? Elem<T>::sign : 0u;
            wf[nb] ^= flip;
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
                mfma_step<T>(acc[nb][mb], wf[nb], pf[mb]);
    };

    // ---- main loop: loads run two stages ahead, one barrier per stage ----
    // Within a stage the fragments of k-step j+1 are read before the MFMAs of
    // k-step j (scheduling fences keep that order).  The loads of stage s+2
    // are issued once every LDS read of stage s has been issued: an LDS DMA
    // holds back the issuing wave's later LDS reads until it lands, so issued
    // there it only has to land before the next stage's reads, with the
    // remaining MFMAs of this stage in between.
    const int S = a.stages;
    issue(0);
    if (S > 1)
        issue(1);
    for (int s = 0; s < S; ++s) {
        // Wait for the loads of stage s; only those of stage s+1 (issued in
        // the previous step: a weight block if s+1 opens one, then the
        // activations) may stay in flight.
        if (s + 1 >= S) {
            wait_vmcnt<0>();
        } else if ((s + 1) % NQG != 0) {
            wait_vmcnt<A_PER_WAVE>();
        } else if (b_full) {
            wait_vmcnt<A_PER_WAVE + LB_HI>();
        } else {
            wait_vmcnt<A_PER_WAVE + LB_LO>();
        }
        block_barrier();
        const int blk = s / NQG;
        const unsigned char *As = a_ring + (s % A_ST) * A_BYTES;
        const unsigned char *Bs = b_ring + (blk % B_ST) * B_BYTES;
        const int qbase = (s - blk * NQG) * QS;
        u32x4 wf0[NB], pf0[MB], wf1[NB], pf1[MB];
        read_frags(As, Bs, qbase, 0, wf0, pf0);
        read_frags(As, Bs, qbase, 1, wf1, pf1);
        __builtin_amdgcn_sched_barrier(0);
        mfmas(qbase, 0, wf0, pf0);
        __builtin_amdgcn_sched_barrier(0);
        read_frags(As, Bs, qbase, 2, wf0, pf0);
        __builtin_amdgcn_sched_barrier(0);
        mfmas(qbase, 1, wf1, pf1);
        __builtin_amdgcn_sched_barrier(0);
        read_frags(As, Bs, qbase, 3, wf1, pf1);
        __builtin_amdgcn_sched_barrier(0);
        // Stage s+2 reuses buffers every wave finished before this step's
        // barrier.
        if (s + 2 < S)
            issue(s + 2);
        __builtin_amdgcn_sched_barrier(0);
        mfmas(qbase, 2, wf0, pf0);
        __builtin_amdgcn_sched_barrier(0);
        mfmas(qbase, 3, wf1, pf1);
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
    if (tap < k_h * k_w && o < c_out && c < c_in)  // the zero tail past the last tap stays 0
        v = src[((o * c_in + c) * k_h + ky) * k_w + kx];
    wp[idx] = v;
}

// ----------------------------- kernel table -------------------------------

struct KernelEntry {
    int bm, bnc, qs, threads;  // qs: input components per K stage (pack block = 128 B / qs)
    DType dt;
    bool dma;  // pipelined direct-to-LDS kernel (needs c_in % vector == 0)
    const void *fn;
    const char *name;
};

#define QCONV_REG(T, DT, BM, BNC, WM, WN, BKC)                                                 \
    KernelEntry                                                                                \
    {                                                                                          \
        BM, BNC, 4, 64 * WM * WN, DT, false, (const void *)&qconv2d_igemm<T, BM, BNC, WM, WN, BKC>, \
            "reg_" #T "_bm" #BM "_bnc" #BNC "_w" #WM "x" #WN "_bkc" #BKC                       \
    }
#define QCONV_DMA(T, DT, BM, BNC, WM, WN, QS)                                                     \
    KernelEntry                                                                                   \
    {                                                                                             \
        BM, BNC, QS, 64 * WM * WN, DT, true, (const void *)&qconv2d_igemm_dma<T, BM, BNC, WM, WN, QS>, \
            "dma_" #T "_bm" #BM "_bnc" #BNC "_w" #WM "x" #WN "_qs" #QS                            \
    }
#define QCONV_DMA3(T, DT, BM, BNC, WM, WN) \
    QCONV_DMA(T, DT, BM, BNC, WM, WN, 1), QCONV_DMA(T, DT, BM, BNC, WM, WN, 2), QCONV_DMA(T, DT, BM, BNC, WM, WN, 4)

// Register-staged kernels use the 4-component stage (qs 4); every entry's BNC
// divides kPackCoutAlign.  DMA entries come in qs = 1, 2, 4 triples.
enum KernelId {
    kRegBf16N64 = 0,
    kRegBf16N32,
    kRegBf16N16,
    kRegF32,
    kDmaBf16M256N64 = 4,   // +0/+1/+2 for qs 1/2/4
    kDmaBf16M128N64 = 7,
    kDmaBf16M128N32 = 10,
    kDmaBf16M128N16 = 13,
    kDmaF32M64N16 = 16,
    kNumKernels = 19,
};
const KernelEntry kKernels[] = {
    QCONV_REG(__bf16, DType::BF16, 128, 64, 2, 2, 16),
    QCONV_REG(__bf16, DType::BF16, 128, 32, 2, 2, 16),
    QCONV_REG(__bf16, DType::BF16, 128, 16, 2, 2, 16),
    QCONV_REG(float, DType::F32, 64, 16, 2, 2, 8),
    QCONV_DMA3(__bf16, DType::BF16, 256, 64, 4, 2),
    QCONV_DMA3(__bf16, DType::BF16, 128, 64, 2, 2),
    QCONV_DMA3(__bf16, DType::BF16, 128, 32, 2, 2),
    QCONV_DMA3(__bf16, DType::BF16, 128, 16, 2, 2),
    QCONV_DMA3(float, DType::F32, 64, 16, 2, 2),
};
static_assert(sizeof(kKernels) / sizeof(kKernels[0]) == kNumKernels, "kernel table");

int qs_index(int qs)
{
    return qs == 1 ? 0 : (qs == 2 ? 1 : 2);
}

// Input components per stage for c_in: the widest 128-byte stage whose
// channel block divides c_in (no zero padding), else the narrowest.
int choose_qs(int c_in, DType dt)
{
    const int es = dt == DType::BF16 ? 2 : 4;
    const int epc = 16 / es;
    if (c_in % epc != 0)
        return 4;
    for (int qs : {1, 2})
        if (c_in % (128 / (qs * es)) == 0)
            return qs;
    return 4;
}

}  // namespace

PackGeom qconv2d_pack_geom(int c_in, int c_out, int k_h, int k_w, DType dt)
{
    PackGeom pg;
    const int es = dt == DType::BF16 ? 2 : 4;
    pg.pk = 128 / (choose_qs(c_in, dt) * es);
    pg.n_cblk = (c_in + pg.pk - 1) / pg.pk;
    pg.cout_pad = (c_out + kPackCoutAlign - 1) / kPackCoutAlign * kPackCoutAlign;
    pg.zero_offset = size_t(k_h) * k_w * pg.n_cblk * 4 * pg.cout_pad * pg.pk * es;
    pg.bytes = pg.zero_offset + kPackZeroTail;
    return pg;
}

ConvPlan qconv2d_plan(const ConvGeom &g, DType dt)
{
    const int epc = dt == DType::BF16 ? 8 : 4;
    const bool vec = g.c_in % epc == 0;
    const int qi = qs_index(choose_qs(g.c_in, dt));
    const int64_t m = g.m();
    int id;
    if (dt == DType::F32) {
        id = vec ? kDmaF32M64N16 + qi : kRegF32;
    } else if (g.c_out >= 64) {
        // 256-pixel tiles when they still give the 256 CUs two rounds of work.
        const int64_t tiles256 = (m + 255) / 256 * ((g.c_out + 63) / 64);
        id = !vec ? kRegBf16N64 : (tiles256 >= 512 ? kDmaBf16M256N64 : kDmaBf16M128N64) + qi;
    } else if (g.c_out > 16) {
        id = vec ? kDmaBf16M128N32 + qi : kRegBf16N32;
    } else {
        id = vec ? kDmaBf16M128N16 + qi : kRegBf16N16;
    }
#ifdef QUAN_TUNING
    // Tuning builds only: force a tile family (QUAN_QCONV_KERNEL=<id of its
    // qs-1 entry>); the qs member still follows c_in.
    if (const char *force = getenv("QUAN_QCONV_KERNEL")) {
        const int f = atoi(force);
        if (f >= kDmaBf16M256N64 && f < kNumKernels && kKernels[f].dt == dt && vec)
            id = f + qi;
    }
#endif
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
    const int es = dt == DType::BF16 ? 2 : 4;
    if (128 / (k.qs * es) != pg.pk || kPackCoutAlign % k.bnc != 0 || k.dt != dt ||
        (k.dma && g.c_in % epc != 0))
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
    a.stages = g.k_h * g.k_w * pg.n_cblk * (k.dma ? 4 / k.qs : 1);
    a.n_cblk = pg.n_cblk;
    a.cout_pad = pg.cout_pad;
    a.n_tiles = plan.n_tiles;
    a.vec_in = (g.c_in % epc) == 0;
    void *args[] = {&a};
    const unsigned blocks = unsigned(plan.m_tiles) * unsigned(plan.n_tiles);
    return hipLaunchKernel(k.fn, dim3(blocks), dim3(k.threads), args, 0, stream);
}

}  // namespace quan
