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
//   - K runs over stages.  A stage is one tap and one block of CS channels
//     of all four input components, 4*CS*sizeof(T) = 128 bytes: each
//     activation row of a stage is one contiguous 128-byte piece of the
//     channels-last pixel (one cache line);
//   - only the four shared real kernels are staged: a stage's weights are
//     W_0..W_3 [BNC][CS] (4*BNC rows of 32 bytes).  The signed 4x4 Hamilton
//     block is formed on the LDS->register read: the fragment for (output
//     component p, input component q) reads kernel p xor q and flips its
//     sign bits with one XOR;
//   - the work-group is four compute waves and two producer waves (four
//     for the separable form and narrow tiles).  The producers move stages from global
//     memory straight into LDS (buffer_load ... lds, 1 KB per instruction;
//     each producer moves its share of every stage), three stages ahead of
//     the compute waves, into a four-stage ring.  One wave can keep at most
//     63 loads in flight (its 6-bit vmcnt), too few to cover the latency at
//     this bandwidth, hence more than one producer.  Rows outside the image
//     read past the buffer range and land as zeros.  Compute waves only read
//     fragments from LDS and issue MFMAs, one fragment read between
//     consecutive MFMAs (a burst of LDS reads stalls the matrix pipe);
//   - one barrier per stage, in the middle of the compute waves' step: the
//     fragments of the next stage's first k-step are read after it while the
//     current stage's last MFMAs run;
//   - v_mfma_f32_32x32x16_bf16 (bf16) / v_mfma_f32_32x32x2f32 (fp32), fp32
//     accumulators in AGPRs; the epilogue adds the bias, rounds to the output
//     type (RNE) and stores channels-last.
#include <hip/hip_runtime.h>

#include <mutex>
#include <type_traits>

#include "gfx950_dma.h"
#include "quan_launch.h"

namespace quan {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));


// Bit 4*p + q is set when the separable form (eq. 7) subtracts W_q (*) x_q
// from output component p.  Row r: + - - -, row i: + + + -, row j: + - + +,
// row k: + + - +.
constexpr unsigned kSeparableNeg =
    (1u << 1) | (1u << 2) | (1u << 3) | (1u << 7) | (1u << 9) | (1u << 14);

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

// Channels per component in one stage (4 components x CS x sizeof(T) = 128 B).
template <typename T>
constexpr int stage_channels()
{
    return 128 / (4 * int(sizeof(T)));
}

struct KArgs {
    const void *x;
    const void *wpack;
    const void *bias;
    void *out;
    int c_in, h, w, c_out, k_h, k_w;
    int s_h, s_w, p_h, p_w, d_h, d_w;
    int h_out, w_out;
    int m;       // n * h_out * w_out output pixels
    int stages;  // taps * n_cblk
    int n_cblk;
    int cout_pad;
    int m_tiles, n_tiles;
    // Work split of a persistent launch: the first full_tiles tiles are
    // dealt to the work-groups (full_tiles = m_tiles * n_tiles unless
    // tail_blocks is non-zero).  tail_blocks (the 64-channel all-components
    // tile with DMA loads, Hamilton form, one N-tile, full_tiles a multiple
    // of the grid of at least one tile and 8 steps per work-group,
    // tail_blocks <= grid): the 32-pixel blocks past
    // those tiles; each work-group claims one once its tiles are nearly
    // done, so the first to get there take them, and its four waves then
    // compute one output component of the block each.  claim (tail_blocks >
    // 0): claim[0] the claim counter, zero when the launch starts and left
    // zero by its last claimant; claim[1 + b] work-group b's mailbox, its
    // ticket posted as (epoch << 16) | ticket; epoch: the launch's tag (16
    // bits, not 0), which tells a post of this launch from an earlier one.
    int full_tiles, tail_blocks;
    unsigned *claim;
    unsigned epoch;
    unsigned w_bytes;   // bytes of packed weights
    long long x_elems;  // elements of x (n * h * w * 4 * c_in)
    // Optional IQBN statistics of the output, per run of consecutive output
    // pixels (an M-tile, or with ALLP waves a tile's 32-pixel sub-tile):
    // stats[0][col][t] = mean and stats[1][col][t] = sum of squared
    // deviations of column col = p * c_out + o over run t's pixels (after
    // rounding to T).  Written only by kernels with the deferred epilogue;
    // NULL: none.
    float *stats;
    int stat_tiles;  // partials per column: ceil(m / rows per partial)
    // Optional per-column affine map applied in the epilogue instead of the
    // bias (inference IQBN folded in): out = scale[col] * acc + shift[col],
    // then max(0, .) when relu is non-zero.  NULL scale: out = acc + bias.
    const float *scale;
    const float *shift;
    int relu;
};

// Work-groups a launch with tail blocks may have (the claim buffer's
// mailboxes).
constexpr int kClaimMaxGroups = 2048;

// XOR swizzle of the 16-byte chunk index within an LDS row of CPR chunks.
// A ds_read_b128 from a wave reads one chunk from each of 16 consecutive rows
// per group of 16 lanes (256 bytes, the full bank width) and from 8
// consecutive rows per group of 8 lanes (128 bytes); the swizzle puts every
// such group on distinct 16-byte bank slots in both views, so the MFMA
// fragment reads are conflict free.  It depends on row % 16 only, so a row
// offset by a multiple of 16 keeps its swizzle.
template <int CPR>
__device__ __forceinline__ int swz(int row)
{
    static_assert(CPR == 2 || CPR == 8, "swizzle defined for 32- and 128-byte rows");
    if constexpr (CPR == 8)
        return (row & 7) ^ ((row >> 3) & 1);
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

// Instruction classes of __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedValu = 0x002, kSchedMfma = 0x008, kSchedDsRead = 0x100;

// Orders one k-step's scheduling region: the VALU sign flips first, then
// every MFMA followed by up to RPM LDS reads while any remain.  A burst of
// LDS reads between MFMA groups stalls the matrix pipe on gfx950; a few reads
// behind each MFMA hide it, and issuing them early in the k-step gives them
// time to land before the next k-step needs them.
template <int NMFMA, int NFLIP, int NDSR, int RPM = 2>
__device__ __forceinline__ void interleave_kstep()
{
    if constexpr (NFLIP > 0)
        __builtin_amdgcn_sched_group_barrier(kSchedValu, NFLIP, 0);
#pragma unroll
    for (int i = 0; i < NMFMA; ++i) {
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
#pragma unroll
        for (int r = 0; r < RPM; ++r)
            if (i * RPM + r < NDSR)
                __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
    }
    if constexpr (NDSR > NMFMA * RPM)
        __builtin_amdgcn_sched_group_barrier(kSchedDsRead, NDSR - NMFMA * RPM, 0);
}

// One work-group: WAVES_M x WAVES_N compute waves, each MB x NB blocks of 32
// pixels x 32 output reals, and NPROD producer waves.  Tile: BM = 32*MB*WAVES_M
// pixels x BN = 32*NB*WAVES_N output reals (BN/4 output channels, all four
// components).  VEC: c_in is a multiple of the 16-byte chunk, so activations
// move by DMA; otherwise the producer loads partial chunks element-wise.
// EPI: what the epilogue applies (kEpiBias, kEpiStats, kEpiFold); fixed at
// compile time so the common bias-only kernel carries none of the others'
// state through its main loop.
//
// SEP: the separable convolution of eq. 7 instead of the Hamilton product.
// Each wave then keeps the four real convolutions c_q = W_q (*) x_q of its
// MB x NB blocks (32 pixels x 32 output channels each) in separate
// accumulators: k-step q multiplies only x_q by W_q (a quarter of the
// Hamilton MFMAs), and the epilogue mixes y_p = sum_q S[p][q] c_q in fp32.
// The tile is BM pixels x BN/4 = 32*NB*WAVES_N output channels, all four
// output components.
//
// PAIR (separable form, bf16, c_in a multiple of 32): a stage's 128-byte
// activation row is 32 channels of two input components (q = 2*pair,
// 2*pair + 1) instead of 16 channels of all four, so every 64-byte request
// the L1 sends to L2 is fully used (half the requests per stage).  The
// stages of a tap alternate pair 0 and 1 over the 32-channel blocks; the
// separable form needs only W_q beside x_q, so a stage's weights are still
// four 16-channel row groups (kernel 2*pair + g/2, channel half g%2).
// K-step j of a stage then belongs to component 2*pair + j/2.
enum : int { kEpiBias = 0, kEpiStats = 1, kEpiFold = 2 };
// Producer waves per work-group.  A tile with few MFMAs per stage (the
// separable form, a quarter of the Hamilton MFMAs; tiles of 32 or fewer
// output channels) runs at the pace of its activation loads, and four
// producers, each issuing half as many DMA instructions per stage, make it
// 3-33% faster; the 64-channel Hamilton tile gains nothing and keeps two.
// Four need every stage's activation and weight DMAs to split evenly.
template <typename T, int MB, int NB, int WM, int WN, bool SEP, bool ALLP = false>
constexpr int producer_waves()
{
    constexpr int bnc = (SEP || ALLP) ? 32 * NB * WN : 8 * NB * WN;  // output channels per tile
    constexpr int cs = 128 / (4 * int(sizeof(T)));                   // channels per stage
    constexpr int a_instr = 32 * MB * WM / 8;
    constexpr int b_instr = 4 * bnc * cs * int(sizeof(T)) / 1024;
    return ((SEP || bnc <= 32) && a_instr % 4 == 0 && b_instr % 4 == 0) ? 4 : 2;
}
// ALLP (Hamilton form, bf16): each compute wave holds 32 pixels x all four
// output components of the tile's BNC = 32*NB channels (4 x NB accumulator
// blocks), instead of all BM pixels of one component.  A stage's four kernel
// fragments are then read once and serve all sixteen Hamilton blocks, and
// one activation fragment (input component q) feeds the four blocks of its
// column of eq. 6: a quarter of the LDS fragment reads per MFMA of the
// one-component layout's k-steps for weights, and one activation read per
// k-step instead of MB.  The MFMAs of a stage run grouped by kernel m = p xor q,
// so a group needs only W_m: the fragments of W_2 and W_3 are read while the
// groups of W_0 and W_1 run.  Negative entries of eq. 6 use a sign-flipped
// copy of the activation fragment (one XOR per dword).
// FORM (Hamilton layouts, not SEP): which signed kernel block (p, q) of the
// 4x4 block weight holds.  kFormHamilton: eq. 6, kernel p xor q with the
// Hamilton sign.  kFormSepGrad: the input gradient of the separable form
// (eqs. 8-10), dX_p = sum_q M[p][q] (W'_p (*) dY_q) with the backward mixing
// matrix M = S^T (S eq. 7's signs): kernel p with sign M[p][q] = S[q][p], so
// the mixing is accumulated in fp32 with the products.
enum : int { kFormHamilton = 0, kFormSepGrad = 1 };
// POINCARE (the stem layer, one input channel, element-wise loads): x is
// the colour planes [N][3][H][W] of the input images, and the producer
// forms the input quaternion of eq. 4 at each tap pixel, q = ((1 - n2), 2r,
// 2g, 2b) / (1 + n2) with n2 = r^2 + g^2 + b^2, in fp32 rounded once to T,
// instead of reading a mapped activation: the quaternion map never goes to
// memory.
template <typename T, int MB, int NB, int WAVES_M, int WAVES_N, bool VEC, int EPI, bool SEP, bool PAIR = false,
          bool ALLP = false, int FORM = kFormHamilton, bool POINCARE = false>
__global__ __launch_bounds__(64 * (WAVES_M * WAVES_N + producer_waves<T, MB, NB, WAVES_M, WAVES_N, SEP, ALLP>())) void qconv2d_igemm(KArgs a)
{
    constexpr int ES = int(sizeof(T));
    constexpr int EPC = Elem<T>::per_chunk;
    constexpr int CS = stage_channels<T>();
    constexpr int CPQ = CS / EPC;  // 16-byte chunks per component (2)
    constexpr int NCW = WAVES_M * WAVES_N;
    constexpr int NPROD = producer_waves<T, MB, NB, WAVES_M, WAVES_N, SEP, ALLP>();
    constexpr int WTM = 32 * MB;
    constexpr int WTN = 32 * NB;
    constexpr int BM = WTM * WAVES_M;
    constexpr int BN = ((SEP || ALLP) ? 4 : 1) * WTN * WAVES_N;  // output reals per tile
    constexpr int BNC = BN / 4;
    constexpr int QS = (SEP || ALLP) ? 4 : 1;  // accumulator sets per block
    constexpr int NBUF = 4;                     // stages in the LDS ring
    constexpr int A_BYTES = BM * 128;           // one stage of activations
    constexpr int B_BYTES = 4 * BNC * CS * ES;  // one stage of weights
    constexpr int A_INSTR = BM / 8;             // DMA instructions per stage (8 rows of 128 B each)
    constexpr int B_INSTR = B_BYTES / 1024;
    // DMA instructions of one producer per stage (producer pr takes the
    // instructions with index = pr mod NPROD)
    constexpr int PER_STAGE = (A_INSTR + NPROD - 1) / NPROD + (B_INSTR + NPROD - 1) / NPROD;
    constexpr int LOOKAHEAD = 3;                // stages issued ahead of the one being read
    constexpr int N_MFMA = MB * NB * (ES == 2 ? 1 : 4);  // MFMA instructions per k-step
    // Tail blocks (see KArgs) are taken by the 64-channel DMA tile (two
    // producers) only, and carry two K-blocks per ring slot: a tail stage
    // fills only rows 0..31 of the slot's
    // activation region, so K-block t's activations go to rows 0..31, K-block
    // t+1's to rows 32..63 and K-block t+1's weights (laid out as in the
    // weight region) to the region's upper half, which the A instructions
    // of rows 64..127 load instead.  A producer issues as many instructions
    // per step as for a tile, and a tail block takes ceil(S / 2) steps.
    constexpr bool TAIL2 = ALLP && FORM == kFormHamilton && VEC && !POINCARE && NPROD == 2 &&
                           A_INSTR == 2 * B_INSTR && A_BYTES == 2 * B_BYTES;
    constexpr bool P_UNIFORM = BNC >= 32;       // a 32-wide N block lies in one output component
    static_assert(CPQ == 2 && CS * 4 * ES == 128, "stage row is 128 bytes");
    static_assert(BNC % 16 == 0 && kPackCoutAlign % BNC == 0 && B_BYTES % 1024 == 0, "tile geometry");
    static_assert(LOOKAHEAD * PER_STAGE <= 63, "the stages in flight must fit the vmcnt counter");
    static_assert(A_INSTR % NPROD == 0 && B_INSTR % NPROD == 0, "producers split every stage evenly");
    static_assert(!PAIR || (SEP && VEC && ES == 2), "paired stages: separable bf16 with 16-byte chunks");
    static_assert(BNC == ((SEP || ALLP) ? 32 * NB * WAVES_N : 8 * NB * WAVES_N) && CS == 128 / (4 * ES),
                  "producer_waves sees the tile geometry");
    static_assert(!ALLP || (!SEP && !PAIR && ES == 2 && MB == 1 && WAVES_N == 1),
                  "all-components waves: Hamilton form, bf16, 32 pixels per wave");
    static_assert(FORM == kFormHamilton || (!SEP && EPI == kEpiBias), "block tables: Hamilton layouts, bias epilogue");
    static_assert(!POINCARE || (!VEC && !SEP && EPI == kEpiBias), "Poincare stem: element loads, bias epilogue");
    // kernel component and sign of block (output p, input q)
    auto blk_kernel = [](int p, int q) { return FORM == kFormHamilton ? (p ^ q) : p; };
    auto blk_neg = [](int p, int q) -> bool {
        return FORM == kFormHamilton ? ((kHamiltonNeg >> (4 * p + q)) & 1u) : ((kSeparableNeg >> (4 * q + p)) & 1u);
    };

    // Deferred epilogue (DEFER): when a wave holds one output component for
    // all BM pixels, it parks each finished tile in its own LDS region and
    // drains it with full-line 16-byte stores during the next tile's steps,
    // instead of every work-group writing its tile at the same moment.
    // With ALLP a wave parks its 32 pixels x all four components (rows of
    // 4 x BNC values, component-major) and drains them itself.  The 16-byte
    // chunks of one component's BNC values are XOR-swizzled with the pixel
    // index modulo SWZ (their count), which spreads a wave's park stores
    // over the banks and leaves the component segments in place.
    constexpr bool DEFER = ALLP || (WAVES_M == 1 && WTN == BNC && P_UNIFORM && !SEP);
    constexpr int SWZ = BNC * ES / 16;                  // chunks of one component's channels
    constexpr int OUT_ROW = (ALLP ? 4 : 1) * BNC * ES;  // bytes of one pixel in a wave's region
    constexpr int OUT_CPR = OUT_ROW / 16;               // 16-byte chunks per pixel
    constexpr int OUT_PIX = ALLP ? WTM : BM;            // pixels of a wave's region
    constexpr int OUT_WAVE = OUT_PIX * OUT_ROW;
    constexpr int N_DRAIN = OUT_WAVE / 1024;  // 1 KB stores per wave per tile
    constexpr int PPS = 64 / OUT_CPR;         // pixels per drain store
    constexpr int OUT_BYTES = DEFER ? NCW * OUT_WAVE : 0;
    static_assert(!DEFER || (OUT_CPR >= 2 && PPS >= 1 && (ALLP || PPS % OUT_CPR == 0)), "drain geometry");

    __shared__ __attribute__((aligned(1024))) unsigned char smem[NBUF * (A_BYTES + B_BYTES) + OUT_BYTES];
    unsigned char *const a_lds = smem;
    unsigned char *const b_lds = smem + NBUF * A_BYTES;
    unsigned char *const o_lds = smem + NBUF * (A_BYTES + B_BYTES);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    // Persistent work-groups (at most one per tile).  Work-groups are dealt
    // to the 8 XCDs round-robin, block b to XCD b % 8; XCD x owns a
    // contiguous range of tiles in proportion to its work-groups, so
    // neighbouring tiles share its L2, and its work-groups take that range's
    // tiles in turn.  The split only steers locality: every tile belongs to
    // exactly one work-group whatever the placement.
    const int n_wg = gridDim.x, bid = blockIdx.x;
    const int xcd = bid & 7, xslot = bid >> 3;
    const int cnt_x = (n_wg >> 3) + (xcd < (n_wg & 7) ? 1 : 0);
    const int before_x = xcd * (n_wg >> 3) + (xcd < (n_wg & 7) ? xcd : (n_wg & 7));
    const int tiles = a.full_tiles;
    const int x_lo = int((long long)tiles * before_x / n_wg);
    const int x_hi = int((long long)tiles * (before_x + cnt_x) / n_wg);
    const int n_mine = x_hi - x_lo > xslot ? (x_hi - x_lo - xslot + cnt_x - 1) / cnt_x : 0;
    // (with tail blocks every work-group has at least one tile, so none
    // leaves here and every one takes part in the claims)
    if (n_mine == 0)
        return;  // the whole work-group leaves: no barrier is pending
    auto tile_of = [&](int k) { return x_lo + xslot + k * cnt_x; };
    const bool tails = TAIL2 && a.tail_blocks > 0;
    // first pixel of tail block c
    auto tail_m0 = [&](int c) { return ((BM / WTM) * a.full_tiles + c) * WTM; };
    const int S = a.stages;
    const int ST = TAIL2 ? (S + 1) / 2 : S;  // steps of a tail block

    if (wave >= NCW) {
        // ================= producer waves =================
        const int pr = wave - NCW;
        const int hw_out = a.h_out * a.w_out;
        const int row_elems = 4 * a.c_in;
        const long long img_elems = (long long)a.h * a.w * row_elems;
        const unsigned a_base = lds_addr(a_lds), b_base = lds_addr(b_lds);
        const unsigned w_stage_bytes = unsigned(4 * a.cout_pad * CS * ES);
        constexpr int A_MINE = A_INSTR / NPROD, B_MINE = B_INSTR / NPROD;

        // Issue cursor: tile k (of this work-group), stage t of that tile at
        // tap (ky, kx) and channel block cblk, and the tile's DMA plan.
        int k = 0, ky = 0, kx = 0, cblk = 0;
        int n_items = n_mine;  // items known so far: the tiles, then each claimed tail block
        const T *xt = nullptr;
        unsigned x_bytes = 0;  // bytes of x from xt on (capped at 2^31 - 1)
        int p_off[A_MINE], p_iy[A_MINE], p_ix[A_MINE], p_cl[A_MINE];
        int p_comp[A_MINE];  // POINCARE: the quaternion component of the lane's chunk
        unsigned p_woff[B_MINE];
        int p_wodd[B_MINE];  // PAIR: the instruction's channel half
        // Activation DMA i covers rows 8i..8i+7 of the tile: lane l loads
        // row 8i + l/8 into physical chunk l%8, i.e. logical chunk
        // lc = (l%8) ^ swz(row): component lc/2, channels 8*(lc%2).. of the
        // stage's channel block (bf16; 4*(lc%2).. for fp32).  Offsets are
        // relative to the first image of the tile.  Weight DMA j covers LDS
        // slots 64j..64j+63 of the stage's weights: slot = row * 2 +
        // physical chunk, row = kernel * BNC + o.
        // (item kt past the tiles: tail block c)
        auto plan_tile = [&](int kt, int c) {
            const int m0 = kt < n_mine ? (tile_of(kt) / a.n_tiles) * BM : tail_m0(c);
            const int o0 = kt < n_mine ? (tile_of(kt) % a.n_tiles) * BNC : 0;
            const int img0 = m0 / hw_out;
            xt = static_cast<const T *>(a.x) + img0 * (POINCARE ? 3LL * a.h * a.w : img_elems);
            const long long rest = (a.x_elems - img0 * img_elems) * ES;
            x_bytes = rest <= 0 ? 0u : (rest < 0x7fffffffLL ? unsigned(rest) : 0x7fffffffu);
#pragma unroll
            for (int ii = 0; ii < A_MINE; ++ii) {
                const int i = ii * NPROD + pr;  // instruction index within the stage
                const int row = 8 * i + (lane >> 3);
                const int lc = (lane & 7) ^ swz<8>(row);
                // PAIR: chunks 0-3 are component 2*pair, 4-7 component 2*pair+1
                const int comp = PAIR ? lc / 4 : lc / CPQ, cin = PAIR ? (lc % 4) * EPC : (lc % CPQ) * EPC;
                // (TAIL2 tail block: rows 32..63 hold the block's rows 0..31
                // again, for the second K-block; the same swizzle)
                const int m = m0 + ((TAIL2 && kt >= n_mine) ? 8 * (i & 3) + (lane >> 3) : row);
                p_cl[ii] = a.c_in - cin;  // channels of this chunk left before block 0
                p_comp[ii] = comp;
                if (m < a.m) {
                    const int img = m / hw_out;
                    const int rr = m - img * hw_out;
                    const int oy = rr / a.w_out;
                    const int ox = rr - oy * a.w_out;
                    p_iy[ii] = oy * a.s_h - a.p_h;
                    p_ix[ii] = ox * a.s_w - a.p_w;
                    const int e = (((img - img0) * a.h + p_iy[ii]) * a.w + p_ix[ii]) * row_elems +
                                  comp * a.c_in + cin;
                    p_off[ii] = VEC ? e * ES : e;
                    if constexpr (POINCARE)  // the pixel's red sample in the planes [img][3][h][w]
                        p_off[ii] = ((img - img0) * 3 * a.h + p_iy[ii]) * a.w + p_ix[ii];
                } else {
                    p_iy[ii] = -0x20000000;  // rows past M never load
                    p_ix[ii] = 0;
                    p_off[ii] = 0;
                }
            }
#pragma unroll
            for (int jj = 0; jj < B_MINE; ++jj) {
                const int j = jj * NPROD + pr;
                const int slot = 64 * j + lane;
                const int row = slot / CPQ;
                const int lc = (slot % CPQ) ^ swz<CPQ>(row);
                const int ws = row / BNC, o = row - (row / BNC) * BNC;
                if constexpr (PAIR) {
                    // row group ws: kernel 2*pair + ws/2 of channel block
                    // 2*(cblk/2) + ws%2 (one group per instruction)
                    p_woff[jj] = unsigned((((ws >> 1) * a.cout_pad + o0 + o) * CS + lc * EPC) * ES);
                    p_wodd[jj] = ws & 1;
                } else {
                    p_woff[jj] = unsigned(((ws * a.cout_pad + o0 + o) * CS + lc * EPC) * ES);
                }
            }
        };
        // Tail block: when its cursor passes the end of its last tile,
        // producer 0 claims one: lane 0 takes a ticket from the counter and
        // posts it, with the launch tag, in the work-group's mailbox.  Both
        // atomics return before the producer goes on, so the post is in
        // memory before its next barrier; after that barrier both producers
        // read it (at the top of their next iteration: resolve_claim) and
        // the compute waves (after the last tile).  A ticket below
        // tail_blocks is the block; the last of the grid's tickets (every
        // work-group claims once) sets the counter back to zero for the next
        // launch.  (System scope, as every access to the claim buffer.)  The
        // claim comes at step n_mine * S - 1, issued in iteration n_mine * S
        // - 4 >= 0 (the host takes tail blocks only then), so a barrier
        // always lies between post and read.
        unsigned *const mbox = a.claim + 1 + bid;
        bool pending = false;  // cursor past the last tile, the claim not yet read
        auto post_claim = [&]() {
            unsigned c = 0;
            if (lane == 0)
                c = __hip_atomic_fetch_add(a.claim, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
            c = __builtin_amdgcn_readfirstlane(c);
            unsigned posted = 0;
            if (lane == 0)
                posted = __hip_atomic_exchange(mbox, (a.epoch << 16) | c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
            asm volatile("" ::"v"(posted));  // wait for the exchange
            if (c == unsigned(n_wg) - 1 && lane == 0)
                __hip_atomic_exchange(a.claim, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        };
        plan_tile(0, 0);
        // Issues the cursor's stage into ring slot g % NBUF and advances the
        // cursor (to the next item after its last stage).
        // The cursor one K-block on; past an item's last one, to the next
        // item (or, past the last tile, the claim of a tail block).
        auto advance = [&]() {
            if (++cblk == a.n_cblk) {
                cblk = 0;
                if (++kx == a.k_w) {
                    kx = 0;
                    if (++ky == a.k_h) {
                        ++k;
                        if (k < n_items) {
                            ky = 0;
                            plan_tile(k, 0);
                        } else if (tails && k == n_mine) {
                            if (pr == 0)
                                post_claim();
                            pending = true;
                        }
                    }
                }
            }
        };
        // TAIL2 tail step: K-blocks t and t + 1 (the second past the last
        // K-block on an odd stage count: its loads land as zeros, unread).
        auto issue_tail2 = [&](int buf) {
            const int t = (ky * a.k_w + kx) * a.n_cblk + cblk;
            const bool two = t + 1 < S;
            int cb2 = cblk + 1, kx2 = kx, ky2 = ky;
            if (cb2 == a.n_cblk) {
                cb2 = 0;
                if (++kx2 == a.k_w) {
                    kx2 = 0;
                    ++ky2;
                }
            }
#pragma unroll
            for (int jj = 0; jj < B_MINE; ++jj)
                dma16(a.wpack, a.w_bytes, p_woff[jj], unsigned(t) * w_stage_bytes,
                      b_base + buf * B_BYTES + (jj * NPROD + pr) * 1024);
            const int dy = ky * a.d_h, dx = kx * a.d_w, cbase = cblk * CS;
            const int dy2 = ky2 * a.d_h, dx2 = kx2 * a.d_w, cbase2 = cb2 * CS;
            const int shift = (dy * a.w + dx) * row_elems + cbase;
            const int shift2 = (dy2 * a.w + dx2) * row_elems + cbase2;
#pragma unroll
            for (int ii = 0; ii < A_MINE; ++ii) {
                const int i = ii * NPROD + pr;  // ii >= A_MINE / 2: i >= 8; ii >= A_MINE / 4: i >= 4
                if (ii >= A_MINE / 2) {
                    // K-block t + 1's weights, to the upper half of the slot's activation region
                    dma16(a.wpack, a.w_bytes, two ? p_woff[ii - A_MINE / 2] : 0x80000000u,
                          two ? unsigned(t + 1) * w_stage_bytes : 0u, a_base + buf * A_BYTES + i * 1024);
                } else {
                    const bool second = ii >= A_MINE / 4;
                    const int ddy = second ? dy2 : dy, ddx = second ? dx2 : dx;
                    const bool inside = ((unsigned)(p_iy[ii] + ddy) < (unsigned)a.h) &
                                        ((unsigned)(p_ix[ii] + ddx) < (unsigned)a.w) &
                                        ((second ? cbase2 : cbase) < p_cl[ii]) & (!second || two);
                    const unsigned off = inside ? unsigned(p_off[ii] + (second ? shift2 : shift) * ES) : 0x80000000u;
                    dma16(xt, x_bytes, off, 0u, a_base + buf * A_BYTES + i * 1024);
                }
            }
            // the cursor one or two K-blocks on; the tail block is a
            // work-group's last item, so its end only moves k past it
            bool end = false;
            for (int r = 0; r < (two ? 2 : 1); ++r) {
                if (++cblk == a.n_cblk) {
                    cblk = 0;
                    if (++kx == a.k_w) {
                        kx = 0;
                        end = ++ky == a.k_h;
                    }
                }
            }
            if (end)
                ++k;
        };
        auto issue = [&](int g) {
            const int buf = g & (NBUF - 1);
            if constexpr (TAIL2) {
                if (k >= n_mine) {
                    issue_tail2(buf);
                    return;
                }
            }
            const int t = (ky * a.k_w + kx) * a.n_cblk + cblk;  // stage within the tile
#pragma unroll
            for (int jj = 0; jj < B_MINE; ++jj) {
                if constexpr (PAIR)
                    dma16(a.wpack, a.w_bytes, p_woff[jj],
                          unsigned(t - (cblk & 1) + p_wodd[jj]) * w_stage_bytes +
                              unsigned(cblk & 1) * (w_stage_bytes / 2),
                          b_base + buf * B_BYTES + (jj * NPROD + pr) * 1024);
                else
                    dma16(a.wpack, a.w_bytes, p_woff[jj], unsigned(t) * w_stage_bytes,
                          b_base + buf * B_BYTES + (jj * NPROD + pr) * 1024);
            }
            // PAIR: stage cblk is channels 32*(cblk/2).. of components
            // 2*(cblk%2) and 2*(cblk%2) + 1
            const int dy = ky * a.d_h, dx = kx * a.d_w, cbase = PAIR ? (cblk >> 1) * 2 * CS : cblk * CS;
            const int shift = (dy * a.w + dx) * row_elems + cbase + (PAIR ? (cblk & 1) * 2 * a.c_in : 0);  // elements
#pragma unroll
            for (int ii = 0; ii < A_MINE; ++ii) {
                const int i = ii * NPROD + pr;
                const bool inside = ((unsigned)(p_iy[ii] + dy) < (unsigned)a.h) &
                                    ((unsigned)(p_ix[ii] + dx) < (unsigned)a.w) & (cbase < p_cl[ii]);
                if constexpr (VEC) {
                    const unsigned off = inside ? unsigned(p_off[ii] + shift * ES) : 0x80000000u;
                    dma16(xt, x_bytes, off, 0u, a_base + buf * A_BYTES + i * 1024);
                } else if constexpr (POINCARE) {
                    // one input channel: the lane of component q's first chunk
                    // holds q's value in element 0, everything else is zero
                    u32x4 v = {0u, 0u, 0u, 0u};
                    if (inside) {
                        const int hw = a.h * a.w;
                        const T *px = xt + p_off[ii] + dy * a.w + dx;
                        const float r = float(px[0]), g = float(px[hw]), b = float(px[2 * hw]);
                        const float n2 = r * r + g * g + b * b;
                        const float den = 1.0f + n2;
                        const int qc = p_comp[ii];
                        const float num = qc == 0 ? 1.0f - n2 : 2.0f * (qc == 1 ? r : qc == 2 ? g : b);
                        T e[Elem<T>::per_chunk];
#pragma unroll
                        for (int k = 0; k < Elem<T>::per_chunk; ++k)
                            e[k] = T(0);
                        e[0] = T(num / den);
                        __builtin_memcpy(&v, e, 16);
                    }
                    *reinterpret_cast<u32x4 *>(a_lds + buf * A_BYTES + i * 1024 + lane * 16) = v;
                } else {
                    u32x4 v = {0u, 0u, 0u, 0u};
                    if (inside)
                        v = load_chunk_masked<T>(xt + (p_off[ii] + shift), p_cl[ii] - cbase);
                    *reinterpret_cast<u32x4 *>(a_lds + buf * A_BYTES + i * 1024 + lane * 16) = v;
                }
            }
            advance();
        };
        // Waits until all but this producer's DMAs of the `later` most
        // recently issued stages have landed.
        auto wait_landed = [&](int later) {
            if constexpr (VEC) {
                if (later >= 2)
                    wait_vmcnt<2 * PER_STAGE>();
                else if (later == 1)
                    wait_vmcnt<PER_STAGE>();
                else
                    wait_vmcnt<0>();
            } else {
                wait_vmcnt<0>();
            }
        };
        // steps of the items known so far (claims add to them as the
        // cursor reaches the end of the tiles)
        auto total = [&]() { return n_mine * S + (n_items - n_mine) * ST; };
        // prologue: steps 0..2; step 0 lands before the first barrier
        for (int g = 0; g < LOOKAHEAD && g < total(); ++g)
            issue(g);
        wait_landed(total() - 1 < LOOKAHEAD - 1 ? total() - 1 : LOOKAHEAD - 1);
        __syncthreads();
        // Iteration g: step g+3 goes into the slot step g-1 left before the
        // barrier of step g-1; step g+1 lands before the barrier of step g,
        // after which the compute waves first read it.  Steps run on across
        // tiles, so the next tile's first stages arrive during this tile's
        // last steps and epilogue.
        // the claim posted before the last barrier: a block is item k
        auto resolve_claim = [&]() {
            const unsigned v = __builtin_amdgcn_readfirstlane(
                __hip_atomic_load(mbox, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM));
            const unsigned c = v & 0xffffu;
            pending = false;
            if ((v >> 16) == a.epoch && c < unsigned(a.tail_blocks)) {
                ++n_items;
                ky = 0;
                plan_tile(k, int(c));
            }
        };
        for (int g = 0; g < total(); ++g) {
            if (pending)
                resolve_claim();
            if (g + LOOKAHEAD < total())
                issue(g + LOOKAHEAD);
            wait_landed(g + 3 < total() ? 2 : (g + 2 < total() ? 1 : 0));
            __syncthreads();
        }
        return;
    }

    // ================= compute waves =================
    const int wm = wave % WAVES_M;
    const int wn = wave / WAVES_M;
    const int khalf = lane >> 5;
    const int l32 = lane & 31;

    // K-step j of a stage is input component q = j: chunks 2j + {0, 1} of the
    // activation row and chunks {0, 1} of weight row (p ^ j) * BNC + o (the
    // Hamilton block), or j * BNC + o (separable: W_j only).  Lane l reads
    // chunk 2j + l/32 (activations) / chunk l/32 (weights) of row l%32 of
    // its 32-row block.
    int a_rd[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
        a_rd[j] = (wm * WTM + l32) * 128 + (((2 * j + khalf) ^ swz<8>(l32)) * 16);
    // When all N blocks of a wave lie in one output component (SHARED_P),
    // block nb's weight rows are block 0's plus 32*nb: an immediate offset.
    constexpr bool SHARED_P = SEP || ALLP || (P_UNIFORM && WTN <= BNC);
    constexpr int NB_RD = SHARED_P ? 1 : NB;
    int b_rd[NB_RD][4];
    unsigned flip[NB][4];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        if constexpr (SEP || ALLP) {
            // row j * BNC + o: kernel j (separable: the k-step's own kernel;
            // ALLP: kernel m = j, read once per stage)
            const int o = wn * WTN + nb * 32 + l32;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (nb < NB_RD)
                    b_rd[nb][j] = (j * BNC + o) * CPQ * 16 + ((khalf ^ swz<CPQ>(o)) * 16);
                flip[nb][j] = 0u;
            }
        } else {
            const int tn = wn * WTN + nb * 32 + l32;
            const int p = P_UNIFORM ? __builtin_amdgcn_readfirstlane(tn / BNC) : tn / BNC;
            const int o = tn % BNC;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int row = blk_kernel(p, j) * BNC + o;
                if (nb < NB_RD)
                    b_rd[nb][j] = row * CPQ * 16 + ((khalf ^ swz<CPQ>(o)) * 16);
                flip[nb][j] = blk_neg(p, j) ? Elem<T>::sign : 0u;
            }
        }
    }

    f32x16 acc[QS][NB][MB];
    struct Frags {
        u32x4 w[NB];
        u32x4 p[MB];
    };
    auto read_frags = [&](int buf, int j, Frags &f) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const int rd = SHARED_P ? b_rd[0][j] + nb * 32 * CPQ * 16 : b_rd[nb < NB_RD ? nb : 0][j];
            f.w[nb] = *reinterpret_cast<const u32x4 *>(b_lds + buf * B_BYTES + rd);
        }
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
            f.p[mb] = *reinterpret_cast<const u32x4 *>(a_lds + buf * A_BYTES + mb * 32 * 128 + a_rd[j]);
    };
    // Sign of block (p, q = j) applied to the weight fragments, then the
    // MFMAs (separable: into the accumulators of c_j, no signs).
    auto mfmas = [&](int j, Frags &f) {
        if constexpr (SEP) {
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
                    mfma_step<T>(acc[j][nb][mb], f.w[nb], f.p[mb]);
        } else {
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                f.w[nb] ^= flip[nb][j];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
                    mfma_step<T>(acc[0][nb][mb], f.w[nb], f.p[mb]);
        }
    };

    // ---- all-components waves (ALLP): stage fragments ----
    // xa0 / xa1: this wave's 32 pixels of input components 0..3 for
    // alternate stages; xn: sign-flipped copies of the current stage's; wk[m]:
    // the tile's rows of kernel m.  Block (p, q) of eq. 6 multiplies
    // W_{p xor q} by x_q into output component p's accumulators.
    u32x4 xa0[4][MB], xa1[4][MB], xn[4][MB], wk[4][NB];
    auto rd_act = [&](unsigned off, u32x4 (&dst)[4][MB]) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
                dst[q][mb] = *reinterpret_cast<const u32x4 *>(a_lds + off + mb * 32 * 128 + a_rd[q]);
    };
    auto rd_ker = [&](unsigned off, int m, u32x4 (&dst)[NB]) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
            dst[nb] = *reinterpret_cast<const u32x4 *>(b_lds + off + b_rd[0][m] + nb * 32 * CPQ * 16);
    };
    auto flip_act = [&](const u32x4 (&src)[MB], u32x4 (&dst)[MB]) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
            dst[mb] = src[mb] ^ Elem<T>::sign;
    };
    // the four blocks of kernel M: (q xor M, q) for the Hamilton product,
    // (M, q) for the separable input gradient, q = 0..3
    auto group = [&](auto mc, const u32x4 (&x)[4][MB], const u32x4 (&xneg)[4][MB], const u32x4 (&w)[NB]) {
        constexpr int M = decltype(mc)::value;
        // (compiled into the all-components kernels only; the others hold
        // one component's accumulators and never call it)
        if constexpr (ALLP)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int p = FORM == kFormHamilton ? q ^ M : M;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) {
                    if (blk_neg(p, q))
                        mfma_step<T>(acc[p][nb][mb], w[nb], xneg[q][mb]);
                    else
                        mfma_step<T>(acc[p][nb][mb], w[nb], x[q][mb]);
                }
        }
    };

    // ---- deferred-epilogue drain ----
    // Store i of a wave's region covers pixels i*PPS + l/OUT_CPR, chunk
    // l%OUT_CPR (its physical chunk is XOR-swizzled with the pixel).  Stores
    // past N_DRAIN, pixels past M and channels past c_out get an offset
    // outside the buffer and are dropped.
    constexpr int CPC = 16 / ES;  // channels per 16-byte chunk
    const bool defer = DEFER && a.c_out % CPC == 0;
    const int region = ALLP ? wm : wn;  // the wave's parking region
    const int d_pix = lane / OUT_CPR, d_chk = lane % OUT_CPR;
    // ALLP: logical chunk d_chk is component d_chk / SWZ, chunk d_chk % SWZ
    // of its channels; the swizzle then depends on the store's pixel
    const int d_p = d_chk / SWZ, d_k = d_chk % SWZ;
    const unsigned char *const d_lds =
        ALLP ? o_lds + region * OUT_WAVE
             : o_lds + region * OUT_WAVE + d_pix * OUT_ROW + ((d_chk ^ (d_pix % OUT_CPR)) * 16);
    const int row_bytes = 4 * a.c_out * ES;
    int d_next = N_DRAIN;        // next store of the pending tile
    const T *d_base = nullptr;   // pending tile: first pixel's output row
    unsigned d_bytes = 0;        // bytes of output from d_base on (capped)
    unsigned d_lane = 0;         // lane's byte offset in a store, or out of range
    auto drain_read = [&](int i) {
        const int ic = i < N_DRAIN ? i : N_DRAIN - 1;
        if constexpr (ALLP) {
            const int pix = ic * PPS + d_pix;
            return *reinterpret_cast<const u32x4 *>(d_lds + pix * OUT_ROW + ((d_p * SWZ + (d_k ^ (pix % SWZ))) * 16));
        } else {
            return *reinterpret_cast<const u32x4 *>(d_lds + ic * 1024);
        }
    };
    // The stores carry device scope (sc1): each line goes on to memory as it
    // is written, instead of every dirty line of the L2 being written back
    // by the release at the kernel's end (measured on MI355X: 3x3 stride-2
    // layer 76-79 -> 71-74 us, 1x1 layer 30.6-31.6 -> 29.1 us, the
    // 64 x 56 x 56 layer with IQBN behind it 271.7 -> 269 us; non-temporal
    // stores were as fast alone but slowed the IQBN pass that reads them).
    constexpr int kStoreDeviceScope = 16;
    auto drain_store = [&](int i, u32x4 v) {
        const unsigned off = (i < N_DRAIN && d_lane != 0x80000000u)
                                 ? d_lane + unsigned(i * (64 / OUT_CPR) * row_bytes)
                                 : 0x80000000u;
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), make_rsrc(d_base, d_bytes), off, 0,
                                               kStoreDeviceScope);
    };

    // Step g (its stage in ring slot g % 4):
    //   k-step 0 on f0, reading k-step 1 into f1;
    //   k-step 1 on f1, reading k-step 2 into f0;
    //   k-step 2 on f0, reading k-step 3 into f1;
    //   barrier (step g+1's stage has landed; step g's is read no more);
    //   k-step 3 on f1, reading step g+1's k-step 0 into f0.
    // Past the last step that read fetches unused data from an idle slot.
    //
    // Separable form: a k-step has only MB x NB MFMAs, too few to cover one
    // fragment read, so each read is issued two k-steps ahead into one of
    // four fragment sets (fa..fd hold k-steps 0..3):
    //   k-step 0 on fa, reading k-step 2 into fc;
    //   k-step 1 on fb, reading k-step 3 into fd;
    //   barrier;
    //   k-step 2 on fc, reading step g+1's k-step 0 into fa;
    //   k-step 3 on fd, reading step g+1's k-step 1 into fb.
    //
    // All-components waves (ALLP): a stage's 16 x NB x MB MFMAs run in four
    // groups by kernel m (group m: blocks (q xor m, q), q = 0..3), with the
    // stage's activations and W_0, W_1 read during the previous stage:
    //   group 0 (W_0; sign flips of x_1..x_3), reading W_2;
    //   group 1 (W_1), reading W_3;
    //   barrier;
    //   group 2 (W_2), reading step g+1's x_0..x_3 and W_0;
    //   group 3 (W_3), reading step g+1's W_1.
    constexpr int N_READ = MB + NB;
    constexpr int N_FLIP = SEP ? 0 : NB * 4;
    Frags f0, f1;
    Frags fc, fd;  // separable form only
    __syncthreads();
    if constexpr (ALLP) {
        rd_act(0, xa0);
        rd_ker(0, 0, wk[0]);
        rd_ker(0, 1, wk[1]);
    } else {
        read_frags(0, 0, f0);
    }
    if constexpr (SEP)
        read_frags(0, 1, f1);
    using G0 = std::integral_constant<int, 0>;
    using G1 = std::integral_constant<int, 1>;
    using G2 = std::integral_constant<int, 2>;
    using G3 = std::integral_constant<int, 3>;
    constexpr int G_MFMA = 4 * NB * MB;  // MFMAs of one kernel group
    // ALLP steps keep the ring slot at run time (one wave-uniform value, a
    // few address adds per stage) rather than unrolling the tile loop per
    // ring phase: the phase copies of the loop cost more registers than an
    // ALLP wave has to spare.
    int slot = 0;  // ring slot of the next ALLP step's stage
    auto step_allp = [&](const u32x4 (&cur)[4][MB], u32x4 (&nxt)[4][MB]) {
        const int ns = (slot + 1) & (NBUF - 1);
        const unsigned cb = unsigned(slot) * B_BYTES;
        const unsigned na = unsigned(ns) * A_BYTES, nb_ = unsigned(ns) * B_BYTES;
        u32x4 dv0;
        if constexpr (DEFER)
            dv0 = drain_read(d_next);
        __builtin_amdgcn_sched_barrier(0);
        rd_ker(cb, 2, wk[2]);
        if constexpr (FORM != kFormHamilton)
            flip_act(cur[0], xn[0]);  // eq. 6 never negates input component r
        flip_act(cur[1], xn[1]);
        flip_act(cur[2], xn[2]);
        flip_act(cur[3], xn[3]);
        group(G0{}, cur, xn, wk[0]);
        interleave_kstep<G_MFMA, (FORM == kFormHamilton ? 12 : 16) * MB, NB>();
        __builtin_amdgcn_sched_barrier(0);
        rd_ker(cb, 3, wk[3]);
        group(G1{}, cur, xn, wk[1]);
        interleave_kstep<G_MFMA, 0, NB>();
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (DEFER) {
            drain_store(d_next, dv0);
            d_next = d_next < N_DRAIN ? d_next + 1 : N_DRAIN;
        }
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        rd_act(na, nxt);
        rd_ker(nb_, 0, wk[0]);
        group(G2{}, cur, xn, wk[2]);
        interleave_kstep<G_MFMA, 0, 4 * MB + NB>();
        __builtin_amdgcn_sched_barrier(0);
        rd_ker(nb_, 1, wk[1]);
        group(G3{}, cur, xn, wk[3]);
        interleave_kstep<G_MFMA, 0, NB>();
        __builtin_amdgcn_sched_barrier(0);
        slot = ns;
    };
    // Tail block: the work-group's 32 pixels and wave wm computes output
    // component p = wm alone, block (p, q = p xor m) of each kernel group m
    // (a quarter of a tile's MFMAs per wave), with the sign of eq. 6 for that
    // block.
    // TAIL2 tail step: the slot's K-block t (activation rows 0..31, the
    // weight region) and, with `two`, K-block t + 1 (rows 32..63, weights in
    // the activation region's upper half); every fragment is read after the
    // previous step's barrier, the slot is free after this one's.
    auto step_tail2 = [&](bool two) {
        const int ns = slot + 1 == NBUF ? 0 : slot + 1;
        const unsigned char *const ab = a_lds + unsigned(slot) * A_BYTES;
        const unsigned char *const bb = b_lds + unsigned(slot) * B_BYTES;
        u32x4 dv0;
        if constexpr (DEFER)
            dv0 = drain_read(d_next);
        auto kblock = [&](const unsigned char *act, const unsigned char *ker) {
            u32x4 x[4], w[4][NB];
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int q = wm ^ m;
                x[m] = *reinterpret_cast<const u32x4 *>(act + l32 * 128 + (((2 * q + khalf) ^ swz<8>(l32)) * 16));
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
                    w[m][nb] = *reinterpret_cast<const u32x4 *>(ker + b_rd[0][m] + nb * 32 * CPQ * 16);
            }
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const unsigned fl = ((kHamiltonNeg >> (4 * wm + (wm ^ m))) & 1u) ? Elem<T>::sign : 0u;
                const u32x4 xs = x[m] ^ fl;
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
                    mfma_step<T>(acc[0][nb][0], w[m][nb], xs);
            }
        };
        kblock(ab, bb);
        if (two)
            kblock(ab + 32 * 128, ab + A_BYTES / 2);
        if constexpr (DEFER) {
            drain_store(d_next, dv0);
            d_next = d_next < N_DRAIN ? d_next + 1 : N_DRAIN;
        }
        __syncthreads();
        slot = ns;
    };
    // One tile: its S steps, two per iteration (activation sets alternate);
    // an odd last step leaves the next stage's activations in xa1, moved
    // back to xa0.
    auto run_tile_allp = [&](auto stepf) {
        int t = 0;
        for (; t + 2 <= S; t += 2) {
            stepf(xa0, xa1);
            stepf(xa1, xa0);
        }
        if (t < S) {
            stepf(xa0, xa1);
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
                    xa0[q][mb] = xa1[q][mb];
        }
    };
    auto step_sep = [&](auto slot) {
        constexpr int B = decltype(slot)::value;
        // accumulator set of k-step j: component j, or with paired stages
        // component 2*pair + j/2, pair = the stage's parity (every tile has
        // an even number of stages, so it equals the ring slot's)
        constexpr int QA0 = PAIR ? 2 * (B & 1) : 0, QA1 = PAIR ? 2 * (B & 1) : 1;
        constexpr int QA2 = PAIR ? 2 * (B & 1) + 1 : 2, QA3 = PAIR ? 2 * (B & 1) + 1 : 3;
        __builtin_amdgcn_sched_barrier(0);
        read_frags(B, 2, fc);
        mfmas(QA0, f0);
        interleave_kstep<N_MFMA, 0, N_READ, 1>();
        __builtin_amdgcn_sched_barrier(0);
        read_frags(B, 3, fd);
        mfmas(QA1, f1);
        interleave_kstep<N_MFMA, 0, N_READ, 1>();
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        read_frags((B + 1) & (NBUF - 1), 0, f0);
        mfmas(QA2, fc);
        interleave_kstep<N_MFMA, 0, N_READ, 1>();
        __builtin_amdgcn_sched_barrier(0);
        read_frags((B + 1) & (NBUF - 1), 1, f1);
        mfmas(QA3, fd);
        interleave_kstep<N_MFMA, 0, N_READ, 1>();
        __builtin_amdgcn_sched_barrier(0);
    };
    auto step = [&](auto slot) {
        if constexpr (SEP) {
            step_sep(slot);
            return;
        }

        constexpr int B = decltype(slot)::value;  // ring slot of this step's stage
        // one drain store per step: read from LDS now, stored after k-step 1
        u32x4 dv0;
        if constexpr (DEFER)
            dv0 = drain_read(d_next);
        __builtin_amdgcn_sched_barrier(0);
        read_frags(B, 1, f1);
        mfmas(0, f0);
        interleave_kstep<N_MFMA, N_FLIP, N_READ>();
        __builtin_amdgcn_sched_barrier(0);
        read_frags(B, 2, f0);
        mfmas(1, f1);
        interleave_kstep<N_MFMA, N_FLIP, N_READ>();
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (DEFER) {
            drain_store(d_next, dv0);
            d_next = d_next < N_DRAIN ? d_next + 1 : N_DRAIN;
        }
        __builtin_amdgcn_sched_barrier(0);
        read_frags(B, 3, f1);
        mfmas(2, f0);
        interleave_kstep<N_MFMA, N_FLIP, N_READ>();
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        read_frags((B + 1) & (NBUF - 1), 0, f0);
        mfmas(3, f1);
        interleave_kstep<N_MFMA, N_FLIP, N_READ>();
        __builtin_amdgcn_sched_barrier(0);
    };
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    using P2 = std::integral_constant<int, 2>;
    using P3 = std::integral_constant<int, 3>;
    // The S steps of one tile whose first stage sits in ring slot PH.
    const int s_main = S & ~(NBUF - 1);
    const int tail = S - s_main;
    auto run_tile = [&](auto ph) {
        constexpr int PH = decltype(ph)::value;
        using Q0 = std::integral_constant<int, PH>;
        using Q1 = std::integral_constant<int, (PH + 1) & 3>;
        using Q2 = std::integral_constant<int, (PH + 2) & 3>;
        using Q3 = std::integral_constant<int, (PH + 3) & 3>;
        for (int s = 0; s < s_main; s += NBUF) {
            step(Q0{});
            step(Q1{});
            step(Q2{});
            step(Q3{});
        }
        if (tail > 0)
            step(Q0{});
        if (tail > 1)
            step(Q1{});
        if (tail > 2)
            step(Q2{});
    };

    // IQBN statistics of a parked tile, read back from the wave's own LDS
    // region with transposing reads (ds_read_b64_tr_b16): in each 16-lane
    // group, lane 4a+b receives element b of the 8-byte pieces addressed by
    // lanes a, a+4, a+8, a+12.  With those four lanes pointing at one
    // 4-channel group of four consecutive pixels, every lane ends up with
    // one channel (lane % BNC) of four pixels per read, two per dword, and
    // reduces over pixels without talking to other lanes.  Two passes: the
    // exact tile mean per column (pairs summed by v_dot2 with ones), then
    // the squared deviations from it, so nothing cancels.  Rows past M of a
    // partial tile hold one and the same parked value (their activations
    // load as zeros); it is read back once and its share taken out of both
    // sums.
    auto tile_stats = [&](const auto *w_lds, int m0, int o0) {  // generic: instantiated where called
        static_assert(ES == 2 && (BNC == 64 || BNC == 32), "statistics read-back geometry");
        typedef short s16x4 __attribute__((ext_vector_type(4)));
        typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
        constexpr int NCG = BNC / 4;     // 4-channel groups per pixel
        constexpr int LPS = 4 * NCG;     // lanes per pixel set: one per channel
        constexpr int SETS = 64 / LPS;   // pixel sets read side by side
        constexpr int PPR = 4 * SETS;    // pixels per read
        constexpr int NR = BM / PPR;     // reads per lane
        const int q = 4 * (lane >> 4) + (lane & 3);
        const int cg = q % NCG, set = q / NCG, r = (lane & 15) >> 2;
        const int p_lane = 4 * set + r;  // pixel of the piece this lane addresses, within a read
        // physical chunk = logical chunk ^ (pixel % OUT_CPR); the read's own
        // share of the pixel index, (PPR * i) % OUT_CPR, is 0 or 4 and shares
        // no bit with p_lane % OUT_CPR
        auto piece = [&](int xr) {
            return w_lds + p_lane * OUT_ROW + ((((cg >> 1) ^ (p_lane % OUT_CPR)) ^ xr) * 16) + (cg & 1) * 8;
        };
        const unsigned char *const src0 = piece(0);
        const unsigned char *const src4 = piece(4 % OUT_CPR);
        unsigned dw[2 * NR];
#pragma unroll
        for (int i = 0; i < NR; ++i) {
            const int xr = (PPR * i) % OUT_CPR;
            const unsigned char *p = (xr == 0 ? src0 : src4) + i * PPR * OUT_ROW;
            const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4 *)(p));
            __builtin_memcpy(&dw[2 * i], &v, 8);
        }
        const int ch = lane % LPS;  // channel within the tile's BNC
        const int n_valid = a.m - m0 < BM ? a.m - m0 : BM;
        const float n_inv = float(BM - n_valid);
        float v_inv = 0.0f;
        if (n_valid < BM) {
            const int pm = BM - 1;
            const T t = *reinterpret_cast<const T *>(w_lds + pm * OUT_ROW + (((ch / 8) ^ (pm % OUT_CPR)) * 16) +
                                                     (ch % 8) * 2);
            v_inv = float(t);
        }
        const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);
        float s[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int i = 0; i < 2 * NR; ++i)
            s[i & 3] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, dw[i]), ones, s[i & 3], false);
        float sum = (s[0] + s[1]) + (s[2] + s[3]);
        if constexpr (SETS == 2)
            sum += __shfl_xor(sum, 32);
        const float mean = (sum - n_inv * v_inv) / float(n_valid);
        float m[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int i = 0; i < 2 * NR; ++i) {
            const float lo = __builtin_bit_cast(float, dw[i] << 16) - mean;
            const float hi = __builtin_bit_cast(float, dw[i] & 0xffff0000u) - mean;
            m[i & 3] = fmaf(lo, lo, m[i & 3]);
            m[(i + 2) & 3] = fmaf(hi, hi, m[(i + 2) & 3]);
        }
        float m2 = (m[0] + m[1]) + (m[2] + m[3]);
        if constexpr (SETS == 2)
            m2 += __shfl_xor(m2, 32);
        const float dv = v_inv - mean;
        m2 = fmaxf(m2 - n_inv * dv * dv, 0.0f);
        if (lane < LPS && o0 + ch < a.c_out) {
            const int mt = m0 / BM;
            const size_t cols = size_t(4) * a.c_out;
            const size_t col = size_t(wn) * a.c_out + o0 + ch;
            a.stats[col * a.stat_tiles + mt] = mean;
            a.stats[(cols + col) * a.stat_tiles + mt] = m2;
        }
    };

    // The same statistics for an ALLP wave's region: 32 pixels (from mw on)
    // x four components, each component's BNC channels read back and reduced
    // as above; one partial per 32-pixel sub-tile (index mw / 32) and column.
    // p_only >= 0 (a tail block): that component alone.
    auto tile_stats_allp = [&](const auto *w_lds, int mw, int o0, int p_only) {
        static_assert(ES == 2 && (BNC == 64 || BNC == 32), "statistics read-back geometry");
        typedef short s16x4 __attribute__((ext_vector_type(4)));
        typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
        constexpr int NCG = BNC / 4;     // 4-channel groups per component
        constexpr int LPS = 4 * NCG;     // lanes per pixel set: one per channel
        constexpr int SETS = 64 / LPS;   // pixel sets read side by side
        constexpr int PPR = 4 * SETS;    // pixels per read
        constexpr int NR = WTM / PPR;    // reads per lane and component
        static_assert(SWZ % PPR == 0 || PPR % SWZ == 0, "swizzle splits into lane and read parts");
        const int n_valid = a.m - mw < WTM ? a.m - mw : WTM;
        if (n_valid <= 0)
            return;  // the whole sub-tile lies past M (wave-uniform)
        const int q = 4 * (lane >> 4) + (lane & 3);
        const int cg = q % NCG, set = q / NCG, r = (lane & 15) >> 2;
        const int p_lane = 4 * set + r;
        const int ch = lane % LPS;
        const float n_inv = float(WTM - n_valid);
        const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);
        const int st = mw / WTM;
        const size_t cols = size_t(4) * a.c_out;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            if (p_only >= 0 && p != p_only)
                continue;
            // physical chunk = p * SWZ + (logical ^ (pixel % SWZ)); pixel =
            // p_lane + PPR * i, whose two parts share no bit below SWZ
            auto piece = [&](int xr) {
                return w_lds + p_lane * OUT_ROW + ((p * SWZ + (((cg >> 1) ^ (p_lane % SWZ)) ^ xr)) * 16) +
                       (cg & 1) * 8;
            };
            const unsigned char *const src0 = piece(0);
            const unsigned char *const src4 = piece(4 % SWZ);
            unsigned dw[2 * NR];
#pragma unroll
            for (int i = 0; i < NR; ++i) {
                const int xr = (PPR * i) % SWZ;
                const unsigned char *pp = (xr == 0 ? src0 : src4) + i * PPR * OUT_ROW;
                const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4 *)(pp));
                __builtin_memcpy(&dw[2 * i], &v, 8);
            }
            float v_inv = 0.0f;
            if (n_valid < WTM) {
                const int pm = WTM - 1;
                const T t = *reinterpret_cast<const T *>(w_lds + pm * OUT_ROW +
                                                         ((p * SWZ + ((ch / 8) ^ (pm % SWZ))) * 16) + (ch % 8) * 2);
                v_inv = float(t);
            }
            float sacc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int i = 0; i < 2 * NR; ++i)
                sacc[i & 3] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, dw[i]), ones, sacc[i & 3], false);
            float sum = (sacc[0] + sacc[1]) + (sacc[2] + sacc[3]);
            if constexpr (SETS == 2)
                sum += __shfl_xor(sum, 32);
            const float mean = (sum - n_inv * v_inv) / float(n_valid);
            float m[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int i = 0; i < 2 * NR; ++i) {
                const float lo = __builtin_bit_cast(float, dw[i] << 16) - mean;
                const float hi = __builtin_bit_cast(float, dw[i] & 0xffff0000u) - mean;
                m[i & 3] = fmaf(lo, lo, m[i & 3]);
                m[(i + 2) & 3] = fmaf(hi, hi, m[(i + 2) & 3]);
            }
            float m2 = (m[0] + m[1]) + (m[2] + m[3]);
            if constexpr (SETS == 2)
                m2 += __shfl_xor(m2, 32);
            const float dv = v_inv - mean;
            m2 = fmaxf(m2 - n_inv * dv * dv, 0.0f);
            if (lane < LPS && o0 + ch < a.c_out) {
                const size_t col = size_t(p) * a.c_out + o0 + ch;
                a.stats[col * a.stat_tiles + st] = mean;
                a.stats[(cols + col) * a.stat_tiles + st] = m2;
            }
        }
    };

    const T *__restrict__ bias = static_cast<const T *>(a.bias);
    T *__restrict__ out = static_cast<T *>(a.out);
    // Per-column epilogue map: (1, bias) or the folded (scale, shift).  With
    // scale 1 the fma is exactly acc + bias.
    auto col_affine = [&](int col, bool inside, float &sc, float &sh) {
        if constexpr (EPI == kEpiFold) {
            sc = inside ? a.scale[col] : 0.0f;
            sh = inside ? a.shift[col] : 0.0f;
        } else {
            sc = 1.0f;
            sh = (bias != nullptr && inside) ? float(bias[col]) : 0.0f;
        }
    };
    auto epi = [&](float v, float sc, float sh) {
        const float y = fmaf(v, sc, sh);
        if constexpr (EPI == kEpiFold)
            return a.relu ? fmaxf(y, 0.0f) : y;
        return y;
    };
    const bool vec_out = (a.c_out & 3) == 0;
    // ALLP deferred epilogue: parks the wave's 32 pixels from mw on in its
    // LDS region w_lds (row l%32, component p, chunk nb*4 + g of its
    // channels, swizzled, half l/32 of it) with the bias added (or the
    // folded map and ReLU applied), rounded to T, takes the statistics and
    // sets up the drain.  TAIL: accumulator set 0 is output component wm
    // alone, parked in place of that component; the region's other chunks
    // keep stale values, which are never read for statistics nor stored.
    auto park_allp_at = [&](unsigned char *w_lds, int mw, int o0, auto tailc) {
        constexpr bool TAIL = decltype(tailc)::value;
        auto park = [&](auto affine) {
            constexpr bool AFFINE = decltype(affine)::value;
#pragma unroll
            for (int pb = 0; pb < (TAIL ? 1 : 4) * NB; ++pb) {
                // one 32-channel block of one component; its per-column map
                // is loaded before any of it is used (one memory latency per
                // block)
                const int pa = pb / NB, nb = pb % NB;
                const int p = TAIL ? wm : pa;
                float sc[4][4], sh[4][4];
                if constexpr (AFFINE) {
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int oc = nb * 32 + 8 * g + 4 * khalf;
                        const bool in4 = o0 + oc < a.c_out;
                        const int col = in4 ? p * a.c_out + o0 + oc : 0;
                        if constexpr (EPI == kEpiFold) {
                            const f32x4 s4 = *reinterpret_cast<const f32x4 *>(a.scale + col);
                            const f32x4 h4 = *reinterpret_cast<const f32x4 *>(a.shift + col);
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                sc[g][e] = in4 ? s4[e] : 0.0f;
                                sh[g][e] = in4 ? h4[e] : 0.0f;
                            }
                        } else {
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                sc[g][e] = 1.0f;
                                const float b = float(bias[col + e]);
                                sh[g][e] = in4 ? b : 0.0f;
                            }
                        }
                    }
                }
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    T v[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        if constexpr (AFFINE)
                            v[e] = T(epi(acc[pa][nb][0][4 * g + e], sc[g][e], sh[g][e]));
                        else
                            v[e] = T(acc[pa][nb][0][4 * g + e]);
                    }
                    unsigned char *dst =
                        w_lds + l32 * OUT_ROW + ((p * SWZ + ((nb * 4 + g) ^ (l32 % SWZ))) * 16) + khalf * 8;
                    uint2 pk;
                    __builtin_memcpy(&pk, v, 8);
                    *reinterpret_cast<uint2 *>(dst) = pk;
                }
            }
        };
        if (EPI == kEpiFold || bias != nullptr)
            park(std::true_type{});
        else
            park(std::false_type{});
        if constexpr (EPI == kEpiStats)
            tile_stats_allp(w_lds, mw, o0, TAIL ? wm : -1);
        const long long rows_left = (long long)(a.m - mw) * row_bytes;
        d_base = out + (size_t)mw * 4 * a.c_out;
        d_bytes = rows_left <= 0 ? 0u : rows_left < 0x7fffffffLL ? unsigned(rows_left) : 0x7fffffffu;
        const int ch = o0 + d_k * CPC;  // first channel of the lane's chunk
        d_lane = (ch < a.c_out && (!TAIL || d_p == wm)) ? unsigned(d_pix * row_bytes + (d_p * a.c_out + ch) * ES)
                                                        : 0x80000000u;
        d_next = 0;
    };
    // ---- epilogue: bias, round, channels-last store ----
    // Accumulator register 4*g + e of lane l holds output channel row
    // 8*g + 4*(l/32) + e of the 32x32 block and pixel column l%32.
    // Writes the four channels o..o+3 of component p at pixel m.
    auto store4 = [&](int m, int p, int o, const float *y) {
        float sc[4], sh[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
            col_affine(p * a.c_out + o + e, o + e < a.c_out, sc[e], sh[e]);
        T *dst = out + ((size_t)m * 4 * a.c_out + p * a.c_out + o);
        T v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
            v[e] = T(epi(y[e], sc[e], sh[e]));
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
    };
    int ph = 0;  // ring slot of the current tile's first stage
    for (int kt = 0; kt < n_mine; ++kt) {
        const int tile = tile_of(kt);
        const int m0 = (tile / a.n_tiles) * BM;
        const int o0 = (tile % a.n_tiles) * BNC;
#pragma unroll
        for (int qs = 0; qs < QS; ++qs)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                    for (int e = 0; e < 16; ++e)
                        acc[qs][nb][mb][e] = 0.0f;
        if constexpr (ALLP) {
            run_tile_allp(step_allp);
        } else {
            if (ph == 0)
                run_tile(P0{});
            else if (ph == 1)
                run_tile(P1{});
            else if (ph == 2)
                run_tile(P2{});
            else
                run_tile(P3{});
            ph = (ph + S) & 3;
        }

        if (defer) {
            // finish the previous tile's stores before its region is reused
            for (; d_next < N_DRAIN; ++d_next)
                drain_store(d_next, drain_read(d_next));
            // park this tile: accumulator register 4*g + e of lane l holds
            // channel 8*g + 4*(l/32) + e of the 32-channel block nb and pixel
            // l%32 of block mb; bias added (or the folded affine map and
            // ReLU applied), rounded to T
            unsigned char *const w_lds = o_lds + region * OUT_WAVE;
            if constexpr (ALLP) {
                park_allp_at(w_lds, m0 + wm * WTM, o0, std::false_type{});
                continue;
            }
            // AFFINE: a per-column map to apply (bias or the folded IQBN);
            // without one the accumulators are only rounded.
            auto park = [&](auto affine) {
                constexpr bool AFFINE = decltype(affine)::value;
                // the lane's per-column map of one 32-channel block, loaded
                // before any of it is used (one memory latency per block,
                // not per channel group); the four channels of a group are
                // all inside c_out or all past it (c_out is a multiple of the
                // 16-byte chunk here)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    float sc[4][4], sh[4][4];
                    if constexpr (AFFINE) {
#pragma unroll
                        for (int g = 0; g < 4; ++g) {
                            const int oc = nb * 32 + 8 * g + 4 * khalf;
                            const bool in4 = o0 + oc < a.c_out;
                            const int col = in4 ? wn * a.c_out + o0 + oc : 0;
                            if constexpr (EPI == kEpiFold) {
                                const f32x4 s4 = *reinterpret_cast<const f32x4 *>(a.scale + col);
                                const f32x4 h4 = *reinterpret_cast<const f32x4 *>(a.shift + col);
#pragma unroll
                                for (int e = 0; e < 4; ++e) {
                                    sc[g][e] = in4 ? s4[e] : 0.0f;
                                    sh[g][e] = in4 ? h4[e] : 0.0f;
                                }
                            } else {
#pragma unroll
                                for (int e = 0; e < 4; ++e) {
                                    sc[g][e] = 1.0f;
                                    const float b = float(bias[col + e]);
                                    sh[g][e] = in4 ? b : 0.0f;
                                }
                            }
                        }
                    }
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int oc = nb * 32 + 8 * g + 4 * khalf;  // channel within the tile's BNC
#pragma unroll
                        for (int mb = 0; mb < MB; ++mb) {
                            const int m = mb * 32 + l32;
                            T v[4];
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                if constexpr (AFFINE)
                                    v[e] = T(epi(acc[0][nb][mb][4 * g + e], sc[g][e], sh[g][e]));
                                else
                                    v[e] = T(acc[0][nb][mb][4 * g + e]);
                            }
                            const int c = oc * ES / 16, within = (oc * ES) % 16;
                            unsigned char *dst = w_lds + m * OUT_ROW + ((c ^ (m % OUT_CPR)) * 16) + within;
                            if constexpr (ES == 2) {
                                uint2 pk;
                                __builtin_memcpy(&pk, v, 8);
                                *reinterpret_cast<uint2 *>(dst) = pk;
                            } else {
                                u32x4 pk;
                                __builtin_memcpy(&pk, v, 16);
                                *reinterpret_cast<u32x4 *>(dst) = pk;
                            }
                        }
                    }
                }
            };
            if (EPI == kEpiFold || bias != nullptr)
                park(std::true_type{});
            else
                park(std::false_type{});
            if constexpr (EPI == kEpiStats)
                tile_stats(w_lds, m0, o0);
            const long long rows_left = (long long)(a.m - m0) * row_bytes;
            d_base = out + (size_t)m0 * 4 * a.c_out;
            d_bytes = rows_left < 0x7fffffffLL ? unsigned(rows_left) : 0x7fffffffu;
            const int ch = o0 + d_chk * CPC;  // first channel of the lane's chunk
            d_lane = ch < a.c_out ? unsigned(d_pix * row_bytes + (wn * a.c_out + ch) * ES) : 0x80000000u;
            d_next = 0;
            continue;
        }

        if constexpr (SEP && sizeof(T) == 2 && NB == 2) {
            if (vec_out && (a.c_out & 7) == 0) {
                // Separable bf16, 64-channel tile, whole 8-channel groups:
                // for channel groups g0 = 2t and g1 = 2t+1 lane l (l < 32)
                // holds channels 8*g0 + 0..3 and 8*g1 + 0..3 of pixel l,
                // lane l+32 the channels 4..7 of both.  One v_permlane32_swap
                // per dword hands lane l the upper half of g0 and lane l+32
                // the lower half of g1, so every lane stores 8 channels (16
                // bytes): 3-9% faster here, 40% slower on the 32-channel
                // tile, which keeps the 8-byte stores.
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
                    for (int t = 0; t < 2; ++t) {
#pragma unroll
                        for (int mb = 0; mb < MB; ++mb) {
                            const int m = m0 + wm * WTM + mb * 32 + l32;
#pragma unroll
                            for (int p = 0; p < 4; ++p) {
                                unsigned h[2][2];  // [g - 2t][dword]: bf16 channel pairs
#pragma unroll
                                for (int gh = 0; gh < 2; ++gh) {
                                    const int g = 2 * t + gh;
                                    const int o = o0 + wn * WTN + nb * 32 + 8 * g + 4 * khalf;
                                    T v[4];
#pragma unroll
                                    for (int e = 0; e < 4; ++e) {
                                        // eq. 7: y_p = sum_q S[p][q] c_q, in fp32
                                        float y = 0.0f;
#pragma unroll
                                        for (int q = 0; q < 4; ++q) {
                                            const float c = acc[q][nb][mb][4 * g + e];
                                            y = ((kSeparableNeg >> (4 * p + q)) & 1u) ? y - c : y + c;
                                        }
                                        float sc, sh;
                                        col_affine(p * a.c_out + o + e, o + e < a.c_out, sc, sh);
                                        v[e] = T(epi(y, sc, sh));
                                    }
                                    __builtin_memcpy(h[gh], v, 8);
                                }
#pragma unroll
                                for (int d = 0; d < 2; ++d) {
                                    const auto r = __builtin_amdgcn_permlane32_swap(h[0][d], h[1][d], false, false);
                                    h[0][d] = r[0];
                                    h[1][d] = r[1];
                                }
                                const int o8 = o0 + wn * WTN + nb * 32 + 8 * (2 * t + khalf);
                                if (m < a.m && o8 < a.c_out)
                                    *reinterpret_cast<u32x4 *>(out + ((size_t)m * 4 * a.c_out + p * a.c_out + o8)) =
                                        u32x4{h[0][0], h[0][1], h[1][0], h[1][1]};
                            }
                        }
                    }
                }
                continue;
            }
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                if constexpr (ALLP) {
                    // c_out not a whole number of 16-byte chunks: direct stores
                    const int o = o0 + nb * 32 + 8 * g + 4 * khalf;
                    const int m = m0 + wm * WTM + l32;
                    if (o >= a.c_out || m >= a.m)
                        continue;
#pragma unroll
                    for (int p = 0; p < 4; ++p) {
                        float y[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            y[e] = acc[p][nb][0][4 * g + e];
                        store4(m, p, o, y);
                    }
                } else if constexpr (SEP) {
                    const int o = o0 + wn * WTN + nb * 32 + 8 * g + 4 * khalf;
                    if (o >= a.c_out)
                        continue;
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) {
                        const int m = m0 + wm * WTM + mb * 32 + l32;
                        if (m >= a.m)
                            continue;
                        // eq. 7: y_p = sum_q S[p][q] c_q, in fp32
#pragma unroll
                        for (int p = 0; p < 4; ++p) {
                            float y[4];
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                float t = 0.0f;
#pragma unroll
                                for (int q = 0; q < 4; ++q) {
                                    const float c = acc[q][nb][mb][4 * g + e];
                                    t = ((kSeparableNeg >> (4 * p + q)) & 1u) ? t - c : t + c;
                                }
                                y[e] = t;
                            }
                            store4(m, p, o, y);
                        }
                    }
                } else {
                    const int tn = wn * WTN + nb * 32 + 8 * g + 4 * khalf;
                    const int p = tn / BNC;
                    const int o = o0 + (tn - p * BNC);
                    if (o >= a.c_out)
                        continue;
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) {
                        const int m = m0 + wm * WTM + mb * 32 + l32;
                        if (m >= a.m)
                            continue;
                        float y[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            y[e] = acc[0][nb][mb][4 * g + e];
                        store4(m, p, o, y);
                    }
                }
            }
        }
    }
    // tail block: wave wm computes output component wm of the block's 32
    // pixels (all four waves read the same activation rows).  The claim was
    // posted before the producers' barrier of step n_mine * S - 4 and is
    // read here after the barrier of step n_mine * S - 1.
    if constexpr (TAIL2) {
        if (tails) {
            const unsigned v = __builtin_amdgcn_readfirstlane(
                __hip_atomic_load(a.claim + 1 + bid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM));
            const unsigned c = v & 0xffffu;
            // (a post of another launch cannot be read here; were it, the
            // block would be left undone rather than the barriers broken)
            if ((v >> 16) == a.epoch && c < unsigned(a.tail_blocks)) {
                const int m0 = tail_m0(int(c));
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int e = 0; e < 16; ++e)
                        acc[0][nb][0][e] = 0.0f;
                for (int st = 0; st < ST; ++st)
                    step_tail2(2 * st + 1 < S);
                if (defer) {
                    for (; d_next < N_DRAIN; ++d_next)
                        drain_store(d_next, drain_read(d_next));
                    park_allp_at(o_lds + region * OUT_WAVE, m0, 0, std::true_type{});
                } else {
                    const int m = m0 + l32;
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                        for (int g = 0; g < 4; ++g) {
                            const int o = nb * 32 + 8 * g + 4 * khalf;
                            if (o >= a.c_out || m >= a.m)
                                continue;
                            float y[4];
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                y[e] = acc[0][nb][0][4 * g + e];
                            store4(m, wm, o, y);
                        }
                }
            }
        }
    }
    if constexpr (DEFER) {
        for (; d_next < N_DRAIN; ++d_next)
            drain_store(d_next, drain_read(d_next));
    }
}

// Packs W_r, W_i, W_j, W_k (each OIHW) into [tap][cblk][kernel][cout_pad][CS]
// so that one stage of one N-tile is four contiguous runs; padding is zero.
// c_in, c_out are the packed convolution's.  The transposed modes pack the
// kernel of an input-gradient convolution instead: with W [c_in][c_out] of
// the forward layer (c_in, c_out here being the forward's c_out, c_in),
// entry (o, c, ky, kx) is the forward kernel W[c][o] at the flipped tap
// (k_h-1-ky, k_w-1-kx); kPackHamiltonGrad takes its conjugate (w_r, -w_i,
// -w_j, -w_k), since the Hamilton matrix of the conjugate is the transpose,
// kPackSeparableGrad the four real kernels as they are.
enum : int { kPackForward = 0, kPackHamiltonGrad = 1, kPackSeparableGrad = 2 };
//
// A transposed mode may pack a sub-kernel instead (one output phase of a
// strided layer's input gradient): tap (ky, kx) of the k_h x k_w sub-kernel
// is tap (ky0 + ky * step_h, kx0 + kx * step_w) of the full_kh x full_kw
// transposed kernel.
template <typename T, int MODE>
__global__ __launch_bounds__(256) void qconv2d_pack(const T *__restrict__ w0, const T *__restrict__ w1,
                                                    const T *__restrict__ w2, const T *__restrict__ w3,
                                                    T *__restrict__ wp, int c_in, int c_out, int k_h,
                                                    int k_w, int n_cblk, int cout_pad, int total, int ky0,
                                                    int kx0, int step_h, int step_w, int full_kh, int full_kw)
{
    constexpr int CS = stage_channels<T>();
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    int t = idx;
    const int cc = t % CS;
    t /= CS;
    const int o = t % cout_pad;
    t /= cout_pad;
    const int ws = t & 3;
    t >>= 2;
    const int cblk = t % n_cblk;
    const int tap = t / n_cblk;
    const int c = cblk * CS + cc;
    const int ky = tap / k_w, kx = tap - (tap / k_w) * k_w;
    const T *src = ws == 0 ? w0 : ws == 1 ? w1 : ws == 2 ? w2 : w3;
    T v = T(0);
    if (o < c_out && c < c_in) {
        if constexpr (MODE != kPackForward) {
            const int kyf = ky0 + ky * step_h, kxf = kx0 + kx * step_w;
            const T u = src[((c * c_out + o) * full_kh + (full_kh - 1 - kyf)) * full_kw + (full_kw - 1 - kxf)];
            v = (MODE == kPackSeparableGrad || ws == 0) ? u : T(-float(u));
        } else {
            v = src[((o * c_in + c) * k_h + ky) * k_w + kx];
        }
    }
    wp[idx] = v;
}

// Scatters dY [n][ho][wo][row] into the zero-filled z [n][hz][wz][row] at
// rows and columns (oy * s_h, ox * s_w): the input of the input-gradient
// convolution of a strided layer.  One thread per VW elements.
// The forward pack of bf16 kernels whose input channels come in whole
// 8-channel octets, TAPS taps: one thread per (channel block, kernel, output
// row, octet).  The thread's source is 8 x TAPS consecutive elements
// ([o][c..c+7][taps]), read as TAPS 16-byte pieces; it writes one 16-byte
// piece per tap (the octet's 8 channels at that tap), consecutive threads
// writing consecutive pieces.  Sources must be 16-byte aligned.
template <int TAPS>
__global__ __launch_bounds__(64) void qconv2d_pack_octets(const __bf16 *__restrict__ w0, const __bf16 *__restrict__ w1,
                                                          const __bf16 *__restrict__ w2, const __bf16 *__restrict__ w3,
                                                          __bf16 *__restrict__ wp, int c_in, int c_out, int n_cblk,
                                                          int cout_pad, int threads)
{
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= threads)
        return;
    const int g = t & 1;
    int r = t >> 1;
    const int o = r % cout_pad;
    r /= cout_pad;
    const int ws = r & 3;
    const int cblk = r >> 2;
    const int c = cblk * 16 + 8 * g;
    const __bf16 *src = ws == 0 ? w0 : ws == 1 ? w1 : ws == 2 ? w2 : w3;
    unsigned d[4 * TAPS];
    if (o < c_out && c < c_in) {
        const u32x4 *p = reinterpret_cast<const u32x4 *>(src + (size_t(o) * c_in + c) * TAPS);
#pragma unroll
        for (int i = 0; i < TAPS; ++i) {
            const u32x4 v = p[i];
            d[4 * i + 0] = v[0];
            d[4 * i + 1] = v[1];
            d[4 * i + 2] = v[2];
            d[4 * i + 3] = v[3];
        }
    } else {
#pragma unroll
        for (int i = 0; i < 4 * TAPS; ++i)
            d[i] = 0u;
    }
    // element e * TAPS + tap of the source is channel c + e at that tap
    auto half = [&](int i) { return (d[i / 2] >> (16 * (i % 2))) & 0xffffu; };
#pragma unroll
    for (int tap = 0; tap < TAPS; ++tap) {
        u32x4 v;
#pragma unroll
        for (int k = 0; k < 4; ++k)
            v[k] = half((2 * k) * TAPS + tap) | (half((2 * k + 1) * TAPS + tap) << 16);
        *reinterpret_cast<u32x4 *>(wp + ((size_t(tap) * n_cblk + cblk) * 4 + ws) * cout_pad * 16 + size_t(o) * 16 +
                                   8 * g) = v;
    }
}

template <typename T, int VW>
__global__ __launch_bounds__(256) void qconv2d_grad_dilate(const T *__restrict__ dy, T *__restrict__ z, int ho,
                                                           int wo, int hz, int wz, int s_h, int s_w, int row_vecs,
                                                           int64_t total)
{
    const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (idx >= total)
        return;
    int64_t t = idx;
    const int v = int(t % row_vecs);
    t /= row_vecs;
    const int zx = int(t % wz);
    t /= wz;
    const int zy = int(t % hz);
    const int64_t n = t / hz;
    struct alignas(sizeof(T) * VW) Chunk {
        T e[VW];
    };
    Chunk c;
    const int oy = zy / s_h, ox = zx / s_w;
    if (zy % s_h == 0 && zx % s_w == 0 && oy < ho && ox < wo) {
        c = reinterpret_cast<const Chunk *>(dy)[((n * ho + oy) * wo + ox) * row_vecs + v];
    } else {
#pragma unroll
        for (int e = 0; e < VW; ++e)
            c.e[e] = T(0);
    }
    reinterpret_cast<Chunk *>(z)[idx] = c;
}

// The output phases of a strided layer's input gradient, computed apart:
// phase (ry, rx) holds dX at rows ry, ry + s_h, ... and columns rx, rx + s_w,
// ... as a dense [n][hp][wp][row] block `off` elements into the stage buffer;
// hp == 0 marks a phase that no kernel tap reaches (its pixels are zero).
constexpr int kMaxPhases = 16;
struct PhaseMap {
    int64_t off[kMaxPhases];
    int hp[kMaxPhases], wp[kMaxPhases];
};

// Interleaves the phases into dX [n][h][w][row].  One thread per VW elements.
template <typename T, int VW>
__global__ __launch_bounds__(256) void qconv2d_grad_interleave(const T *__restrict__ stage, T *__restrict__ dx,
                                                               PhaseMap pm, int h, int w, int s_h, int s_w,
                                                               int row_vecs, int64_t total)
{
    const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (idx >= total)
        return;
    int64_t t = idx;
    const int v = int(t % row_vecs);
    t /= row_vecs;
    const int ix = int(t % w);
    t /= w;
    const int iy = int(t % h);
    const int64_t n = t / h;
    struct alignas(sizeof(T) * VW) Chunk {
        T e[VW];
    };
    Chunk c;
    const int ph = (iy % s_h) * s_w + ix % s_w;
    if (pm.hp[ph] > 0) {
        const int64_t at = ((n * pm.hp[ph] + iy / s_h) * pm.wp[ph] + ix / s_w) * row_vecs + v;
        c = reinterpret_cast<const Chunk *>(stage + pm.off[ph])[at];
    } else {
#pragma unroll
        for (int e = 0; e < VW; ++e)
            c.e[e] = T(0);
    }
    reinterpret_cast<Chunk *>(dx)[idx] = c;
}

// ----------------------------- kernel table -------------------------------

struct KernelEntry {
    int bm, bnc, mb, nb, threads;
    int form;    // a ConvForm: Hamilton product, separable (eq. 7), separable unmixed
    bool defer;  // deferred epilogue (one output component per wave); writes IQBN statistics
    int stat_rows;  // output pixels per statistics partial
    DType dt;
    // [epilogue kind][variant]: variant 0 when c_in is a multiple of the
    // 16-byte vector (activations move by DMA), 1 for element loads with
    // channel masking, 2 for paired stages (separable bf16, c_in a multiple
    // of 32), 3 for the Poincare stem (element loads of eq. 4 from colour
    // planes); NULL where the kind or variant does not apply (statistics need
    // the deferred epilogue).
    const void *fn[3][4];
    const char *name;
    bool allp;   // all-components waves in the Hamilton form: takes tail blocks
};

#define QCONV_DEFER(NB, WM, WN, SEP) (!(SEP) && (WM) == 1 && (WN) == 4 && 8 * (NB) * (WN) >= 32)
// the statistics variant exists only for tiles with the deferred epilogue
template <typename T, int MB, int NB, int WM, int WN, bool VEC, bool SEP>
constexpr const void *stats_fn()
{
    if constexpr (QCONV_DEFER(NB, WM, WN, SEP))
        return (const void *)&qconv2d_igemm<T, MB, NB, WM, WN, VEC, kEpiStats, SEP>;
    else
        return nullptr;
}
#define QCONV_STATS_FN(T, MB, NB, WM, WN, VEC, SEP) stats_fn<T, MB, NB, WM, WN, VEC, SEP>()
// the paired-stage variant exists only for the separable form in bf16
template <typename T, int MB, int NB, int WM, int WN, int EPI, bool SEP>
constexpr const void *pair_fn()
{
    if constexpr (SEP && sizeof(T) == 2 && EPI == kEpiBias)
        return (const void *)&qconv2d_igemm<T, MB, NB, WM, WN, true, EPI, SEP, true>;
    else
        return nullptr;
}
// the Poincare stem variant exists for the Hamilton form
template <typename T, int MB, int NB, int WM, int WN, bool SEP>
constexpr const void *stem_fn()
{
    if constexpr (SEP)
        return nullptr;
    else
        return (const void *)&qconv2d_igemm<T, MB, NB, WM, WN, false, kEpiBias, SEP, false, false, kFormHamilton, true>;
}
// the folded-IQBN epilogue serves the Hamilton form only (inference
// convolution + IQBN); the separable form has a bias epilogue
template <typename T, int MB, int NB, int WM, int WN, bool VEC, bool SEP>
constexpr const void *fold_fn()
{
    if constexpr (SEP)
        return nullptr;
    else
        return (const void *)&qconv2d_igemm<T, MB, NB, WM, WN, VEC, kEpiFold, SEP>;
}
#define QCONV_K(T, DT, MB, NB, WM, WN, SEP)                                                            \
    KernelEntry                                                                                        \
    {                                                                                                  \
        32 * (MB) * (WM), ((SEP) ? 32 : 8) * (NB) * (WN), MB, NB, 64 * ((WM) * (WN) + producer_waves<T, MB, NB, WM, WN, SEP>()), (SEP) ? 1 : 0, \
            QCONV_DEFER(NB, WM, WN, SEP), 32 * (MB) * (WM), DT,                                        \
            {{(const void *)&qconv2d_igemm<T, MB, NB, WM, WN, true, kEpiBias, SEP>,                    \
              (const void *)&qconv2d_igemm<T, MB, NB, WM, WN, false, kEpiBias, SEP>,                   \
              pair_fn<T, MB, NB, WM, WN, kEpiBias, SEP>(), stem_fn<T, MB, NB, WM, WN, SEP>()},           \
             {QCONV_STATS_FN(T, MB, NB, WM, WN, true, SEP), QCONV_STATS_FN(T, MB, NB, WM, WN, false, SEP), \
              nullptr, nullptr},                                                                         \
             {fold_fn<T, MB, NB, WM, WN, true, SEP>(),                                                 \
              fold_fn<T, MB, NB, WM, WN, false, SEP>(),                                                \
              pair_fn<T, MB, NB, WM, WN, kEpiFold, SEP>(), nullptr}},                                    \
            #T "_mb" #MB "x" #WM "_nb" #NB "x" #WN #SEP                                                \
    }

// Hamilton product in bf16 with all-components waves (4 waves of 32 pixels
// x all four components of 32*NB channels); statistics per 32-pixel wave.
#define QCONV_KA(NB)                                                                                   \
    KernelEntry                                                                                        \
    {                                                                                                  \
        128, 32 * (NB), 1, NB, 64 * (4 + producer_waves<__bf16, 1, NB, 4, 1, false, true>()), 0, true, 32, \
            DType::BF16,                                                                               \
            {{(const void *)&qconv2d_igemm<__bf16, 1, NB, 4, 1, true, kEpiBias, false, false, true>,    \
              (const void *)&qconv2d_igemm<__bf16, 1, NB, 4, 1, false, kEpiBias, false, false, true>,   \
              nullptr,                                                                                 \
              (const void *)&qconv2d_igemm<__bf16, 1, NB, 4, 1, false, kEpiBias, false, false, true,    \
                                           kFormHamilton, true>},                                      \
             {(const void *)&qconv2d_igemm<__bf16, 1, NB, 4, 1, true, kEpiStats, false, false, true>,   \
              (const void *)&qconv2d_igemm<__bf16, 1, NB, 4, 1, false, kEpiStats, false, false, true>,  \
              nullptr, nullptr},                                                                       \
             {(const void *)&qconv2d_igemm<__bf16, 1, NB, 4, 1, true, kEpiFold, false, false, true>,    \
              (const void *)&qconv2d_igemm<__bf16, 1, NB, 4, 1, false, kEpiFold, false, false, true>,   \
              nullptr, nullptr}},                                                                      \
            "bf16_allp_nb" #NB, true                                                                   \
    }

// The input gradient of the separable form (eqs. 8-10) on the Hamilton
// layouts with the kFormSepGrad block table: bias epilogue only.
#define QCONV_KG(T, DT, MB, NB, WM, WN, ALLPW)                                                         \
    KernelEntry                                                                                        \
    {                                                                                                  \
        32 * (MB) * (WM), ((ALLPW) ? 32 : 8) * (NB) * (WN), MB, NB,                                    \
            64 * ((WM) * (WN) + producer_waves<T, MB, NB, WM, WN, false, ALLPW>()), 2, false,          \
            32 * (MB) * (WM), DT,                                                                      \
            {{(const void *)&qconv2d_igemm<T, MB, NB, WM, WN, true, kEpiBias, false, false, ALLPW, kFormSepGrad>,  \
              (const void *)&qconv2d_igemm<T, MB, NB, WM, WN, false, kEpiBias, false, false, ALLPW, kFormSepGrad>, \
              nullptr, nullptr},                                                                       \
             {nullptr, nullptr, nullptr, nullptr},                                                     \
             {nullptr, nullptr, nullptr, nullptr}},                                                    \
            #T "_sepgrad_mb" #MB "x" #WM "_nb" #NB "x" #WN                                             \
    }

const KernelEntry kKernels[] = {
    // Hamilton product (eq. 5)
    QCONV_KA(2),  // 128 px x 64 channels
    QCONV_KA(1),  // 128 px x 32 channels
    // (no bf16 16-channel tile: with four producers the 32-channel tile is
    // faster at 16 output channels too: 27.5 vs 32.3 us on 128 images of
    // 32x32, 16 -> 16 channels)
    QCONV_K(float, DType::F32, 1, 1, 2, 2, false),    // 64 px x 16 channels
    // separable form (eq. 7): each wave all four c_q of 32 px x 32*NB channels
    QCONV_K(__bf16, DType::BF16, 1, 2, 4, 1, true),   // 128 px x 64 channels
    QCONV_K(__bf16, DType::BF16, 1, 1, 4, 1, true),   // 128 px x 32 channels
    QCONV_K(float, DType::F32, 1, 1, 4, 1, true),     // 128 px x 32 channels
    // the separable form's input gradient (kernel p, sign M[p][q])
    QCONV_KG(__bf16, DType::BF16, 1, 2, 4, 1, true),  // 128 px x 64 channels, all-components waves
    QCONV_KG(__bf16, DType::BF16, 1, 1, 4, 1, true),  // 128 px x 32 channels
    QCONV_KG(float, DType::F32, 1, 1, 2, 2, false),   // 64 px x 16 channels
};
constexpr int kNumKernels = int(sizeof(kKernels) / sizeof(kKernels[0]));

// Compute units of the current device (cached per device; the library may
// be called from several threads, so the caches are guarded).
std::mutex g_cache_mutex;

int device_cus()
{
    static int cached[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return 256;
    std::lock_guard<std::mutex> lock(g_cache_mutex);
    if (cached[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        cached[dev] = n;
    }
    return cached[dev];
}

// Work-groups of `fn` one compute unit holds at once (cached per kernel;
// at least 1).
int resident_wgs(const void *fn, int threads)
{
    static const void *fns[16 * kNumKernels] = {};
    static int counts[16 * kNumKernels] = {};
    std::lock_guard<std::mutex> lock(g_cache_mutex);
    for (int i = 0; i < 16 * kNumKernels; ++i) {
        if (fns[i] == fn)
            return counts[i];
        if (fns[i] == nullptr) {
            int n = 0;
            if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, threads, 0) != hipSuccess || n < 1)
                n = 1;
            counts[i] = n;
            fns[i] = fn;
            return n;
        }
    }
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, threads, 0) != hipSuccess || n < 1)
        n = 1;
    return n;
}

// Estimated cycles of a launch: rounds of one tile per CU times the tile's
// K loop (MFMA cycles per wave with an allowance for fragment reads), its
// fill latency and its epilogue stores.
double plan_cost(const KernelEntry &k, int64_t m, int c_out, int stages, int cus)
{
    const int64_t tiles = (m + k.bm - 1) / k.bm * ((c_out + k.bnc - 1) / k.bnc);
    const int64_t rounds = (tiles + cus - 1) / cus;
    const double mfma_cycles = k.dt == DType::BF16 ? 32.0 : 4 * 64.0;
    const double stage = 4.0 * k.mb * k.nb * mfma_cycles * 1.15 + 150.0;
    const double tile = stages * stage + 6000.0 + 0.3 * k.bm * 4.0 * k.bnc;
    return double(rounds) * tile;
}

}  // namespace

PackGeom qconv2d_pack_geom(int c_in, int c_out, int k_h, int k_w, DType dt)
{
    PackGeom pg;
    const int es = dt == DType::BF16 ? 2 : 4;
    pg.pk = 128 / (4 * es);
    pg.n_cblk = (c_in + pg.pk - 1) / pg.pk;
    pg.cout_pad = (c_out + kPackCoutAlign - 1) / kPackCoutAlign * kPackCoutAlign;
    pg.bytes = size_t(k_h) * k_w * pg.n_cblk * 4 * pg.cout_pad * pg.pk * es;
    return pg;
}

ConvPlan qconv2d_plan(const ConvGeom &g, DType dt, ConvForm form)
{
    const bool sep = form != ConvForm::Hamilton;
    const int64_t m = g.m();
    if (form == ConvForm::Hamilton && qconv2d_pointwise_takes(g, dt)) {
        // 1x1 layers stream through the pointwise kernel
        ConvPlan p;
        p.id = -1;
        p.pointwise = true;
        p.group_stages = qconv2d_pointwise_group_stages(m, device_cus());
        p.bm = qconv2d_pointwise_stage_pixels();
        p.bnc = g.c_out;
        p.n_tiles = 1;
        p.m_tiles = int((m + p.bm - 1) / p.bm);
        p.stat_rows = p.bm * p.group_stages;
        p.stat_tiles = int((m + p.stat_rows - 1) / p.stat_rows);
        p.name = "bf16_pointwise";
        return p;
    }
    const int pk = dt == DType::BF16 ? 16 : 8;
    const int stages = g.k_h * g.k_w * ((g.c_in + pk - 1) / pk);
    int id = -1;
    double best = 0.0;
    const int cus = device_cus();
    for (int i = 0; i < kNumKernels; ++i) {
        const KernelEntry &k = kKernels[i];
        if (k.dt != dt || k.form != int(form))
            continue;
        // the narrow tile only where the output channels leave a wide one idle
        if (dt == DType::BF16 && k.bnc == 64 && g.c_out <= 32)
            continue;
        if (sep && k.bnc == 64 && g.c_out <= 32)
            continue;
        const double cost = plan_cost(k, m, g.c_out, stages, cus);
        if (id < 0 || cost < best) {
            best = cost;
            id = i;
        }
    }
    const KernelEntry &k = kKernels[id];
    ConvPlan p;
    p.id = id;
    p.pointwise = false;
    p.group_stages = 0;
    p.bm = k.bm;
    p.bnc = k.bnc;
    p.n_tiles = (g.c_out + k.bnc - 1) / k.bnc;
    p.m_tiles = int((m + k.bm - 1) / k.bm);
    p.stat_rows = k.stat_rows;
    p.stat_tiles = int((m + k.stat_rows - 1) / k.stat_rows);
    p.name = k.name;
    return p;
}

namespace {
// (ky0, kx0, step_h, step_w, full_kh, full_kw): the sub-kernel of a
// transposed mode (the whole kernel: 0, 0, 1, 1, k_h, k_w)
template <int MODE>
hipError_t pack_weights(const PackGeom &pg, int c_in, int c_out, int k_h, int k_w, DType dt, const void *w_r,
                        const void *w_i, const void *w_j, const void *w_k, void *wpack, hipStream_t stream,
                        int ky0 = 0, int kx0 = 0, int step_h = 1, int step_w = 1, int full_kh = 0,
                        int full_kw = 0)
{
    const int total = int(pg.bytes / (dt == DType::BF16 ? 2 : 4));
    const int blocks = (total + 255) / 256;
    const bool aligned16 = ((reinterpret_cast<uintptr_t>(w_r) | reinterpret_cast<uintptr_t>(w_i) |
                             reinterpret_cast<uintptr_t>(w_j) | reinterpret_cast<uintptr_t>(w_k)) & 15) == 0;
    if (MODE == kPackForward && dt == DType::BF16 && c_in % 8 == 0 && aligned16 && pg.pk == 16 &&
        (k_h * k_w == 9 || k_h * k_w == 1)) {
        const int threads = pg.n_cblk * 4 * pg.cout_pad * 2;
        const int b64 = (threads + 63) / 64;
        if (k_h * k_w == 9)
            hipLaunchKernelGGL((qconv2d_pack_octets<9>), dim3(b64), dim3(64), 0, stream, (const __bf16 *)w_r,
                               (const __bf16 *)w_i, (const __bf16 *)w_j, (const __bf16 *)w_k, (__bf16 *)wpack, c_in,
                               c_out, pg.n_cblk, pg.cout_pad, threads);
        else
            hipLaunchKernelGGL((qconv2d_pack_octets<1>), dim3(b64), dim3(64), 0, stream, (const __bf16 *)w_r,
                               (const __bf16 *)w_i, (const __bf16 *)w_j, (const __bf16 *)w_k, (__bf16 *)wpack, c_in,
                               c_out, pg.n_cblk, pg.cout_pad, threads);
        return hipGetLastError();
    }
    if (full_kh == 0) {
        full_kh = k_h;
        full_kw = k_w;
    }
    if (dt == DType::BF16)
        hipLaunchKernelGGL((qconv2d_pack<__bf16, MODE>), dim3(blocks), dim3(256), 0, stream,
                           (const __bf16 *)w_r, (const __bf16 *)w_i, (const __bf16 *)w_j,
                           (const __bf16 *)w_k, (__bf16 *)wpack, c_in, c_out, k_h, k_w, pg.n_cblk,
                           pg.cout_pad, total, ky0, kx0, step_h, step_w, full_kh, full_kw);
    else
        hipLaunchKernelGGL((qconv2d_pack<float, MODE>), dim3(blocks), dim3(256), 0, stream,
                           (const float *)w_r, (const float *)w_i, (const float *)w_j,
                           (const float *)w_k, (float *)wpack, c_in, c_out, k_h, k_w, pg.n_cblk,
                           pg.cout_pad, total, ky0, kx0, step_h, step_w, full_kh, full_kw);
    return hipGetLastError();
}
}  // namespace

hipError_t qconv2d_pack_weights(const PackGeom &pg, int c_in, int c_out, int k_h, int k_w, DType dt,
                                const void *w_r, const void *w_i, const void *w_j, const void *w_k,
                                void *wpack, hipStream_t stream)
{
    return pack_weights<kPackForward>(pg, c_in, c_out, k_h, k_w, dt, w_r, w_i, w_j, w_k, wpack, stream);
}

ConvGeom qconv2d_grad_data_geom(const ConvGeom &g)
{
    ConvGeom t;
    t.n = g.n;
    t.c_in = g.c_out;
    t.c_out = g.c_in;
    t.k_h = g.k_h;
    t.k_w = g.k_w;
    t.s_h = t.s_w = 1;
    t.d_h = g.d_h;
    t.d_w = g.d_w;
    t.p_h = g.d_h * (g.k_h - 1) - g.p_h;
    t.p_w = g.d_w * (g.k_w - 1) - g.p_w;
    t.h = g.h + 2 * g.p_h - g.d_h * (g.k_h - 1);
    t.w = g.w + 2 * g.p_w - g.d_w * (g.k_w - 1);
    t.h_out = g.h;
    t.w_out = g.w;
    return t;
}

size_t qconv2d_grad_data_stage_bytes(const ConvGeom &g, DType dt)
{
    if (g.s_h == 1 && g.s_w == 1)
        return 0;
    const ConvGeom t = qconv2d_grad_data_geom(g);
    const size_t es = dt == DType::BF16 ? 2 : 4;
    // the zero-inserted gradient (dilated layers), or the output phases (dX's size)
    const size_t z = size_t(t.n) * t.h * t.w * 4 * t.c_in * es;
    // (each phase starts on a 16-byte boundary)
    const size_t phases = size_t(g.n) * g.h * g.w * 4 * g.c_in * es + size_t(16) * kMaxPhases;
    return z > phases ? z : phases;
}

namespace {
// One output phase of a strided layer's input gradient along one axis: with
// the transposed kernel W'[u] = W[k-1-u] and its stride-1 padding
// tp = k-1-p, dX[s*j + r] = sum over taps u = u0 + m*s (u < k) of
// W'[u] dY[j + c + m] for c = (r - tp + u0) / s, u0 = (tp - r) mod s:
// a stride-1 correlation of dY with the sub-kernel of `taps` taps and
// padding -c.  (Unit dilation.)
struct AxisPhase {
    int u0, taps, pad, size;
};
AxisPhase axis_phase(int k, int p, int s, int in, int r)
{
    AxisPhase a;
    const int tp = k - 1 - p;
    a.u0 = ((tp - r) % s + s) % s;
    a.taps = a.u0 < k ? (k - 1 - a.u0) / s + 1 : 0;
    a.pad = -((r - tp + a.u0) / s);  // exact: r - tp + u0 is a multiple of s
    a.size = in > r ? (in - r + s - 1) / s : 0;
    return a;
}

// The strided input gradient as s_h x s_w stride-1 convolutions of dY, one
// per output phase (only the taps that reach it: the MFMA work of the layer
// once, where the zero-inserted gradient does it s_h * s_w times), then one
// pass that interleaves the phases into dX.
hipError_t backward_data_phases(const ConvGeom &g, DType dt, const void *dy, const void *w_r, const void *w_i,
                                const void *w_j, const void *w_k, void *dx, void *wpack, void *stage,
                                hipStream_t stream, bool sep, ConvClaim *claim)
{
    const size_t es = dt == DType::BF16 ? 2 : 4;
    const int row = 4 * g.c_in;
    PhaseMap pm;
    int64_t off = 0;          // elements into the stage buffer
    size_t wp_off = 0;        // bytes into the packed-weight buffer
    for (int ry = 0; ry < g.s_h; ++ry)
        for (int rx = 0; rx < g.s_w; ++rx) {
            const int ph = ry * g.s_w + rx;
            const AxisPhase ay = axis_phase(g.k_h, g.p_h, g.s_h, g.h, ry);
            const AxisPhase ax = axis_phase(g.k_w, g.p_w, g.s_w, g.w, rx);
            pm.off[ph] = off;
            pm.hp[ph] = pm.wp[ph] = 0;
            if (ay.size == 0 || ax.size == 0 || ay.taps == 0 || ax.taps == 0)
                continue;  // no pixels, or no tap reaches them: zeros
            ConvGeom t;
            t.n = g.n;
            t.c_in = g.c_out;
            t.c_out = g.c_in;
            t.k_h = ay.taps;
            t.k_w = ax.taps;
            t.s_h = t.s_w = 1;
            t.d_h = t.d_w = 1;
            t.p_h = ay.pad;
            t.p_w = ax.pad;
            t.h = g.h_out;
            t.w = g.w_out;
            t.h_out = ay.size;
            t.w_out = ax.size;
            const PackGeom pg = qconv2d_pack_geom(t.c_in, t.c_out, t.k_h, t.k_w, dt);
            void *wp = static_cast<unsigned char *>(wpack) + wp_off;
            hipError_t e = sep ? pack_weights<kPackSeparableGrad>(pg, t.c_in, t.c_out, t.k_h, t.k_w, dt, w_r, w_i,
                                                                   w_j, w_k, wp, stream, ay.u0, ax.u0, g.s_h, g.s_w,
                                                                   g.k_h, g.k_w)
                               : pack_weights<kPackHamiltonGrad>(pg, t.c_in, t.c_out, t.k_h, t.k_w, dt, w_r, w_i,
                                                                  w_j, w_k, wp, stream, ay.u0, ax.u0, g.s_h, g.s_w,
                                                                  g.k_h, g.k_w);
            if (e != hipSuccess)
                return e;
            e = qconv2d_run(qconv2d_plan(t, dt, sep ? ConvForm::SeparableGradData : ConvForm::Hamilton), pg, t, dt,
                            dy, wp, nullptr, static_cast<unsigned char *>(stage) + size_t(off) * es, nullptr,
                            nullptr, stream, false, claim);
            if (e != hipSuccess)
                return e;
            pm.hp[ph] = ay.size;
            pm.wp[ph] = ax.size;
            // the next phase starts on a 16-byte boundary
            off += int64_t(g.n) * ay.size * ax.size * row;
            off = (off * int64_t(es) + 15) / 16 * 16 / int64_t(es);
            wp_off += pg.bytes;
        }
    const int vw = row % (dt == DType::BF16 ? 8 : 4) == 0 ? (dt == DType::BF16 ? 8 : 4) : 1;
    const int64_t total = int64_t(g.n) * g.h * g.w * (row / vw);
    const unsigned blocks = unsigned((total + 255) / 256);
    if (dt == DType::BF16) {
        if (vw == 8)
            hipLaunchKernelGGL((qconv2d_grad_interleave<__bf16, 8>), dim3(blocks), dim3(256), 0, stream,
                               (const __bf16 *)stage, (__bf16 *)dx, pm, g.h, g.w, g.s_h, g.s_w, row / vw, total);
        else
            hipLaunchKernelGGL((qconv2d_grad_interleave<__bf16, 1>), dim3(blocks), dim3(256), 0, stream,
                               (const __bf16 *)stage, (__bf16 *)dx, pm, g.h, g.w, g.s_h, g.s_w, row, total);
    } else {
        if (vw == 4)
            hipLaunchKernelGGL((qconv2d_grad_interleave<float, 4>), dim3(blocks), dim3(256), 0, stream,
                               (const float *)stage, (float *)dx, pm, g.h, g.w, g.s_h, g.s_w, row / vw, total);
        else
            hipLaunchKernelGGL((qconv2d_grad_interleave<float, 1>), dim3(blocks), dim3(256), 0, stream,
                               (const float *)stage, (float *)dx, pm, g.h, g.w, g.s_h, g.s_w, row, total);
    }
    return hipGetLastError();
}
}  // namespace

hipError_t qconv2d_backward_data_run(const ConvGeom &g, DType dt, const void *dy, const void *w_r, const void *w_i,
                                     const void *w_j, const void *w_k, void *dx, void *wpack, void *stage,
                                     hipStream_t stream, bool sep, ConvClaim *claim)
{
    const ConvGeom t = qconv2d_grad_data_geom(g);
    if (t.p_h < 0 || t.p_w < 0 || t.h < 1 || t.w < 1)
        return hipErrorInvalidValue;
    const PackGeom pg = qconv2d_pack_geom(t.c_in, t.c_out, t.k_h, t.k_w, dt);
    hipError_t e = sep ? pack_weights<kPackSeparableGrad>(pg, t.c_in, t.c_out, t.k_h, t.k_w, dt, w_r, w_i, w_j, w_k,
                                                          wpack, stream)
                       : pack_weights<kPackHamiltonGrad>(pg, t.c_in, t.c_out, t.k_h, t.k_w, dt, w_r, w_i, w_j, w_k,
                                                         wpack, stream);
    if (e != hipSuccess)
        return e;
    if ((g.s_h != 1 || g.s_w != 1) && g.d_h == 1 && g.d_w == 1 && g.s_h * g.s_w <= kMaxPhases)
        return backward_data_phases(g, dt, dy, w_r, w_i, w_j, w_k, dx, wpack, stage, stream, sep, claim);
    const void *z = dy;
    if (g.s_h != 1 || g.s_w != 1) {
        const int row = 4 * g.c_out;
        const int vw = row % (dt == DType::BF16 ? 8 : 4) == 0 ? (dt == DType::BF16 ? 8 : 4) : 1;
        const int64_t total = int64_t(t.n) * t.h * t.w * (row / vw);
        const unsigned blocks = unsigned((total + 255) / 256);
        if (dt == DType::BF16) {
            if (vw == 8)
                hipLaunchKernelGGL((qconv2d_grad_dilate<__bf16, 8>), dim3(blocks), dim3(256), 0, stream,
                                   (const __bf16 *)dy, (__bf16 *)stage, g.h_out, g.w_out, t.h, t.w, g.s_h, g.s_w,
                                   row / vw, total);
            else
                hipLaunchKernelGGL((qconv2d_grad_dilate<__bf16, 1>), dim3(blocks), dim3(256), 0, stream,
                                   (const __bf16 *)dy, (__bf16 *)stage, g.h_out, g.w_out, t.h, t.w, g.s_h, g.s_w,
                                   row, total);
        } else {
            if (vw == 4)
                hipLaunchKernelGGL((qconv2d_grad_dilate<float, 4>), dim3(blocks), dim3(256), 0, stream,
                                   (const float *)dy, (float *)stage, g.h_out, g.w_out, t.h, t.w, g.s_h, g.s_w,
                                   row / vw, total);
            else
                hipLaunchKernelGGL((qconv2d_grad_dilate<float, 1>), dim3(blocks), dim3(256), 0, stream,
                                   (const float *)dy, (float *)stage, g.h_out, g.w_out, t.h, t.w, g.s_h, g.s_w,
                                   row, total);
        }
        e = hipGetLastError();
        if (e != hipSuccess)
            return e;
        z = stage;
    }
    return qconv2d_run(qconv2d_plan(t, dt, sep ? ConvForm::SeparableGradData : ConvForm::Hamilton), pg, t, dt, z,
                       wpack, nullptr, dx, nullptr, nullptr, stream, false, claim);
}

bool qconv2d_writes_stats(const ConvPlan &plan, const ConvGeom &g, DType dt)
{
    if (plan.pointwise)
        return qconv2d_pointwise_takes(g, dt);
    if (plan.id < 0 || plan.id >= kNumKernels)
        return false;
    const KernelEntry &k = kKernels[plan.id];
    // deferred epilogue and whole 16-byte output chunks
    return k.defer && g.c_out % (dt == DType::BF16 ? 8 : 4) == 0;
}

size_t qconv2d_claim_bytes()
{
    return sizeof(unsigned) * (1 + size_t(kClaimMaxGroups));
}

hipError_t qconv2d_run(const ConvPlan &plan, const PackGeom &pg, const ConvGeom &g, DType dt,
                       const void *x, const void *wpack, const void *bias, void *out,
                       float *stats, const ConvFold *fold, hipStream_t stream, bool poincare, ConvClaim *claim)
{
    if (plan.pointwise) {
        if (poincare)
            return hipErrorInvalidValue;
        return qconv2d_pointwise_run(g, pg, plan.group_stages, x, wpack, bias, out, stats, plan.stat_tiles, fold,
                                     stream);
    }
    if (plan.id < 0 || plan.id >= kNumKernels)
        return hipErrorInvalidValue;
    const KernelEntry &k = kKernels[plan.id];
    const int epc = dt == DType::BF16 ? 8 : 4;
    const int es = dt == DType::BF16 ? 2 : 4;
    if (128 / (4 * es) != pg.pk || kPackCoutAlign % k.bnc != 0 || k.dt != dt || pg.bytes > 0x7fffffffu)
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
    a.m = int(g.m());
    a.stages = g.k_h * g.k_w * pg.n_cblk;
    a.n_cblk = pg.n_cblk;
    a.cout_pad = pg.cout_pad;
    a.m_tiles = plan.m_tiles;
    a.n_tiles = plan.n_tiles;
    a.w_bytes = unsigned(pg.bytes);
    a.x_elems = (long long)g.n * g.h * g.w * 4 * g.c_in;
    a.stats = stats;
    a.stat_tiles = plan.stat_tiles;
    a.scale = fold != nullptr ? fold->scale : nullptr;
    a.shift = fold != nullptr ? fold->shift : nullptr;
    a.relu = fold != nullptr && fold->relu ? 1 : 0;
    if (stats != nullptr && !qconv2d_writes_stats(plan, g, dt))
        return hipErrorInvalidValue;
    if (fold != nullptr && (fold->scale == nullptr || fold->shift == nullptr))
        return hipErrorInvalidValue;
    void *args[] = {&a};
    const int epi = stats != nullptr ? kEpiStats : fold != nullptr ? kEpiFold : kEpiBias;
    const bool paired = k.fn[epi][2] != nullptr && g.c_in % 32 == 0;
    if (poincare && (g.c_in != 1 || epi != kEpiBias))
        return hipErrorInvalidValue;
    const void *fn = k.fn[epi][poincare ? 3 : (g.c_in % epc) != 0 ? 1 : paired ? 2 : 0];
    if (fn == nullptr)
        return hipErrorInvalidValue;
    // Persistent grid: as many work-groups as fit on the device at once, at
    // most one per tile.
    const long long tiles = (long long)plan.m_tiles * plan.n_tiles;
    const long long slots = (long long)device_cus() * resident_wgs(fn, k.threads);
    const unsigned blocks = unsigned(tiles < slots ? tiles : slots);
    // With all-components waves and one N-tile, a last round that would
    // leave work-groups idle goes out as 32-pixel tail blocks instead:
    // every work-group takes `full` tiles, then claims one tail block (a
    // quarter of a tile's MFMAs) while any are left, so the work-groups that
    // finish first take them.
    a.full_tiles = int(tiles);
    a.tail_blocks = 0;
    a.claim = claim != nullptr ? claim->buf : nullptr;
    // 1..65535: never the zero of a mailbox that was never written; each
    // launch on the buffer takes the next tag
    a.epoch = claim != nullptr ? claim->epoch++ % 0xffffu + 1u : 0u;
    // Only the 64-channel tile with DMA loads takes them (two K-blocks per
    // tail stage): on the 32-channel tile a tail block costs about two
    // thirds of a tile and the claim then outweighs the gain (measured:
    // the four phase convolutions of a 3x3 stride-2 input gradient 183 ->
    // 191 us).
    const bool tail_kernel = k.allp && k.bnc == 64 && !poincare && (g.c_in % epc) == 0;
    if (tail_kernel && plan.n_tiles == 1 && a.claim != nullptr && blocks <= unsigned(kClaimMaxGroups)) {
        const long long blk = (a.m + 31) / 32;
        const long long full = blk / (4LL * blocks);
        const long long rest = blk - full * 4 * blocks;
        // (at least 8 steps of tiles per work-group: the first claim then
        // falls after the producers' first barrier, and the tiles outweigh
        // the claim)
        if (full >= 1 && rest > 0 && rest <= blocks && full * a.stages >= 8) {
            a.full_tiles = int(full * blocks);
            a.tail_blocks = int(rest);
        }
    }
    return hipLaunchKernel(fn, dim3(blocks), dim3(k.threads), args, 0, stream);
}

}  // namespace quan
