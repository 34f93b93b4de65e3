// rvq_kernels.hip -- per-head residual vector quantization (assignment) on
// gfx950 matrix cores.
//
// Method (Sec. 3 "Setup" of the paper): an archived K or V head vector x is
// stored as S codebook indices whose centroids sum to its reconstruction.
// Greedy residual VQ: r_0 = x; for stage s, i_s = argmin_j ||r_s - C_s[j]||^2
// (lowest j on exact ties), then r_{s+1} = r_s - C_s[i_s].
//
// Formulation.  For a token with residual r and stage codebook C:
//     u_j = r.c_j - ||c_j||^2/2 - b  =  -||r - c_j||^2/2 - (b - ||r||^2/2),
// with a per-token bias b >= ||r||^2/2, so every u_j is a negative float whose
// magnitude orders like the squared distance.  All of u_j comes out of the
// matrix cores (v_mfma_f32_32x32x16_f16, codebook = A operand from LDS,
// 32 tokens = B operand in registers):
//   * one "bias step" per 32x32 tile: A row i = (-||c_i||^2/2 split exactly
//     into three fp16 parts, 1, 2^14), B column j = (1, 1, 1, b_j parts), so
//     the tile starts at -||c_i||^2/2 - b_j.  b only has to be an upper bound
//     of ||r||^2/2 (it shifts every score of a token equally), so it is
//     rounded up into fp16 freely;
//   * the d/16 data steps add r.c_i.
// In the 32x32 accumulator layout lane l owns token l%32 and 16 of the tile's
// 32 codewords, so the argmin is in-lane: a negative float's bits, read as an
// unsigned integer, grow with its magnitude; with the low 5 bits replaced by
// the codeword's position among the 32 that the lane holds in a pair of
// consecutive tiles, they form a key whose minimum (v_min3_u32) is the
// nearest codeword and carries its index.  Dropping 5 mantissa bits coarsens
// the comparison to 2^-18 relative, inside the 1e-5 near-tie band.  Tile pairs
// merge on the value bits (earlier pair wins ties), then lane l with lane
// l^32.  Stage s's bias is the winning |u| of stage s-1 (||r_s||^2/2 plus the
// previous margin), grown by 2^-10.
//
// Exact operands.  Stage 0 multiplies fp16 x by fp16 codewords (every product
// exact in fp32).  Stage 1 uses r_1 = x - c_0 as two fp16 passes, x.c and
// (-c_0).c, both exact.  From stage 2 on the residual is carried as an fp16
// pair hi + lo (about 22 bits, rebuilt in fp32 and split again after every
// stage) and both halves go through the matrix cores.
//
// Codebooks.  Each stage's codebook is copied global -> LDS with the
// asynchronous global_load_lds_dwordx4 into two alternating buffers, so the
// next stage's book streams in while the current one is in use.  An LDS row
// holds a codeword's 16-byte chunks followed by its bias-step chunk; the odd
// chunk count per row spreads the 32 rows of an A fragment over distinct banks.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>
#include <mutex>

#include "fkv.h"
#include "fkv_hip_common.h"
#include "fkv_internal.h"

namespace fkv {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2 __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kLdsBudget = 160 * 1024;
constexpr float kBiasHiScale = 16384.0f;   // weight of the bias's second fp16 slot
constexpr int kMaxGroup = 256;             // streams per group in the grouped form (<= threads per block)

// One LDS book buffer: Kp rows of row_p bytes, then a 16-byte zero pad.
__host__ __device__ constexpr size_t buf_bytes_of(int row_p, int Kp)
{
    return (size_t)Kp * row_p + 16;
}

template <int D>
struct Cfg {
    static constexpr int KS = D / 16;                    // 16-deep matrix steps along d
    static constexpr int NCH = D / 8;                    // 16-byte chunks of a codeword
    // LDS row: the codeword's NCH chunks, then its bias-step A chunk.  The odd
    // number of 16-byte chunks per row puts any 16 consecutive rows on 16
    // distinct bank groups, so fragment reads are conflict-free without a
    // swizzle and a lane's fragments sit at fixed offsets from one base.
    static constexpr int ROW_P = (NCH + 1) * 16;
    static constexpr int TILE_P = 32 * ROW_P;            // one 32-codeword tile
    static constexpr int TT = D <= 64 ? 2 : 1;           // 32-token tiles per wave
    static constexpr int WAVES = D <= 64 ? 4 : 8;
    static constexpr int THREADS = 64 * WAVES;
    static constexpr int TOK = WAVES * TT * 32;          // tokens per block
    static constexpr int MIN_BLOCKS = 8 / WAVES;         // two waves per SIMD
    // two book buffers when two full (K = 256) books fit, else one
    static constexpr int NBUF = 2 * buf_bytes_of(ROW_P, 256) <= kLdsBudget ? 2 : 1;
};

template <int D>
size_t lds_bytes(int Kp)
{
    return (size_t)Cfg<D>::NBUF * buf_bytes_of(Cfg<D>::ROW_P, Kp);
}

// Asynchronously copies stage codebook C ([K][D] fp16) into an LDS buffer of
// Kp rows.  Each 64-lane copy fills 64 consecutive 16-byte LDS chunks; a
// row's bias-step slot gets a placeholder (its last data chunk) that
// book_bias_rows overwrites, and rows >= K are copies of row K-1, so they tie
// with it and lose to its lower index.
template <int D>
__device__ __forceinline__ void book_to_lds_async(const _Float16* __restrict__ C, int K, int Kp,
                                                  uint8_t* buf, int wave, int lane)
{
    constexpr int NCH = Cfg<D>::NCH, CH = NCH + 1, STEP = Cfg<D>::WAVES * 64;
    const int chunks = Kp * CH;   // a multiple of 64 (Kp is)
    for (int q0 = __builtin_amdgcn_readfirstlane(wave) * 64; q0 < chunks; q0 += STEP) {
        const uint32_t q = (uint32_t)(q0 + lane);
        const uint32_t row = q / CH, slot = q - row * CH;
        const uint32_t off = min(row, (uint32_t)K - 1) * D + min(slot, (uint32_t)NCH - 1) * 8;
        const _Float16* src = C + off;
        __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)src,
                                         (void __attribute__((address_space(3)))*)(buf + (size_t)q0 * 16),
                                         16, 0, 0);
    }
}

// Bias-step A chunk of every row of NB buffers: (-||c||^2/2 as hi + mid + lo
// fp16 parts, 1, 2^14, 0, 0, 0), written into the row's last slot.  All rows'
// LDS reads are issued before any norm is formed, so their latencies overlap.
template <int D, int NB>
__device__ __forceinline__ void book_bias_rows(uint8_t* buf0, uint8_t* buf1, int Kp)
{
    constexpr int NCH = Cfg<D>::NCH;
    for (int r = threadIdx.x; r < Kp; r += Cfg<D>::THREADS) {
        uint8_t* row[2] = {buf0 + (size_t)r * Cfg<D>::ROW_P, buf1 + (size_t)r * Cfg<D>::ROW_P};
        half8 v[NB][NCH];
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int p = 0; p < NCH; ++p) v[b][p] = *(const half8*)(row[b] + p * 16);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            float acc = 0.0f;
#pragma unroll
            for (int p = 0; p < NCH; ++p) {
#pragma unroll
                for (int e = 0; e < 8; e += 2) {
                    const half2 h = {v[b][p][e], v[b][p][e + 1]};
                    acc = __builtin_amdgcn_fdot2(h, h, acc, false);
                }
            }
            const float n = -0.5f * acc;
            const _Float16 hi = (_Float16)n;
            const float rem = n - (float)hi;
            const _Float16 mid = (_Float16)rem;
            const _Float16 lo = (_Float16)(rem - (float)mid);
            half8 a = (half8)(_Float16)0;
            a[0] = hi;
            a[1] = mid;
            a[2] = lo;
            a[3] = (_Float16)1.0f;
            a[4] = (_Float16)kBiasHiScale;
            *(half8*)(row[b] + NCH * 16) = a;
        }
    }
}

// The value lane l ^ 32 holds (hh: this lane's half-wave).
__device__ __forceinline__ uint32_t lane_xor32(uint32_t v, int hh)
{
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return hh ? r[0] : r[1];
}

// Bias-step B column of a token: slots 0-2 multiply the norm parts (1, 1, 1),
// slots 3-4 hold -b rounded up in magnitude, b <= 32768 in slot 3 directly,
// larger b in slot 4 in units of 2^14.  Lanes holding k = 8..15 give zeros.
__device__ __forceinline__ half8 bias_column(float b, int hh)
{
    half8 v = (half8)(_Float16)0;
    if (hh == 0) {
        const float bu = fmaxf(b * (1.0f + 0x1p-9f), 0x1p-24f);
        v[0] = v[1] = v[2] = (_Float16)1.0f;
        if (bu <= 32768.0f)
            v[3] = (_Float16)(-bu);
        else
            v[4] = (_Float16)(-fminf(bu * (1.0f / kBiasHiScale), 65504.0f));
    }
    return v;
}

__device__ __forceinline__ void wait_all_and_sync()
{
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
}

// A-operand fragments of one 32-codeword tile: its d/16 data steps and the
// bias step.
template <int D>
struct Frag {
    half8 a[Cfg<D>::KS];
    half8 bias;
};

// A lane's fragments of tile ct start at buf + base + ct * TILE_P, with
// base = col * ROW_P + 16 hh: data step ks at +32 ks, the bias chunk at
// +16 NCH.  For the upper half-wave (k = 8..15 of the bias step) that chunk is
// the next row's first chunk or the buffer's zero pad: finite values that
// meet the zero half of the token's bias column.
template <int D>
__device__ __forceinline__ void load_frag(Frag<D>& f, const uint8_t* buf, uint32_t base, int ct)
{
    const uint8_t* tile = buf + base + (size_t)ct * Cfg<D>::TILE_P;
#pragma unroll
    for (int ks = 0; ks < Cfg<D>::KS; ++ks) f.a[ks] = *(const half8*)(tile + ks * 32);
    f.bias = *(const half8*)(tile + Cfg<D>::NCH * 16);
}

// acc[tt] = bias step + A(tile) x B(tt) over all k-steps; with TWO a second B
// operand accumulates into the same tile.
template <int D, int TT, bool TWO>
__device__ __forceinline__ void issue_tile(const Frag<D>& f, const half8 (&bz)[TT],
                                           const half8 (&bA)[TT][Cfg<D>::KS],
                                           const half8 (&bB)[TT][Cfg<D>::KS], floatx16 (&acc)[TT])
{
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
        acc[tt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(f.bias, bz[tt], (floatx16)0.0f, 0, 0, 0);
#pragma unroll
    for (int ks = 0; ks < Cfg<D>::KS; ++ks) {
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
            acc[tt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(f.a[ks], bA[tt][ks], acc[tt], 0, 0, 0);
        if (TWO) {
#pragma unroll
            for (int tt = 0; tt < TT; ++tt)
                acc[tt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(f.a[ks], bB[tt][ks], acc[tt], 0, 0, 0);
        }
    }
}

// Minimum over a lane's 16 scores of (float bits with the low 5 bits replaced
// by base + register index), as a tree of three-input minima.
template <uint32_t BASE>
__device__ __forceinline__ uint32_t tile_min_key(const floatx16& a)
{
    uint32_t k[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) k[v] = (__float_as_uint(a[v]) & ~31u) | (BASE + (uint32_t)v);
    const uint32_t m0 = min(min(k[0], k[1]), k[2]);
    const uint32_t m1 = min(min(k[3], k[4]), k[5]);
    const uint32_t m2 = min(min(k[6], k[7]), k[8]);
    const uint32_t m3 = min(min(k[9], k[10]), k[11]);
    const uint32_t m4 = min(min(k[12], k[13]), k[14]);
    const uint32_t m5 = min(min(m0, m1), m2);
    const uint32_t m6 = min(min(m3, m4), k[15]);
    return min(m5, m6);
}

// Key minimum of the first tile of a pair (positions 0..15).
template <int TT>
__device__ __forceinline__ void pair_first(const floatx16 (&acc)[TT], uint32_t (&pk)[TT])
{
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) pk[tt] = tile_min_key<0>(acc[tt]);
}

// Adds the second tile of pair `pair` (positions 16..31) and folds the pair
// into the running best; an earlier pair wins ties on the value bits.
template <int TT>
__device__ __forceinline__ void pair_second(const floatx16 (&acc)[TT], const uint32_t (&pk)[TT], int pair,
                                            uint32_t (&bkey)[TT], int (&bpair)[TT])
{
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
        const uint32_t k = min(pk[tt], tile_min_key<16>(acc[tt]));
        if ((k & ~31u) < (bkey[tt] & ~31u)) {
            bkey[tt] = k;
            bpair[tt] = pair;
        }
    }
}

// Instruction-interleaving hints for one pipelined step: every MFMA of the tile
// being issued is followed by a few VALU ops of the previous tile's argmin and,
// early on, the LDS reads of the next tile's fragments, so one wave keeps its
// matrix core busy while its vector ALU and LDS work proceed.
template <int NMFMA, int NVALU, int NDS>
__device__ __forceinline__ void interleave_hint()
{
    constexpr int per = (NVALU + NMFMA - 1) / NMFMA;
#pragma unroll
    for (int i = 0; i < NMFMA; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);      // one MFMA
        if (i < NDS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
        __builtin_amdgcn_sched_group_barrier(0x002, per, 0);    // a few VALU
    }
}

// One stage's scores over all nct (even) codeword tiles, software-pipelined:
// the fragments of tile ct+2 load and the MFMAs of tile ct+1 run while the
// argmin of tile ct executes on the VALU.  Tiles 2p and 2p+1 form pair p.
template <int D, int TT, bool TWO>
__device__ __forceinline__ void stage_scan(const uint8_t* buf, uint32_t fa, int nct,
                                           const half8 (&bz)[TT], const half8 (&bA)[TT][Cfg<D>::KS],
                                           const half8 (&bB)[TT][Cfg<D>::KS], uint32_t (&bkey)[TT],
                                           int (&bpair)[TT])
{
    constexpr int NM = TT * (1 + Cfg<D>::KS * (TWO ? 2 : 1));   // MFMAs per tile
    constexpr int NV = TT * 26;                                 // VALU ops of one tile's argmin
    constexpr int ND = Cfg<D>::KS + 1;                          // LDS reads of one tile's fragments
    Frag<D> f0, f1;
    floatx16 acc0[TT], acc1[TT];
    uint32_t pk[TT];
    load_frag<D>(f0, buf, fa, 0);
    load_frag<D>(f1, buf, fa, 1);
    issue_tile<D, TT, TWO>(f0, bz, bA, bB, acc0);
    int ct = 0;
    for (; ct + 2 < nct; ct += 2) {
        issue_tile<D, TT, TWO>(f1, bz, bA, bB, acc1);
        load_frag<D>(f0, buf, fa, ct + 2);
        pair_first<TT>(acc0, pk);
        interleave_hint<NM, NV, ND>();
        issue_tile<D, TT, TWO>(f0, bz, bA, bB, acc0);
        load_frag<D>(f1, buf, fa, min(ct + 3, nct - 1));
        pair_second<TT>(acc1, pk, ct >> 1, bkey, bpair);
        interleave_hint<NM, NV, ND>();
    }
    issue_tile<D, TT, TWO>(f1, bz, bA, bB, acc1);
    pair_first<TT>(acc0, pk);
    pair_second<TT>(acc1, pk, ct >> 1, bkey, bpair);
}

// Re-split of a residual pair: for the two fp16 lanes q of the words a (hi),
// b (lo) and c (chosen codeword), rv = (a + b) - c in fp32 (each operation
// rounded once, as written), then hi' = fp16(rv) and lo' = fp16(rv - hi'),
// with the mixed-precision FMAs (fp16 operands read from either half of a
// word, fp32 arithmetic, an fp16 result written into one half).
__device__ __forceinline__ void resplit2(uint32_t a, uint32_t b, uint32_t c, uint32_t& na, uint32_t& nb)
{
    float t0, t1, r0, r1;
    asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel:[0,0,0] op_sel_hi:[1,0,1]" : "=v"(t0) : "v"(a), "v"(b));
    asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel:[1,0,1] op_sel_hi:[1,0,1]" : "=v"(t1) : "v"(a), "v"(b));
    asm("v_fma_mix_f32 %0, %1, -1.0, %2 op_sel:[0,0,0] op_sel_hi:[1,0,0]" : "=v"(r0) : "v"(c), "v"(t0));
    asm("v_fma_mix_f32 %0, %1, -1.0, %2 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "=v"(r1) : "v"(c), "v"(t1));
    uint32_t h, l;
    asm("v_fma_mixlo_f16 %0, %1, 1.0, 0 op_sel_hi:[0,0,0]" : "=&v"(h) : "v"(r0));
    asm("v_fma_mixhi_f16 %0, %1, 1.0, 0 op_sel_hi:[0,0,0]" : "+v"(h) : "v"(r1));
    asm("v_fma_mixlo_f16 %0, %1, -1.0, %2 op_sel:[0,0,0] op_sel_hi:[1,0,0]" : "=&v"(l) : "v"(h), "v"(r0));
    asm("v_fma_mixhi_f16 %0, %1, -1.0, %2 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "+v"(l) : "v"(h), "v"(r1));
    na = h;
    nb = l;
}

// GRP: a work item is a group of G streams that share one book (groups[g * G
// + e] is member e of group g) and its tokens are the members' archived
// tokens, member by member, so that one block serves all of them with a single
// copy of the book (the per-token arithmetic is that of the per-stream form).
template <int D, bool HILO, bool ENC, bool GRP>
__global__ __launch_bounds__(Cfg<D>::THREADS, Cfg<D>::MIN_BLOCKS) void rvq_assign_kernel(
    const _Float16* __restrict__ x, const _Float16* __restrict__ books,
    const int32_t* __restrict__ stream_book, uint8_t* __restrict__ symbols,
    float* __restrict__ residual, uint32_t* __restrict__ n_bad, int64_t T, int64_t t_begin,
    int64_t Ta, int S, int NS, int K, int Kp, int n_books, int64_t blocks_per_stream, int64_t tpb,
    double2* __restrict__ points, const double2* __restrict__ vtab, double cr, int cN, int cL, int64_t n_spans,
    const int32_t* __restrict__ groups, int G, int64_t n_streams, int64_t ipb, int64_t n_items)
{
    static_assert(!(GRP && ENC), "the grouped form has no fused encode");
    using C = Cfg<D>;
    // PERS: a block takes ipb consecutive work items (token ranges, mostly of
    // one stream) and loads the next item's token rows into registers during
    // the current item's last stage, so a new item does not start by waiting
    // on HBM.  Only the hi/lo per-stream instances hold the extra registers
    // without spilling.
    constexpr bool PERS = HILO && !ENC && !GRP;
    constexpr int KS = C::KS, TT = C::TT, TOK = C::TOK, NBUF = C::NBUF;
    extern __shared__ __align__(16) uint8_t lds[];
    // LDS: NBUF buffers of Kp rows (codeword + bias-step chunk) and a zero
    // pad; addressed from `lds` so every access stays an LDS access.
    const size_t buf_bytes = buf_bytes_of(C::ROW_P, Kp);

    // XCD-aware order: blocks dispatched to one XCD (every 8th) take consecutive
    // work items, so the blocks of one stream share that XCD's L2 copy of its book.
    const uint32_t nblk = gridDim.x, q8 = nblk / 8, r8 = nblk % 8;
    const uint32_t xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
    const int64_t bidx = (int64_t)xcd * q8 + min(xcd, r8) + slot;
    const int64_t it0 = PERS ? bidx * ipb : bidx;
    const int64_t it1 = PERS ? min(it0 + ipb, n_items) : it0 + 1;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int col = lane & 31, hh = lane >> 5;
    half8 bN[TT][KS];   // PERS: the next item's token rows
    bool have_next = false;
    for (int64_t item = it0; item < it1; ++item) {
        const int64_t s = item / blocks_per_stream;                // the stream (GRP: the group)
        const int64_t Tv = GRP ? (int64_t)G * Ta : Ta;             // the item's tokens
        const int64_t tb = (item - s * blocks_per_stream) * tpb;   // first token of the block
        const int64_t te = min(Tv, tb + tpb);                      // one past its last

        uint8_t* sym_s = symbols + s * Ta * S;
        int b = GRP ? -1 : stream_book[s];

        // this lane's tokens (independent of the book id, so their loads overlap its)
        int64_t tok[TT];
        bool valid[TT];
        int64_t srow[TT];               // GRP: the token's row in the [n_streams][Ta] outputs
        half8 bA[TT][KS], bB[TT][KS];   // B operands of the current stage's passes
        half8 bz[TT];                   // bias-step B operand
        const bool prefetched = PERS && have_next;
        have_next = false;
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
            tok[tt] = tb + (int64_t)(wave * TT + tt) * 32 + col;
            valid[tt] = tok[tt] < te;
            int64_t xr;
            if constexpr (GRP) {
                // member e's token t; a member id out of range rejects the group
                // below, and meanwhile reads stream 0
                const int64_t tv = valid[tt] ? tok[tt] : tb;
                const int64_t e = tv / Ta, t = tv - e * Ta;
                const int64_t m = groups[s * G + e];
                const int64_t mm = (m >= 0 && m < n_streams) ? m : 0;
                srow[tt] = mm * Ta + t;
                xr = mm * T + t_begin + t;
            } else {
                srow[tt] = 0;
                xr = s * T + t_begin + (valid[tt] ? tok[tt] : 0);
            }
            const _Float16* row = x + xr * D + 8 * hh;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                if (prefetched)
                    bA[tt][ks] = bN[tt][ks];
                else
                    bA[tt][ks] = valid[tt] ? *(const half8*)(row + 16 * ks) : (half8)(_Float16)0;
                bB[tt][ks] = (half8)(_Float16)0;
            }
        }
        if constexpr (GRP) {
            // the group's book: its first member's, which every member must share
            const int32_t m0 = groups[s * G];
            const int gb = (m0 >= 0 && m0 < n_streams) ? stream_book[m0] : -1;
            int bad = gb < 0 || gb >= n_books;
            if (tid < G) {
                const int32_t m = groups[s * G + tid];
                bad |= m < 0 || m >= n_streams || stream_book[m] != gb;
            }
            b = __syncthreads_or(bad) ? -1 : gb;
        }

        if (b < 0 || b >= n_books) {
            if constexpr (GRP) {
                // every in-range member's symbols (and residual) of the block's tokens
                for (int64_t i = tb * S + tid; i < te * S; i += C::THREADS) {
                    const int64_t j = i / S, e = j / Ta, m = groups[s * G + e];
                    if (m >= 0 && m < n_streams) symbols[(m * Ta + (j - e * Ta)) * S + (i - j * S)] = 0xFF;
                }
                if (residual)
                    for (int64_t i = tb * D + tid; i < te * D; i += C::THREADS) {
                        const int64_t j = i / D, e = j / Ta, m = groups[s * G + e];
                        if (m >= 0 && m < n_streams) residual[(m * Ta + (j - e * Ta)) * D + (i - j * D)] = NAN;
                    }
                if (tid == 0 && tb == 0 && n_bad) atomicAdd(n_bad, 1u);
                return;
            }
            for (int64_t i = tb * S + tid; i < te * S; i += C::THREADS) sym_s[i] = 0xFF;
            if (ENC)   // the block's spans encode 0xFF symbols: NaN points, as a separate encode gives
                for (int64_t j = tb * S / cL + tid; j < (te * S + cL - 1) / cL; j += C::THREADS)
                    points[s * n_spans + j] = make_double2(NAN, NAN);
            if (residual)
                for (int64_t i = tb * D + tid; i < te * D; i += C::THREADS) residual[s * Ta * D + i] = NAN;
            if (tid == 0 && tb == 0 && n_bad) atomicAdd(n_bad, 1u);
            continue;
        }
        const _Float16* bk = books + (int64_t)b * S * K * D;

        // Fused span encode: the vertex table (NaN beyond the alphabet) and the
        // block's symbols live after the book buffers.
        double2* V_l = (double2*)(lds + NBUF * buf_bytes);
        uint8_t* sym_l = (uint8_t*)(V_l + 256);
        if (ENC && tid < 256) V_l[tid] = tid < cN ? vtab[tid] : make_double2(NAN, NAN);

        // start the first books' copies; zero the buffers' end pads
        book_to_lds_async<D>(bk, K, Kp, lds, wave, lane);
        if (NBUF > 1 && NS > 1) book_to_lds_async<D>(bk + (size_t)K * D, K, Kp, lds + buf_bytes, wave, lane);
        if (tid < NBUF) *(half8*)(lds + tid * buf_bytes + (size_t)Kp * C::ROW_P) = (half8)(_Float16)0;

#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
            float n2 = 0.0f;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
                for (int e = 0; e < 8; e += 2) {
                    const half2 h = {bA[tt][ks][e], bA[tt][ks][e + 1]};
                    n2 = __builtin_amdgcn_fdot2(h, h, n2, false);
                }
            }
            n2 += __uint_as_float(lane_xor32(__float_as_uint(n2), hh));
            bz[tt] = bias_column(0.5f * n2 * (1.0f + 0x1p-10f), hh);
        }
        const uint32_t fa = (uint32_t)(col * C::ROW_P + hh * 16);

        wait_all_and_sync();
        if (NBUF > 1 && NS > 1)
            book_bias_rows<D, 2>(lds, lds + buf_bytes, Kp);
        else
            book_bias_rows<D, 1>(lds, lds, Kp);
        __syncthreads();

        const int nct = Kp / 32;  // even
        // GRP: a wave without tokens (short items, such as one token per member)
        // skips the scans and only takes part in the book pipeline
        const bool wave_on = !GRP || __builtin_amdgcn_readfirstlane((int)(tb + (int64_t)wave * TT * 32 < te));
        // One stage: TWO (stages 1..) scans with two passes per tile.  Stage 0 is
        // issued on its own, ahead of the loop over the later stages: with one
        // loop body holding both scan forms the register allocator kept both
        // forms' values live across the loop and spilled (d = 128, three stages:
        // 256 VGPRs and 32 bytes of scratch per lane, against 188 and none).
        auto stage = [&](const int st, auto two_c) {
            constexpr bool TWO = decltype(two_c)::value;
            if (PERS && st + 1 == NS && item + 1 < it1) {
                // the next item's token rows, in flight during this stage
                const int64_t sn = (item + 1) / blocks_per_stream;
                const int64_t tbn = (item + 1 - sn * blocks_per_stream) * tpb;
                const int64_t ten = min(Ta, tbn + tpb);
#pragma unroll
                for (int tt = 0; tt < TT; ++tt) {
                    const int64_t tk = tbn + (int64_t)(wave * TT + tt) * 32 + col;
                    const bool v = tk < ten;
                    const _Float16* row = x + (sn * T + t_begin + (v ? tk : 0)) * D + 8 * hh;
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks)
                        bN[tt][ks] = v ? *(const half8*)(row + 16 * ks) : (half8)(_Float16)0;
                }
                have_next = true;
            }
            const int cur = NBUF > 1 ? (st & 1) : 0;
            const uint8_t* buf = lds + cur * buf_bytes;
            uint32_t bkey[TT];
            int bpair[TT];
#pragma unroll
            for (int tt = 0; tt < TT; ++tt) {
                bkey[tt] = 0xFFFFFFFFu;
                bpair[tt] = 0;
            }
            if (wave_on) {
                stage_scan<D, TT, TWO>(buf, fa, nct, bz, bA, bB, bkey, bpair);
#pragma unroll
                for (int tt = 0; tt < TT; ++tt) {
                    const int li = (int)(bkey[tt] & 31u);
                    int cw = (2 * bpair[tt] + (li >> 4)) * 32 + 8 * ((li & 15) >> 2) + 4 * hh + (li & 3);
                    cw = min(cw, K - 1);  // only reachable with all-NaN scores; keeps reads in bounds
                    uint32_t val = bkey[tt] & ~31u;
                    const uint32_t oval = lane_xor32(val, hh);
                    const int ocw = (int)lane_xor32((uint32_t)cw, hh);
                    if (oval < val || (oval == val && ocw < cw)) {
                        val = oval;
                        cw = ocw;
                    }
                    if (hh == 0 && valid[tt]) {
                        if (GRP)
                            symbols[srow[tt] * S + st] = (uint8_t)cw;
                        else
                            sym_s[tok[tt] * S + st] = (uint8_t)cw;
                        if (ENC) sym_l[(tok[tt] - tb) * S + st] = (uint8_t)cw;
                    }
                    // next stage's bias: this stage's winning |u| grown by 2^-10
                    bz[tt] = bias_column(-__uint_as_float(val) * (1.0f + 0x1p-10f), hh);
                    // this lane's chunks of the chosen codeword
                    half8 cv[KS];
                    const uint8_t* crow = buf + (size_t)cw * C::ROW_P + hh * 16;
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) cv[ks] = *(const half8*)(crow + ks * 32);
                    const bool last = st + 1 == NS;
                    if (HILO && TWO && !last) {
                        // r = (hi + lo) - c for st >= 2, (x - c_0) - c_1 for st == 1; split again
#pragma unroll
                        for (int ks = 0; ks < KS; ++ks) {
                            typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
                            const u32x4 a = __builtin_bit_cast(u32x4, bA[tt][ks]), b = __builtin_bit_cast(u32x4, bB[tt][ks]),
                                        c = __builtin_bit_cast(u32x4, cv[ks]);
                            u32x4 na, nb;
#pragma unroll
                            for (int w = 0; w < 4; ++w) {
                                uint32_t x, y;
                                resplit2(a[w], b[w], c[w], x, y);
                                na[w] = x;
                                nb[w] = y;
                            }
                            bA[tt][ks] = __builtin_bit_cast(half8, na);
                            bB[tt][ks] = __builtin_bit_cast(half8, nb);
                        }
                    }
                    if (last && residual && valid[tt]) {
                        float* out = residual + (GRP ? srow[tt] : s * Ta + tok[tt]) * D + 8 * hh;
#pragma unroll
                        for (int ks = 0; ks < KS; ++ks) {
                            floatx4 lo4, hi4;
#pragma unroll
                            for (int e = 0; e < 8; ++e) {
                                const float rv = (float)bA[tt][ks][e] + (TWO ? (float)bB[tt][ks][e] : 0.0f) -
                                                 (float)cv[ks][e];
                                if (e < 4) lo4[e] = rv; else hi4[e - 4] = rv;
                            }
                            *(floatx4*)(out + 16 * ks) = lo4;
                            *(floatx4*)(out + 16 * ks + 4) = hi4;
                        }
                    }
                    if (!TWO && !last) {
#pragma unroll
                        for (int ks = 0; ks < KS; ++ks) bB[tt][ks] = -cv[ks];
                    }
                }
            }   // wave_on
            if (st + 1 < NS && (NBUF == 1 || st >= 1 || st + 2 < NS)) {
                // Book pipeline: buffer `cur` is free once every wave is past here.
                wait_all_and_sync();
                if (NBUF == 1) {
                    book_to_lds_async<D>(bk + (size_t)(st + 1) * K * D, K, Kp, lds, wave, lane);
                    wait_all_and_sync();
                } else if (st + 2 < NS) {
                    book_to_lds_async<D>(bk + (size_t)(st + 2) * K * D, K, Kp, lds + cur * buf_bytes, wave, lane);
                }
                if (NBUF == 1 || st >= 1) {
                    uint8_t* nb = lds + (NBUF > 1 ? ((st + 1) & 1) : 0) * buf_bytes;
                    book_bias_rows<D, 1>(nb, nb, Kp);
                }
                __syncthreads();
            }
        };
        stage(0, std::false_type{});
        for (int st = 1; st < NS; ++st) stage(st, std::true_type{});
        if (ENC) {
            // Span encode of the block's symbols (Sec. 1 "The code"): the block's
            // token range holds whole spans, each walked from the anchor (0,0) with
            // p <- V + r (p - V), operation for operation as the encode kernel, and
            // stored with a streaming store (measured: faster on the four-stage
            // d = 64 shape, neutral elsewhere; slower in the small-book kernel).
            __syncthreads();
            const int64_t n_sym = Ta * S;
            for (int64_t j = tb * S / cL + tid; j < (te * S + cL - 1) / cL; j += C::THREADS) {
                const int64_t a = j * cL;
                const int len = (int)min((int64_t)cL, n_sym - a);
                const uint8_t* my = sym_l + (a - tb * S);
                double px = 0.0, py = 0.0;
                for (int k0 = 0; k0 < len; k0 += 8) {
                    // the vertices of up to 8 symbols first (they do not depend on p),
                    // then the dependent steps
                    double2 v[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) v[u] = k0 + u < len ? V_l[my[k0 + u]] : make_double2(0.0, 0.0);
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        if (k0 + u < len) {
                            const double tx = px - v[u].x, ty = py - v[u].y;
                            const double ux = cr * tx, uy = cr * ty;
                            px = v[u].x + ux;
                            py = v[u].y + uy;
                        }
                    }
                }
                store_point_stream(points + s * n_spans + j, px, py);
            }
        }
        if (item + 1 < it1) __syncthreads();   // the next item's book copies overwrite the buffers
    }
}

// LDS after the book buffers for the fused span encode: 256 vertices and the
// block's symbols.
template <int D>
constexpr size_t enc_lds_bytes()
{
    return 256 * 16 + (size_t)Cfg<D>::TOK * 8;
}

// ---- small books: at most 64 codewords and two stages (d <= 64) ----------
// Every stage's book then fits in LDS for the whole block, so one block walks
// several token items of one stream: the books are copied and their norms
// formed once, no barrier separates the stages or the items, and the next
// item's token rows load while the current item is assigned.  The block's
// symbols are staged in LDS and its spans encoded once, after its last item.
constexpr int kSmallK = 64;
constexpr int kSmallBlocks = 3;     // resident blocks per compute unit
constexpr int kSmallMaxItems = 8;   // token items per block (bounds the symbol staging)

// One stage over the two codeword tiles of a small book with a single
// fragment buffer.
template <int D, bool TWO>
__device__ __forceinline__ void stage_scan_small(const uint8_t* buf, uint32_t fa, const half8 (&bz)[1],
                                                 const half8 (&bA)[1][Cfg<D>::KS], const half8 (&bB)[1][Cfg<D>::KS],
                                                 uint32_t (&bkey)[1], int (&bpair)[1])
{
    Frag<D> f;
    floatx16 acc0[1], acc1[1];
    uint32_t pk[1];
    load_frag<D>(f, buf, fa, 0);
    issue_tile<D, 1, TWO>(f, bz, bA, bB, acc0);
    load_frag<D>(f, buf, fa, 1);
    issue_tile<D, 1, TWO>(f, bz, bA, bB, acc1);
    pair_first<1>(acc0, pk);
    pair_second<1>(acc1, pk, 0, bkey, bpair);
}

// A block barrier that orders LDS only: each wave's LDS operations complete
// before it, while its global loads (the next item's token rows) and stores
// stay in flight (__syncthreads also waits for those).
__device__ __forceinline__ void lds_barrier()
{
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int D>
__device__ __forceinline__ void load_rows(half8 (&dst)[Cfg<D>::KS], const _Float16* __restrict__ x, int64_t row,
                                          bool valid, int hh)
{
    const _Float16* p = x + row * D + 8 * hh;
#pragma unroll
    for (int ks = 0; ks < Cfg<D>::KS; ++ks) dst[ks] = valid ? *(const half8*)(p + 16 * ks) : (half8)(_Float16)0;
}

template <int D, bool ENC>
__global__ __launch_bounds__(Cfg<D>::THREADS, kSmallBlocks) void rvq_small_kernel(
    const _Float16* __restrict__ x, const _Float16* __restrict__ books, const int32_t* __restrict__ stream_book,
    uint8_t* __restrict__ symbols, float* __restrict__ residual, uint32_t* __restrict__ n_bad, int64_t T,
    int64_t t_begin, int64_t Ta, int S, int NS, int K, int Kp, int n_books, int64_t blocks_per_stream, int64_t tpi,
    int64_t ipb, double2* __restrict__ points, const double2* __restrict__ vtab, double cr, int cN, int cL,
    int64_t n_spans)
{
    using C = Cfg<D>;
    constexpr int KS = C::KS, TOK = C::WAVES * 32;
    extern __shared__ __align__(16) uint8_t lds[];
    const size_t buf_bytes = buf_bytes_of(C::ROW_P, Kp);

    // XCD-aware order, as in rvq_assign_kernel
    const uint32_t nblk = gridDim.x, q8 = nblk / 8, r8 = nblk % 8;
    const uint32_t xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
    const int64_t item = (int64_t)xcd * q8 + min(xcd, r8) + slot;
    const int64_t s = item / blocks_per_stream;
    const int64_t tb0 = (item - s * blocks_per_stream) * ipb * tpi;   // the block's first token
    const int64_t te0 = min(Ta, tb0 + ipb * tpi);                      // one past its last

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int col = lane & 31, hh = lane >> 5;
    uint8_t* sym_s = symbols + s * Ta * S;
    const int b = stream_book[s];
    const _Float16* xs = x + (s * T + t_begin) * D;

    half8 bA[1][KS];   // token rows of the block's first item
    load_rows<D>(bA[0], xs, tb0 + wave * 32 + col, tb0 + wave * 32 + col < min(te0, tb0 + tpi), hh);

    if (b < 0 || b >= n_books) {
        for (int64_t i = tb0 * S + tid; i < te0 * S; i += C::THREADS) sym_s[i] = 0xFF;
        if (ENC)
            for (int64_t j = tb0 * S / cL + tid; j < (te0 * S + cL - 1) / cL; j += C::THREADS)
                points[s * n_spans + j] = make_double2(NAN, NAN);
        if (residual)
            for (int64_t i = tb0 * D + tid; i < te0 * D; i += C::THREADS) residual[s * Ta * D + i] = NAN;
        if (tid == 0 && tb0 == 0 && n_bad) atomicAdd(n_bad, 1u);
        return;
    }
    const _Float16* bk = books + (int64_t)b * S * K * D;

    double2* V_l = (double2*)(lds + 2 * buf_bytes);
    uint8_t* sym_l = (uint8_t*)(V_l + 256);   // the block's symbols, token-major from tb0
    if (ENC && tid < 256) V_l[tid] = tid < cN ? vtab[tid] : make_double2(NAN, NAN);
    book_to_lds_async<D>(bk, K, Kp, lds, wave, lane);
    if (NS > 1) book_to_lds_async<D>(bk + (size_t)K * D, K, Kp, lds + buf_bytes, wave, lane);
    if (tid < 2) *(half8*)(lds + tid * buf_bytes + (size_t)Kp * C::ROW_P) = (half8)(_Float16)0;
    wait_all_and_sync();
    if (NS > 1)
        book_bias_rows<D, 2>(lds, lds + buf_bytes, Kp);
    else
        book_bias_rows<D, 1>(lds, lds, Kp);
    __syncthreads();

    const uint32_t fa = (uint32_t)(col * C::ROW_P + hh * 16);
    // One token item on rows `cur`; the next item's rows load into `nxt`
    // (the two register sets alternate, so the load is first waited for when
    // the next item starts).
    auto run_item = [&](int64_t tb, half8 (&cur)[1][KS], half8 (&nxt)[1][KS]) {
        const int64_t te = min(te0, tb + tpi);
        const int64_t tok = tb + wave * 32 + col;
        const bool valid = tok < te;
        const int64_t tbn = tb + tpi;
        if (tbn < te0) load_rows<D>(nxt[0], xs, tbn + wave * 32 + col, tbn + wave * 32 + col < min(te0, tbn + tpi), hh);

        half8 bz[1], bB[1][KS];
        float n2 = 0.0f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            bB[0][ks] = (half8)(_Float16)0;
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
                const half2 h = {cur[0][ks][e], cur[0][ks][e + 1]};
                n2 = __builtin_amdgcn_fdot2(h, h, n2, false);
            }
        }
        n2 += __uint_as_float(lane_xor32(__float_as_uint(n2), hh));
        bz[0] = bias_column(0.5f * n2 * (1.0f + 0x1p-10f), hh);

        // stage 0, then stage 1 (as in rvq_assign_kernel: one body per scan form)
        auto stage = [&](const int st, auto two_c) {
            constexpr bool TWO = decltype(two_c)::value;
            const uint8_t* buf = lds + st * buf_bytes;
            uint32_t bkey[1] = {0xFFFFFFFFu};
            int bpair[1] = {0};
            stage_scan_small<D, TWO>(buf, fa, bz, cur, bB, bkey, bpair);
            const int li = (int)(bkey[0] & 31u);
            int cw = (li >> 4) * 32 + 8 * ((li & 15) >> 2) + 4 * hh + (li & 3);
            cw = min(cw, K - 1);  // only reachable with all-NaN scores; keeps reads in bounds
            uint32_t val = bkey[0] & ~31u;
            const uint32_t oval = lane_xor32(val, hh);
            const int ocw = (int)lane_xor32((uint32_t)cw, hh);
            if (oval < val || (oval == val && ocw < cw)) {
                val = oval;
                cw = ocw;
            }
            if (hh == 0 && valid) {
                sym_s[tok * S + st] = (uint8_t)cw;
                if (ENC) sym_l[(tok - tb0) * S + st] = (uint8_t)cw;
            }
            bz[0] = bias_column(-__uint_as_float(val) * (1.0f + 0x1p-10f), hh);
            half8 cv[KS];
            const uint8_t* crow = buf + (size_t)cw * C::ROW_P + hh * 16;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) cv[ks] = *(const half8*)(crow + ks * 32);
            const bool last = st + 1 == NS;
            if (last && residual && valid) {
                float* out = residual + (s * Ta + tok) * D + 8 * hh;
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    floatx4 lo4, hi4;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float rv = (float)cur[0][ks][e] + (TWO ? (float)bB[0][ks][e] : 0.0f) -
                                         (float)cv[ks][e];
                        if (e < 4) lo4[e] = rv; else hi4[e - 4] = rv;
                    }
                    *(floatx4*)(out + 16 * ks) = lo4;
                    *(floatx4*)(out + 16 * ks + 4) = hi4;
                }
            }
            if (!TWO && !last) {
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) bB[0][ks] = -cv[ks];
            }
        };
        stage(0, std::false_type{});
        if (NS > 1) stage(1, std::true_type{});
    };
    half8 rB[1][KS];
    for (int64_t tb = tb0; tb < te0; tb += 2 * tpi) {
        run_item(tb, bA, rB);
        if (tb + tpi < te0) run_item(tb + tpi, rB, bA);
    }
    if (ENC) {
        // the block's token range holds whole spans (tpi is a multiple of
        // L / gcd(L, S)), each walked from the anchor (0,0) with
        // p <- V + r (p - V), operation for operation as the encode kernel
        lds_barrier();
        const int64_t n_sym = Ta * S;
        for (int64_t j = tb0 * S / cL + tid; j < (te0 * S + cL - 1) / cL; j += C::THREADS) {
            const int64_t a = j * cL;
            const int len = (int)min((int64_t)cL, n_sym - a);
            const uint8_t* my = sym_l + (a - tb0 * S);
            double px = 0.0, py = 0.0;
            for (int k0 = 0; k0 < len; k0 += 8) {
                double2 v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) v[u] = k0 + u < len ? V_l[my[k0 + u]] : make_double2(0.0, 0.0);
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    if (k0 + u < len) {
                        const double tx = px - v[u].x, ty = py - v[u].y;
                        const double ux = cr * tx, uy = cr * ty;
                        px = v[u].x + ux;
                        py = v[u].y + uy;
                    }
                }
            }
            points[s * n_spans + j] = make_double2(px, py);
        }
    }
}

// Fused encode parameters (points == nullptr: assignment only).
struct EncArgs {
    double2* points;
    const double2* vtab;
    double r;
    int N, L;
};

// Stream groups of the grouped form (on = false: the per-stream form).
struct GroupArgs {
    bool on;
    const int32_t* groups;
    int64_t n_groups;
    int G;
};

template <int D, bool HILO, bool ENC, bool GRP>
int launch_rvq_t(const fkv_rvq_desc* dsc, int ns, const uint16_t* x, const uint16_t* books,
                 const int32_t* stream_book, uint8_t* symbols, float* residual, uint32_t* n_bad,
                 const EncArgs& enc, const GroupArgs& grp, hipStream_t stream)
{
    static std::once_flag once;
    const int Kp = (dsc->K + 63) / 64 * 64;  // whole pairs of 32-codeword tiles
    std::call_once(once, [] {
        (void)hipFuncSetAttribute((const void*)rvq_assign_kernel<D, HILO, ENC, GRP>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize,
                                  (int)(lds_bytes<D>(256) + (ENC ? enc_lds_bytes<D>() : 0)));
    });
    (void)hipGetLastError();
    const int64_t Ta = dsc->t_end - dsc->t_begin;
    // Tokens per block: with the fused encode, a multiple of L / gcd(L, S) so
    // that every block holds whole spans.
    int64_t tpb = Cfg<D>::TOK;
    if (ENC) {
        int a = enc.L, b = dsc->S;
        while (b) {
            const int t = a % b;
            a = b;
            b = t;
        }
        const int unit = enc.L / a;
        tpb = (int64_t)(Cfg<D>::TOK / unit) * unit;
    }
    const int64_t items = GRP ? grp.n_groups : dsc->n_streams;
    const int64_t bps = ((GRP ? grp.G * Ta : Ta) + tpb - 1) / tpb;
    const int64_t n_items = bps * items;
    // 16 items per block once there are at least 64 blocks' worth per compute
    // unit (2-3.5% faster at the long-context shape than one item per block)
    const int64_t ipb = (HILO && !ENC && !GRP && n_items >= 256 * 64) ? 16 : 1;
    const int64_t nblk = (n_items + ipb - 1) / ipb;
    if (nblk > 0x7fffffff) return FKV_ERR_UNSUPPORTED;
    const int64_t n_spans = ENC ? (Ta * dsc->S + enc.L - 1) / enc.L : 0;
    const size_t shm = lds_bytes<D>(Kp) + (ENC ? enc_lds_bytes<D>() : 0);
    hipLaunchKernelGGL((rvq_assign_kernel<D, HILO, ENC, GRP>), dim3((unsigned)nblk), dim3(Cfg<D>::THREADS), shm,
                       stream, (const _Float16*)x, (const _Float16*)books, stream_book, symbols, residual, n_bad,
                       dsc->T, dsc->t_begin, Ta, dsc->S, ns, dsc->K, Kp, dsc->n_books, bps, tpb, enc.points, enc.vtab,
                       enc.r, enc.N, enc.L, n_spans, grp.groups, grp.G, dsc->n_streams, ipb, n_items);
    return launch_status();
}

// Small books: token items of 128 (whole spans with the fused encode) per
// wave set, several per block, blocks balanced within a stream so that the
// grid is about four rounds of resident blocks.
template <int D, bool ENC>
int launch_rvq_small(const fkv_rvq_desc* dsc, int ns, const uint16_t* x, const uint16_t* books,
                     const int32_t* stream_book, uint8_t* symbols, float* residual, uint32_t* n_bad,
                     const EncArgs& enc, hipStream_t stream)
{
    constexpr int TOK = Cfg<D>::WAVES * 32;
    const int Kp = 64;
    const int64_t Ta = dsc->t_end - dsc->t_begin;
    int64_t tpi = TOK;
    if (ENC) {
        int a = enc.L, b = dsc->S;
        while (b) {
            const int t = a % b;
            a = b;
            b = t;
        }
        const int unit = enc.L / a;
        if (unit > TOK) return FKV_ERR_UNSUPPORTED;
        tpi = (int64_t)(TOK / unit) * unit;
    }
    const int64_t ips = (Ta + tpi - 1) / tpi;                   // items per stream
    const int64_t target = 256 * kSmallBlocks * 4;             // about four rounds of resident blocks
    const int64_t want = std::min<int64_t>(kSmallMaxItems, std::max<int64_t>(1, (dsc->n_streams * ips + target - 1) / target));
    const int64_t bps = (ips + want - 1) / want;               // blocks per stream
    const int64_t ipb = (ips + bps - 1) / bps;                 // items per block
    const int64_t nblk = bps * dsc->n_streams;
    if (nblk > 0x7fffffff) return FKV_ERR_UNSUPPORTED;
    const int64_t n_spans = ENC ? (Ta * dsc->S + enc.L - 1) / enc.L : 0;
    const size_t shm = 2 * buf_bytes_of(Cfg<D>::ROW_P, Kp) + (ENC ? 256 * 16 + (size_t)kSmallMaxItems * TOK * 2 : 0);
    hipLaunchKernelGGL((rvq_small_kernel<D, ENC>), dim3((unsigned)nblk), dim3(Cfg<D>::THREADS), shm, stream,
                       (const _Float16*)x, (const _Float16*)books, stream_book, symbols, residual, n_bad, dsc->T,
                       dsc->t_begin, Ta, dsc->S, ns, dsc->K, Kp, dsc->n_books, bps, tpi, ipb, enc.points, enc.vtab, enc.r,
                       enc.N, enc.L, n_spans);
    return launch_status();
}

template <int D>
int launch_rvq(const fkv_rvq_desc* dsc, int ns, const uint16_t* x, const uint16_t* books,
               const int32_t* stream_book, uint8_t* symbols, float* residual, uint32_t* n_bad,
               const EncArgs& enc, const GroupArgs& grp, hipStream_t stream)
{
    // ns stages are assigned (the first ns of the S in the layout); the hi/lo
    // residual is needed only from a third stage on
    if (grp.on) {
        if (ns <= 2)
            return launch_rvq_t<D, false, false, true>(dsc, ns, x, books, stream_book, symbols, residual, n_bad, enc,
                                                       grp, stream);
        return launch_rvq_t<D, true, false, true>(dsc, ns, x, books, stream_book, symbols, residual, n_bad, enc, grp,
                                                  stream);
    }
    if constexpr (D <= 64) {
        if (dsc->K <= kSmallK && ns <= 2) {
            if (enc.points)
                return launch_rvq_small<D, true>(dsc, ns, x, books, stream_book, symbols, residual, n_bad, enc, stream);
            return launch_rvq_small<D, false>(dsc, ns, x, books, stream_book, symbols, residual, n_bad, enc, stream);
        }
    }
    if (enc.points) {
        if (ns <= 2)
            return launch_rvq_t<D, false, true, false>(dsc, ns, x, books, stream_book, symbols, residual, n_bad, enc,
                                                       grp, stream);
        return launch_rvq_t<D, true, true, false>(dsc, ns, x, books, stream_book, symbols, residual, n_bad, enc, grp,
                                                  stream);
    }
    if (ns <= 2)
        return launch_rvq_t<D, false, false, false>(dsc, ns, x, books, stream_book, symbols, residual, n_bad, enc,
                                                    grp, stream);
    return launch_rvq_t<D, true, false, false>(dsc, ns, x, books, stream_book, symbols, residual, n_bad, enc, grp,
                                               stream);
}

int rvq_dispatch(const fkv_rvq_desc* desc, int ns, const uint16_t* x_f16, const uint16_t* books_f16,
                 const int32_t* stream_book, uint8_t* symbols, float* residual, uint32_t* n_bad_streams,
                 const EncArgs& enc, void* stream, const GroupArgs& grp = GroupArgs{false, nullptr, 0, 0})
{
    if (!desc) return FKV_ERR_INVALID_ARG;
    const fkv_rvq_desc& d = *desc;
    if (d.n_streams < 0 || d.T < 0 || d.t_begin < 0 || d.t_end < d.t_begin || d.t_end > d.T)
        return FKV_ERR_INVALID_ARG;
    if (d.d < 16 || d.d > 256 || d.d % 16 != 0) return FKV_ERR_INVALID_ARG;
    if (d.S < 1 || d.S > 8 || d.K < 1 || d.K > 256 || d.n_books < 1) return FKV_ERR_INVALID_ARG;
    if (ns < 1 || ns > d.S || (enc.points && ns != d.S)) return FKV_ERR_INVALID_ARG;
    if (grp.on && (grp.n_groups < 0 || grp.G < 1 || grp.G > kMaxGroup || enc.points)) return FKV_ERR_INVALID_ARG;
    if (grp.on && grp.n_groups > 0 && (!grp.groups || !aligned(grp.groups, 4))) return FKV_ERR_INVALID_ARG;
    if (d.n_streams == 0 || d.t_end == d.t_begin || (grp.on && grp.n_groups == 0)) return FKV_OK;
    if (!x_f16 || !books_f16 || !stream_book || !symbols) return FKV_ERR_INVALID_ARG;
    if (!aligned(x_f16, 16) || !aligned(books_f16, 16) || !aligned(stream_book, 4))
        return FKV_ERR_INVALID_ARG;
    if (residual && !aligned(residual, 16)) return FKV_ERR_INVALID_ARG;
    if (n_bad_streams && !aligned(n_bad_streams, 4)) return FKV_ERR_INVALID_ARG;
    const hipStream_t st = (hipStream_t)stream;
#define FKV_RVQ_CASE(DD) \
    case DD: return launch_rvq<DD>(desc, ns, x_f16, books_f16, stream_book, symbols, residual, n_bad_streams, enc, grp, st);
    switch (d.d) {
        FKV_RVQ_CASE(16) FKV_RVQ_CASE(32) FKV_RVQ_CASE(48) FKV_RVQ_CASE(64)
        FKV_RVQ_CASE(80) FKV_RVQ_CASE(96) FKV_RVQ_CASE(112) FKV_RVQ_CASE(128)
        FKV_RVQ_CASE(144) FKV_RVQ_CASE(160) FKV_RVQ_CASE(176) FKV_RVQ_CASE(192)
        FKV_RVQ_CASE(208) FKV_RVQ_CASE(224) FKV_RVQ_CASE(240) FKV_RVQ_CASE(256)
    default: return FKV_ERR_INVALID_ARG;
    }
#undef FKV_RVQ_CASE
}

// From this many head vectors per call on, fkv_rvq_assign_encode runs the
// assignment and then the span encode as two kernels.  The fused kernel's
// encode tail sits on every block's critical path (one block per compute unit
// at d = 128, so about 1,000 blocks in a row per compute unit at the
// long-context shape: 0.85 ms more than the separate encode's 0.12 ms);
// below a few thousand blocks the one launch and the symbols never read back
// win (GPT-2 shape: 37 us fused against 41 us).
constexpr int64_t kSplitHeadVectors = (int64_t)1 << 23;

bool encode_split(const fkv_rvq_desc* desc, const uint8_t* symbols)
{
    return desc && desc->n_streams > 0 && desc->t_end > desc->t_begin &&
           desc->n_streams * (desc->t_end - desc->t_begin) >= kSplitHeadVectors && aligned(symbols, 4);
}

}  // namespace
}  // namespace fkv

using namespace fkv;

extern "C" int fkv_rvq_assign_encode_fused(const fkv_rvq_desc* desc, const uint8_t* symbols)
{
    if (!desc) return FKV_ERR_INVALID_ARG;
    return encode_split(desc, symbols) ? 0 : 1;
}

extern "C" int fkv_rvq_assign(const fkv_rvq_desc* desc, const uint16_t* x_f16, const uint16_t* books_f16,
                              const int32_t* stream_book, uint8_t* symbols, float* residual,
                              uint32_t* n_bad_streams, void* stream)
{
    const EncArgs none = {nullptr, nullptr, 0.0, 0, 1};
    return rvq_dispatch(desc, desc ? desc->S : 0, x_f16, books_f16, stream_book, symbols, residual, n_bad_streams,
                        none, stream);
}

extern "C" int fkv_rvq_assign_stages(const fkv_rvq_desc* desc, int32_t n_stages, const uint16_t* x_f16,
                                     const uint16_t* books_f16, const int32_t* stream_book, uint8_t* symbols,
                                     float* residual, uint32_t* n_bad_streams, void* stream)
{
    const EncArgs none = {nullptr, nullptr, 0.0, 0, 1};
    return rvq_dispatch(desc, n_stages, x_f16, books_f16, stream_book, symbols, residual, n_bad_streams, none,
                        stream);
}

extern "C" int fkv_rvq_assign_encode(const fkv_rvq_desc* desc, const uint16_t* x_f16, const uint16_t* books_f16,
                                     const int32_t* stream_book, const fkv_codec* c, const void* dev_table,
                                     uint8_t* symbols, double* points, float* residual, uint32_t* n_bad_streams,
                                     void* stream)
{
    if (!c || c->N < 3 || c->N > 256 || c->L < 1 || c->L > 64 || !(c->r > 0.0 && c->r < 1.0) ||
        !(c->r_max > 0.0 && c->r <= c->r_max * (1.0 + 1e-12)))
        return FKV_ERR_INVALID_ARG;
    if (!dev_table || !points || !aligned(dev_table, 16) || !aligned(points, 16)) return FKV_ERR_INVALID_ARG;
    if (encode_split(desc, symbols)) {
        // assignment, then the encode of its symbols on the same stream: the
        // same symbols and points as the fused kernel, bit for bit (an invalid
        // stream's 0xFF symbols encode to NaN points there too)
        const EncArgs none = {nullptr, nullptr, 0.0, 0, 1};
        const int rc = rvq_dispatch(desc, desc->S, x_f16, books_f16, stream_book, symbols, residual, n_bad_streams,
                                    none, stream);
        if (rc != FKV_OK) return rc;
        return fkv_cgr_encode_spans(c, dev_table, symbols, desc->n_streams, (desc->t_end - desc->t_begin) * desc->S,
                                    points, stream);
    }
    const EncArgs enc = {(double2*)points, (const double2*)((const uint8_t*)dev_table + table_off_V(c->N)), c->r,
                         c->N, c->L};
    return rvq_dispatch(desc, desc ? desc->S : 0, x_f16, books_f16, stream_book, symbols, residual, n_bad_streams,
                        enc, stream);
}

extern "C" int fkv_rvq_assign_groups(const fkv_rvq_desc* desc, const int32_t* groups, int64_t n_groups,
                                     int32_t group_size, const uint16_t* x_f16, const uint16_t* books_f16,
                                     const int32_t* stream_book, uint8_t* symbols, float* residual,
                                     uint32_t* n_bad_groups, void* stream)
{
    const EncArgs none = {nullptr, nullptr, 0.0, 0, 1};
    const GroupArgs grp = {true, groups, n_groups, group_size};
    return rvq_dispatch(desc, desc ? desc->S : 0, x_f16, books_f16, stream_book, symbols, residual, n_bad_groups,
                        none, stream, grp);
}
