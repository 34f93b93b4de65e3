// cgr_kernels.hip -- fixed-span chaos-game (iterated-map) encode, bulk span
// decode and O(1) random access for gfx950.
//
// Method (Sec. 1 "The code" and Sec. 2 of the paper): symbol c maps the running
// point by p <- V(c) + r (p - V(c)); a span of L symbols starting at the anchor
// (0,0) is stored as its final point.  Decoding reads the symbol off the cell
// (sector) that holds the point and inverts the map, p <- (p - (1-r)V(c)) / r,
// walking back to the anchor.
//
// Layout: one span per lane; the spans of a tile are contiguous in both the
// symbol bytes and the 16-byte points, so every global access of a tile is a
// coalesced stream.  Encode reads each span's bytes straight from the aligned
// dwords that cover it (spans of up to 16 symbols); longer spans, and decode's
// output, go through LDS.  The per-alphabet tables (vertices, cell centres,
// sector look-up) live in LDS for the whole persistent block.
//
// Floating point: the encode recurrence must be bit-reproducible, so this file
// is compiled without FP contraction, and fused multiply-adds appear only where
// written explicitly (decode's inverse map, whose points are never compared --
// only the symbols they yield).
#include "cgr_device.h"

namespace fkv {
namespace {

// ------------------------------------------------------------------ encode --

// Span encode through an LDS tile of 256 spans (spans longer than 16 symbols).
__global__ __launch_bounds__(kBlock, 8) void cgr_encode_tiles_kernel(
    const uint8_t* __restrict__ sym, double2* __restrict__ pts, const uint8_t* __restrict__ gtab,
    CodecArgs cd, int64_t n_sym, int64_t n_spans, int64_t tiles_per_stream, int64_t n_tiles)
{
    extern __shared__ __align__(16) uint8_t lds[];
    const int N = cd.N, L = cd.L;
    // LDS: the 256-entry vertex table (entries >= N are NaN, so a symbol
    // outside the alphabet yields a NaN point), then the symbol tile.
    static_assert(kBlock == 256, "one vertex entry per thread");
    double2* V = (double2*)lds;
    uint8_t* tile = lds + 256 * sizeof(double2);
    // This thread's vertex entry: loaded first, stored once the first tile's
    // symbol loads are in flight, so the two memory latencies overlap.
    const double2 vreg = (int)threadIdx.x < N ? ((const double2*)(gtab + table_off_V(N)))[threadIdx.x]
                                              : make_double2(NAN, NAN);
    bool staged = false;
    TileWalk cur;
    cur.init(blockIdx.x, gridDim.x, tiles_per_stream);
    for (int64_t tl = blockIdx.x; tl < n_tiles; tl += gridDim.x, cur.next()) {
        const int64_t s = cur.s;
        const int64_t j0 = cur.j * kBlock;
        const int64_t nsp = min((int64_t)kBlock, n_spans - j0);
        const int64_t g0 = s * n_sym + j0 * L;
        const int64_t g1 = s * n_sym + min(n_sym, (j0 + nsp) * L);
        __syncthreads();  // previous tile consumed
        bytes_to_lds(sym, g0, g1, tile);
        if (!staged) {
            V[threadIdx.x] = vreg;
            staged = true;
        }
        __syncthreads();
        if (threadIdx.x < nsp) {
            const int64_t a = (j0 + threadIdx.x) * L;
            const int len = (int)min((int64_t)L, n_sym - a);
            const uint8_t* my = tile + (g0 & 3) + threadIdx.x * L;
            double px = 0.0, py = 0.0;
            for (int k = 0; k < len; ++k) encode_step(px, py, V[my[k]], cd.r);
            store_point_stream(pts + s * n_spans + j0 + threadIdx.x, px, py);
        }
    }
}

// Span encode for spans of up to 16 symbols, with no LDS staging: a wave
// takes 256 consecutive spans of one stream (a wave tile), four per lane (j,
// j + 64, j + 128, j + 192), loads the aligned dwords that cover each span,
// extracts the symbols and walks the four spans from the anchor as independent
// chains; the points go out with streaming stores.  Wave tiles are walked
// without division.
constexpr int kEncSpl = 4;
constexpr int kEncTile = 64 * kEncSpl;

__device__ __forceinline__ void span_dwords(const uint8_t* __restrict__ sym, const uint32_t* __restrict__ s32,
                                            int64_t a, int len, int64_t n_dw, int64_t total_bytes, uint32_t (&e)[4])
{
    const int off = (int)(a & 3);
    const int64_t d0 = a >> 2;
    uint32_t dw[5];
#pragma unroll
    for (int q = 0; q < 5; ++q) {
        const int64_t d = d0 + q;
        dw[q] = 0;
        if (q * 4 < off + len) {
            if (d < n_dw) {
                dw[q] = s32[d];
            } else {   // the array's last, partial dword, byte by byte
                for (int b = 0; b < 4 && d * 4 + b < total_bytes; ++b) dw[q] |= (uint32_t)sym[d * 4 + b] << (8 * b);
            }
        }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) e[c] = __builtin_amdgcn_alignbyte(dw[c + 1], dw[c], off);
}

// LC > 0: the span length is LC, known at compile time; a lane whose four
// spans are all whole walks them fully unrolled with no per-step predicate, so
// the four chains' steps interleave (the predicated walk puts each chain's
// step in its own branch region).
template <int LC>
__global__ __launch_bounds__(kBlock, 8) void cgr_encode_kernel(
    const uint8_t* __restrict__ sym, double2* __restrict__ pts, const uint8_t* __restrict__ gtab,
    CodecArgs cd, int64_t n_sym, int64_t n_spans, int64_t wtiles_per_stream, int64_t n_wtiles, int64_t total_bytes)
{
    __shared__ double2 V[256];   // entries >= N are NaN: a symbol outside the alphabet gives a NaN point
    const int N = cd.N, L = cd.L;
    static_assert(kBlock == 256, "one vertex entry per thread");
    V[threadIdx.x] = (int)threadIdx.x < N ? ((const double2*)(gtab + table_off_V(N)))[threadIdx.x]
                                          : make_double2(NAN, NAN);
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int64_t wave = (int64_t)blockIdx.x * (kBlock / 64) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t n_waves = (int64_t)gridDim.x * (kBlock / 64);
    const uint32_t* s32 = (const uint32_t*)sym;
    const int64_t n_dw = total_bytes >> 2;   // whole dwords of the symbol array
    TileWalk w;
    w.init(wave, n_waves, wtiles_per_stream);
    for (int64_t t = wave; t < n_wtiles; t += n_waves, w.next()) {
        int64_t jj[kEncSpl];
        int len[kEncSpl];
        uint32_t e[kEncSpl][4];
#pragma unroll
        for (int h = 0; h < kEncSpl; ++h) {
            jj[h] = w.j * kEncTile + h * 64 + lane;
            len[h] = jj[h] < n_spans ? (int)min((int64_t)L, n_sym - jj[h] * L) : 0;
            e[h][0] = e[h][1] = e[h][2] = e[h][3] = 0;
            if (len[h] > 0) span_dwords(sym, s32, w.s * n_sym + jj[h] * L, len[h], n_dw, total_bytes, e[h]);
        }
        double px[kEncSpl], py[kEncSpl];
#pragma unroll
        for (int h = 0; h < kEncSpl; ++h) px[h] = py[h] = 0.0;
        bool whole = LC > 0;
#pragma unroll
        for (int h = 0; h < kEncSpl; ++h) whole = whole && len[h] == LC;
        if (whole) {
#pragma unroll
            for (int k = 0; k < (LC > 0 ? LC : 1); ++k)
#pragma unroll
                for (int h = 0; h < kEncSpl; ++h)
                    encode_step(px[h], py[h], V[(e[h][k >> 2] >> (8 * (k & 3))) & 0xFF], cd.r);
        } else {
#pragma unroll
            for (int k = 0; k < 16; ++k)
#pragma unroll
                for (int h = 0; h < kEncSpl; ++h)
                    if (k < len[h]) encode_step(px[h], py[h], V[(e[h][k >> 2] >> (8 * (k & 3))) & 0xFF], cd.r);
        }
#pragma unroll
        for (int h = 0; h < kEncSpl; ++h)
            if (len[h] > 0) store_point_stream(pts + w.s * n_spans + jj[h], px[h], py[h]);
    }
}

// ------------------------------------------------------------------ decode --

// Bulk decode with no block barrier after the table staging: a wave decodes
// 128 consecutive spans of one stream (a wave tile), two per lane walked as
// independent chains so that the look-ups of one overlap the arithmetic of
// the other.  With 6-symbol spans at an even offset (and no verification,
// which re-reads the symbols), each lane keeps its chains' symbols in
// registers and stores them as three 16-bit pairs per span; otherwise they go
// to the wave's LDS staging area and back out as aligned dwords (bytes at
// either end).  The points of the next wave tile are loaded while the current
// one decodes.  Points are read and symbols written with streaming accesses:
// each is touched once, and the tables stay in LDS.
constexpr int kDecodeSpl = 2;                  // spans per lane
constexpr int kDecodeTile = 64 * kDecodeSpl;   // spans per wave tile

template <bool EXACT, bool VERIFY>
__device__ inline bool decode_finish(double qx, double qy, const double2 P, const uint8_t* my, int len,
                                     const Tables& t, const CodecArgs& cd)
{
    bool ok = anchor_ok(qx, qy);
    if (VERIFY) {
        double px = 0.0, py = 0.0;
        for (int k = 0; k < len; ++k) encode_step(px, py, t.V[my[k]], cd.r);
        ok = ok && (__double_as_longlong(px) == __double_as_longlong(P.x)) &&
             (__double_as_longlong(py) == __double_as_longlong(P.y));
    }
    return ok;
}

// Two independent backward walks of `len` steps (LC > 0: the length fixed at
// compile time, so the loop unrolls fully), symbols into my0 / my1.  With an
// even LC each chain's symbols 2p + 1 and 2p are staged together as one
// 16-bit write when the staging addresses are even (they are whenever the
// stream length is), else byte by byte.
template <int LC, bool EXACT>
__device__ __forceinline__ void walk_two(double& ax, double& ay, double& bx, double& by, uint8_t* my0, uint8_t* my1,
                                         int len, const Tables& t, const CodecArgs& cd)
{
    constexpr bool PACK = LC > 0 && LC % 2 == 0;
    const int n = LC > 0 ? LC : len;
    const bool even = ((uintptr_t)my0 & 1) == 0;   // my1 - my0 is even
    uint32_t ha = 0, hb = 0;
#pragma unroll
    for (int k = n - 1; k >= 0; --k) {
        int ca, cb;
        if (EXACT) {
            ca = sector_of<EXACT>(ax, ay, t, cd);
            cb = sector_of<EXACT>(bx, by, t, cd);
        } else {
            sector_fast2(ax, ay, bx, by, t.lut, cd.lut_bias, ca, cb);
        }
        if (PACK && (k & 1)) {
            ha = (uint32_t)ca;
            hb = (uint32_t)cb;
        } else if (PACK && even) {
            *(uint16_t*)(my0 + k) = (uint16_t)((ha << 8) | (uint32_t)ca);
            *(uint16_t*)(my1 + k) = (uint16_t)((hb << 8) | (uint32_t)cb);
        } else if (PACK) {
            my0[k] = (uint8_t)ca;
            my0[k + 1] = (uint8_t)ha;
            my1[k] = (uint8_t)cb;
            my1[k + 1] = (uint8_t)hb;
        } else {
            my0[k] = (uint8_t)ca;
            my1[k] = (uint8_t)cb;
        }
        const double2 wa = t.Wr[ca], wb = t.Wr[cb];
        decode_step(ax, ay, wa, cd.inv_r);
        decode_step(bx, by, wb, cd.inv_r);
    }
}


// Two backward walks of 6 steps with each chain's symbols kept in registers as
// three 16-bit pairs (symbol 2p in the low byte, 2p + 1 in the high byte).
template <bool EXACT>
__device__ __forceinline__ void walk_two_regs6(double& ax, double& ay, double& bx, double& by, uint32_t (&pa)[3],
                                               uint32_t (&pb)[3], const Tables& t, const CodecArgs& cd)
{
    uint32_t ha = 0, hb = 0;
#pragma unroll
    for (int k = 5; k >= 0; --k) {
        int ca, cb;
        if (EXACT) {
            ca = sector_of<EXACT>(ax, ay, t, cd);
            cb = sector_of<EXACT>(bx, by, t, cd);
        } else {
            sector_fast2(ax, ay, bx, by, t.lut, cd.lut_bias, ca, cb);
        }
        if (k & 1) {
            ha = (uint32_t)ca;
            hb = (uint32_t)cb;
        } else {
            pa[k >> 1] = (ha << 8) | (uint32_t)ca;
            pb[k >> 1] = (hb << 8) | (uint32_t)cb;
        }
        const double2 wa = t.Wr[ca], wb = t.Wr[cb];
        decode_step(ax, ay, wa, cd.inv_r);
        decode_step(bx, by, wb, cd.inv_r);
    }
}

template <bool EXACT, bool VERIFY>
__global__ __launch_bounds__(kBlock, 8) void cgr_decode_kernel(
    const double2* __restrict__ pts, uint8_t* __restrict__ sym, uint8_t* __restrict__ span_ok,
    uint32_t* __restrict__ n_failed, const uint8_t* __restrict__ gtab, CodecArgs cd, int64_t n_sym,
    int64_t n_spans, int64_t wtiles_per_stream, int64_t n_wtiles, int stage_bytes)
{
    extern __shared__ __align__(16) uint8_t lds[];
    const int N = cd.N, L = cd.L;
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t wave = (int64_t)blockIdx.x * (kBlock / 64) + wv;
    const int64_t n_waves = (int64_t)gridDim.x * (kBlock / 64);
    TileWalk cur, nxt;
    cur.init(wave, n_waves, wtiles_per_stream);
    nxt = cur;
    nxt.next();
    // the first wave tile's points are loaded before the tables are staged,
    // so the two memory latencies overlap
    const double2 zero = make_double2(0.0, 0.0);
    double2 P0 = zero, P1 = zero;
    if (wave < n_wtiles) {
        const int64_t j = cur.j * kDecodeTile + lane;
        if (j < n_spans) P0 = load_point_stream(pts + cur.s * n_spans + j);
        if (j + 64 < n_spans) P1 = load_point_stream(pts + cur.s * n_spans + j + 64);
    }
    Tables t = stage_tables(gtab, N, lds, VERIFY, EXACT);
    uint8_t* stage = lds + staged_table_bytes(N, VERIFY, EXACT) + (size_t)wv * stage_bytes;
    __syncthreads();   // tables staged
    for (int64_t tw = wave; tw < n_wtiles; tw += n_waves, cur.next(), nxt.next()) {
        const int64_t s = cur.s;
        const int64_t j0 = cur.j * kDecodeTile;
        const int64_t nsp = min((int64_t)kDecodeTile, n_spans - j0);
        const int64_t g0 = s * n_sym + j0 * L;
        const int64_t g1 = s * n_sym + min(n_sym, (j0 + nsp) * L);
        double2 N0 = zero, N1 = zero;
        if (tw + n_waves < n_wtiles) {
            const int64_t j = nxt.j * kDecodeTile + lane;
            if (j < n_spans) N0 = load_point_stream(pts + nxt.s * n_spans + j);
            if (j + 64 < n_spans) N1 = load_point_stream(pts + nxt.s * n_spans + j + 64);
        }
        uint8_t* my0 = stage + (g0 & 3) + lane * L;
        uint8_t* my1 = my0 + 64 * L;
        bool f0 = false, f1 = false;
        bool direct = false;   // the tile's symbols already stored
        if (nsp == kDecodeTile && (j0 + kDecodeTile) * L <= n_sym) {
            // every span of the tile is whole: both chains run L steps in lockstep
            double ax = P0.x, ay = P0.y, bx = P1.x, by = P1.y;
            if (!VERIFY && L == 6 && (g0 & 1) == 0) {
                // symbols straight from registers to global memory, three
                // 16-bit stores per span (no LDS staging)
                uint32_t pa[3], pb[3];
                walk_two_regs6<EXACT>(ax, ay, bx, by, pa, pb, t, cd);
                uint16_t* da = (uint16_t*)(sym + g0 + lane * 6);
                uint16_t* db = (uint16_t*)(sym + g0 + (64 + lane) * 6);
#pragma unroll
                for (int q = 0; q < 3; ++q) {
                    __builtin_nontemporal_store((uint16_t)pa[q], da + q);
                    __builtin_nontemporal_store((uint16_t)pb[q], db + q);
                }
                direct = true;
            } else if (L == 6)   // N = 256, 64 and 16 at 0.98 r_N: fixed lengths, fully unrolled
                walk_two<6, EXACT>(ax, ay, bx, by, my0, my1, L, t, cd);
            else if (!EXACT && !VERIFY && L == 9)   // (unrolled, the checking instances would spill)
                walk_two<9, EXACT>(ax, ay, bx, by, my0, my1, L, t, cd);
            else if (!EXACT && !VERIFY && L == 16)
                walk_two<16, EXACT>(ax, ay, bx, by, my0, my1, L, t, cd);
            else
                walk_two<0, EXACT>(ax, ay, bx, by, my0, my1, L, t, cd);
            f0 = !decode_finish<EXACT, VERIFY>(ax, ay, P0, my0, L, t, cd);
            f1 = !decode_finish<EXACT, VERIFY>(bx, by, P1, my1, L, t, cd);
            if (span_ok) {
                span_ok[s * n_spans + j0 + lane] = f0 ? 0 : 1;
                span_ok[s * n_spans + j0 + 64 + lane] = f1 ? 0 : 1;
            }
        } else {
            // the stream's last tile: spans may be missing or short
            for (int h = 0; h < kDecodeSpl; ++h) {
                const int64_t jj = j0 + h * 64 + lane;
                if (jj >= j0 + nsp) continue;
                const int len = (int)min((int64_t)L, n_sym - jj * L);
                uint8_t* my = h ? my1 : my0;
                const double2 P = h ? P1 : P0;
                double qx = P.x, qy = P.y;
                for (int k = len - 1; k >= 0; --k) {
                    const int c = sector_of<EXACT>(qx, qy, t, cd);
                    my[k] = (uint8_t)c;
                    decode_step(qx, qy, t.Wr[c], cd.inv_r);
                }
                const bool bad = !decode_finish<EXACT, VERIFY>(qx, qy, P, my, len, t, cd);
                if (h) f1 = bad; else f0 = bad;
                if (span_ok) span_ok[s * n_spans + jj] = bad ? 0 : 1;
            }
        }
        count_flags(f0, n_failed);
        count_flags(f1, n_failed);
        // the wave's LDS writes above precede its reads below (a wave's LDS
        // operations are performed in order)
        __builtin_amdgcn_wave_barrier();
        if (!direct) lds_to_bytes_wave<true>(stage, g0, g1, sym, lane);
        P0 = N0;
        P1 = N1;
    }
}

// ------------------------------------------------------------------ lookup --

template <bool EXACT>
__global__ __launch_bounds__(kBlock) void span_lookup_kernel(
    const double2* __restrict__ pts, const uint32_t* __restrict__ q_stream,
    const uint32_t* __restrict__ q_token, uint8_t* __restrict__ out, uint8_t* __restrict__ q_status,
    uint32_t* __restrict__ n_failed, const uint8_t* __restrict__ gtab, CodecArgs cd, int64_t n_streams,
    int64_t n_sym, int64_t n_spans, int S, int64_t n_q)
{
    extern __shared__ __align__(16) uint8_t lds[];
    const int N = cd.N, L = cd.L;
    const int64_t n_tok = n_sym / S;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t n_iter = (n_q + stride - 1) / stride;  // same trip count for every lane
    // The first query and the point of its first span are loaded before the
    // tables are staged, so the memory latencies overlap.
    const int64_t q0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t s0 = 0, tk0 = 0;
    double2 P0 = make_double2(0.0, 0.0);
    if (q0 < n_q) {
        s0 = q_stream[q0];
        tk0 = q_token[q0];
        if (s0 < n_streams && tk0 < n_tok) P0 = pts[s0 * n_spans + tk0 * S / L];
    }
    Tables t = stage_tables(gtab, N, lds, false, EXACT);
    __syncthreads();
    for (int64_t it = 0; it < n_iter; ++it) {
        const int64_t q = it * stride + q0;
        int status = 0;
        uint64_t got = 0;
        if (q < n_q) {
            const int64_t s = it == 0 ? s0 : (int64_t)q_stream[q];
            const int64_t tk = it == 0 ? tk0 : (int64_t)q_token[q];
            if (s >= n_streams || tk >= n_tok)
                status = 2;
            else
                status = lookup_token<EXACT>(pts, t, cd, s, tk, S, n_sym, n_spans, it == 0, P0, &got);
            for (int k = 0; k < S; ++k) out[q * S + k] = (uint8_t)(got >> (8 * k));
            if (q_status) q_status[q] = (uint8_t)status;
        }
        count_flags(status != 0, n_failed);
    }
}

}  // namespace
}  // namespace fkv

using namespace fkv;

extern "C" int fkv_cgr_encode_spans(const fkv_codec* c, const void* dev_table, const uint8_t* symbols,
                                    int64_t n_streams, int64_t n_sym, double* points, void* stream)
{
    if (!codec_ok(c) || !dev_table || n_streams < 0 || n_sym < 0) return FKV_ERR_INVALID_ARG;
    if (n_streams == 0 || n_sym == 0) return FKV_OK;
    if (!symbols || !points || !aligned(dev_table, 16) || !aligned(points, 16) || !aligned(symbols, 4))
        return FKV_ERR_INVALID_ARG;
    if (n_sym % c->L == 0) {
        // whole spans: the streams sit back to back in both arrays, so they
        // are tiled as one run of spans (no partial tile at each stream's end)
        n_sym *= n_streams;
        n_streams = 1;
    }
    const int64_t n_spans = (n_sym + c->L - 1) / c->L;
    if (c->L <= 16) {
        const int64_t wtps = (n_spans + kEncTile - 1) / kEncTile;
        const int64_t n_wtiles = wtps * n_streams;
        const int64_t nb = min((int64_t)kMaxBlocks, (n_wtiles + kBlock / 64 - 1) / (kBlock / 64));
        auto go = [&](auto kern) {
            hipLaunchKernelGGL(kern, dim3((unsigned)nb), dim3(kBlock), 0, (hipStream_t)stream, symbols,
                               (double2*)points, (const uint8_t*)dev_table, codec_args(c), n_sym, n_spans, wtps,
                               n_wtiles, n_streams * n_sym);
        };
        if (c->L == 6)   // N = 256, 64 and 16 at 0.98 r_N
            go(cgr_encode_kernel<6>);
        else if (c->L == 9)
            go(cgr_encode_kernel<9>);
        else if (c->L == 16)
            go(cgr_encode_kernel<16>);
        else
            go(cgr_encode_kernel<0>);
        return launch_status();
    }
    const int64_t tps = (n_spans + kBlock - 1) / kBlock;
    const int64_t n_tiles = tps * n_streams;
    const size_t shm = 256 * 16 + (size_t)kBlock * c->L + 16;
    hipLaunchKernelGGL(cgr_encode_tiles_kernel, dim3((unsigned)blocks_for(n_tiles)), dim3(kBlock), shm,
                       (hipStream_t)stream, symbols, (double2*)points, (const uint8_t*)dev_table,
                       codec_args(c), n_sym, n_spans, tps, n_tiles);
    return launch_status();
}

extern "C" int fkv_cgr_decode_spans(const fkv_codec* c, const void* dev_table, const double* points,
                                    int64_t n_streams, int64_t n_sym, uint8_t* symbols, uint8_t* span_ok,
                                    uint32_t* n_failed, int32_t verify, void* stream)
{
    if (!codec_ok(c) || !dev_table || n_streams < 0 || n_sym < 0) return FKV_ERR_INVALID_ARG;
    if (verify != 0 && verify != 1) return FKV_ERR_INVALID_ARG;
    if (n_streams == 0 || n_sym == 0) return FKV_OK;
    if (!symbols || !points || !aligned(dev_table, 16) || !aligned(points, 16) || !aligned(symbols, 4))
        return FKV_ERR_INVALID_ARG;
    if (n_failed && !aligned(n_failed, 4)) return FKV_ERR_INVALID_ARG;
    if (n_sym % c->L == 0) {
        // whole spans: the streams sit back to back in all three arrays, so
        // they are tiled as one run of spans (no partial tile at each stream's
        // end, which would take the per-span path)
        n_sym *= n_streams;
        n_streams = 1;
    }
    const int64_t n_spans = (n_sym + c->L - 1) / c->L;
    const int64_t wtps = (n_spans + kDecodeTile - 1) / kDecodeTile;
    const int64_t n_wtiles = wtps * n_streams;
    const int stage_bytes = (kDecodeTile * c->L + 4 + 15) / 16 * 16;   // one wave tile's symbols, dword-shifted
    const bool exact = needs_exact_sectors(c);
    const size_t shm = staged_table_bytes(c->N, verify != 0, exact) + (size_t)(kBlock / 64) * stage_bytes;
    const dim3 grid((unsigned)min((int64_t)kMaxBlocks, (n_wtiles + kBlock / 64 - 1) / (kBlock / 64))), block(kBlock);
    const hipStream_t st = (hipStream_t)stream;
    const double2* P = (const double2*)points;
    const uint8_t* tb = (const uint8_t*)dev_table;
    const CodecArgs a = codec_args(c);
    if (exact && verify)
        hipLaunchKernelGGL((cgr_decode_kernel<true, true>), grid, block, shm, st, P, symbols, span_ok,
                           n_failed, tb, a, n_sym, n_spans, wtps, n_wtiles, stage_bytes);
    else if (exact)
        hipLaunchKernelGGL((cgr_decode_kernel<true, false>), grid, block, shm, st, P, symbols, span_ok,
                           n_failed, tb, a, n_sym, n_spans, wtps, n_wtiles, stage_bytes);
    else if (verify)
        hipLaunchKernelGGL((cgr_decode_kernel<false, true>), grid, block, shm, st, P, symbols, span_ok,
                           n_failed, tb, a, n_sym, n_spans, wtps, n_wtiles, stage_bytes);
    else
        hipLaunchKernelGGL((cgr_decode_kernel<false, false>), grid, block, shm, st, P, symbols, span_ok,
                           n_failed, tb, a, n_sym, n_spans, wtps, n_wtiles, stage_bytes);
    return launch_status();
}

extern "C" int fkv_span_lookup(const fkv_codec* c, const void* dev_table, const double* points,
                               int64_t n_streams, int64_t n_sym, int32_t S, const uint32_t* q_stream,
                               const uint32_t* q_token, int64_t n_q, uint8_t* out, uint8_t* q_status,
                               uint32_t* n_failed, void* stream)
{
    if (!codec_ok(c) || !dev_table || n_streams < 0 || n_sym < 0 || n_q < 0) return FKV_ERR_INVALID_ARG;
    if (S < 1 || S > 8 || n_sym % S != 0) return FKV_ERR_INVALID_ARG;
    if (n_q == 0) return FKV_OK;
    if (!q_stream || !q_token || !out || !aligned(dev_table, 16)) return FKV_ERR_INVALID_ARG;
    if (n_streams > 0 && n_sym > 0 && (!points || !aligned(points, 16))) return FKV_ERR_INVALID_ARG;
    if (!aligned(q_stream, 4) || !aligned(q_token, 4)) return FKV_ERR_INVALID_ARG;
    if (n_failed && !aligned(n_failed, 4)) return FKV_ERR_INVALID_ARG;
    const int64_t n_spans = (n_sym + c->L - 1) / c->L;
    const bool exact = needs_exact_sectors(c);
    const size_t shm = staged_table_bytes(c->N, false, exact);
    const int64_t nb = blocks_for((n_q + kBlock - 1) / kBlock);
    const hipStream_t st = (hipStream_t)stream;
    if (exact)
        hipLaunchKernelGGL((span_lookup_kernel<true>), dim3((unsigned)nb), dim3(kBlock), shm, st,
                           (const double2*)points, q_stream, q_token, out, q_status, n_failed,
                           (const uint8_t*)dev_table, codec_args(c), n_streams, n_sym, n_spans, S, n_q);
    else
        hipLaunchKernelGGL((span_lookup_kernel<false>), dim3((unsigned)nb), dim3(kBlock), shm, st,
                           (const double2*)points, q_stream, q_token, out, q_status, n_failed,
                           (const uint8_t*)dev_table, codec_args(c), n_streams, n_sym, n_spans, S, n_q);
    return launch_status();
}
