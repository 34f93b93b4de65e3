// cgr_kernels.hip -- fixed-span chaos-game (iterated-map) encode, bulk span
// decode and O(1) random access for gfx950.
//
// Method (Sec. 1 "The code" and Sec. 2 of the paper): symbol c maps the running
// point by p <- V(c) + r (p - V(c)); a span of L symbols starting at the anchor
// (0,0) is stored as its final point.  Decoding reads the symbol off the cell
// (sector) that holds the point and inverts the map, p <- (p - (1-r)V(c)) / r,
// walking back to the anchor.
//
// Layout: one span per lane, 256 spans per block tile, tiles of one stream are
// contiguous in both the symbol bytes and the 16-byte points, so every global
// access of a tile is a coalesced stream; symbol bytes are staged through LDS.
// The per-alphabet tables (vertices, cell centres, sector look-up) live in LDS
// for the whole persistent block.
//
// Floating point: the encode recurrence must be bit-reproducible, so this file
// is compiled without FP contraction, and fused multiply-adds appear only where
// written explicitly (decode's inverse map, whose points are never compared --
// only the symbols they yield).
#include "cgr_device.h"

namespace fkv {
namespace {

// ------------------------------------------------------------------ encode --

__global__ __launch_bounds__(kBlock) void cgr_encode_kernel(
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
    for (int64_t tl = blockIdx.x; tl < n_tiles; tl += gridDim.x) {
        const int64_t s = tl / tiles_per_stream;
        const int64_t j0 = (tl - s * tiles_per_stream) * kBlock;
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
            pts[s * n_spans + j0 + threadIdx.x] = make_double2(px, py);
        }
    }
}

// ------------------------------------------------------------------ decode --

template <bool EXACT, bool VERIFY>
__global__ __launch_bounds__(kBlock) void cgr_decode_kernel(
    const double2* __restrict__ pts, uint8_t* __restrict__ sym, uint8_t* __restrict__ span_ok,
    uint32_t* __restrict__ n_failed, const uint8_t* __restrict__ gtab, CodecArgs cd, int64_t n_sym,
    int64_t n_spans, int64_t tiles_per_stream, int64_t n_tiles)
{
    extern __shared__ __align__(16) uint8_t lds[];
    const int N = cd.N, L = cd.L;
    // The first tile's point is loaded before the tables are staged, so the
    // two memory latencies overlap.
    double2 P0 = make_double2(0.0, 0.0);
    if ((int64_t)blockIdx.x < n_tiles) {
        const int64_t s = (int64_t)blockIdx.x / tiles_per_stream;
        const int64_t j0 = ((int64_t)blockIdx.x - s * tiles_per_stream) * kBlock;
        if ((int64_t)threadIdx.x < min((int64_t)kBlock, n_spans - j0)) P0 = pts[s * n_spans + j0 + threadIdx.x];
    }
    Tables t = stage_tables(gtab, N, lds, VERIFY, EXACT);
    uint8_t* tile = lds + table_bytes(N);
    for (int64_t tl = blockIdx.x; tl < n_tiles; tl += gridDim.x) {
        const int64_t s = tl / tiles_per_stream;
        const int64_t j0 = (tl - s * tiles_per_stream) * kBlock;
        const int64_t nsp = min((int64_t)kBlock, n_spans - j0);
        const int64_t g0 = s * n_sym + j0 * L;
        const int64_t g1 = s * n_sym + min(n_sym, (j0 + nsp) * L);
        __syncthreads();  // tables staged / previous tile flushed
        bool failed = false;
        if (threadIdx.x < nsp) {
            const int64_t a = (j0 + threadIdx.x) * L;
            const int len = (int)min((int64_t)L, n_sym - a);
            uint8_t* my = tile + (g0 & 3) + threadIdx.x * L;
            const double2 P = tl == (int64_t)blockIdx.x ? P0 : pts[s * n_spans + j0 + threadIdx.x];
            double qx = P.x, qy = P.y;
            for (int k = len - 1; k >= 0; --k) {
                const int c = sector_of<EXACT>(qx, qy, t, N);
                my[k] = (uint8_t)c;
                decode_step(qx, qy, t.Wr[c], cd.inv_r);
            }
            bool ok = anchor_ok(qx, qy);
            if (VERIFY) {
                double px = 0.0, py = 0.0;
                for (int k = 0; k < len; ++k) encode_step(px, py, t.V[my[k]], cd.r);
                ok = ok && (__double_as_longlong(px) == __double_as_longlong(P.x)) &&
                     (__double_as_longlong(py) == __double_as_longlong(P.y));
            }
            if (span_ok) span_ok[s * n_spans + j0 + threadIdx.x] = ok ? 1 : 0;
            failed = !ok;
        }
        count_flags(failed, n_failed);
        __syncthreads();
        lds_to_bytes(tile, g0, g1, sym);
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
    const int64_t n_spans = (n_sym + c->L - 1) / c->L;
    const int64_t tps = (n_spans + kBlock - 1) / kBlock;
    const int64_t n_tiles = tps * n_streams;
    const size_t shm = 256 * 16 + (size_t)kBlock * c->L + 16;
    hipLaunchKernelGGL(cgr_encode_kernel, dim3((unsigned)blocks_for(n_tiles)), dim3(kBlock), shm,
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
    const int64_t n_spans = (n_sym + c->L - 1) / c->L;
    const int64_t tps = (n_spans + kBlock - 1) / kBlock;
    const int64_t n_tiles = tps * n_streams;
    const size_t shm = table_bytes(c->N) + (size_t)kBlock * c->L + 16;
    const bool exact = needs_exact_sectors(c);
    const dim3 grid((unsigned)blocks_for(n_tiles)), block(kBlock);
    const hipStream_t st = (hipStream_t)stream;
    const double2* P = (const double2*)points;
    const uint8_t* tb = (const uint8_t*)dev_table;
    const CodecArgs a = codec_args(c);
    if (exact && verify)
        hipLaunchKernelGGL((cgr_decode_kernel<true, true>), grid, block, shm, st, P, symbols, span_ok,
                           n_failed, tb, a, n_sym, n_spans, tps, n_tiles);
    else if (exact)
        hipLaunchKernelGGL((cgr_decode_kernel<true, false>), grid, block, shm, st, P, symbols, span_ok,
                           n_failed, tb, a, n_sym, n_spans, tps, n_tiles);
    else if (verify)
        hipLaunchKernelGGL((cgr_decode_kernel<false, true>), grid, block, shm, st, P, symbols, span_ok,
                           n_failed, tb, a, n_sym, n_spans, tps, n_tiles);
    else
        hipLaunchKernelGGL((cgr_decode_kernel<false, false>), grid, block, shm, st, P, symbols, span_ok,
                           n_failed, tb, a, n_sym, n_spans, tps, n_tiles);
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
    const size_t shm = table_bytes(c->N);
    const int64_t nb = blocks_for((n_q + kBlock - 1) / kBlock);
    const bool exact = needs_exact_sectors(c);
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
