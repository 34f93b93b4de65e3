// archive_kernels.hip -- reading reconstructions out of the archive and
// appending to it, for gfx950.
//
// Rehydrate (Sec. 3 "Setup": an archived position's K/V vector is replaced by
// the sum of its S codewords; Sec. 5: a matched position is rehydrated from the
// archive alone): random access to the token's S symbols (one query per lane,
// as in span lookup), then a block-cooperative gather of the codeword rows --
// consecutive lanes take consecutive 16-byte chunks of one output row, so the
// codeword reads and the output writes are contiguous runs.  The S codewords
// are summed in fp64 (exact for a few binary16 values) and rounded once to
// binary16, so the result is the correctly rounded reconstruction.
//
// Append (Sec. 2, Table 1): one stream per lane re-walks from its last stored
// point; a span that starts at a multiple of L starts from the anchor (0,0).
// The forward step is the bulk encoder's, operation for operation, so the
// points equal a bulk encode of the whole stream bit for bit.
#include "cgr_device.h"

namespace fkv {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));

// ---------------------------------------------------------------- rehydrate --

// A block takes QB queries at a time (64 while the grid has room for that
// many blocks, else kBlock): its first QB threads look them up (one lane
// each) into LDS, then all kBlock threads rebuild the output rows, up to
// kRehydU (query, 16-byte chunk) tasks per thread with their codebook-row
// loads issued together, two stages at a time.
constexpr int kRehydU = 2;

template <int QB, bool EXACT>
__global__ __launch_bounds__(kBlock) void rehydrate_kernel(
    const double2* __restrict__ pts, const uint32_t* __restrict__ q_stream,
    const uint32_t* __restrict__ q_token, const _Float16* __restrict__ books,
    const int32_t* __restrict__ stream_book, _Float16* __restrict__ out, uint8_t* __restrict__ q_status,
    uint32_t* __restrict__ n_failed, const uint8_t* __restrict__ gtab, CodecArgs cd, int64_t n_streams,
    int64_t n_sym, int64_t n_spans, int S, int K, int d, int n_books, int64_t n_q)
{
    extern __shared__ __align__(16) uint8_t lds[];
    const int N = cd.N;
    // the first batch's query ids load while the tables are staged; each
    // batch loads the next one's
    int64_t qs_n = 0, qt_n = 0;
    {
        const int64_t q0 = (int64_t)blockIdx.x * QB + threadIdx.x;
        if (threadIdx.x < QB && q0 < n_q) {
            qs_n = q_stream[q0];
            qt_n = q_token[q0];
        }
    }
    Tables t = stage_tables(gtab, N, lds, false, EXACT);
    // After the tables: each query of the current batch's book id (-1: no
    // output) and its packed symbols.
    int32_t* qbook = (int32_t*)(lds + staged_table_bytes(N, false, EXACT));
    uint64_t* qsym = (uint64_t*)(lds + staged_table_bytes(N, false, EXACT) + QB * sizeof(int32_t));
    __syncthreads();
    const int64_t n_tok = n_sym / S;
    const int nch = d / 8;   // 16-byte chunks per output row
    for (int64_t base = (int64_t)blockIdx.x * QB; base < n_q; base += (int64_t)gridDim.x * QB) {
        if (threadIdx.x < QB) {
            const int64_t q = base + threadIdx.x;
            const int64_t s = qs_n, tk = qt_n;
            const int64_t qn = q + (int64_t)gridDim.x * QB;
            if (qn < n_q) {
                qs_n = q_stream[qn];
                qt_n = q_token[qn];
            }
            int status = 0;
            uint64_t got = 0;
            int32_t b = -1;
            if (q < n_q) {
                if (s >= n_streams || tk >= n_tok) {
                    status = 2;
                } else {
                    b = stream_book[s];   // loads beside the point
                    status = lookup_token<EXACT>(pts, t, cd, s, tk, S, n_sym, n_spans, false,
                                                 make_double2(0.0, 0.0), &got);
                    if (status == 0) {
                        if (b < 0 || b >= n_books) status = 3;
                        for (int k = 0; k < S; ++k)
                            if ((int)((got >> (8 * k)) & 0xff) >= K) status = 3;
                    }
                }
                if (q_status) q_status[q] = (uint8_t)status;
            }
            count_flags(status != 0, n_failed);
            qbook[threadIdx.x] = status == 0 ? b : -1;
            qsym[threadIdx.x] = got;
        }
        __syncthreads();
        const int nq = (int)min((int64_t)QB, n_q - base);
        const int n_tasks = nq * nch;
        for (int t0 = threadIdx.x; t0 < n_tasks; t0 += kRehydU * kBlock) {
            int ql[kRehydU], ch[kRehydU];
            int32_t bb[kRehydU];
            uint64_t sy[kRehydU];
            double acc[kRehydU][8];
#pragma unroll
            for (int u = 0; u < kRehydU; ++u) {
                const int task = t0 + u * kBlock;
                ql[u] = task < n_tasks ? task / nch : 0;
                ch[u] = task - ql[u] * nch;
                bb[u] = task < n_tasks ? qbook[ql[u]] : -1;
                sy[u] = qsym[ql[u]];
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[u][e] = 0.0;
            }
            // stages k and k + 1: every load first, then the sums in stage order
            for (int k = 0; k < S; k += 2) {
                half8 v0[kRehydU], v1[kRehydU];
#pragma unroll
                for (int u = 0; u < kRehydU; ++u) {
                    v0[u] = v1[u] = (half8)(_Float16)0;
                    if (bb[u] >= 0) {
                        const _Float16* row = books + ((int64_t)bb[u] * S + k) * K * d + ch[u] * 8;
                        v0[u] = *(const half8*)(row + (int64_t)((sy[u] >> (8 * k)) & 0xff) * d);
                        if (k + 1 < S)
                            v1[u] = *(const half8*)(row + (int64_t)K * d +
                                                    (int64_t)((sy[u] >> (8 * (k + 1))) & 0xff) * d);
                    }
                }
#pragma unroll
                for (int u = 0; u < kRehydU; ++u)
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[u][e] = acc[u][e] + (double)v0[u][e];
                if (k + 1 < S) {
#pragma unroll
                    for (int u = 0; u < kRehydU; ++u)
#pragma unroll
                        for (int e = 0; e < 8; ++e) acc[u][e] = acc[u][e] + (double)v1[u][e];
                }
            }
#pragma unroll
            for (int u = 0; u < kRehydU; ++u) {
                if (t0 + u * kBlock < n_tasks) {
                    half8 o;
#pragma unroll
                    for (int e = 0; e < 8; ++e) o[e] = f64_to_f16(acc[u][e]);
                    *(half8*)(out + (base + ql[u]) * d + ch[u] * 8) = o;
                }
            }
        }
        __syncthreads();   // the batch's query table is consumed
    }
}

// ------------------------------------------------------------------- append --

__global__ __launch_bounds__(kBlock) void append_kernel(double2* __restrict__ pts,
                                                         const uint8_t* __restrict__ sym_new,
                                                         const uint8_t* __restrict__ gtab, CodecArgs cd,
                                                         int64_t cap_spans, int64_t n_streams, int64_t n_old,
                                                         int64_t m)
{
    __shared__ double2 V[256];   // entries >= N are NaN: a symbol outside the alphabet gives NaN
    const int N = cd.N, L = cd.L;
    V[threadIdx.x] = (int)threadIdx.x < N ? ((const double2*)(gtab + table_off_V(N)))[threadIdx.x]
                                          : make_double2(NAN, NAN);
    __syncthreads();
    for (int64_t s = (int64_t)blockIdx.x * kBlock + threadIdx.x; s < n_streams;
         s += (int64_t)gridDim.x * kBlock) {
        double2* P = pts + s * cap_spans;
        double px = 0.0, py = 0.0;
        if (n_old % L != 0) {
            const double2 p = P[n_old / L];
            px = p.x;
            py = p.y;
        }
        const uint8_t* my = sym_new + s * m;
        for (int64_t k = 0; k < m; ++k) {
            const int64_t pos = n_old + k;
            if (pos % L == 0) {
                px = 0.0;
                py = 0.0;
            }
            encode_step(px, py, V[my[k]], cd.r);
            if ((pos + 1) % L == 0 || k == m - 1) P[pos / L] = make_double2(px, py);
        }
    }
}

// --------------------------------------------------------------- retrieval --
// Sec. 5: the per-position index holds, for every symbol position k, the
// point of the walk over the W symbols ending at k, from the origin (one lane
// per position: W forward steps over a symbol tile staged in LDS).  A suffix
// query of ell symbols is encoded from the origin to q; every indexed position
// with ell symbols of history whose point lies within 2 r^ell of q is a
// candidate, kept when decoding ell symbols backward from it reproduces the
// query.  The scan streams the index once (16 bytes per position).

// WC > 0: the window length is WC, known at compile time, and full windows
// are walked fully unrolled (the first WC - 1 positions of a stream, with
// shorter windows, take the loop).
template <int WC>
__global__ __launch_bounds__(kBlock) void trajectory_kernel(const uint8_t* __restrict__ sym,
                                                             double2* __restrict__ traj,
                                                             const uint8_t* __restrict__ gtab, CodecArgs cd,
                                                             int64_t n_sym, int W, int64_t tiles_per_stream,
                                                             int64_t n_tiles)
{
    extern __shared__ __align__(16) uint8_t lds[];
    const int N = cd.N;
    double2* V = (double2*)lds;
    uint8_t* tile = lds + 256 * sizeof(double2);
    V[threadIdx.x] = (int)threadIdx.x < N ? ((const double2*)(gtab + table_off_V(N)))[threadIdx.x]
                                          : make_double2(NAN, NAN);
    TileWalk w;
    w.init(blockIdx.x, gridDim.x, tiles_per_stream);
    for (int64_t tl = blockIdx.x; tl < n_tiles; tl += gridDim.x, w.next()) {
        const int64_t s = w.s;
        const int64_t k0 = w.j * kBlock;
        const int64_t a0 = max((int64_t)0, k0 - W + 1);
        const int64_t k1 = min(n_sym, k0 + kBlock);
        const int64_t g0 = s * n_sym + a0, g1 = s * n_sym + k1;
        __syncthreads();   // previous tile consumed
        bytes_to_lds(sym, g0, g1, tile);
        __syncthreads();
        const int64_t k = k0 + threadIdx.x;
        if (k < k1) {
            const int Wn = WC > 0 ? WC : W;
            const int64_t a = max((int64_t)0, k - Wn + 1);
            const uint8_t* my = tile + (g0 & 3) + (int)(a - a0);
            const int len = (int)(k - a) + 1;
            double px = 0.0, py = 0.0;
            if (WC > 0 && len == WC) {
                double2 v[WC > 0 ? WC : 1];
#pragma unroll
                for (int u = 0; u < WC; ++u) v[u] = V[my[u]];
#pragma unroll
                for (int u = 0; u < WC; ++u) encode_step(px, py, v[u], cd.r);
            } else {
                for (int j = 0; j < len; ++j) encode_step(px, py, V[my[j]], cd.r);
            }
            store_point_stream(traj + s * n_sym + k, px, py);
        }
    }
}

template <bool EXACT, bool VERIFY>
__global__ __launch_bounds__(kBlock) void suffix_search_kernel(
    const double2* __restrict__ traj, const uint8_t* __restrict__ query, const uint8_t* __restrict__ gtab,
    CodecArgs cd, int64_t n_streams, int64_t n_sym, int ell, uint32_t* __restrict__ hits, int64_t max_hits,
    uint32_t* __restrict__ n_hits, uint32_t* __restrict__ n_cand)
{
    extern __shared__ __align__(16) uint8_t lds[];
    const int N = cd.N;
    Tables t = stage_tables(gtab, N, lds, true, EXACT);
    uint8_t* qs = lds + staged_table_bytes(N, true, EXACT);
    if ((int)threadIdx.x < ell) qs[threadIdx.x] = query[threadIdx.x];
    __syncthreads();
    // the query's point from the origin and the threshold, as in the index; a
    // query symbol outside the alphabet matches nothing
    bool qok = true;
    for (int j = 0; j < ell; ++j) qok = qok && qs[j] < N;
    double qx = 0.0, qy = 0.0;
    for (int j = 0; j < ell; ++j) encode_step(qx, qy, t.V[qok ? qs[j] : 0], cd.r);
    double rl = 1.0;
    for (int j = 0; j < ell; ++j) rl = rl * cd.r;
    const double thr = 2.0 * rl;
    const double thr2 = thr * thr;
    const int64_t total = n_streams * n_sym;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t n_iter = (total + stride - 1) / stride;   // same trip count for every lane
    const int lane = threadIdx.x & 63;
    // (stream, position) of this thread's index entry, advanced by the grid
    // stride with additions only: the stride is ds streams and dk < n_sym
    // positions
    const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t ds = stride / n_sym, dk = stride - ds * n_sym;
    int64_t s = i0 / n_sym, k = i0 - s * n_sym;
    for (int64_t it = 0; it < n_iter; ++it) {
        const int64_t i = it * stride + i0;
        if (it > 0) {
            s += ds;
            k += dk;
            if (k >= n_sym) {
                k -= n_sym;
                ++s;
            }
        }
        bool cand = false, hit = false;
        if (i < total) {
            if (qok && k >= ell - 1) {
                const double2 p = load_point_stream(traj + i);
                const double dx = p.x - qx, dy = p.y - qy;
                const double d2 = dx * dx + dy * dy;
                cand = d2 <= thr2;
                hit = cand;
                if (VERIFY && cand) {
                    double x = p.x, y = p.y;
                    for (int j = ell - 1; j >= 0; --j) {
                        const int c = sector_of<EXACT>(x, y, t, cd);
                        if (c != qs[j]) {
                            hit = false;
                            break;
                        }
                        decode_step(x, y, t.Wr[c], cd.inv_r);
                    }
                }
            }
        }
        const unsigned long long mc = __ballot(cand), mh = __ballot(hit);
        if (n_cand && mc && lane == 0) atomicAdd(n_cand, (uint32_t)__popcll(mc));
        if (mh) {
            uint32_t base = 0;
            if (lane == 0) base = atomicAdd(n_hits, (uint32_t)__popcll(mh));
            base = __shfl(base, 0);
            if (hit) {
                const int64_t slot = (int64_t)base + __popcll(mh & ((1ull << lane) - 1));
                if (slot < max_hits) {
                    hits[2 * slot] = (uint32_t)s;
                    hits[2 * slot + 1] = (uint32_t)k;
                }
            }
        }
    }
}

}  // namespace
}  // namespace fkv

using namespace fkv;

extern "C" int fkv_rehydrate(const fkv_codec* c, const void* dev_table, const double* points,
                             int64_t n_streams, int64_t n_sym, int32_t S, const uint16_t* books_f16,
                             const int32_t* stream_book, int32_t n_books, int32_t K, int32_t d,
                             const uint32_t* q_stream, const uint32_t* q_token, int64_t n_q,
                             uint16_t* out_f16, uint8_t* q_status, uint32_t* n_failed, void* stream)
{
    if (!codec_ok(c) || !dev_table || n_streams < 0 || n_sym < 0 || n_q < 0) return FKV_ERR_INVALID_ARG;
    if (S < 1 || S > 8 || n_sym % S != 0) return FKV_ERR_INVALID_ARG;
    if (n_books < 1 || K < 1 || K > 256 || d < 8 || d > 256 || d % 8 != 0) return FKV_ERR_INVALID_ARG;
    if (n_q == 0) return FKV_OK;
    if (!q_stream || !q_token || !out_f16 || !books_f16 || !aligned(dev_table, 16)) return FKV_ERR_INVALID_ARG;
    if (n_streams > 0 && n_sym > 0 && (!points || !aligned(points, 16) || !stream_book))
        return FKV_ERR_INVALID_ARG;
    if (!aligned(books_f16, 16) || !aligned(out_f16, 16) || !aligned(q_stream, 4) || !aligned(q_token, 4))
        return FKV_ERR_INVALID_ARG;
    if ((stream_book && !aligned(stream_book, 4)) || (n_failed && !aligned(n_failed, 4)))
        return FKV_ERR_INVALID_ARG;
    const int64_t n_spans = (n_sym + c->L - 1) / c->L;
    const bool small_batches = (n_q + 63) / 64 <= kMaxBlocks;
    const int qb = small_batches ? 64 : kBlock;
    const size_t shm =
        staged_table_bytes(c->N, false, needs_exact_sectors(c)) + (size_t)qb * (sizeof(int32_t) + sizeof(uint64_t));
    const int64_t nb = blocks_for((n_q + qb - 1) / qb);
    const hipStream_t st = (hipStream_t)stream;
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3((unsigned)nb), dim3(kBlock), shm, st, (const double2*)points, q_stream, q_token,
                           (const _Float16*)books_f16, stream_book, (_Float16*)out_f16, q_status, n_failed,
                           (const uint8_t*)dev_table, codec_args(c), n_streams, n_sym, n_spans, S, K, d, n_books,
                           n_q);
    };
    if (needs_exact_sectors(c))
        small_batches ? go(rehydrate_kernel<64, true>) : go(rehydrate_kernel<kBlock, true>);
    else
        small_batches ? go(rehydrate_kernel<64, false>) : go(rehydrate_kernel<kBlock, false>);
    return launch_status();
}

extern "C" int fkv_cgr_append(const fkv_codec* c, const void* dev_table, double* points, int64_t cap_spans,
                              int64_t n_streams, int64_t n_old, const uint8_t* sym_new, int64_t m,
                              void* stream)
{
    if (!codec_ok(c) || !dev_table || cap_spans < 0 || n_streams < 0 || n_old < 0 || m < 0)
        return FKV_ERR_INVALID_ARG;
    if ((n_old + m + c->L - 1) / c->L > cap_spans) return FKV_ERR_INVALID_ARG;
    if (n_streams == 0 || m == 0) return FKV_OK;
    if (!points || !sym_new || !aligned(points, 16) || !aligned(dev_table, 16)) return FKV_ERR_INVALID_ARG;
    const int64_t nb = blocks_for((n_streams + kBlock - 1) / kBlock);
    hipLaunchKernelGGL(append_kernel, dim3((unsigned)nb), dim3(kBlock), 0, (hipStream_t)stream,
                       (double2*)points, sym_new, (const uint8_t*)dev_table, codec_args(c), cap_spans, n_streams,
                       n_old, m);
    return launch_status();
}

extern "C" int fkv_trajectory(const fkv_codec* c, const void* dev_table, const uint8_t* symbols,
                              int64_t n_streams, int64_t n_sym, int32_t W, double* traj, void* stream)
{
    if (!codec_ok(c) || !dev_table || n_streams < 0 || n_sym < 0 || W < 1 || W > 64) return FKV_ERR_INVALID_ARG;
    if (n_streams == 0 || n_sym == 0) return FKV_OK;
    if (!symbols || !traj || !aligned(symbols, 4) || !aligned(traj, 16) || !aligned(dev_table, 16))
        return FKV_ERR_INVALID_ARG;
    const int64_t tps = (n_sym + kBlock - 1) / kBlock;
    const int64_t n_tiles = tps * n_streams;
    const size_t shm = 256 * 16 + (size_t)kBlock + 64 + 16;
    // the codec's own span length L is the usual window: 6, 9 and 16 for N = 256, 64 and 16
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3((unsigned)blocks_for(n_tiles)), dim3(kBlock), shm, (hipStream_t)stream, symbols,
                           (double2*)traj, (const uint8_t*)dev_table, codec_args(c), n_sym, W, tps, n_tiles);
    };
    if (W == 6)
        go(trajectory_kernel<6>);
    else if (W == 9)
        go(trajectory_kernel<9>);
    else if (W == 16)
        go(trajectory_kernel<16>);
    else
        go(trajectory_kernel<0>);
    return launch_status();
}

extern "C" int fkv_suffix_search(const fkv_codec* c, const void* dev_table, const double* traj, int64_t n_streams,
                                 int64_t n_sym, const uint8_t* query, int32_t ell, int32_t verify, uint32_t* hits,
                                 int64_t max_hits, uint32_t* n_hits, uint32_t* n_candidates, void* stream)
{
    if (!codec_ok(c) || !dev_table || n_streams < 0 || n_sym < 0 || max_hits < 0) return FKV_ERR_INVALID_ARG;
    if (ell < 1 || ell > c->L || (verify != 0 && verify != 1) || !query || !n_hits) return FKV_ERR_INVALID_ARG;
    if (max_hits > 0 && (!hits || !aligned(hits, 8))) return FKV_ERR_INVALID_ARG;
    if (!aligned(n_hits, 4) || (n_candidates && !aligned(n_candidates, 4)) || !aligned(dev_table, 16))
        return FKV_ERR_INVALID_ARG;
    if (n_streams == 0 || n_sym == 0) return FKV_OK;
    if (!traj || !aligned(traj, 16)) return FKV_ERR_INVALID_ARG;
    const bool exact = needs_exact_sectors(c);
    const size_t shm = staged_table_bytes(c->N, true, exact) + 64;
    const int64_t nb = blocks_for((n_streams * n_sym + kBlock - 1) / kBlock);
    const dim3 grid((unsigned)nb), block(kBlock);
    const hipStream_t st = (hipStream_t)stream;
    const double2* T = (const double2*)traj;
    const uint8_t* tb = (const uint8_t*)dev_table;
    const CodecArgs a = codec_args(c);
    if (exact && verify)
        hipLaunchKernelGGL((suffix_search_kernel<true, true>), grid, block, shm, st, T, query, tb, a, n_streams,
                           n_sym, ell, hits, max_hits, n_hits, n_candidates);
    else if (exact)
        hipLaunchKernelGGL((suffix_search_kernel<true, false>), grid, block, shm, st, T, query, tb, a, n_streams,
                           n_sym, ell, hits, max_hits, n_hits, n_candidates);
    else if (verify)
        hipLaunchKernelGGL((suffix_search_kernel<false, true>), grid, block, shm, st, T, query, tb, a, n_streams,
                           n_sym, ell, hits, max_hits, n_hits, n_candidates);
    else
        hipLaunchKernelGGL((suffix_search_kernel<false, false>), grid, block, shm, st, T, query, tb, a, n_streams,
                           n_sym, ell, hits, max_hits, n_hits, n_candidates);
    return launch_status();
}
