/*
 * fkv.h -- C ABI of libfkv, the MI355X (gfx950) hot path of the fractal
 * KV-cache archive (Gusev, "Fractal KV-Cache Archives: Lossless Symbolic
 * Storage with In-Place Retrieval for Long-Context LLM Inference",
 * arXiv 2607.07144).
 *
 * The archive stores a quantized KV cache as symbol streams (codebook indices
 * from per-head residual VQ, Sec. 3 "Setup") serialised by a contractive
 * iterated-map (chaos-game) code on a regular N-gon, one fp64 point per
 * fixed-length span (Sec. 1 "The code", Sec. 2).  The calls below are the
 * steps of that path: residual-VQ assignment, span encode, bulk span decode
 * and O(1) random access.
 *
 * Conventions shared by every call:
 *   - Device pointers are plain device addresses owned by the caller (for
 *     example PyTorch tensors); the library never allocates, frees or
 *     synchronises in these calls, and keeps no global mutable state, so
 *     calls are re-entrant -- except fkv_kmeans_update_noalloc, whose device
 *     scratch array is shared by every call on one device (see its comment).
 *     `stream` is a hipStream_t (NULL = the null stream); all device work is
 *     enqueued on it asynchronously.
 *   - Arguments are validated on the host before anything is enqueued.  An
 *     invalid call returns a negative fkv_status and has no side effect.
 *   - Data-dependent outcomes (a span failing its anchor check, an
 *     out-of-range lookup, an invalid book id) are reported on the device
 *     only, through the optional per-item status arrays and counters.
 *     Counters are ACCUMULATED with atomic adds: the caller zeroes them.
 *   - Symbols are bytes (alphabets of at most 256 letters).  A symbol value
 *     >= N in an encode input is invalid input: the affected span's point is
 *     NaN.
 *   - Layouts are row-major C arrays as written in each comment.
 */
#ifndef FKV_H
#define FKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FKV_OK = 0,
    FKV_ERR_INVALID_ARG = -1, /* a null pointer, a size or value out of range, a bad alignment */
    FKV_ERR_UNSUPPORTED = -2, /* valid by the paper but outside what this library implements */
    FKV_ERR_LAUNCH = -3,      /* the HIP runtime refused the launch (hipGetLastError) */
    FKV_ERR_NO_DEVICE = -4,   /* no usable gfx950 device is current */
    FKV_ERR_SCRATCH_TOO_SMALL = -5 /* the input needs more than the library's fixed device scratch
                                      (allocation-free entry points only) */
} fkv_status;

/* Codec parameters of one alphabet (Sec. 1 "The code"; Fig. 1).
 *   N      alphabet size, 3 <= N <= 256; vertex c of the regular N-gon is at
 *          angle 2*pi*c/N on the unit circle centred at the origin
 *   r_max  the packing limit r_N below which the N cells (contracted copies
 *          of the polygon) are pairwise disjoint, r_N = s/(s+m) with
 *          s = sin(pi/N), m = max_j sin((2j+1)pi/N); r_3 = r_4 = 1/2
 *   r      the contraction ratio, r = r_scale * r_N
 *   L      symbols per stored point: floor(44 / log2(1/r)) (the precision
 *          budget of one double, Sec. 1), or an explicit override */
typedef struct {
    int32_t N;
    int32_t L;
    double r;
    double r_max;
} fkv_codec;

/* Fills *out for alphabet N.  r_scale in (0, 1]; L_override = 0 selects
 * floor(44/log2(1/r)), otherwise 1 <= L_override <= 64.  Host only. */
int fkv_codec_init(int32_t N, double r_scale, int32_t L_override, fkv_codec* out);

/* Size in bytes of the codec's device table (opaque layout, 16-byte aligned
 * sections: vertex table V(c), cell centres (1-r)V(c) and their 1/r
 * multiples, and a sector look-up table used by decode). */
size_t fkv_codec_table_bytes(const fkv_codec* c);

/* Writes the device table into caller host memory of fkv_codec_table_bytes()
 * bytes.  The caller copies it once to device memory (16-byte aligned) and
 * passes that copy as `dev_table` below.  Host only. */
int fkv_codec_fill_table(const fkv_codec* c, void* host_table);

/* ceil(n_sym / L): stored points per stream (the last span may be shorter). */
int64_t fkv_num_spans(const fkv_codec* c, int64_t n_sym);

/* ---- a2: per-head residual-VQ assignment (Sec. 3 "Setup") ---------------
 * For every stream s and archived token t in [t_begin, t_end), starting from
 * r = x[s][t] and for stage st = 0..S-1:
 *     i_st = argmin_j ||r - C[b][st][j]||^2   (lowest j on exact ties)
 *     r    = r - C[b][st][i_st]
 * with b = stream_book[s].  The S indices sum (through their centroids) to
 * the reconstruction of the vector.
 *   desc.n_streams, desc.T   x is [n_streams][T][d] IEEE binary16
 *   desc.t_begin, t_end      archived token range (exact-window policy:
 *                            first 4 sinks and last 32 recent stay exact)
 *   desc.d                   head dim, multiple of 16, 16..256
 *   desc.S, desc.K           stages (1..8) and codewords per stage (1..256)
 *   desc.n_books             books is [n_books][S][K][d] binary16
 *   stream_book              device int32 [n_streams]; an id outside
 *                            [0, n_books) marks the stream invalid: its
 *                            symbols are set to 0xFF and *n_bad_streams (if
 *                            given) is incremented
 *   symbols                  device out u8 [n_streams][(t_end-t_begin)*S],
 *                            token-major, stage-minor
 *   residual                 device out f32 [n_streams][t_end-t_begin][d],
 *                            x - sum_st C[b][st][i_st]; nullable
 * Distances are evaluated as ||c||^2/2 - r.c with fp16 operands on matrix
 * cores and fp32 accumulation; residuals beyond the first stage are split
 * into two fp16 parts so both products stay exact.  x, books: 16-byte
 * aligned. */
typedef struct {
    int64_t n_streams;
    int64_t T;
    int64_t t_begin;
    int64_t t_end;
    int32_t d;
    int32_t S;
    int32_t K;
    int32_t n_books;
} fkv_rvq_desc;

int fkv_rvq_assign(const fkv_rvq_desc* desc, const uint16_t* x_f16, const uint16_t* books_f16,
                   const int32_t* stream_book, uint8_t* symbols, float* residual,
                   uint32_t* n_bad_streams, void* stream);

/* The first n_stages (1..desc->S) stages of fkv_rvq_assign's assignment, in
 * the same layout (books [n_books][S][K][d], symbols with stride S): what a
 * k-means update of stage n_stages-1 needs (Sec. 3 "Setup": the later stages
 * do not enter it).  Symbol bytes of stages >= n_stages are left as they are
 * (for an invalid stream all S bytes are set to 0xFF, as fkv_rvq_assign
 * does); the residual, when requested, is the one after n_stages stages.  The
 * assigned stages' symbols equal fkv_rvq_assign's.  FKV_ERR_INVALID_ARG for
 * n_stages outside [1, S]; otherwise as fkv_rvq_assign. */
int fkv_rvq_assign_stages(const fkv_rvq_desc* desc, int32_t n_stages, const uint16_t* x_f16,
                          const uint16_t* books_f16, const int32_t* stream_book, uint8_t* symbols,
                          float* residual, uint32_t* n_bad_streams, void* stream);

/* ---- a2, grouped by book: the per-step eviction form (Sec. 3 "Setup") ------
 * When a position ages out of the exact window at a decoding step, every
 * stream's leaving vector is assigned: one token per stream.  A per-stream
 * block would copy a whole stage book into LDS for that one token, so this
 * form takes groups of streams that share a book and gives each block the
 * tokens [t_begin, t_end) of all members of one group (member by member),
 * served from one copy of the book.  The symbols and residuals of every
 * listed stream are those fkv_rvq_assign gives, bit for bit (the arithmetic of
 * a token does not depend on the other tokens of its block); streams not
 * listed are not touched.
 *   groups        device int32 [n_groups][group_size] (4-byte aligned):
 *                 stream ids; all members of a group must have the same book
 *                 id in stream_book.  A stream listed in two groups is
 *                 assigned twice (the same bytes are written twice).
 *   n_groups      >= 0 (0: nothing to do; groups may then be null)
 *   group_size    1..256
 * A group with a member id outside [0, n_streams), or whose members' book ids
 * differ or lie outside [0, n_books): the symbols of its in-range members are
 * set to 0xFF (residual NaN) and *n_bad_groups (if given) is incremented once
 * per such group.  The other arguments are those of fkv_rvq_assign; errors as
 * fkv_rvq_assign, and FKV_ERR_INVALID_ARG for a group_size outside 1..256, a
 * negative n_groups, or groups null or misaligned with n_groups > 0. */
int fkv_rvq_assign_groups(const fkv_rvq_desc* desc, const int32_t* groups, int64_t n_groups,
                          int32_t group_size, const uint16_t* x_f16, const uint16_t* books_f16,
                          const int32_t* stream_book, uint8_t* symbols, float* residual,
                          uint32_t* n_bad_groups, void* stream);

/* ---- a2 + a3 fused: assignment and span encode in one call -----------------
 * Equivalent to fkv_rvq_assign followed by fkv_cgr_encode_spans of its
 * symbols (n_sym = (t_end - t_begin) * S per stream): the same symbols and the
 * same points, bit for bit.  Below 2^23 head vectors per call (n_streams x
 * (t_end - t_begin)), or when symbols is not 4-byte aligned, one kernel does
 * both: each assignment block takes a token range that holds whole spans (a
 * multiple of L / gcd(L, S) tokens) and encodes them as soon as its last stage
 * is assigned, so the symbols are never read back.  From 2^23 head vectors on
 * the call launches the assignment and then the span encode on the same
 * stream, which is faster there (the encode tail of a fused block holds its
 * compute unit; fkv_rvq_assign_encode_fused says which form a call takes).
 *   c, dev_table  the codec, as for fkv_cgr_encode_spans
 *   points        device f64 [n_streams][n_spans][2] (n_spans = ceil(n_sym / L)),
 *                 16-byte aligned; a stream with an invalid book id gets NaN
 *                 points, as encoding its 0xFF symbols would give
 * The other arguments are those of fkv_rvq_assign. */
int fkv_rvq_assign_encode(const fkv_rvq_desc* desc, const uint16_t* x_f16, const uint16_t* books_f16,
                          const int32_t* stream_book, const fkv_codec* c, const void* dev_table,
                          uint8_t* symbols, double* points, float* residual, uint32_t* n_bad_streams,
                          void* stream);

/* Which form fkv_rvq_assign_encode takes for this descriptor and symbols
 * pointer: 1 the single fused kernel, 0 the assignment kernel and then the
 * span encode kernel.  Host-only (no device call); FKV_ERR_INVALID_ARG for a
 * null descriptor. */
int fkv_rvq_assign_encode_fused(const fkv_rvq_desc* desc, const uint8_t* symbols);

/* ---- a3: fixed-span chaos-game encode (Sec. 1 "The code", Sec. 2) --------
 * symbols [n_streams][n_sym] (device u8) -> points [n_streams][n_spans][2]
 * (device f64, x then y; 16-byte aligned), n_spans = fkv_num_spans().
 * Span j covers symbols [jL, min((j+1)L, n_sym)) and is encoded from the
 * anchor (0,0) by p = V(c) + r (p - V(c)), each coordinate evaluated as
 * t = p - V; u = r*t; p = V + u with round-to-nearest-even and no fused
 * multiply-add, so points are bit-for-bit reproducible. */
int fkv_cgr_encode_spans(const fkv_codec* c, const void* dev_table, const uint8_t* symbols,
                         int64_t n_streams, int64_t n_sym, double* points, void* stream);

/* ---- a4: bulk span decode (Sec. 1 "The code") ----------------------------
 * points [n_streams][n_spans][2] -> symbols [n_streams][n_sym].  Each span
 * is walked backward from its stored point: the symbol is the cell holding
 * the point (nearest cell centre (1-r)V(c), equivalently the angular
 * sector), then p <- (p - (1-r)V(c)) / r.  Anchored reconstruction: after
 * the span's steps the point must be back at the anchor (0,0); a span is
 * accepted when max(|x|,|y|) <= 2^-6 and, with verify != 0, when re-encoding
 * its decoded symbols reproduces the stored point bit for bit.
 *   span_ok   device out u8 [n_streams][n_spans] (1 accepted, 0 failed); nullable
 *   n_failed  device u32 counter, += number of failed spans; nullable
 * Symbols of a failed span are unspecified (but always < N). */
int fkv_cgr_decode_spans(const fkv_codec* c, const void* dev_table, const double* points,
                         int64_t n_streams, int64_t n_sym, uint8_t* symbols, uint8_t* span_ok,
                         uint32_t* n_failed, int32_t verify, void* stream);

/* ---- a5: O(1) random access (Sec. 2, Table 1 "random access") -------------
 * For query q with (s, t) = (q_stream[q], q_token[q]): a = t*S; decode only
 * the span(s) holding symbols [a, a+S) of stream s and write them to
 * out[q][0..S).  n_sym must be a multiple of S (S symbols per token).
 *   q_status  device out u8 [n_q]: 0 ok, 1 a decoded span failed its anchor
 *             check, 2 out of range (s >= n_streams or t >= n_sym/S; out
 *             row left zero); nullable
 *   n_failed  device u32 counter, += number of queries with status != 0; nullable */
int fkv_span_lookup(const fkv_codec* c, const void* dev_table, const double* points,
                    int64_t n_streams, int64_t n_sym, int32_t S, const uint32_t* q_stream,
                    const uint32_t* q_token, int64_t n_q, uint8_t* out, uint8_t* q_status,
                    uint32_t* n_failed, void* stream);

/* ---- rehydrate: reconstruction of archived positions (Sec. 3 "Setup": an
 * archived position is replaced by the sum of its codewords; Sec. 5: matched
 * positions are rehydrated from the archive alone) ---------------------------
 * For query q with (s, t) = (q_stream[q], q_token[q]): the token's S symbols
 * i_0..i_{S-1} are read back by random access (as fkv_span_lookup), then
 *     out[q][e] = sum_{st<S} C[b][st][i_st][e],   b = stream_book[s],
 * formed exactly and rounded once to binary16 (round to nearest, ties to
 * even).
 *   books_f16    device binary16 [n_books][S][K][d], 16-byte aligned
 *   stream_book  device int32 [n_streams]
 *   K, d         codewords per stage (1..256); head dim (multiple of 8, 8..256)
 *   out_f16      device binary16 [n_q][d], 16-byte aligned
 *   q_status     device u8 [n_q], nullable: 0 ok, 1 a decoded span failed its
 *                anchor check, 2 out of range, 3 invalid book id or a decoded
 *                symbol >= K; the out row is zero unless the status is 0
 *   n_failed     device u32 counter, += number of queries with status != 0;
 *                nullable */
int fkv_rehydrate(const fkv_codec* c, const void* dev_table, const double* points, int64_t n_streams,
                  int64_t n_sym, int32_t S, const uint16_t* books_f16, const int32_t* stream_book,
                  int32_t n_books, int32_t K, int32_t d, const uint32_t* q_stream,
                  const uint32_t* q_token, int64_t n_q, uint16_t* out_f16, uint8_t* q_status,
                  uint32_t* n_failed, void* stream);

/* ---- append (Sec. 2 and Table 1, "append") ---------------------------------
 * Extends each of n_streams streams of n_old symbols by m symbols
 * (sym_new [n_streams][m], device u8), re-walking only from the stream's last
 * stored point: a partial last span continues from points[s][n_old / L], a
 * span that starts at a multiple of L starts from the anchor (0,0), and the
 * point of every span the new symbols fall in is written back.  points is
 * [n_streams][cap_spans][2] (device f64, 16-byte aligned) with
 * cap_spans >= ceil((n_old + m) / L); spans before the open one are not
 * touched.  The result is bit-identical to fkv_cgr_encode_spans of the whole
 * stream.  A symbol >= N makes its span's point NaN. */
int fkv_cgr_append(const fkv_codec* c, const void* dev_table, double* points, int64_t cap_spans,
                   int64_t n_streams, int64_t n_old, const uint8_t* sym_new, int64_t m, void* stream);

/* ---- in-archive retrieval (Sec. 5) ---------------------------------------
 * Per-position index: traj[s][k] (device f64 pairs [n_streams][n_sym][2],
 * 16-byte aligned) is the point of the walk over the W symbols ending at
 * position k of stream s (positions max(0, k-W+1)..k), started at the origin
 * (1 <= W <= 64).  symbols: device u8 [n_streams][n_sym], 4-byte aligned. */
int fkv_trajectory(const fkv_codec* c, const void* dev_table, const uint8_t* symbols, int64_t n_streams,
                   int64_t n_sym, int32_t W, double* traj, void* stream);

/* Suffix search on the index: the query (device u8 [ell], 1 <= ell <= L and
 * ell <= the index's W) is encoded from the origin to q; every position k >=
 * ell-1 whose point p has |p - q|^2 <= (2 r^ell)^2 is a candidate (a position
 * whose last ell symbols equal the query lies within r^ell, so none is
 * missed); with verify = 1 a candidate is kept only when decoding ell symbols
 * backward from p reproduces the query, with verify = 0 every candidate is a
 * hit.  Hits are written as (stream, position) u32 pairs to hits
 * [max_hits][2] (8-byte aligned; order unspecified, at most max_hits);
 * *n_hits (device u32, required) += the number of hits, *n_candidates
 * (nullable) += the number of candidates.  A query symbol >= N matches
 * nothing. */
int fkv_suffix_search(const fkv_codec* c, const void* dev_table, const double* traj, int64_t n_streams,
                      int64_t n_sym, const uint8_t* query, int32_t ell, int32_t verify, uint32_t* hits,
                      int64_t max_hits, uint32_t* n_hits, uint32_t* n_candidates, void* stream);

/* ---- k-means codebook update (Sec. 3 "Setup": codebooks are trained by
 * k-means) -------------------------------------------------------------------
 * One Lloyd update of residual stage `stage` (0 <= stage < S) of the books,
 * after an assignment by fkv_rvq_assign (symbols [n_streams][(t_end-t_begin)*S]).
 * fkv_kmeans_accumulate adds, for every archived token of every stream whose
 * book id is valid and whose symbols of stages 0..stage are < K, the stage
 * input r = x_t - sum_{st<stage} C[b][st][i_st] to
 *     sums[b][i_stage][0..d)   (device int64, units of 2^-24: exact integers)
 * and 1 to counts[b][i_stage] (device u32).  The caller zeroes both; desc is
 * read as for fkv_rvq_assign, except that d only has to be a multiple of 8
 * (8..256).  x, books: 16-byte aligned; sums 8-byte aligned.
 * fkv_kmeans_finalize replaces, for every cluster with count > 0, row
 * books[b][stage][j] by the mean sums / count * 2^-24 (fp64) rounded once to
 * binary16 (round to nearest, ties to even); an empty cluster keeps its
 * centroid. */
int fkv_kmeans_accumulate(const fkv_rvq_desc* desc, const uint16_t* x_f16, const uint16_t* books_f16,
                          const int32_t* stream_book, const uint8_t* symbols, int32_t stage, int64_t* sums,
                          uint32_t* counts, void* stream);
int fkv_kmeans_finalize(int32_t n_books, int32_t S, int32_t K, int32_t d, int32_t stage, const int64_t* sums,
                        const uint32_t* counts, uint16_t* books_f16, void* stream);

/* ---- k-means update without allocation ------------------------------------
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same
 * update as fkv_kmeans_accumulate followed by fkv_kmeans_finalize (identical
 * books and counts, bit for bit), but the cluster sums and counts live in a
 * device scratch array owned by the library instead of caller workspace:
 * FKV_NOALLOC_SCRATCH_BYTES per device, held from the first call on that
 * device until the process ends.  The call allocates and frees nothing; it
 * clears the scratch it uses (a fill kernel, no memset) before accumulating.
 *   desc, x_f16, stream_book, symbols, stage   as for fkv_kmeans_accumulate
 *   books_f16   device binary16 [n_books][S][K][d], updated in place
 *   counts_out  device u32 [n_books][K], nullable: the cluster counts
 * Returns FKV_ERR_SCRATCH_TOO_SMALL (with no side effect) when
 * fkv_kmeans_update_noalloc_bytes(n_books, K, d) exceeds the scratch size.
 * Every call on one device shares that device's scratch: calls that overlap
 * in time on one device (different streams, or several host threads) race
 * and must be serialised by the caller. */
#define FKV_NOALLOC_SCRATCH_BYTES (64u << 20)

/* Scratch bytes an update of n_books books of K codewords of dimension d
 * needs: n_books*K*d*8 (sums) + n_books*K*4 (counts). */
size_t fkv_kmeans_update_noalloc_bytes(int32_t n_books, int32_t K, int32_t d);

int fkv_kmeans_update_noalloc(const fkv_rvq_desc* desc, const uint16_t* x_f16, uint16_t* books_f16,
                              const int32_t* stream_book, const uint8_t* symbols, int32_t stage,
                              uint32_t* counts_out, void* stream);

/* ---------------------------------------------------------------------------
 * Measurement aid (not part of the archive path).
 *
 * fkv_diag_mfma_loop runs n_blocks blocks of 256 threads; every wave issues
 * iters rounds of four independent v_mfma_f32_32x32x16_f16 (the instruction
 * of fkv_rvq_assign) from registers, with no memory traffic, and block 0
 * writes one accumulator sum to out[0] (device float).  With random_operands
 * = 0 every operand element is a or b, and out[0] = 4 * 16 * iters * a * b
 * when that is exact; otherwise each lane alternates between two
 * pseudo-random operand sets, so that the multiplier inputs change on every
 * instruction as on real data (a and b are ignored).  The rate of the random
 * form is the device's practical ceiling for that instruction under its
 * power limit; fkv_diag_mfma_loop_flops gives the FLOP count of a launch
 * (2*32*32*16 per instruction).  Errors: FKV_ERR_INVALID_ARG for n_blocks < 1,
 * iters < 0 or a null or misaligned out.
 * --------------------------------------------------------------------------- */
int fkv_diag_mfma_loop(int32_t n_blocks, int32_t iters, int32_t random_operands, float a, float b, float* out,
                       void* stream);
double fkv_diag_mfma_loop_flops(int32_t n_blocks, int32_t iters);

/* Static description of a status code. */
const char* fkv_status_string(int status);

/* Library version string. */
const char* fkv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* FKV_H */
