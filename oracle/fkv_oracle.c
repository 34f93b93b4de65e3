/*
 * fkv_oracle.c -- plain, slow, obviously correct CPU oracle for the fractal
 * KV-archive hot path (Gusev, "Fractal KV-Cache Archives", arXiv 2607.07144).
 *
 * THIS IS TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg may load it.  It shares
 * no source, header, table or helper with the HIP library: it recomputes every
 * constant itself from the paper's definitions.
 *
 * Precision: every floating-point step is IEEE binary64, built with
 * -ffp-contract=off (no fused multiply-add), so each written operation is one
 * round-to-nearest-even result.  Loops run in the order the definitions give.
 * OpenMP is used only across independent streams (the outer loop), never
 * inside one stream's computation.
 *
 * What each function follows:
 *   fkvo_r_max, fkvo_codec_params, fkvo_tables
 *       Sec. 1 ("The code"): regular N-gon, one vertex per symbol; the cells
 *       must be disjoint, which bounds r by a packing constant r_N; the
 *       precision budget of about 44/log2(1/r) symbols per double sets the
 *       span length.  Fig. 1 (cell geometry).
 *       Readings (the paper is silent): unit circumradius, centred at the
 *       origin, vertex c at angle 2*pi*c/N; r_N = s/(s+m) with s = sin(pi/N),
 *       m = max_j sin((2j+1)pi/N) (adjacent cells just touch across the
 *       bisector of their vertices); r = r_scale * r_N; L = floor(44/log2(1/r)).
 *   fkvo_encode_spans
 *       Sec. 1: p_k = V(c_k) + r (p_{k-1} - V(c_k)), evaluated literally as
 *       t = p - V; u = r*t; p = V + u per coordinate.  Sec. 1 / Sec. 2: one
 *       stored point per fixed-length span.  Reading: every span starts from
 *       the anchor (0,0) (a query is encoded "from the origin", Sec. 5), the
 *       last span may be shorter.
 *   fkvo_cell, fkvo_decode_spans
 *       Sec. 1: the decoded symbol is the vertex whose contracted image (cell)
 *       contains the point, then p_{k-1} = (p_k - (1-r)V(c_k))/r.  Reading:
 *       the cell is found as the nearest cell centre W(c) = (1-r)V(c), lowest
 *       index on exact ties (for r <= r_N this equals cell membership for
 *       every point of a cell; the pin tests check it by polygon containment).
 *       Anchored backward reconstruction: after the span's L backward steps
 *       the point must be back at the anchor (0,0); the span is accepted when
 *       max(|x|,|y|) <= 2^-6, and, with verify, when re-encoding the decoded
 *       symbols reproduces the stored point bit for bit.
 *   fkvo_span_lookup
 *       Sec. 2 / Table 1: random access decodes only the span(s) holding the
 *       requested position.
 *   fkvo_rvq_assign
 *       Sec. 3 ("Setup"): residual VQ of depth S stores a vector as S indices
 *       whose centroids sum to the reconstruction; an archived position is
 *       replaced by its nearest codebook entries.  Per stage:
 *       j* = argmin_j ||r - C_s[j]||^2 (lowest j on exact ties), then
 *       r <- r - C_s[j*].  Distances are exact-input fp64 sums in index order.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define FKVO_ANCHOR_TOL (1.0 / 64.0) /* 2^-6 */

/* ---------------------------------------------------------------- codec -- */

double fkvo_r_max(int32_t N)
{
    /* Disjointness of adjacent cells c, c+1 (Sec. 1, Fig. 1).  The mirror line
     * between V(c) and V(c+1) passes through the origin; the centre of cell c
     * is (1-r)*sin(pi/N) away from it and the cell (an r-scaled hull)
     * reaches r*m towards it, m = max_j sin((2j+1)pi/N).  Equality gives r_N. */
    double s = sin(M_PI / (double)N);
    double m = 0.0;
    for (int32_t j = 0; j < N; ++j) {
        double v = sin((2.0 * (double)j + 1.0) * M_PI / (double)N);
        if (v > m) m = v;
    }
    return s / (s + m);
}

int fkvo_codec_params(int32_t N, double r_scale, int32_t L_override,
                      double* r_max, double* r, int32_t* L)
{
    if (N < 3) return -1;
    double rm = fkvo_r_max(N);
    double rr = r_scale * rm;
    if (!(rr > 0.0) || !(rr < 1.0)) return -1;
    int32_t LL = L_override;
    if (LL <= 0) LL = (int32_t)floor(44.0 / log2(1.0 / rr));
    if (LL < 1) LL = 1;
    *r_max = rm;
    *r = rr;
    *L = LL;
    return 0;
}

/* V[c] = (cos t, sin t), t = 2*pi*c/N; W[c] = (1-r) V[c] (cell centres). */
void fkvo_tables(int32_t N, double r, double* V, double* W)
{
    for (int32_t c = 0; c < N; ++c) {
        double t = (2.0 * M_PI * (double)c) / (double)N;
        V[2 * c + 0] = cos(t);
        V[2 * c + 1] = sin(t);
        W[2 * c + 0] = (1.0 - r) * V[2 * c + 0];
        W[2 * c + 1] = (1.0 - r) * V[2 * c + 1];
    }
}

static int64_t n_spans_of(int64_t n_sym, int32_t L)
{
    return (n_sym + L - 1) / L;
}

/* --------------------------------------------------------------- encode -- */

static void encode_one(double r, const double* V, const uint8_t* sym, int64_t len,
                       double* px_out, double* py_out)
{
    double px = 0.0, py = 0.0; /* the span's anchor */
    for (int64_t k = 0; k < len; ++k) {
        int c = sym[k];
        double vx = V[2 * c + 0], vy = V[2 * c + 1];
        double tx = px - vx, ty = py - vy;
        double ux = r * tx, uy = r * ty;
        px = vx + ux;
        py = vy + uy;
    }
    *px_out = px;
    *py_out = py;
}

void fkvo_encode_spans(int32_t N, double r, int32_t L, const double* V,
                       const uint8_t* symbols, int64_t n_streams, int64_t n_sym,
                       double* points, int32_t threads)
{
    (void)N;
    int64_t ns = n_spans_of(n_sym, L);
#pragma omp parallel for schedule(dynamic, 1) num_threads(threads)
    for (int64_t s = 0; s < n_streams; ++s) {
        for (int64_t j = 0; j < ns; ++j) {
            int64_t a = j * L;
            int64_t len = (a + L <= n_sym) ? L : (n_sym - a);
            encode_one(r, V, symbols + s * n_sym + a, len,
                       &points[(s * ns + j) * 2 + 0], &points[(s * ns + j) * 2 + 1]);
        }
    }
}

/* --------------------------------------------------------------- decode -- */

int32_t fkvo_cell(int32_t N, const double* W, double qx, double qy)
{
    int32_t best = 0;
    double dx = qx - W[0], dy = qy - W[1];
    double bd = dx * dx + dy * dy;
    for (int32_t c = 1; c < N; ++c) {
        dx = qx - W[2 * c + 0];
        dy = qy - W[2 * c + 1];
        double d = dx * dx + dy * dy;
        if (d < bd) {
            bd = d;
            best = c;
        }
    }
    return best;
}

/* Decodes one span of length len from its stored point.  Writes len symbols,
 * returns 1 when the span passes the anchor check (and the re-encode check
 * when verify != 0), 0 otherwise.  *resid receives the anchor residual. */
static int decode_one(int32_t N, double r, const double* V, const double* W,
                      double px, double py, int64_t len, uint8_t* sym,
                      int32_t verify, double* resid)
{
    double qx = px, qy = py;
    for (int64_t k = len - 1; k >= 0; --k) {
        int32_t c = fkvo_cell(N, W, qx, qy);
        sym[k] = (uint8_t)c;
        qx = (qx - W[2 * c + 0]) / r;
        qy = (qy - W[2 * c + 1]) / r;
    }
    double ax = fabs(qx), ay = fabs(qy);
    double a = ax > ay ? ax : ay;
    if (ax != ax || ay != ay) a = NAN;
    if (resid) *resid = a;
    int ok = (a <= FKVO_ANCHOR_TOL);
    if (verify) {
        double ex, ey;
        encode_one(r, V, sym, len, &ex, &ey);
        if (memcmp(&ex, &px, sizeof(double)) != 0 || memcmp(&ey, &py, sizeof(double)) != 0)
            ok = 0;
    }
    return ok;
}

int64_t fkvo_decode_spans(int32_t N, double r, int32_t L, const double* V, const double* W,
                          const double* points, int64_t n_streams, int64_t n_sym,
                          uint8_t* symbols, uint8_t* span_ok, double* anchor_resid,
                          int32_t verify, int32_t threads)
{
    int64_t ns = n_spans_of(n_sym, L);
    int64_t failed = 0;
#pragma omp parallel for schedule(dynamic, 1) num_threads(threads) reduction(+ : failed)
    for (int64_t s = 0; s < n_streams; ++s) {
        for (int64_t j = 0; j < ns; ++j) {
            int64_t a = j * L;
            int64_t len = (a + L <= n_sym) ? L : (n_sym - a);
            const double* P = &points[(s * ns + j) * 2];
            int ok = decode_one(N, r, V, W, P[0], P[1], len, symbols + s * n_sym + a, verify,
                                anchor_resid ? &anchor_resid[s * ns + j] : NULL);
            if (span_ok) span_ok[s * ns + j] = (uint8_t)ok;
            if (!ok) failed += 1;
        }
    }
    return failed;
}

/* --------------------------------------------------------------- lookup -- */

int64_t fkvo_span_lookup(int32_t N, double r, int32_t L, const double* V, const double* W,
                         const double* points, int64_t n_streams, int64_t n_sym, int32_t S,
                         const uint32_t* q_stream, const uint32_t* q_token, int64_t n_q,
                         uint8_t* out, uint8_t* q_status, int32_t threads)
{
    int64_t ns = n_spans_of(n_sym, L);
    int64_t n_tok = n_sym / S;
    int64_t failed = 0;
#pragma omp parallel for schedule(static) num_threads(threads) reduction(+ : failed)
    for (int64_t q = 0; q < n_q; ++q) {
        uint8_t buf[64];
        uint8_t st = 0;
        memset(out + q * S, 0, (size_t)S);
        if ((int64_t)q_stream[q] >= n_streams || (int64_t)q_token[q] >= n_tok) {
            st = 2;
        } else {
            int64_t s = q_stream[q];
            int64_t a = (int64_t)q_token[q] * S;
            for (int64_t j = a / L; j <= (a + S - 1) / L; ++j) {
                int64_t b = j * L;
                int64_t len = (b + L <= n_sym) ? L : (n_sym - b);
                const double* P = &points[(s * ns + j) * 2];
                if (!decode_one(N, r, V, W, P[0], P[1], len, buf, 0, NULL)) st = 1;
                for (int64_t k = 0; k < len; ++k) {
                    int64_t pos = b + k;
                    if (pos >= a && pos < a + S) out[q * S + (pos - a)] = buf[k];
                }
            }
        }
        if (q_status) q_status[q] = st;
        if (st) failed += 1;
    }
    return failed;
}

/* ------------------------------------------------------------------ RVQ -- */

/* IEEE-754 binary16 -> binary64, written out from the format definition
 * (1 sign bit, 5 exponent bits with bias 15, 10 fraction bits). */
double fkvo_half_to_double(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int m = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)m, -24); /* zero or subnormal: m * 2^-14 * 2^-10 */
    else if (e == 31)
        v = m ? NAN : INFINITY;
    else
        v = ldexp((double)(m + 1024), e - 25); /* (1 + m/1024) * 2^(e-15) */
    return sign ? -v : v;
}

/*
 * x:      [n_streams][T][d] binary16 bit patterns
 * books:  [n_books][S][K][d] binary16 bit patterns
 * stream_book: [n_streams] book id of each stream
 * symbols:  out [n_streams][(t_end-t_begin)*S], token-major, stage-minor
 * residual: out, nullable [n_streams][t_end-t_begin][d]: x - sum_s C_s[i_s]
 * gaps:     out, nullable [n_streams][t_end-t_begin][S]: (D2 - D1)/D2 of the
 *           two smallest squared distances at each stage (0 when D2 == 0)
 * force:    nullable [n_streams][(t_end-t_begin)*S]: another implementation's
 *           choice.  Where it differs from the exact argmin and its distance is
 *           within relative force_tol of the optimum ((D_g - D1)/D_g < tol) the
 *           oracle continues from the forced choice (teacher forcing) and counts
 *           it in counts[0]; otherwise it keeps its own choice and counts the
 *           disagreement in counts[1].
 */
void fkvo_rvq_assign(int64_t n_streams, int64_t T, int64_t t_begin, int64_t t_end,
                     int32_t d, int32_t S, int32_t K,
                     const uint16_t* x, const uint16_t* books, const int32_t* stream_book,
                     uint8_t* symbols, double* residual, double* gaps,
                     const uint8_t* force, double force_tol, int64_t* counts,
                     int32_t threads)
{
    int64_t Ta = t_end - t_begin;
    int64_t n_forced = 0, n_hard = 0;
#pragma omp parallel for schedule(dynamic, 1) num_threads(threads) reduction(+ : n_forced, n_hard)
    for (int64_t s = 0; s < n_streams; ++s) {
        double* r = (double*)malloc(sizeof(double) * (size_t)d);
        double* D = (double*)malloc(sizeof(double) * (size_t)K);
        const uint16_t* book = books + (int64_t)stream_book[s] * S * K * d;
        for (int64_t t = 0; t < Ta; ++t) {
            const uint16_t* xv = x + (s * T + t_begin + t) * d;
            for (int32_t i = 0; i < d; ++i) r[i] = fkvo_half_to_double(xv[i]);
            for (int32_t st = 0; st < S; ++st) {
                const uint16_t* C = book + (int64_t)st * K * d;
                for (int32_t j = 0; j < K; ++j) {
                    double acc = 0.0;
                    for (int32_t i = 0; i < d; ++i) {
                        double e = r[i] - fkvo_half_to_double(C[(int64_t)j * d + i]);
                        acc = acc + e * e;
                    }
                    D[j] = acc;
                }
                int32_t j1 = 0;
                for (int32_t j = 1; j < K; ++j)
                    if (D[j] < D[j1]) j1 = j;
                double D1 = D[j1], D2 = INFINITY;
                for (int32_t j = 0; j < K; ++j)
                    if (j != j1 && D[j] < D2) D2 = D[j];
                double gap = 0.0;
                if (K > 1 && D2 > 0.0) gap = (D2 - D1) / D2;
                if (gaps) gaps[(s * Ta + t) * S + st] = (K > 1) ? gap : INFINITY;
                int32_t pick = j1;
                if (force) {
                    int32_t g = force[(s * Ta + t) * S + st];
                    if (g != j1) {
                        double rel = (g < K && D[g] > 0.0) ? (D[g] - D1) / D[g] : INFINITY;
                        if (g < K && rel < force_tol) {
                            pick = g;
                            n_forced += 1;
                        } else {
                            n_hard += 1;
                        }
                    }
                }
                symbols[(s * Ta + t) * S + st] = (uint8_t)pick;
                for (int32_t i = 0; i < d; ++i)
                    r[i] = r[i] - fkvo_half_to_double(C[(int64_t)pick * d + i]);
            }
            if (residual)
                for (int32_t i = 0; i < d; ++i) residual[(s * Ta + t) * d + i] = r[i];
        }
        free(r);
        free(D);
    }
    if (counts) {
        counts[0] = n_forced;
        counts[1] = n_hard;
    }
}

/* ------------------------------------------------------------- rehydrate -- */

/*
 * Sec. 3 ("Setup"): an archived position's K or V vector is replaced by the sum
 * of its S codewords; Sec. 5: a matched position is rehydrated from the
 * archive alone.  Query q = (stream, token): its S symbols are read back by
 * random access (fkvo_span_lookup's steps), then
 *     out[q][e] = sum_{st=0..S-1} C[b][st][i_st][e],   b = stream_book[stream],
 * summed in fp64 in stage order (exact: a few binary16 values).
 * q_status: 0 ok, 1 a decoded span failed its anchor check, 2 out of range,
 * 3 invalid book id or a decoded symbol >= K; out row is zero unless 0.
 */
int64_t fkvo_rehydrate(int32_t N, double r, int32_t L, const double* V, const double* W,
                       const double* points, int64_t n_streams, int64_t n_sym, int32_t S,
                       const uint16_t* books, const int32_t* stream_book, int32_t n_books,
                       int32_t K, int32_t d, const uint32_t* q_stream, const uint32_t* q_token,
                       int64_t n_q, double* out, uint8_t* q_status, int32_t threads)
{
    uint8_t* sym = (uint8_t*)malloc((size_t)(n_q > 0 ? n_q : 1) * (size_t)S);
    uint8_t* st = (uint8_t*)malloc((size_t)(n_q > 0 ? n_q : 1));
    fkvo_span_lookup(N, r, L, V, W, points, n_streams, n_sym, S, q_stream, q_token, n_q, sym, st,
                     threads);
    int64_t failed = 0;
#pragma omp parallel for schedule(static) num_threads(threads) reduction(+ : failed)
    for (int64_t q = 0; q < n_q; ++q) {
        uint8_t s_ = st[q];
        int32_t b = 0;
        if (s_ == 0) {
            b = stream_book[q_stream[q]];
            if (b < 0 || b >= n_books) s_ = 3;
            for (int32_t k = 0; k < S; ++k)
                if (sym[q * S + k] >= K) s_ = 3;
        }
        for (int32_t e = 0; e < d; ++e) {
            double acc = 0.0;
            if (s_ == 0)
                for (int32_t k = 0; k < S; ++k) {
                    const uint16_t* row = books + (((int64_t)b * S + k) * K + sym[q * S + k]) * d;
                    acc = acc + fkvo_half_to_double(row[e]);
                }
            out[q * d + e] = acc;
        }
        if (q_status) q_status[q] = s_;
        if (s_) failed += 1;
    }
    free(sym);
    free(st);
    return failed;
}

/* ---------------------------------------------------------------- append -- */

/*
 * Sec. 2 / Table 1 (append): new symbols extend a stream by re-walking only
 * from its last stored point.  Each of n_streams streams holds n_old symbols
 * whose span points sit in points[s][0..][2] (capacity cap_spans spans per
 * stream).  m new symbols per stream (sym_new[s][0..m)) are appended: a partial
 * last span continues from its stored point, every span that starts at a
 * multiple of L starts from the anchor (0,0), and each touched span's point is
 * written back.  The result equals a bulk encode of the whole stream.
 */
void fkvo_append(int32_t N, double r, int32_t L, const double* V, double* points,
                 int64_t cap_spans, int64_t n_streams, int64_t n_old, const uint8_t* sym_new,
                 int64_t m, int32_t threads)
{
#pragma omp parallel for schedule(static) num_threads(threads)
    for (int64_t s = 0; s < n_streams; ++s) {
        double* P = points + s * cap_spans * 2;
        double px = 0.0, py = 0.0;
        if (n_old % L != 0) {
            px = P[(n_old / L) * 2];
            py = P[(n_old / L) * 2 + 1];
        }
        for (int64_t k = 0; k < m; ++k) {
            int64_t pos = n_old + k;
            if (pos % L == 0) {
                px = 0.0;
                py = 0.0;
            }
            int32_t c = sym_new[s * m + k];
            double vx = c < N ? V[2 * c] : NAN, vy = c < N ? V[2 * c + 1] : NAN;
            double tx = px - vx, ty = py - vy;
            double ux = r * tx, uy = r * ty;
            px = vx + ux;
            py = vy + uy;
            P[(pos / L) * 2] = px;
            P[(pos / L) * 2 + 1] = py;
        }
    }
}

/* ------------------------------------------------------------- retrieval -- */

/*
 * Sec. 5: the archive is searchable in place.  Per-position index: for every
 * symbol position k of a stream, traj[k] is the point of the walk over the W
 * symbols ending at k (positions max(0, k-W+1)..k), started at the origin.
 * (The contraction makes older symbols' weight r^age; windows of W symbols
 * keep every position independent, the reading taken for a parallel layout.)
 */
void fkvo_trajectory(int32_t N, double r, const double* V, const uint8_t* symbols,
                     int64_t n_streams, int64_t n_sym, int32_t W, double* traj, int32_t threads)
{
    (void)N;
#pragma omp parallel for schedule(static) num_threads(threads)
    for (int64_t s = 0; s < n_streams; ++s)
        for (int64_t k = 0; k < n_sym; ++k) {
            int64_t a = k - W + 1 > 0 ? k - W + 1 : 0;
            encode_one(r, V, symbols + s * n_sym + a, k - a + 1, &traj[(s * n_sym + k) * 2],
                       &traj[(s * n_sym + k) * 2 + 1]);
        }
}

/*
 * Sec. 5 suffix search: the query (ell symbols, ell <= W and ell <= L) is
 * encoded from the origin to q; every indexed position k >= ell - 1 (one with
 * ell symbols of history) whose point p has |p - q|^2 <= (2 r^ell)^2 is a
 * candidate (two walks sharing their last ell symbols end within r^ell of each
 * other, so no true match is missed while r^ell stays far above the rounding
 * of the points, which ell <= L guarantees).  With verify, a candidate is kept only
 * when decoding ell symbols backward from p reproduces the query.  Hits are
 * written as (stream, position) pairs in stream-major, position order (at most
 * max_hits); returns the number of hits, *n_candidates gets the candidates.
 * The threshold is 2 * r^ell with r^ell formed by ell successive products.
 */
int64_t fkvo_suffix_search(int32_t N, double r, const double* V, const double* W_,
                           const double* traj, int64_t n_streams, int64_t n_sym,
                           const uint8_t* query, int32_t ell, int32_t verify,
                           uint32_t* hits, int64_t max_hits, int64_t* n_candidates)
{
    double qx, qy;
    encode_one(r, V, query, ell, &qx, &qy);
    double rl = 1.0;
    for (int32_t k = 0; k < ell; ++k) rl = rl * r;
    double thr = 2.0 * rl;
    double thr2 = thr * thr;
    int64_t n_hit = 0, n_cand = 0;
    for (int64_t s = 0; s < n_streams; ++s)
        for (int64_t k = ell - 1; k < n_sym; ++k) {
            const double* p = &traj[(s * n_sym + k) * 2];
            double dx = p[0] - qx, dy = p[1] - qy;
            double d2 = dx * dx + dy * dy;
            if (!(d2 <= thr2)) continue;
            n_cand += 1;
            if (verify) {
                /* the cell of the point is the last symbol; invert and repeat */
                double x = p[0], y = p[1];
                int ok = 1;
                for (int32_t j = ell - 1; j >= 0 && ok; --j) {
                    int32_t c = fkvo_cell(N, W_, x, y);
                    if (c != query[j]) ok = 0;
                    x = (x - W_[2 * c]) / r;
                    y = (y - W_[2 * c + 1]) / r;
                }
                if (!ok) continue;
            }
            if (n_hit < max_hits) {
                hits[n_hit * 2] = (uint32_t)s;
                hits[n_hit * 2 + 1] = (uint32_t)k;
            }
            n_hit += 1;
        }
    if (n_candidates) *n_candidates = n_cand;
    return n_hit;
}

/* ---------------------------------------------------------------- k-means -- */

/*
 * Sec. 3 ("Setup"): codebooks are trained by k-means.  One Lloyd update of
 * residual stage `stage` of per-head books: every archived token t of every
 * stream contributes its stage input r = x_t - sum_{st<stage} C[b][st][i_st]
 * to cluster i_stage of its book b = stream_book[s]; the new centroid of a
 * cluster is the mean of its members, and an empty cluster keeps its
 * centroid.  Sums are exact integers in units of 2^-24 (every binary16 value
 * is a multiple of 2^-24); mean = (double)sum / count * 2^-24.
 *   means:  out [n_books][K][d] (the old centroid where count == 0)
 *   counts: out [n_books][K]
 */
void fkvo_kmeans_update(int64_t n_streams, int64_t T, int64_t t_begin, int64_t t_end, int32_t d,
                        int32_t S, int32_t K, int32_t n_books, const uint16_t* x, const uint16_t* books,
                        const int32_t* stream_book, const uint8_t* symbols, int32_t stage,
                        double* means, int64_t* counts)
{
    int64_t Ta = t_end - t_begin;
    int64_t* sums = (int64_t*)calloc((size_t)n_books * K * d, sizeof(int64_t));
    for (int64_t i = 0; i < (int64_t)n_books * K; ++i) counts[i] = 0;
    for (int64_t s = 0; s < n_streams; ++s) {
        int32_t b = stream_book[s];
        if (b < 0 || b >= n_books) continue;
        const uint16_t* book = books + (int64_t)b * S * K * d;
        for (int64_t t = 0; t < Ta; ++t) {
            const uint8_t* sym = symbols + (s * Ta + t) * S;
            int32_t j = sym[stage], bad = 0;
            for (int32_t st = 0; st <= stage; ++st)
                if (sym[st] >= K) bad = 1;
            if (bad) continue; /* a symbol outside the book: the token is skipped */
            const uint16_t* xv = x + (s * T + t_begin + t) * d;
            for (int32_t e = 0; e < d; ++e) {
                double r = fkvo_half_to_double(xv[e]);
                for (int32_t st = 0; st < stage; ++st)
                    r = r - fkvo_half_to_double(book[((int64_t)st * K + sym[st]) * d + e]);
                sums[((int64_t)b * K + j) * d + e] += (int64_t)ldexp(r, 24); /* exact */
            }
            counts[(int64_t)b * K + j] += 1;
        }
    }
    for (int64_t b = 0; b < n_books; ++b)
        for (int32_t j = 0; j < K; ++j)
            for (int32_t e = 0; e < d; ++e) {
                int64_t c = counts[b * K + j];
                double m = c ? ldexp((double)sums[(b * K + j) * d + e] / (double)c, -24)
                             : fkvo_half_to_double(books[(((int64_t)b * S + stage) * K + j) * d + e]);
                means[(b * K + j) * d + e] = m;
            }
    free(sums);
}
