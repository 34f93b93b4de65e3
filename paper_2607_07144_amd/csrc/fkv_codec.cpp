// fkv_codec.cpp -- host-side codec setup of libfkv: contraction limit,
// contraction ratio, span length and the device table of one alphabet.
//
// Geometry (Sec. 1 "The code", Fig. 1 of the paper): a regular N-gon on the
// unit circle, vertex c at angle 2*pi*c/N; symbol c contracts the plane
// towards V(c) by r; its cell is the polygon scaled by r about V(c), centred
// at W(c) = (1-r)V(c).  Cells are pairwise disjoint for r <= r_N; the
// decodable precision of one double (about 44 bits) fixes the span length.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "fkv.h"
#include "fkv_internal.h"

namespace {

// Packing limit of N contracted copies of the polygon.  Adjacent cells c and
// c+1 are mirror images across the line through the origin that bisects
// V(c) and V(c+1).  Cell c's centre lies (1-r) sin(pi/N) from that line,
// and the cell (an r-scaled polygon) reaches r * h towards it, where h is
// the polygon's half-width normal to the line, h = max_j sin((2j+1) pi/N).
// The cells just touch when (1-r) sin(pi/N) = r h.
double packing_limit(int N)
{
    const double s = sin(M_PI / (double)N);
    double h = 0.0;
    for (int j = 0; j < N; ++j) {
        const double v = sin((2.0 * (double)j + 1.0) * M_PI / (double)N);
        h = v > h ? v : h;
    }
    return s / (s + h);
}

// Pseudo-angle of a direction, monotone in its angle over [-pi/2, 3pi/2).
double pseudo_angle(double x, double y)
{
    const double d = y / (fabs(x) + fabs(y));
    return x >= 0.0 ? d : 2.0 - d;
}

}  // namespace

extern "C" int fkv_codec_init(int32_t N, double r_scale, int32_t L_override, fkv_codec* out)
{
    if (!out) return FKV_ERR_INVALID_ARG;
    if (N < 3 || N > 256) return FKV_ERR_INVALID_ARG;
    if (!(r_scale > 0.0) || !(r_scale <= 1.0)) return FKV_ERR_INVALID_ARG;
    if (L_override < 0 || L_override > 64) return FKV_ERR_INVALID_ARG;
    const double rm = packing_limit(N);
    const double r = r_scale * rm;
    int32_t L = L_override;
    if (L == 0) {
        L = (int32_t)floor(44.0 / log2(1.0 / r));
        if (L < 1) L = 1;
        if (L > 64) L = 64;
    }
    out->N = N;
    out->L = L;
    out->r = r;
    out->r_max = rm;
    return FKV_OK;
}

extern "C" size_t fkv_codec_table_bytes(const fkv_codec* c)
{
    if (!c || c->N < 3 || c->N > 256) return 0;
    return fkv::table_bytes(c->N);
}

extern "C" int64_t fkv_num_spans(const fkv_codec* c, int64_t n_sym)
{
    if (!c || c->L < 1 || n_sym < 0) return -1;
    return (n_sym + c->L - 1) / c->L;
}

extern "C" int fkv_codec_fill_table(const fkv_codec* c, void* host_table)
{
    if (!c || !host_table) return FKV_ERR_INVALID_ARG;
    const int N = c->N;
    if (N < 3 || N > 256 || !(c->r > 0.0) || !(c->r < 1.0)) return FKV_ERR_INVALID_ARG;
    const double r = c->r;
    unsigned char* base = (unsigned char*)host_table;
    double* V = (double*)(base + fkv::table_off_V(N));
    double* W = (double*)(base + fkv::table_off_W(N));
    double* Wr = (double*)(base + fkv::table_off_Wr(N));
    uint32_t* lut = (uint32_t*)(base + fkv::table_off_lut(N));
    for (int k = 0; k < N; ++k) {
        const double t = (2.0 * M_PI * (double)k) / (double)N;
        V[2 * k + 0] = cos(t);
        V[2 * k + 1] = sin(t);
        W[2 * k + 0] = (1.0 - r) * V[2 * k + 0];
        W[2 * k + 1] = (1.0 - r) * V[2 * k + 1];
        Wr[2 * k + 0] = W[2 * k + 0] / r;
        Wr[2 * k + 1] = W[2 * k + 1] / r;
    }
    // Sector boundaries (angle (k + 1/2) 2 pi / N) in bucket coordinates
    // u = (P + 1) K + shift, with the sector that starts at each of them; the
    // wrap boundary (sector 0 above it) sits exactly on a bucket edge.
    const double K = (double)fkv::kLutPerUnit;
    const double shift = fkv::lut_shift(N);
    std::vector<std::pair<double, int>> bnd;
    bnd.reserve(N);
    for (int k = 0; k < N; ++k) {
        const double a = ((double)k + 0.5) * 2.0 * M_PI / (double)N;
        const int above = (k + 1) % N;
        double u = (pseudo_angle(cos(a), sin(a)) + 1.0) * K + shift;
        if (above == 0) u = nearbyint(u);
        bnd.push_back({u, above});
    }
    std::sort(bnd.begin(), bnd.end());
    for (int i = 0; i < fkv::kLutEntries; ++i) {
        // sector just above the bucket's lower edge: the one started by the
        // last boundary at or below it (before the first boundary: the
        // sector that the first one ends)
        int c_lo = (bnd.front().second + N - 1) % N;
        for (const auto& b : bnd)
            if (b.first <= (double)i) c_lo = b.second;
        float thr = 2.0f;
        int found = 0;
        for (const auto& b : bnd) {
            if (b.first > (double)i && b.first < (double)(i + 1)) {
                ++found;
                if (b.second != c_lo + 1) return FKV_ERR_UNSUPPORTED;   // cannot happen: no wrap inside
                thr = (float)(b.first - (double)i);
            }
        }
        if (found > 1) return FKV_ERR_UNSUPPORTED;  // cannot happen for N <= 256
        uint32_t w;
        memcpy(&w, &thr, sizeof w);
        lut[i] = (w & ~0xFFu) | (uint32_t)c_lo;
    }
    // the section's padding repeats the last bucket: a coordinate that rounds
    // just past the range's upper end (the direction -pi/2 approached with
    // x < 0) reads the bucket it belongs to, with no clamp in the kernels
    for (size_t i = fkv::kLutEntries; i < (fkv::kLutBytes - fkv::kLutGuard) / sizeof(uint32_t); ++i)
        lut[i] = lut[fkv::kLutEntries - 1];
    // the guard entries before the table: sector 0, no boundary (threshold 2)
    const float two = 2.0f;
    uint32_t gw;
    memcpy(&gw, &two, sizeof gw);
    for (size_t i = 1; i <= fkv::kLutGuard / sizeof(uint32_t); ++i) lut[-(ptrdiff_t)i] = gw & ~0xFFu;
    return FKV_OK;
}

extern "C" const char* fkv_status_string(int status)
{
    switch (status) {
    case FKV_OK: return "ok";
    case FKV_ERR_INVALID_ARG: return "invalid argument";
    case FKV_ERR_UNSUPPORTED: return "unsupported configuration";
    case FKV_ERR_LAUNCH: return "kernel launch failed";
    case FKV_ERR_NO_DEVICE: return "no usable gfx950 device";
    case FKV_ERR_SCRATCH_TOO_SMALL: return "input exceeds the fixed device scratch of the allocation-free entry point";
    default: return "unknown status";
    }
}

extern "C" const char* fkv_version(void)
{
    return "fkv 0.1.0 (gfx950)";
}
