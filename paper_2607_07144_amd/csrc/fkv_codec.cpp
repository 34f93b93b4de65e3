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
    fkv::LutEntry* lut = (fkv::LutEntry*)(base + fkv::table_off_lut(N));
    for (int k = 0; k < N; ++k) {
        const double t = (2.0 * M_PI * (double)k) / (double)N;
        V[2 * k + 0] = cos(t);
        V[2 * k + 1] = sin(t);
        W[2 * k + 0] = (1.0 - r) * V[2 * k + 0];
        W[2 * k + 1] = (1.0 - r) * V[2 * k + 1];
        Wr[2 * k + 0] = W[2 * k + 0] / r;
        Wr[2 * k + 1] = W[2 * k + 1] / r;
    }
    // Sector boundaries (angle (k + 1/2) 2 pi / N) in pseudo-angle space,
    // with the sector that starts at each of them.
    std::vector<std::pair<double, int>> bnd;
    bnd.reserve(N);
    for (int k = 0; k < N; ++k) {
        const double a = ((double)k + 0.5) * 2.0 * M_PI / (double)N;
        bnd.push_back({pseudo_angle(cos(a), sin(a)), (k + 1) % N});
    }
    std::sort(bnd.begin(), bnd.end());
    for (int i = 0; i < fkv::kLutBuckets; ++i) {
        const double lo = -1.0 + (double)i / fkv::kLutPerUnit;
        const double hi = -1.0 + (double)(i + 1) / fkv::kLutPerUnit;
        // sector just above lo: the one started by the last boundary <= lo
        // (before the first boundary: the sector that the first one ends)
        int c_lo = (bnd.front().second + N - 1) % N;
        for (const auto& b : bnd)
            if (b.first <= lo) c_lo = b.second;
        fkv::LutEntry e;
        e.thr = INFINITY;
        e.lo = (uint16_t)c_lo;
        e.hi = (uint16_t)c_lo;
        int found = 0;
        for (const auto& b : bnd) {
            if (b.first > lo && b.first <= hi) {
                ++found;
                e.thr = (float)b.first;
                e.hi = (uint16_t)b.second;
            }
        }
        if (found > 1) return FKV_ERR_UNSUPPORTED;  // cannot happen for N <= 256
        lut[i] = e;
    }
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
    default: return "unknown status";
    }
}

extern "C" const char* fkv_version(void)
{
    return "fkv 0.1.0 (gfx950)";
}
