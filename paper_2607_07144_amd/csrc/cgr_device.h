// cgr_device.h -- codec helpers shared by the span kernels (encode, decode,
// lookup, rehydrate, append): per-alphabet tables in LDS, the forward step,
// the cell (sector) of a point, the inverse step, the anchor check, random
// access to one token's symbols, and the host-side launch helpers.
//
// Floating point: the forward step must be bit-reproducible, so every file
// including this header is compiled without FP contraction; fused
// multiply-adds appear only where written explicitly (the inverse map, whose
// points are never compared -- only the symbols they yield).
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "fkv.h"
#include "fkv_hip_common.h"
#include "fkv_internal.h"

#pragma clang fp contract(off)

namespace fkv {
namespace {

constexpr int kBlock = 256;        // threads per block = spans per tile
constexpr int kMaxBlocks = 2048;   // persistent grid cap (8 blocks per CU)

struct CodecArgs {
    int N;
    int L;
    double r;
    double inv_r;
    float lut_bias;   // 2 kLutPerUnit + lut_shift(N): bucket coordinate at R = 0
};

// LDS image of the device table, sized for the alphabet.
struct Tables {
    double2* V;
    double2* W;
    double2* Wr;
    uint32_t* lut;
};

// Bytes of LDS the staged table occupies: Wr and the look-up table always,
// then V and W when needed (sections keep their table offsets).
__host__ __device__ constexpr size_t staged_table_bytes(int N, bool needV, bool needW)
{
    return needW ? table_bytes(N) : needV ? table_off_W(N) : table_fast_bytes(N);
}

// Copies the needed sections of the device table into LDS at the same
// offsets (sections not needed are left unwritten).
__device__ inline Tables stage_tables(const uint8_t* __restrict__ gtab, int N, uint8_t* lds,
                                      bool needV, bool needW)
{
    Tables t;
    t.V = (double2*)(lds + table_off_V(N));
    t.W = (double2*)(lds + table_off_W(N));
    t.Wr = (double2*)(lds + table_off_Wr(N));
    t.lut = (uint32_t*)(lds + table_off_lut(N));
    const uint4* g = (const uint4*)gtab;
    uint4* l = (uint4*)lds;
    const int iV = (int)(table_off_V(N) / 16), iW = (int)(table_off_W(N) / 16);
    const int n16 = (int)(staged_table_bytes(N, needV, needW) / 16);
    // four loads in flight per thread before any is stored (indices clamped
    // into the staged range; only the wanted ones are stored)
    const int bd = blockDim.x;
    for (int i0 = threadIdx.x; i0 < n16; i0 += 4 * bd) {
        const int i1 = i0 + bd, i2 = i0 + 2 * bd, i3 = i0 + 3 * bd;
        const uint4 v0 = g[i0];
        const uint4 v1 = g[min(i1, n16 - 1)];
        const uint4 v2 = g[min(i2, n16 - 1)];
        const uint4 v3 = g[min(i3, n16 - 1)];
        auto put = [&](int i, const uint4& v) {
            if (i < n16 && (needV || i < iV || i >= iW)) l[i] = v;
        };
        put(i0, v0);
        put(i1, v1);
        put(i2, v2);
        put(i3, v3);
    }
    return t;
}

// One forward step p <- V + r (p - V), each operation rounded on its own.
__device__ inline void encode_step(double& px, double& py, const double2 v, const double r)
{
    const double tx = px - v.x;
    const double ty = py - v.y;
    const double ux = r * tx;
    const double uy = r * ty;
    px = v.x + ux;
    py = v.y + uy;
}

// The bucket word at coordinate u: the conversion to unsigned saturates
// (negative and NaN give 0, +inf gives 2^32 - 1), and the index times four is
// added to the table's LDS address modulo 2^32, so 2^32 - 1 lands on the
// guard entry just before the table.  For every other input u < 516.
__device__ __forceinline__ uint32_t lut_word(const uint32_t* lut, float u)
{
    uint32_t idx;
    asm("v_cvt_u32_f32 %0, %1" : "=v"(idx) : "v"(u));
    const uint32_t addr = (uint32_t)(uintptr_t)lut + (idx << 2);
    return *(const __attribute__((address_space(3))) uint32_t*)(size_t)addr;
}

// Sector of a point from the pseudo-angle look-up table.  Exact for every
// point at least kFastSectorMargin away from the sector lines (the fp32
// pseudo-angle errs by < 1e-6 there); never leaves [0, N).
__device__ inline int sector_fast(double qx, double qy, const uint32_t* __restrict__ lut, float lut_bias)
{
    const float fx = (float)qx;
    const float fy = (float)qy;
    const float rs = __builtin_amdgcn_rcpf(fabsf(fx) + fabsf(fy));
    // R = 1 - P = copysign(1 - y/(|x|+|y|), x).  For a point whose |x|+|y| is
    // a normal fp32 number, |y| rs <= 1 up to rounding, so u lies within
    // [shift - 2^-14, 4 kLutPerUnit + 1 + 2^-14) and the table repeats its last
    // bucket in its padding.  Other inputs occur only in corrupted points:
    // zero gives NaN, a sum too small for the reciprocal gives R = +-inf, and
    // lut_word maps those to bucket 0 or the guard word, so the look-up stays
    // inside the table and the sector inside [0, N).
    const float R = __builtin_copysignf(__builtin_fmaf(-fy, rs, 1.0f), fx);
    const float u = __builtin_fmaf(R, -(float)kLutPerUnit, lut_bias);
    const uint32_t e = lut_word(lut, u);
    // lower-edge sector (the word's low byte), plus one when the point lies
    // past the bucket's boundary: the compare sets the carry that an add with
    // byte-0 operand select consumes, so no separate mask of the low byte
    const float f = __builtin_amdgcn_fractf(u);
    uint32_t c;
    asm("v_cmp_ge_f32 vcc, %1, %2\n\t"
        "v_addc_co_u32_sdwa %0, vcc, %3, %2, vcc dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0"
        : "=v"(c)
        : "v"(f), "v"(e), "v"(0u)
        : "vcc");
    return (int)c;
}

// Exact nearest cell centre, lowest index on exact ties (used when the margin
// cannot be certified, e.g. touching cells at r = r_N).
__device__ inline int sector_exact(double qx, double qy, const double2* __restrict__ W, int N)
{
    int best = 0;
    double dx = qx - W[0].x, dy = qy - W[0].y;
    double bd = dx * dx + dy * dy;
    for (int c = 1; c < N; ++c) {
        dx = qx - W[c].x;
        dy = qy - W[c].y;
        const double d = dx * dx + dy * dy;
        if (d < bd) {
            bd = d;
            best = c;
        }
    }
    return best;
}

// Sectors of two independent points at once: both reciprocals, both table
// reads, then both compares, so that one point's look-up latency overlaps the
// other's arithmetic.  Same result as two sector_fast calls.
__device__ inline void sector_fast2(double ax, double ay, double bx, double by, const uint32_t* __restrict__ lut,
                                    float lut_bias, int& ca, int& cb)
{
    const float fxa = (float)ax, fya = (float)ay, fxb = (float)bx, fyb = (float)by;
    const float rsa = __builtin_amdgcn_rcpf(fabsf(fxa) + fabsf(fya));
    const float rsb = __builtin_amdgcn_rcpf(fabsf(fxb) + fabsf(fyb));
    const float Ra = __builtin_copysignf(__builtin_fmaf(-fya, rsa, 1.0f), fxa);
    const float Rb = __builtin_copysignf(__builtin_fmaf(-fyb, rsb, 1.0f), fxb);
    const float ua = __builtin_fmaf(Ra, -(float)kLutPerUnit, lut_bias);
    const float ub = __builtin_fmaf(Rb, -(float)kLutPerUnit, lut_bias);
    const uint32_t ea = lut_word(lut, ua);
    const uint32_t eb = lut_word(lut, ub);
    const float fa = __builtin_amdgcn_fractf(ua), fb = __builtin_amdgcn_fractf(ub);
    uint32_t xa, xb;
    asm("v_cmp_ge_f32 vcc, %2, %3\n\t"
        "v_addc_co_u32_sdwa %0, vcc, %6, %3, vcc dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0\n\t"
        "v_cmp_ge_f32 vcc, %4, %5\n\t"
        "v_addc_co_u32_sdwa %1, vcc, %6, %5, vcc dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0"
        : "=&v"(xa), "=&v"(xb)
        : "v"(fa), "v"(ea), "v"(fb), "v"(eb), "v"(0u)
        : "vcc");
    ca = (int)xa;
    cb = (int)xb;
}

template <bool EXACT>
__device__ inline int sector_of(double qx, double qy, const Tables& t, const CodecArgs& cd)
{
    if (EXACT) return sector_exact(qx, qy, t.W, cd.N);
    return sector_fast(qx, qy, t.lut, cd.lut_bias);
}

// Inverse map q <- (q - W(c)) / r, as q * (1/r) - W(c)/r with one rounding per
// coordinate.
__device__ inline void decode_step(double& qx, double& qy, const double2 wr, const double inv_r)
{
    qx = __builtin_fma(qx, inv_r, -wr.x);
    qy = __builtin_fma(qy, inv_r, -wr.y);
}

__device__ inline bool anchor_ok(double qx, double qy)
{
    const double a = fmax(fabs(qx), fabs(qy));
    return a <= kAnchorTol && qx == qx && qy == qy;
}

// Random access to one token (Sec. 2, Table 1): decodes only the span(s) of
// stream s holding symbols [tk*S, tk*S + S) and packs them into *got (byte k =
// symbol k).  P0 is the point of the first such span when the caller already
// loaded it (has_p0).  Returns 1 when a decoded span fails its anchor check.
template <bool EXACT>
__device__ inline int lookup_token(const double2* __restrict__ pts, const Tables& t, const CodecArgs& cd,
                                   int64_t s, int64_t tk, int S, int64_t n_sym, int64_t n_spans,
                                   bool has_p0, double2 P0, uint64_t* got)
{
    const int L = cd.L;
    const int64_t a = tk * S;
    const int64_t j0 = a / L, j1 = (a + S - 1) / L;
    int status = 0;
    uint64_t g = 0;
    for (int64_t j = j0; j <= j1; ++j) {
        const int64_t b = j * L;
        const int len = (int)min((int64_t)L, n_sym - b);
        const double2 P = (has_p0 && j == j0) ? P0 : pts[s * n_spans + j];
        double qx = P.x, qy = P.y;
        for (int k = len - 1; k >= 0; --k) {
            const int c = sector_of<EXACT>(qx, qy, t, cd);
            const int64_t off = b + k - a;   // position within the token's S symbols
            if (off >= 0 && off < S) g |= (uint64_t)c << (8 * off);
            decode_step(qx, qy, t.Wr[c], cd.inv_r);
        }
        if (!anchor_ok(qx, qy)) status = 1;
    }
    *got = g;
    return status;
}

// The tiles tl = blockIdx.x + i gridDim.x of a persistent block as (stream,
// tile within the stream), advanced with additions only: a 64-bit division
// per tile is emulated on the scalar unit and costs more than the tile's own
// scalar work.
struct TileWalk {
    int64_t s, j;           // stream, tile within the stream
    int64_t ds, dj, tps;    // the grid stride as (streams, tiles); tiles per stream

    __device__ void init(int64_t tl, int64_t stride, int64_t tiles_per_stream)
    {
        tps = tiles_per_stream;
        s = tl / tps;
        j = tl - s * tps;
        ds = stride / tps;
        dj = stride - ds * tps;
    }
    __device__ void next()
    {
        s += ds;
        j += dj;
        if (j >= tps) {
            j -= tps;
            ++s;
        }
    }
};

int64_t blocks_for(int64_t n_tiles)
{
    return n_tiles < kMaxBlocks ? (n_tiles > 0 ? n_tiles : 1) : kMaxBlocks;
}

bool codec_ok(const fkv_codec* c)
{
    return c && c->N >= 3 && c->N <= 256 && c->L >= 1 && c->L <= 64 && c->r > 0.0 && c->r < 1.0 &&
           c->r_max > 0.0 && c->r <= c->r_max * (1.0 + 1e-12);
}

CodecArgs codec_args(const fkv_codec* c)
{
    CodecArgs a;
    a.N = c->N;
    a.L = c->L;
    a.r = c->r;
    a.inv_r = 1.0 / c->r;
    a.lut_bias = (float)(2.0 * kLutPerUnit + lut_shift(c->N));
    return a;
}

// The look-up path is exact when every valid point keeps a margin of at least
// kFastSectorMargin from the sector lines: that margin is sin(pi/N) (1 - r/r_N).
bool needs_exact_sectors(const fkv_codec* c)
{
    const double margin = sin(M_PI / (double)c->N) * (1.0 - c->r / c->r_max);
    return !(margin >= kFastSectorMargin);
}

}  // namespace
}  // namespace fkv
