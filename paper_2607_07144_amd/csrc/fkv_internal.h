// fkv_internal.h -- private layout shared by libfkv's host code and kernels.
#pragma once

#include <math.h>
#include <stddef.h>
#include <stdint.h>

namespace fkv {

// Sector look-up table: the plane is cut into angular sectors around the
// cell centres; decode finds a point's sector through a monotone
// pseudo-angle  P = y/(|x|+|y|)  (x >= 0)  or  2 - y/(|x|+|y|)  (x < 0),
// which runs from -1 (angle -pi/2) to 3 (angle 3pi/2).  P is cut into
// kLutPerUnit buckets per unit; a sector is at least pi/N wide in P, wider
// than a bucket for N <= 256, so a bucket holds at most one boundary.
//
// The bucket grid is shifted by lut_shift(N) buckets so that the boundary at
// angle -pi/N, where the sector numbering wraps from N-1 to 0, falls on a
// bucket edge: inside every bucket the sector above a boundary is then the
// one below it plus one, and an entry is a single 32-bit word -- the
// boundary's position within the bucket as an fp32 fraction (2 when the
// bucket has none) whose low 8 mantissa bits are replaced by the sector at
// the bucket's lower edge (the threshold moves by < 2^-15 of a bucket).
//
// The kernels evaluate the mirrored coordinate R = 1 - P, which is
// copysign(1 - y/(|x|+|y|), x) (one fused multiply-add and a sign copy); the
// bucket coordinate is u = (P + 1) kLutPerUnit + shift
// = 2 kLutPerUnit + shift - R kLutPerUnit, in [0, 4 kLutPerUnit + 1).
constexpr int kLutPerUnit = 128;
constexpr int kLutEntries = 4 * kLutPerUnit + 1;
// The section: 16 bytes whose last word is a guard entry (sector 0, no
// boundary) right before the table, then the entries, padded to 16 bytes.
constexpr size_t kLutGuard = 16;
constexpr size_t kLutBytes = kLutGuard + (sizeof(uint32_t) * kLutEntries + 15) / 16 * 16;
static_assert((kLutBytes - kLutGuard) / sizeof(uint32_t) >= kLutEntries + 1, "the look-up table needs a padding entry");

// (P + 1) kLutPerUnit of the wrap boundary is c/(c+s) kLutPerUnit with
// c = cos(pi/N), s = sin(pi/N); the shift lifts it to the next integer.
inline double lut_shift(int N)
{
    const double s = sin(M_PI / (double)N), c = cos(M_PI / (double)N);
    const double u = c / (c + s) * (double)kLutPerUnit;
    return ceil(u) - u;
}

// Device table, one per alphabet, 16-byte aligned sections, ordered so that
// the inverse map's fast path needs only the first two:
//   [0,             16N)            Wr[c] = W[c] / r                double2
//   [16N,           16N + B)        16 bytes ending in a guard word, then the
//                                   sector look-up table            uint32_t[513]
//   [16N + B,       32N + B)        V[c]  = (cos 2 pi c/N, sin 2 pi c/N)
//   [32N + B,       48N + B)        W[c]  = (1 - r) V[c]  (cell centres)
// with B = kLutBytes.
constexpr size_t table_off_Wr(int) { return 0; }
constexpr size_t table_off_lut(int N) { return (size_t)16 * N + kLutGuard; }
constexpr size_t table_off_V(int N) { return (size_t)16 * N + kLutBytes; }
constexpr size_t table_off_W(int N) { return (size_t)32 * N + kLutBytes; }
constexpr size_t table_bytes(int N) { return (size_t)48 * N + kLutBytes; }
// the prefix holding Wr and the look-up table
constexpr size_t table_fast_bytes(int N) { return (size_t)16 * N + kLutBytes; }

// Decode may take a sector straight from the look-up table only when every
// valid point keeps a margin of at least this much (absolute, in the unit
// disk) from the sector lines; otherwise it compares exact distances.
constexpr double kFastSectorMargin = 1e-4;

// Anchor acceptance threshold after a span's backward walk (2^-6).
constexpr double kAnchorTol = 1.0 / 64.0;

}  // namespace fkv
