// fkv_internal.h -- private layout shared by libfkv's host code and kernels.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace fkv {

// Sector look-up table: the plane is cut into angular sectors around the
// cell centres; decode finds a point's sector through a monotone
// pseudo-angle  P = y/(|x|+|y|)  (x >= 0)  or  2 - y/(|x|+|y|)  (x < 0),
// which runs from -1 (angle -pi/2) to 3 (angle 3pi/2).  P is cut into
// kLutPerUnit buckets per unit; each bucket holds the sector at its lower
// edge and, when one sector boundary falls inside it, that boundary and
// the sector above it.  A sector is at least pi/N wide in P, wider than a
// bucket for N <= 256, so a bucket never holds two boundaries.
constexpr int kLutPerUnit = 128;
constexpr int kLutBuckets = 4 * kLutPerUnit;

struct LutEntry {
    float thr;      // P at the sector boundary inside this bucket, or +inf
    uint16_t lo;    // sector for P < thr
    uint16_t hi;    // sector for P >= thr
};
static_assert(sizeof(LutEntry) == 8, "LutEntry layout");

// Device table, one per alphabet, 16-byte aligned sections:
//   [0,      16N)  V[c]   = (cos 2 pi c/N, sin 2 pi c/N)        double2
//   [16N,    32N)  W[c]   = (1 - r) V[c]   (cell centres)        double2
//   [32N,    48N)  Wr[c]  = W[c] / r                             double2
//   [48N, 48N+4096) sector look-up table                         LutEntry[512]
constexpr size_t table_off_V(int) { return 0; }
constexpr size_t table_off_W(int N) { return (size_t)16 * N; }
constexpr size_t table_off_Wr(int N) { return (size_t)32 * N; }
constexpr size_t table_off_lut(int N) { return (size_t)48 * N; }
constexpr size_t table_bytes(int N) { return (size_t)48 * N + sizeof(LutEntry) * kLutBuckets; }

// Decode may take a sector straight from the look-up table only when every
// valid point keeps a margin of at least this much (absolute, in the unit
// disk) from the sector lines; otherwise it compares exact distances.
constexpr double kFastSectorMargin = 1e-4;

// Anchor acceptance threshold after a span's backward walk (2^-6).
constexpr double kAnchorTol = 1.0 / 64.0;

}  // namespace fkv
