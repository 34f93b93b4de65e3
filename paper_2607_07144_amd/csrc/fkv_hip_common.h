// fkv_hip_common.h -- small device/host helpers shared by libfkv's kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fkv.h"

namespace fkv {

// Maps the last HIP error of this thread to a status code.
inline int launch_status()
{
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) return FKV_OK;
    if (e == hipErrorNoDevice || e == hipErrorInvalidDevice) return FKV_ERR_NO_DEVICE;
    return FKV_ERR_LAUNCH;
}

inline bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

// Streaming (non-temporal) 16-byte point load and store: the access carries
// the non-temporal hint, so lines that a kernel touches exactly once do not
// displace what it re-reads (its tables, the symbol lines that neighbouring
// lanes share).  Values are those of a plain access.
typedef double fkv_v2d __attribute__((ext_vector_type(2)));
__device__ __forceinline__ double2 load_point_stream(const double2* p)
{
    const fkv_v2d v = __builtin_nontemporal_load((const fkv_v2d*)p);
    return make_double2(v.x, v.y);
}
__device__ __forceinline__ void store_point_stream(double2* p, double x, double y)
{
    const fkv_v2d v = {x, y};
    __builtin_nontemporal_store(v, (fkv_v2d*)p);
}

// Copies global bytes [g0, g1) of `src` into LDS so that global byte g sits at
// LDS byte (g - (g0 & ~3)).  Whole aligned dwords are moved as dwords; the
// partial dwords at either end byte by byte, so nothing outside [g0, g1) is
// touched.  `src` must be 4-byte aligned.  Block-cooperative, no barrier.
__device__ inline void bytes_to_lds(const uint8_t* __restrict__ src, int64_t g0, int64_t g1,
                                    uint8_t* lds)
{
    const int tid = threadIdx.x, nt = blockDim.x;
    const int64_t base = g0 & ~(int64_t)3;
    const int64_t a0 = (g0 + 3) & ~(int64_t)3;
    const int64_t a1 = g1 & ~(int64_t)3;
    if (a0 >= a1) {
        for (int64_t g = g0 + tid; g < g1; g += nt) lds[g - base] = src[g];
        return;
    }
    const uint32_t* s32 = (const uint32_t*)src;
    uint32_t* l32 = (uint32_t*)(lds + (a0 - base));
    for (int64_t w = (a0 >> 2) + tid; w < (a1 >> 2); w += nt) l32[w - (a0 >> 2)] = s32[w];
    if (tid < a0 - g0) lds[g0 + tid - base] = src[g0 + tid];
    if (tid < g1 - a1) lds[a1 + tid - base] = src[a1 + tid];
}

// Inverse of bytes_to_lds: writes LDS bytes back to global [g0, g1).
__device__ inline void lds_to_bytes(const uint8_t* lds, int64_t g0, int64_t g1,
                                    uint8_t* __restrict__ dst)
{
    const int tid = threadIdx.x, nt = blockDim.x;
    const int64_t base = g0 & ~(int64_t)3;
    const int64_t a0 = (g0 + 3) & ~(int64_t)3;
    const int64_t a1 = g1 & ~(int64_t)3;
    if (a0 >= a1) {
        for (int64_t g = g0 + tid; g < g1; g += nt) dst[g] = lds[g - base];
        return;
    }
    uint32_t* d32 = (uint32_t*)dst;
    const uint32_t* l32 = (const uint32_t*)(lds + (a0 - base));
    for (int64_t w = (a0 >> 2) + tid; w < (a1 >> 2); w += nt) d32[w] = l32[w - (a0 >> 2)];
    if (tid < a0 - g0) dst[g0 + tid] = lds[g0 + tid - base];
    if (tid < g1 - a1) dst[a1 + tid] = lds[a1 + tid - base];
}

// One wave's counterpart of lds_to_bytes: its 64 lanes write LDS bytes back to
// global [g0, g1), whole aligned dwords as dwords (streaming stores when NT)
// and the partial dwords at either end byte by byte (so nothing outside
// [g0, g1) is written).
template <bool NT = false>
__device__ inline void lds_to_bytes_wave(const uint8_t* lds, int64_t g0, int64_t g1, uint8_t* __restrict__ dst,
                                         int lane)
{
    const int64_t base = g0 & ~(int64_t)3;
    const int64_t a0 = (g0 + 3) & ~(int64_t)3;
    const int64_t a1 = g1 & ~(int64_t)3;
    if (a0 >= a1) {
        for (int64_t g = g0 + lane; g < g1; g += 64) dst[g] = lds[g - base];
        return;
    }
    uint32_t* d32 = (uint32_t*)dst;
    const uint32_t* l32 = (const uint32_t*)(lds + (a0 - base));
    for (int64_t w = (a0 >> 2) + lane; w < (a1 >> 2); w += 64) {
        if (NT)
            __builtin_nontemporal_store(l32[w - (a0 >> 2)], d32 + w);
        else
            d32[w] = l32[w - (a0 >> 2)];
    }
    if (lane < a0 - g0) dst[g0 + lane] = lds[g0 + lane - base];
    if (lane < g1 - a1) dst[a1 + lane] = lds[a1 + lane - base];
}

// Correctly rounded binary64 -> binary16 (round to nearest, ties to even): the
// conversion to binary32 is made round-to-odd (truncate, then set the last
// bit when inexact), which carries enough information for the final
// round-to-nearest-even step to binary16 (binary32 has 13 more bits).
__device__ inline _Float16 f64_to_f16(double v)
{
    const float f = (float)v;
    uint32_t u = __float_as_uint(f);
    if ((double)f != v) {
        if (fabs((double)f) > fabs(v)) u -= 1;   // towards zero
        u |= 1u;
    }
    return (_Float16)__uint_as_float(u);
}

// Adds the number of lanes of the block with `flag` set to *counter, one
// atomic per wave that has any.
__device__ inline void count_flags(bool flag, uint32_t* counter)
{
    if (!counter) return;
    const unsigned long long m = __ballot(flag);
    if (m && (threadIdx.x & 63) == 0) atomicAdd(counter, (uint32_t)__popcll(m));
}

}  // namespace fkv
