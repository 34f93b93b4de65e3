// diag_kernels.hip -- a measurement aid, not part of the archive path: the
// rate the matrix cores sustain on the instruction the RVQ assignment uses
// (v_mfma_f32_32x32x16_f16), issued from registers in independent chains with
// no memory traffic.  It is the device's practical ceiling for that kernel
// under the board's power limit, reported beside the datasheet peak.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fkv.h"
#include "fkv_hip_common.h"

namespace fkv {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
constexpr int kDiagThreads = 256;
constexpr int kDiagChains = 4;   // independent accumulators per wave

// Pseudo-random binary16 in [-1, 1) from a 32-bit counter (a multiplicative
// hash; the values only need to make the multiplier inputs change).
__device__ __forceinline__ _Float16 hash_half(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return (_Float16)((float)(x >> 8) * (1.0f / 8388608.0f) - 1.0f);
}

// RANDOM = false: every operand element is a_val or b_val (the accumulators
// have a closed form).  RANDOM = true: each lane's operands are two
// pseudo-random sets used alternately, so the multiplier inputs change on
// every instruction as they do on real data (the power the matrix cores draw
// depends on it).
template <bool RANDOM>
__global__ __launch_bounds__(kDiagThreads) void mfma_loop_kernel(float a_val, float b_val, int32_t iters,
                                                                  float* __restrict__ out)
{
    half8 a0, b0, a1, b1;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const uint32_t base = (blockIdx.x * kDiagThreads + threadIdx.x) * 32u + (uint32_t)e;
        a0[e] = RANDOM ? hash_half(base) : (_Float16)a_val;
        b0[e] = RANDOM ? hash_half(base + 8) : (_Float16)b_val;
        a1[e] = RANDOM ? hash_half(base + 16) : (_Float16)a_val;
        b1[e] = RANDOM ? hash_half(base + 24) : (_Float16)b_val;
    }
    floatx16 acc[kDiagChains];
#pragma unroll
    for (int c = 0; c < kDiagChains; ++c) acc[c] = (floatx16)0.0f;
    for (int32_t i = 0; i < iters; ++i) {
        const half8 a = (i & 1) ? a1 : a0;
        const half8 b = (i & 1) ? b1 : b0;
#pragma unroll
        for (int c = 0; c < kDiagChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc[c], 0, 0, 0);
    }
    float s = 0.0f;
#pragma unroll
    for (int c = 0; c < kDiagChains; ++c) s += acc[c][0];
    if (blockIdx.x == 0 && threadIdx.x == 0) out[0] = s;
}

}  // namespace
}  // namespace fkv

using namespace fkv;

extern "C" int fkv_diag_mfma_loop(int32_t n_blocks, int32_t iters, int32_t random_operands, float a_val, float b_val,
                                  float* out, void* stream)
{
    if (n_blocks < 1 || iters < 0 || !out || !aligned(out, 4)) return FKV_ERR_INVALID_ARG;
    if (random_operands)
        hipLaunchKernelGGL(mfma_loop_kernel<true>, dim3((unsigned)n_blocks), dim3(kDiagThreads), 0,
                           (hipStream_t)stream, a_val, b_val, iters, out);
    else
        hipLaunchKernelGGL(mfma_loop_kernel<false>, dim3((unsigned)n_blocks), dim3(kDiagThreads), 0,
                           (hipStream_t)stream, a_val, b_val, iters, out);
    return launch_status();
}

extern "C" double fkv_diag_mfma_loop_flops(int32_t n_blocks, int32_t iters)
{
    if (n_blocks < 1 || iters < 0) return 0.0;
    return (double)n_blocks * (kDiagThreads / 64) * kDiagChains * (double)iters * (2.0 * 32 * 32 * 16);
}
