// rvq_kernels.hip -- per-head residual vector quantization (assignment) on
// gfx950 matrix cores.
//
// Method (Sec. 3 "Setup" of the paper): an archived K or V head vector x is
// stored as S codebook indices whose centroids sum to its reconstruction.
// Greedy residual VQ: r = x; for each stage st, i_st = argmin_j ||r - C_st[j]||^2
// (lowest j on exact ties), then r -= C_st[i_st].
//
// Formulation.  argmin_j ||r - c_j||^2 = argmin_j (||c_j||^2/2 - r.c_j): a dense
// contraction of the token block against the stage's codebook, plus a per-
// codeword bias.  The contraction runs on v_mfma_f32_32x32x16_f16 with the
// codebook as the A operand (32 codewords x 16 dims per instruction, staged in
// LDS with a 16-byte row pad so the 32 rows of a fragment hit distinct banks)
// and 32 tokens as the B operand (held in registers for all stages).  The
// accumulator is seeded with ||c||^2/2, so the finished tile already holds the
// scores.  In the 32x32 accumulator layout lane l owns token l%32 and 16 of
// the 32 codewords of the tile, so the argmin is an in-lane scan followed by
// one exchange with lane l^32.
//
// Precision.  Stage 0 multiplies fp16 x by fp16 codewords: every product is
// exact in fp32.  From stage 1 on the residual is an fp32 value; it is split
// as r = hi + lo with hi = fp16(r), lo = fp16(r - hi), and both halves go
// through the matrix cores into the same accumulator, so the scores keep
// about 22 bits of the residual instead of fp16's 11.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "fkv.h"
#include "fkv_hip_common.h"

namespace fkv {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

template <int D>
struct Shape {
    static constexpr int KS = D / 16;              // 16-deep matrix steps along d
    static constexpr int ROW = D + 8;              // LDS row stride in halfs (16-byte pad)
    static constexpr int TT = D <= 64 ? 2 : 1;     // 32-token tiles per wave
    static constexpr int TOK = kWaves * TT * 32;   // tokens per block
};

inline size_t rvq_lds_bytes(int D, int Kp)
{
    return (size_t)Kp * (D + 8) * sizeof(_Float16) + (size_t)Kp * sizeof(float);
}

template <int D>
__global__ __launch_bounds__(kThreads) void rvq_assign_kernel(
    const _Float16* __restrict__ x, const _Float16* __restrict__ books,
    const int32_t* __restrict__ stream_book, uint8_t* __restrict__ symbols,
    float* __restrict__ residual, uint32_t* __restrict__ n_bad, int64_t T, int64_t t_begin,
    int64_t Ta, int S, int K, int Kp, int n_books, int64_t blocks_per_stream)
{
    constexpr int KS = Shape<D>::KS, ROW = Shape<D>::ROW, TT = Shape<D>::TT, TOK = Shape<D>::TOK;
    extern __shared__ __align__(16) uint8_t lds[];
    _Float16* sB = (_Float16*)lds;
    float* sN = (float*)(lds + (size_t)Kp * ROW * sizeof(_Float16));

    const int64_t s = blockIdx.x / blocks_per_stream;
    const int64_t tb = (blockIdx.x - s * blocks_per_stream) * TOK;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int col = lane & 31, hh = lane >> 5;
    uint8_t* sym_s = symbols + s * Ta * S;
    const int b = stream_book[s];
    if (b < 0 || b >= n_books) {
        const int64_t te = min(Ta, tb + TOK);
        for (int64_t i = tb * S + tid; i < te * S; i += kThreads) sym_s[i] = 0xFF;
        if (residual)
            for (int64_t i = tb * D + tid; i < te * D; i += kThreads) residual[s * Ta * D + i] = NAN;
        if (tid == 0 && tb == 0 && n_bad) atomicAdd(n_bad, 1u);
        return;
    }
    const _Float16* bk = books + (int64_t)b * S * K * D;

    int64_t tok[TT];
    bool valid[TT];
    float r32[TT][KS][8];
    half8 bh[TT][KS], bl[TT][KS];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
        tok[tt] = tb + (int64_t)(wave * TT + tt) * 32 + col;
        valid[tt] = tok[tt] < Ta;
        const _Float16* row = x + (s * T + t_begin + (valid[tt] ? tok[tt] : 0)) * D + 8 * hh;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            half8 v = valid[tt] ? *(const half8*)(row + 16 * ks) : (half8)(_Float16)0;
            bh[tt][ks] = -v;
            bl[tt][ks] = (half8)(_Float16)0;
#pragma unroll
            for (int e = 0; e < 8; ++e) r32[tt][ks][e] = (float)v[e];
        }
    }

    for (int st = 0; st < S; ++st) {
        // Stage this stage's codebook (rows >= K zero) and its half norms.
        __syncthreads();
        const _Float16* C = bk + (int64_t)st * K * D;
        for (int i = tid; i < Kp * (D / 8); i += kThreads) {
            const int rw = i / (D / 8), c8 = i - rw * (D / 8);
            half8 v = rw < K ? *(const half8*)(C + (int64_t)rw * D + c8 * 8) : (half8)(_Float16)0;
            *(half8*)(sB + rw * ROW + c8 * 8) = v;
        }
        __syncthreads();
        for (int i = tid; i < Kp; i += kThreads) {
            float acc = 0.0f;
            for (int c8 = 0; c8 < D / 8; ++c8) {
                const half8 v = *(const half8*)(sB + i * ROW + c8 * 8);
#pragma unroll
                for (int e = 0; e < 8; ++e) acc += (float)v[e] * (float)v[e];
            }
            sN[i] = i < K ? 0.5f * acc : INFINITY;
        }
        __syncthreads();

        float best[TT];
        int bidx[TT];
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
            best[tt] = INFINITY;
            bidx[tt] = 0;
        }
        for (int ct = 0; ct < Kp / 32; ++ct) {
            const float* nb = sN + ct * 32 + 4 * hh;
            const floatx4 n0 = *(const floatx4*)(nb + 0), n1 = *(const floatx4*)(nb + 8);
            const floatx4 n2 = *(const floatx4*)(nb + 16), n3 = *(const floatx4*)(nb + 24);
            floatx16 acc[TT];
#pragma unroll
            for (int tt = 0; tt < TT; ++tt) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[tt][e] = n0[e];
                    acc[tt][4 + e] = n1[e];
                    acc[tt][8 + e] = n2[e];
                    acc[tt][12 + e] = n3[e];
                }
            }
            const _Float16* arow = sB + (ct * 32 + col) * ROW + 8 * hh;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const half8 a = *(const half8*)(arow + 16 * ks);
#pragma unroll
                for (int tt = 0; tt < TT; ++tt)
                    acc[tt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bh[tt][ks], acc[tt], 0, 0, 0);
                if (st > 0) {
#pragma unroll
                    for (int tt = 0; tt < TT; ++tt)
                        acc[tt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bl[tt][ks], acc[tt], 0, 0, 0);
                }
            }
            // acc[tt][v] is the score of codeword ct*32 + 8(v/4) + 4*hh + v%4 for
            // token col: increasing v visits this lane's codewords in index order.
#pragma unroll
            for (int tt = 0; tt < TT; ++tt) {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const float val = acc[tt][v];
                    if (val < best[tt]) {
                        best[tt] = val;
                        bidx[tt] = ct * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
                    }
                }
            }
        }
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
            const float ob = __shfl_xor(best[tt], 32);
            const int oi = __shfl_xor(bidx[tt], 32);
            if (ob < best[tt] || (ob == best[tt] && oi < bidx[tt])) {
                best[tt] = ob;
                bidx[tt] = oi;
            }
            if (hh == 0 && valid[tt]) sym_s[tok[tt] * S + st] = (uint8_t)bidx[tt];
            const _Float16* crow = sB + bidx[tt] * ROW + 8 * hh;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const half8 cv = *(const half8*)(crow + 16 * ks);
#pragma unroll
                for (int e = 0; e < 8; ++e) r32[tt][ks][e] -= (float)cv[e];
            }
            if (st + 1 < S) {
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const _Float16 h = (_Float16)r32[tt][ks][e];
                        const _Float16 l = (_Float16)(r32[tt][ks][e] - (float)h);
                        bh[tt][ks][e] = -h;
                        bl[tt][ks][e] = -l;
                    }
                }
            }
        }
    }

    if (residual) {
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
            if (!valid[tt]) continue;
            float* out = residual + (s * Ta + tok[tt]) * D + 8 * hh;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                floatx4 lo4, hi4;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    lo4[e] = r32[tt][ks][e];
                    hi4[e] = r32[tt][ks][4 + e];
                }
                *(floatx4*)(out + 16 * ks) = lo4;
                *(floatx4*)(out + 16 * ks + 4) = hi4;
            }
        }
    }
}

template <int D>
int launch_rvq(const fkv_rvq_desc* dsc, const uint16_t* x, const uint16_t* books,
               const int32_t* stream_book, uint8_t* symbols, float* residual, uint32_t* n_bad,
               hipStream_t stream)
{
    static std::once_flag once;
    const int Kp = (dsc->K + 31) / 32 * 32;
    const size_t shm = rvq_lds_bytes(D, Kp);
    std::call_once(once, [] {
        (void)hipFuncSetAttribute((const void*)rvq_assign_kernel<D>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)rvq_lds_bytes(D, 256));
    });
    (void)hipGetLastError();
    const int64_t Ta = dsc->t_end - dsc->t_begin;
    const int64_t bps = (Ta + Shape<D>::TOK - 1) / Shape<D>::TOK;
    const int64_t nblk = bps * dsc->n_streams;
    if (nblk > 0x7fffffff) return FKV_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(rvq_assign_kernel<D>, dim3((unsigned)nblk), dim3(kThreads), shm, stream,
                       (const _Float16*)x, (const _Float16*)books, stream_book, symbols, residual,
                       n_bad, dsc->T, dsc->t_begin, Ta, dsc->S, dsc->K, Kp, dsc->n_books, bps);
    return launch_status();
}

}  // namespace
}  // namespace fkv

using namespace fkv;

extern "C" int fkv_rvq_assign(const fkv_rvq_desc* desc, const uint16_t* x_f16, const uint16_t* books_f16,
                              const int32_t* stream_book, uint8_t* symbols, float* residual,
                              uint32_t* n_bad_streams, void* stream)
{
    if (!desc) return FKV_ERR_INVALID_ARG;
    const fkv_rvq_desc& d = *desc;
    if (d.n_streams < 0 || d.T < 0 || d.t_begin < 0 || d.t_end < d.t_begin || d.t_end > d.T)
        return FKV_ERR_INVALID_ARG;
    if (d.d < 16 || d.d > 256 || d.d % 16 != 0) return FKV_ERR_INVALID_ARG;
    if (d.S < 1 || d.S > 8 || d.K < 1 || d.K > 256 || d.n_books < 1) return FKV_ERR_INVALID_ARG;
    if (d.n_streams == 0 || d.t_end == d.t_begin) return FKV_OK;
    if (!x_f16 || !books_f16 || !stream_book || !symbols) return FKV_ERR_INVALID_ARG;
    if (!aligned(x_f16, 16) || !aligned(books_f16, 16) || !aligned(stream_book, 4))
        return FKV_ERR_INVALID_ARG;
    if (residual && !aligned(residual, 16)) return FKV_ERR_INVALID_ARG;
    if (n_bad_streams && !aligned(n_bad_streams, 4)) return FKV_ERR_INVALID_ARG;
    const hipStream_t st = (hipStream_t)stream;
#define FKV_RVQ_CASE(DD) \
    case DD: return launch_rvq<DD>(desc, x_f16, books_f16, stream_book, symbols, residual, n_bad_streams, st);
    switch (d.d) {
        FKV_RVQ_CASE(16) FKV_RVQ_CASE(32) FKV_RVQ_CASE(48) FKV_RVQ_CASE(64)
        FKV_RVQ_CASE(80) FKV_RVQ_CASE(96) FKV_RVQ_CASE(112) FKV_RVQ_CASE(128)
        FKV_RVQ_CASE(144) FKV_RVQ_CASE(160) FKV_RVQ_CASE(176) FKV_RVQ_CASE(192)
        FKV_RVQ_CASE(208) FKV_RVQ_CASE(224) FKV_RVQ_CASE(240) FKV_RVQ_CASE(256)
    default: return FKV_ERR_INVALID_ARG;
    }
#undef FKV_RVQ_CASE
}
