// kmeans_kernels.hip -- one Lloyd update of a residual stage of per-head
// codebooks (Sec. 3 "Setup": codebooks are trained by k-means), for gfx950.
//
// The assignment step is fkv_rvq_assign.  Accumulate: one block per book and
// 64-dimension slice; one lane per 8 dimensions of a member token forms the
// stage input r = x - (codewords of the earlier stages) exactly in fp64 and
// adds it, as an integer in units of 2^-24 (every binary16 value is a multiple
// of 2^-24), to its cluster's sum with 64-bit LDS atomics -- integer addition,
// so the sums do not depend on the order of the atomics.  Finalize: mean = sum / count * 2^-24 in fp64, rounded once to
// binary16; an empty cluster keeps its centroid.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>

#include "fkv.h"
#include "fkv_hip_common.h"

#pragma clang fp contract(off)

namespace fkv {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
constexpr int kThreads = 256;
// Accumulate: one 1024-thread block per (book, slice), so that enough member
// tokens' loads are in flight to cover their latency (a block's tokens are
// walked in 1024-task steps, each task waiting on its symbol, row and earlier
// codewords).
constexpr int kAccThreads = 1024;
constexpr int kAccBatch = 4;   // tasks per thread whose loads are in flight together

// One block per (book, 64-dimension slice): the block owns that slice of the
// book's cluster sums, accumulates every member token of every stream of the
// book into LDS (64-bit LDS atomics), then adds the slice to the global sums
// with plain read-modify-writes (no other block touches it in this launch).
// A cluster's row in LDS is dc + 1 words long: with an odd number of 8-byte
// words per row, the same dimension of different clusters falls in different
// banks (with dc words, every cluster's dimension e shared one bank, so the
// atomics of a wave's tokens, which hit random clusters, serialised).
constexpr int kSlice = 64;

// ST >= 0: the stage is fixed at compile time, so the loops over the earlier
// stages unroll and all their codeword reads of a task batch are issued
// together (one dependent memory round instead of one per earlier stage;
// measured at the long-context shape: stage 1 from 8.1 to 6.5 ms, stage 2
// from 10.6 to 7.6 ms).  ST = -1 takes the stage at run time (stages 5..7,
// where the unrolled form would spill).
template <int ST>
__global__ __launch_bounds__(kAccThreads) void kmeans_accumulate_kernel(
    const _Float16* __restrict__ x, const _Float16* __restrict__ books, const int32_t* __restrict__ stream_book,
    const uint8_t* __restrict__ symbols, unsigned long long* __restrict__ sums, uint32_t* __restrict__ counts,
    int64_t n_streams, int64_t T, int64_t t_begin, int64_t Ta, int d, int S, int K, int stage_rt)
{
    const int stage = ST >= 0 ? ST : stage_rt;
    extern __shared__ __align__(16) uint8_t lds[];
    const int n_slices = (d + kSlice - 1) / kSlice;
    const int b = blockIdx.x / n_slices, slice = blockIdx.x - b * n_slices;
    const int e0 = slice * kSlice, dc = min(kSlice, d - e0);   // this block's dimensions [e0, e0 + dc)
    const int nch = dc / 8;
    const int pitch = dc + 1;                                    // words per cluster row
    unsigned long long* ls = (unsigned long long*)lds;           // [K][pitch]
    uint32_t* lc = (uint32_t*)(ls + (size_t)K * pitch);          // [K]
    int* match = (int*)(lc + K);                                 // [kAccThreads]: streams of a chunk using book b
    int* n_match = match + kAccThreads;
    for (int i = threadIdx.x; i < K * pitch; i += kAccThreads) ls[i] = 0;
    for (int i = threadIdx.x; i < K; i += kAccThreads) lc[i] = 0;
    // The streams are scanned kAccThreads at a time, one per thread, and those
    // of book b listed in LDS (their order does not matter: integer sums).
    for (int64_t s0 = 0; s0 < n_streams; s0 += kAccThreads) {
        if (threadIdx.x == 0) *n_match = 0;
        __syncthreads();
        if (s0 + threadIdx.x < n_streams && stream_book[s0 + threadIdx.x] == b)
            match[atomicAdd(n_match, 1)] = (int)threadIdx.x;
        __syncthreads();
        const int nm = *n_match;
        for (int m = 0; m < nm; ++m) {
            const int64_t s = s0 + match[m];
            // 32-bit task walk (the host checks that Ta * nch fits).  Each thread
            // takes kAccBatch tasks at a time and issues all their loads before
            // any sum, so the latencies of the batch overlap.
            const int n_task = (int)(Ta * nch);
            for (int task0 = threadIdx.x; task0 < n_task; task0 += kAccThreads * kAccBatch) {
                int cl[kAccBatch];          // cluster of each task, -1: none (past the end, or skipped)
                int64_t row[kAccBatch];     // token row of x
                const uint8_t* sym[kAccBatch];
                int chn[kAccBatch];
#pragma unroll
                for (int u = 0; u < kAccBatch; ++u) {
                    const int task = task0 + u * kAccThreads;
                    const int t = task / nch;
                    chn[u] = task - t * nch;
                    sym[u] = symbols + (s * Ta + (task < n_task ? t : 0)) * S;
                    row[u] = s * T + t_begin + (task < n_task ? t : 0);
                    cl[u] = task < n_task ? 0 : -1;
                }
                uint64_t sy[kAccBatch];     // the task's symbols of stages 0..stage, one byte each
#pragma unroll
                for (int u = 0; u < kAccBatch; ++u) {
                    sy[u] = 0;
                    for (int st = 0; st <= stage; ++st) sy[u] |= (uint64_t)sym[u][st] << (8 * st);
                }
                half8 xv[kAccBatch];
#pragma unroll
                for (int u = 0; u < kAccBatch; ++u) xv[u] = *(const half8*)(x + row[u] * d + e0 + chn[u] * 8);
#pragma unroll
                for (int u = 0; u < kAccBatch; ++u) {
                    bool bad = cl[u] < 0;
                    for (int st = 0; st <= stage; ++st) bad = bad || (int)((sy[u] >> (8 * st)) & 255u) >= K;
                    cl[u] = bad ? -1 : (int)((sy[u] >> (8 * stage)) & 255u);   // outside the book: skipped
                }
                double r[kAccBatch][8];
#pragma unroll
                for (int u = 0; u < kAccBatch; ++u)
#pragma unroll
                    for (int e = 0; e < 8; ++e) r[u][e] = (double)xv[u][e];
#pragma unroll
                for (int st = 0; st < stage; ++st) {
                    half8 c[kAccBatch];
#pragma unroll
                    for (int u = 0; u < kAccBatch; ++u)
                        c[u] = *(const half8*)(books +
                                               (((int64_t)b * S + st) * K + (cl[u] < 0 ? 0 : (int)((sy[u] >> (8 * st)) & 255u))) * d +
                                               e0 + chn[u] * 8);
#pragma unroll
                    for (int u = 0; u < kAccBatch; ++u)
#pragma unroll
                        for (int e = 0; e < 8; ++e) r[u][e] = r[u][e] - (double)c[u][e];
                }
#pragma unroll
                for (int u = 0; u < kAccBatch; ++u) {
                    if (cl[u] < 0) continue;
                    unsigned long long* dst = ls + (size_t)cl[u] * pitch + chn[u] * 8;
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        atomicAdd(dst + e, (unsigned long long)(long long)ldexp(r[u][e], 24));
                    if (chn[u] == 0 && slice == 0) atomicAdd(lc + cl[u], 1u);
                }
            }
        }
        __syncthreads();   // the list is rewritten for the next chunk
    }
    for (int i = threadIdx.x; i < K * dc; i += kAccThreads) {
        const int j = i / dc, e = i - j * dc;
        const unsigned long long v = ls[j * pitch + e];
        if (v) sums[((int64_t)b * K + j) * d + e0 + e] += v;
    }
    if (slice == 0)
        for (int j = threadIdx.x; j < K; j += kAccThreads)
            if (lc[j]) counts[(int64_t)b * K + j] += lc[j];
}

__global__ __launch_bounds__(kThreads) void kmeans_finalize_kernel(
    const unsigned long long* __restrict__ sums, const uint32_t* __restrict__ counts, _Float16* __restrict__ books,
    int d, int S, int K, int stage, int64_t n_elems)
{
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n_elems; i += (int64_t)gridDim.x * kThreads) {
        const int64_t bj = i / d;   // book * K + j
        const int e = (int)(i - bj * d);
        const uint32_t c = counts[bj];
        if (c == 0) continue;
        const int64_t b = bj / K, j = bj - b * K;
        const double m = ldexp((double)(long long)sums[i] / (double)c, -24);
        books[((b * S + stage) * K + j) * d + e] = f64_to_f16(m);
    }
}

int64_t grid_for(int64_t n)
{
    const int64_t b = (n + kThreads - 1) / kThreads;
    return b < 1 ? 1 : (b > 4096 ? 4096 : b);
}

// Zero fill of n 8-byte words (the scratch sums and counts before an update;
// a kernel rather than a memset so that the call can be captured in a graph).
__global__ __launch_bounds__(kThreads) void zero_words_kernel(unsigned long long* __restrict__ p, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads) p[i] = 0;
}

// Device scratch of the allocation-free k-means update: the cluster sums
// (int64, [n_books][K][d]) followed by the counts (u32, [n_books][K]).  Each
// device the library runs on holds its own copy until the process ends.  In
// host code this name is not a device address: kernels get the per-device
// address taken once with hipGetSymbolAddress.
static __device__ __align__(256) unsigned long long scratch[FKV_NOALLOC_SCRATCH_BYTES / 8];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices];

// Address of the current device's scratch array (taken once per device);
// nullptr when the device is unknown or the runtime refuses.
void* scratch_address()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return nullptr;
        }
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

}  // namespace
}  // namespace fkv

using namespace fkv;

extern "C" int fkv_kmeans_accumulate(const fkv_rvq_desc* desc, const uint16_t* x_f16, const uint16_t* books_f16,
                                     const int32_t* stream_book, const uint8_t* symbols, int32_t stage,
                                     int64_t* sums, uint32_t* counts, void* stream)
{
    if (!desc) return FKV_ERR_INVALID_ARG;
    const fkv_rvq_desc& D = *desc;
    if (D.n_streams < 0 || D.T < 0 || D.t_begin < 0 || D.t_end < D.t_begin || D.t_end > D.T) return FKV_ERR_INVALID_ARG;
    if (D.d < 8 || D.d > 256 || D.d % 8 != 0 || D.S < 1 || D.S > 8 || D.K < 1 || D.K > 256 || D.n_books < 1)
        return FKV_ERR_INVALID_ARG;
    if (stage < 0 || stage >= D.S) return FKV_ERR_INVALID_ARG;
    const int64_t Ta = D.t_end - D.t_begin;
    if (D.n_streams == 0 || Ta == 0) return FKV_OK;
    if (!x_f16 || !books_f16 || !stream_book || !symbols || !sums || !counts) return FKV_ERR_INVALID_ARG;
    if (!aligned(x_f16, 16) || !aligned(books_f16, 16) || !aligned(sums, 8) || !aligned(counts, 4) ||
        !aligned(stream_book, 4))
        return FKV_ERR_INVALID_ARG;
    const int n_slices = (D.d + kSlice - 1) / kSlice;
    if (Ta * (std::min(kSlice, (int)D.d) / 8) > 0x7fffffff - kAccThreads * kAccBatch) return FKV_ERR_UNSUPPORTED;
    const size_t shm = (size_t)D.K * (std::min(kSlice, (int)D.d) + 1) * 8 + (size_t)D.K * 4 + (kAccThreads + 1) * 4;
    static std::once_flag once[6];   // one per kernel instance below
    auto go = [&](int slot, auto kern) {
        std::call_once(once[slot], [&] {
            (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                      256 * (kSlice + 1) * 8 + 256 * 4 + (kAccThreads + 1) * 4);
        });
        (void)hipGetLastError();
        hipLaunchKernelGGL(kern, dim3((unsigned)(D.n_books * n_slices)), dim3(kAccThreads), shm, (hipStream_t)stream,
                           (const _Float16*)x_f16, (const _Float16*)books_f16, stream_book, symbols,
                           (unsigned long long*)sums, counts, D.n_streams, D.T, D.t_begin, Ta, D.d, D.S, D.K, stage);
        return launch_status();
    };
    switch (stage) {
    case 0: return go(0, kmeans_accumulate_kernel<0>);
    case 1: return go(1, kmeans_accumulate_kernel<1>);
    case 2: return go(2, kmeans_accumulate_kernel<2>);
    case 3: return go(3, kmeans_accumulate_kernel<3>);
    case 4: return go(4, kmeans_accumulate_kernel<4>);
    default: return go(5, kmeans_accumulate_kernel<-1>);
    }
}

extern "C" int fkv_kmeans_finalize(int32_t n_books, int32_t S, int32_t K, int32_t d, int32_t stage,
                                   const int64_t* sums, const uint32_t* counts, uint16_t* books_f16, void* stream)
{
    if (n_books < 1 || S < 1 || S > 8 || K < 1 || K > 256 || d < 8 || d > 256 || d % 8 != 0) return FKV_ERR_INVALID_ARG;
    if (stage < 0 || stage >= S || !sums || !counts || !books_f16) return FKV_ERR_INVALID_ARG;
    if (!aligned(sums, 8) || !aligned(counts, 4) || !aligned(books_f16, 2)) return FKV_ERR_INVALID_ARG;
    const int64_t n_elems = (int64_t)n_books * K * d;
    hipLaunchKernelGGL(kmeans_finalize_kernel, dim3((unsigned)grid_for(n_elems)), dim3(kThreads), 0,
                       (hipStream_t)stream, (const unsigned long long*)sums, counts, (_Float16*)books_f16, d, S, K,
                       stage, n_elems);
    return launch_status();
}

extern "C" size_t fkv_kmeans_update_noalloc_bytes(int32_t n_books, int32_t K, int32_t d)
{
    if (n_books < 1 || K < 1 || d < 1) return 0;
    return (size_t)n_books * K * d * 8 + (size_t)n_books * K * 4;
}

extern "C" int fkv_kmeans_update_noalloc(const fkv_rvq_desc* desc, const uint16_t* x_f16, uint16_t* books_f16,
                                         const int32_t* stream_book, const uint8_t* symbols, int32_t stage,
                                         uint32_t* counts_out, void* stream)
{
    if (!desc) return FKV_ERR_INVALID_ARG;
    const fkv_rvq_desc& D = *desc;
    if (D.n_streams < 0 || D.T < 0 || D.t_begin < 0 || D.t_end < D.t_begin || D.t_end > D.T) return FKV_ERR_INVALID_ARG;
    if (D.d < 8 || D.d > 256 || D.d % 8 != 0 || D.S < 1 || D.S > 8 || D.K < 1 || D.K > 256 || D.n_books < 1)
        return FKV_ERR_INVALID_ARG;
    if (stage < 0 || stage >= D.S) return FKV_ERR_INVALID_ARG;
    if (!x_f16 || !books_f16 || !stream_book || !symbols) return FKV_ERR_INVALID_ARG;
    if (!aligned(x_f16, 16) || !aligned(books_f16, 16) || !aligned(stream_book, 4) ||
        (counts_out && !aligned(counts_out, 4)))
        return FKV_ERR_INVALID_ARG;
    const size_t need = fkv_kmeans_update_noalloc_bytes(D.n_books, D.K, D.d);
    if (need > (size_t)FKV_NOALLOC_SCRATCH_BYTES) return FKV_ERR_SCRATCH_TOO_SMALL;
    const int64_t Ta = D.t_end - D.t_begin;
    if (Ta * (std::min(kSlice, (int)D.d) / 8) > 0x7fffffff - kAccThreads * kAccBatch) return FKV_ERR_UNSUPPORTED;
    void* base = scratch_address();
    if (!base) return FKV_ERR_NO_DEVICE;
    const hipStream_t st = (hipStream_t)stream;
    unsigned long long* sums = (unsigned long long*)base;
    const int64_t n_sum = (int64_t)D.n_books * D.K * D.d;
    uint32_t* counts = (uint32_t*)(sums + n_sum);
    // the previous call's contents are cleared first: sums and counts start at zero
    const int64_t n_words = (int64_t)((need + 7) / 8);
    hipLaunchKernelGGL(zero_words_kernel, dim3((unsigned)grid_for(n_words)), dim3(kThreads), 0, st, sums, n_words);
    int rc = launch_status();
    if (rc != FKV_OK) return rc;
    if (D.n_streams > 0 && Ta > 0) {
        rc = fkv_kmeans_accumulate(desc, x_f16, books_f16, stream_book, symbols, stage, (int64_t*)sums, counts,
                                   stream);
        if (rc != FKV_OK) return rc;
    }
    rc = fkv_kmeans_finalize(D.n_books, D.S, D.K, D.d, stage, (const int64_t*)sums, counts, books_f16, stream);
    if (rc != FKV_OK) return rc;
    if (counts_out) {
        if (hipMemcpyAsync(counts_out, counts, (size_t)D.n_books * D.K * 4, hipMemcpyDeviceToDevice, st) != hipSuccess) {
            (void)hipGetLastError();
            return FKV_ERR_LAUNCH;
        }
    }
    return FKV_OK;
}
