/*
 * wsr_copy.hip - the per-use copy of the staged sweep (Sec. 8.1's copy endpoint, Table 2's
 * pipelined double-buffered copy), read from pinned host pages across PCIe by the shaders.
 *
 * The copy engines moved the same pinned pages at 55 GB/s in some processes and at 29 GB/s in
 * others, while the shaders' own reads of those pages (the mapped arm) held 56 GB/s in every run;
 * a copy kernel takes that path.  It runs on the staged sweep's copy stream, so the ordering by
 * events is unchanged.
 */
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "wsr_copy.h"

namespace wsr {

typedef uint32_t c4_t __attribute__((ext_vector_type(4)));

constexpr int COPY_THREADS = 256;
constexpr int COPY_UNROLL = 4;                  /* 16-byte units in flight per thread            */
constexpr int64_t COPY_BLOCKS = 256;            /* one block per CU: 4 MiB in flight, the rest of
                                                   the chip free for the sweep's GEMV beside it  */

/* dst[i] = src[i] for i < n16 (16-byte units): each round a block moves COPY_UNROLL runs of 4 KiB,
   every wave 1 KiB of one run, loads first. */
__global__ __launch_bounds__(COPY_THREADS) void k_copy16(const c4_t* __restrict__ src, c4_t* __restrict__ dst,
                                                         int64_t n16) {
    const int64_t per_round = (int64_t)gridDim.x * COPY_THREADS * COPY_UNROLL;
    for (int64_t i = (int64_t)blockIdx.x * COPY_THREADS * COPY_UNROLL + threadIdx.x; i < n16; i += per_round) {
        c4_t v[COPY_UNROLL];
#pragma unroll
        for (int k = 0; k < COPY_UNROLL; ++k) {
            const int64_t j = i + (int64_t)k * COPY_THREADS;
            if (j < n16) v[k] = __builtin_nontemporal_load(src + j);
        }
#pragma unroll
        for (int k = 0; k < COPY_UNROLL; ++k) {
            const int64_t j = i + (int64_t)k * COPY_THREADS;
            if (j < n16) dst[j] = v[k];
        }
    }
}

hipError_t launch_copy16(const void* src, void* dst, size_t bytes, hipStream_t s) {
    if (bytes == 0) return hipSuccess;
    if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst) | bytes) & 15)
        return hipErrorInvalidValue;
    const int64_t n16 = (int64_t)(bytes / 16);
    const int64_t blocks = std::min<int64_t>(COPY_BLOCKS, (n16 + COPY_THREADS * COPY_UNROLL - 1) /
                                                              (COPY_THREADS * COPY_UNROLL));
    hipLaunchKernelGGL(k_copy16, dim3((unsigned)blocks), dim3(COPY_THREADS), 0, s,
                       static_cast<const c4_t*>(src), static_cast<c4_t*>(dst), n16);
    return hipGetLastError();
}

}  // namespace wsr
