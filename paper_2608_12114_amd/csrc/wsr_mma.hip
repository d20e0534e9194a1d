/*
 * wsr_mma.hip - the batched decode sweep on the matrix cores: kernel and launcher.
 *
 *  k_sweep_mma   up to 16 tokens of the sweep per pass over the weights, one wave per workgroup,
 *                each wave taking the whole 64-row groups that start in its span of the stream
 */
#include <hip/hip_runtime.h>

#include <algorithm>

#include "wsr_mma.h"

namespace wsr {

constexpr int MMA_TILES = 4;                  /* 16-row tiles per wave and row group (64 rows)     */
constexpr int64_t SWEEP_SPAN_MMA = 64 << 10;  /* least bytes of the weight stream per wave         */

/* One wave per workgroup, so that a wave whose span holds no row group frees its slot at once. */
template <int FMT>
__global__ __launch_bounds__(WAVE) void k_sweep_mma(const DevMat* __restrict__ tab, const int64_t* __restrict__ cost,
                                                    int nmat, int64_t total, int32_t token0, int ntok) {
    const int lane = threadIdx.x;
    const int64_t nw = gridDim.x, w = blockIdx.x;
    const int64_t q = total / nw, r = total % nw;
    const int64_t lo = q * w + (int64_t)((uint64_t)r * (uint64_t)w / nw);
    const int64_t hi = q * (w + 1) + (int64_t)((uint64_t)r * (uint64_t)(w + 1) / nw);
    int hint = 0;
    if (lo < hi) stream_range_mma<FMT, MMA_TILES>(tab, cost, nmat, lo, hi, token0, ntok, lane, hint);
}

int64_t mma_group_rows() { return 16 * MMA_TILES; }

hipError_t launch_sweep_mma(const DevMat* tab, const int64_t* cost, int nmat, int64_t total, int64_t max_group,
                            int fmt_all, int32_t token0, int ntok, hipStream_t s) {
    if (nmat == 0 || total == 0) return hipSuccess;
    if (ntok < 1 || ntok > MMA_TOKENS) return hipErrorInvalidValue;
    /* a wave's span holds at least the largest row group: a row group is never split, so a smaller
       span leaves most waves without one */
    const int64_t span = std::max(SWEEP_SPAN_MMA, max_group);
    const int64_t waves = (total + span - 1) / span;
    if (waves > INT32_MAX) return hipErrorInvalidValue;
#define WSR_MMA(F) \
    hipLaunchKernelGGL((k_sweep_mma<F>), dim3((unsigned)waves), dim3(WAVE), 0, s, tab, cost, nmat, total, token0, ntok)
    switch (fmt_all) {
        case FMT_F16: WSR_MMA(FMT_F16); break;
        case FMT_BF16: WSR_MMA(FMT_BF16); break;
        case FMT_Q4: WSR_MMA(FMT_Q4); break;
        case FMT_I8: WSR_MMA(FMT_I8); break;
        default: WSR_MMA(0); break;
    }
#undef WSR_MMA
    return hipGetLastError();
}

}  // namespace wsr
