/*
 * wsr_mma.hip - the batched decode sweep on the matrix cores: kernel and launcher.
 *
 *  k_sweep_mma   up to 16 tokens of the sweep per pass over the weights, one wave per workgroup,
 *                each wave taking the whole 64-row groups that start in its span of the stream
 */
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "wsr_mma.h"
#include "wsr_mma_launch.h"

namespace wsr {

constexpr int MMA_TAIL_TILES = 1;             /* 16-row tiles per row group in the tail of the stream */
constexpr int64_t SWEEP_SPAN_MMA = 64 << 10;  /* least bytes of the weight stream per wave             */

/* One wave per workgroup, so that a wave whose span holds no row group frees its slot at once.
   Waves w < w1 split the stream's bytes [0, tail) into equal spans of whole row groups of 16 NT
   rows; the others split [tail, total) into spans of 16-row groups.  The launcher sets a tail only
   where the main spans would leave the last round of wave slots at most a quarter full (the
   protocol pass: 2,304 groups of 64 rows on 2,048 slots); then the last waves to finish hold a
   quarter of a group's work.  A matrix's rows from the first main-group boundary at or after byte
   `tail` on belong to the tail, the rows before it to the main spans. */
template <int FMT, int NT>
__global__ __launch_bounds__(WAVE) __attribute__((amdgpu_waves_per_eu(FMT == FMT_Q4_WHOLE ? 2 : 1)))
void k_sweep_mma(const DevMat* __restrict__ tab, const int64_t* __restrict__ cost,
                                                    int nmat, int64_t total, int64_t tail, int64_t w1,
                                                    int32_t token0, int ntok) {
    const int lane = threadIdx.x;
    const int64_t w = blockIdx.x;
    const bool main = w < w1;
    const int64_t base = main ? 0 : tail, len = main ? tail : total - tail;
    const int64_t nw = main ? w1 : (int64_t)gridDim.x - w1, k = main ? w : w - w1;
    const int64_t q = len / nw, r = len % nw;
    const int64_t lo = base + q * k + (int64_t)((uint64_t)r * (uint64_t)k / nw);
    const int64_t hi = base + q * (k + 1) + (int64_t)((uint64_t)r * (uint64_t)(k + 1) / nw);
    int hint = 0;
    if (lo >= hi) return;
    /* the LDS ring: slots of 64 16-byte chunks (at four tiles q4 20 KiB, int8 8 KiB, 16-bit
       4 KiB; the kernel for mixed tables holds the largest); the tail's one-tile groups need no
       more */
    constexpr int F = mma_base_fmt(FMT);
    constexpr int RING = F == 0 ? mma_ring_slots<FMT_Q4, NT>() : mma_ring_slots<F, NT>();
    __shared__ u32x4 xlds[RING * WAVE];
    if (main)
        stream_range_mma<FMT, NT>(tab, cost, nmat, lo, hi, 0, 16 * NT, token0, ntok, lane, hint, xlds);
    else
        stream_range_mma<FMT, MMA_TAIL_TILES>(tab, cost, nmat, lo, hi, tail, 16 * NT, token0, ntok, lane, hint, xlds);
}

/* Tiles per row group.  Eight tiles (128 rows) halve the activation reads per weight byte but hold
   one wave per SIMD instead of two; measured in one process against four tiles, outputs bitwise
   equal: int8 protocol +8.6 % at 16 tokens, 0 at 8, -5 % at 4; 70B bf16 +1.2 to +1.3 % at 2 and
   16; 8B q4 -2.3 % at 16 and -4 % at 8 (506 registers).  q4 and the kernel for mixed tables (which
   spills at eight) stay at four, and so does any table with rows whose 128-row group would pass
   2^31 bytes (the matrix-core loops' 32-bit lane offsets). */
int mma_tiles(int fmt_all, int ntok, int64_t max_row_bytes) {
    const int f = mma_base_fmt(fmt_all);
    if (f == 0 || f == FMT_Q4 || max_row_bytes * 128 > (int64_t{1} << 31)) return 4;
    if (f == FMT_F16 || f == FMT_BF16) return 8;
    return ntok >= 12 ? 8 : 4;
}
int64_t mma_tail_rows() { return 16 * MMA_TAIL_TILES; }

template <int FMT>
static hipError_t occupancy_of(int tiles, int& per_cu) {
    if constexpr (FMT == 0 || mma_base_fmt(FMT) == FMT_Q4) {
        return hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_sweep_mma<0, 4>, WAVE, 0);
    } else {
        return tiles == 8 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_sweep_mma<FMT, 8>, WAVE, 0)
                          : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_sweep_mma<FMT, 4>, WAVE, 0);
    }
}

/* Wave slots of the device for the kernel of format fmt_all and its tile count (its occupancy
   times the CU count), found once per device, format and tile count. */
static hipError_t mma_slots(int fmt_all, int tiles, int64_t& slots) {
    static std::mutex mu;
    static int64_t cache[64][9][2] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const int f = (fmt_all >= 0 && fmt_all <= 4) || fmt_all == FMT_Q4_WHOLE ? fmt_all : 0;
    const int ti = tiles == 8 ? 1 : 0;
    std::lock_guard<std::mutex> lock(mu);
    if (dev >= 0 && dev < 64 && cache[dev][f][ti] > 0) {
        slots = cache[dev][f][ti];
        return hipSuccess;
    }
    int cus = 0, per_cu = 0;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    switch (f) {
        case FMT_F16: e = occupancy_of<FMT_F16>(tiles, per_cu); break;
        case FMT_BF16: e = occupancy_of<FMT_BF16>(tiles, per_cu); break;
        case FMT_Q4: e = occupancy_of<FMT_Q4>(4, per_cu); break;
        case FMT_I8: e = occupancy_of<FMT_I8>(tiles, per_cu); break;
        case FMT_Q4_WHOLE: e = occupancy_of<FMT_Q4_WHOLE>(4, per_cu); break;
        default: e = occupancy_of<0>(4, per_cu); break;
    }
    if (e != hipSuccess) return e;
    slots = (int64_t)cus * per_cu;
    if (dev >= 0 && dev < 64) cache[dev][f][ti] = slots;
    return hipSuccess;
}

hipError_t launch_sweep_mma(const DevMat* tab, const int64_t* cost, int nmat, int64_t total, int tiles,
                            int64_t max_group, int64_t max_tail_group, int fmt_all, int32_t token0, int ntok,
                            hipStream_t s) {
    if (nmat == 0 || total == 0) return hipSuccess;
    if (ntok < 1 || ntok > MMA_TOKENS) return hipErrorInvalidValue;
    if (tiles != 4 && tiles != 8) return hipErrorInvalidValue;
    if (mma_tiles(fmt_all, ntok, 0) == 4) tiles = 4;            /* formats held at four tiles */
    /* a wave's span holds at least the largest row group: a row group is never split, so a smaller
       span leaves most waves without one */
    const int64_t span = std::max(SWEEP_SPAN_MMA, max_group);
    const int64_t span_t = std::max(SWEEP_SPAN_MMA / 4, max_tail_group);
    const int64_t waves = (total + span - 1) / span;
    int64_t slots = 0;
    const hipError_t e = mma_slots(fmt_all, tiles, slots);
    if (e != hipSuccess) return e;
    /* whole rounds of spans, and a tail only where the last round would be at most a quarter full
       (measured on int8 passes: 1/8 full 323 -> 265 us per pass with the tail; 1/2 full 356 -> 381) */
    int64_t tail = total, w1 = waves, w2 = 0;
    const int64_t rounds = slots > 0 ? waves / slots : 0, rest = slots > 0 ? waves % slots : 0;
    if (rounds >= 1 && rounds < 8 && rest > 0 && 4 * rest <= slots) {
        tail = rounds * slots * span;
        w1 = rounds * slots;
        w2 = (total - tail + span_t - 1) / span_t;
    }
    if (w1 + w2 > INT32_MAX) return hipErrorInvalidValue;
#define WSR_MMA(F, NT)                                                                                             \
    hipLaunchKernelGGL((k_sweep_mma<F, NT>), dim3((unsigned)(w1 + w2)), dim3(WAVE), 0, s, tab, cost, nmat, total, \
                       tail, w1, token0, ntok)
#define WSR_MMA_T(F) \
    if (tiles == 8) WSR_MMA(F, 8); else WSR_MMA(F, 4)
    switch (fmt_all) {
        case FMT_F16: WSR_MMA_T(FMT_F16); break;
        case FMT_BF16: WSR_MMA_T(FMT_BF16); break;
        case FMT_Q4: WSR_MMA(FMT_Q4, 4); break;
        case FMT_I8: WSR_MMA_T(FMT_I8); break;
        case FMT_Q4_WHOLE: WSR_MMA(FMT_Q4_WHOLE, 4); break;
        default: WSR_MMA(0, 4); break;
    }
#undef WSR_MMA_T
#undef WSR_MMA
    return hipGetLastError();
}

}  // namespace wsr
