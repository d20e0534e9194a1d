/*
 * wsr_kernels.hip - HIP kernels of the weight-streaming read path for gfx950 and their launchers.
 *
 *  k_probe_part / k_probe_final   pure-read reference: fp32 buffer -> fp64 sum (paper Sec. 3.1, 3.3)
 *  k_gemv16    single-token GEMV, fp16 / bf16 weights and activations, fp32 accumulate (Sec. 3.1)
 *  k_gemv_q4   single-token GEMV over 4-bit block-quantised weights, decoded in registers
 *  k_sweep     one decode token: every matrix of a table in one persistent launch (Sec. 6.2)
 *  k_put_table writes the sweep's matrix table into the caller's workspace from kernel arguments
 *              and clears the sweep's tile counters, so a sweep needs no host copy or host
 *              synchronisation (C3, Table 1)
 *
 * Streaming layout.  HBM3E serves long sequential runs best.  Each probe block walks its own
 * contiguous region.  The 16-bit sweep hands out tiles of the weight stream (64 KiB to 2 MiB) in
 * order from a counter, so the waves in flight work on one moving front of memory and finish
 * together.  The q4 sweep gives each wave an equal contiguous span instead, which measured faster
 * for its heavier per-byte work; its waves keep several steps of loads in flight in registers.
 */
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "wsr_device.h"

namespace wsr {

constexpr int BLOCK = 256;
constexpr int WAVES_PER_BLOCK = BLOCK / WAVE;

/* ======================================= probe ================================================ */

constexpr int PROBE_UNROLL = 4;            /* 16-byte loads in flight per thread               */
constexpr int PROBE_ACC = 4;               /* independent fp64 accumulators per thread          */
constexpr int64_t PROBE_MAX_GRID = 512;    /* two blocks per CU: few, long sequential streams   */

int64_t probe_grid(int64_t n) {
    const int64_t n4 = n / 4;
    const int64_t per_block = (int64_t)BLOCK * PROBE_UNROLL * 4;
    const int64_t g = (n4 + per_block - 1) / per_block;
    return std::max<int64_t>(1, std::min(g, PROBE_MAX_GRID));
}

/* Elements are reinterpreted through __uint_as_float: applying __builtin_bit_cast to an element of
   an ext_vector_type value makes this compiler read element 0 for every component. */
__device__ __forceinline__ double sum4(u32x4 v, double acc) {
    acc += (double)__uint_as_float(v.x);
    acc += (double)__uint_as_float(v.y);
    acc += (double)__uint_as_float(v.z);
    acc += (double)__uint_as_float(v.w);
    return acc;
}

/* Sum over a block's threads, in a fixed order: valid in thread 0. */
__device__ __forceinline__ double block_sum(double v, double* red) {
    v = wave_sum(v);
    if ((threadIdx.x & (WAVE - 1)) == 0) red[threadIdx.x / WAVE] = v;
    __syncthreads();
    double s = 0.0;
    if (threadIdx.x == 0)
        for (int i = 0; i < WAVES_PER_BLOCK; ++i) s += red[i];
    return s;
}

/* Block b sums 16-byte groups [b * chunk, (b + 1) * chunk): per step its 256 threads read 16 KiB of
   consecutive memory, thread t taking groups t, t + 256, t + 512, t + 768 into accumulators 0..3. */
__global__ __launch_bounds__(BLOCK) void k_probe_part(const u32x4* __restrict__ buf, int64_t n4,
                                                      double* __restrict__ part) {
    __shared__ double red[WAVES_PER_BLOCK];
    g_u32x4* b = as_global<g_u32x4*>(buf);
    const int64_t chunk = (n4 + gridDim.x - 1) / gridDim.x;
    const int64_t beg = (int64_t)blockIdx.x * chunk;
    const int64_t end = std::min<int64_t>(n4, beg + chunk);
    double acc[PROBE_ACC];
#pragma unroll
    for (int a = 0; a < PROBE_ACC; ++a) acc[a] = 0.0;
    int64_t i = beg + threadIdx.x;
    for (; i + (PROBE_UNROLL - 1) * BLOCK < end; i += PROBE_UNROLL * BLOCK) {
        u32x4 v[PROBE_UNROLL];
#pragma unroll
        for (int j = 0; j < PROBE_UNROLL; ++j) v[j] = load_once(b + i + j * BLOCK);
#pragma unroll
        for (int j = 0; j < PROBE_UNROLL; ++j) acc[j % PROBE_ACC] = sum4(v[j], acc[j % PROBE_ACC]);
    }
    for (; i < end; i += BLOCK) acc[0] = sum4(load_once(b + i), acc[0]);
    double t = 0.0;
#pragma unroll
    for (int a = 0; a < PROBE_ACC; ++a) t += acc[a];
    t = block_sum(t, red);
    if (threadIdx.x == 0) part[blockIdx.x] = t;
}

/* One block: the partials in index order, then the n % 4 trailing elements. */
__global__ __launch_bounds__(BLOCK) void k_probe_final(const double* __restrict__ part, int G,
                                                       const float* __restrict__ tail, int ntail,
                                                       double* __restrict__ out) {
    __shared__ double red[WAVES_PER_BLOCK];
    double a = 0.0;
    for (int j = threadIdx.x; j < G; j += BLOCK) a += part[j];
    double s = block_sum(a, red);
    if (threadIdx.x == 0) {
        for (int j = 0; j < ntail; ++j) s += (double)tail[j];
        *out = s;
    }
}

hipError_t launch_probe(const float* buf, int64_t n, double* sum_dev, void* ws, hipStream_t s) {
    const int64_t g = probe_grid(n);
    const int64_t n4 = n / 4;
    double* part = static_cast<double*>(ws);
    hipLaunchKernelGGL(k_probe_part, dim3((unsigned)g), dim3(BLOCK), 0, s,
                       reinterpret_cast<const u32x4*>(buf), n4, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_probe_final, dim3(1), dim3(BLOCK), 0, s, part, (int)g, buf + 4 * n4,
                       (int)(n % 4), sum_dev);
    return hipGetLastError();
}

/* ======================================= GEMVs ================================================ */

/* One wave per R consecutive rows. */
template <int FMT, int R, int U>
__global__ __launch_bounds__(BLOCK) void k_gemv16(DevMat d) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int64_t wave = (int64_t)blockIdx.x * WAVES_PER_BLOCK + wave_in_block();
    const int64_t r0 = wave * R;
    if (r0 >= d.M) return;
    rows16<FMT, R, U>(d, r0, std::min<int64_t>(r0 + R, d.M), 0, lane);
}

template <int R, int U>
__global__ __launch_bounds__(BLOCK) void k_gemv_q4(DevMat d) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int64_t wave = (int64_t)blockIdx.x * WAVES_PER_BLOCK + wave_in_block();
    const int64_t r0 = wave * R;
    if (r0 >= d.M) return;
    rows_q4<R, U>(d, r0, std::min<int64_t>(r0 + R, d.M), 0, lane);
}

template <typename K>
static hipError_t launch_rows(K kernel, const DevMat& m, int R, hipStream_t s) {
    const int64_t waves = (m.M + R - 1) / R;
    const int64_t blocks = (waves + WAVES_PER_BLOCK - 1) / WAVES_PER_BLOCK;
    hipLaunchKernelGGL(kernel, dim3((unsigned)blocks), dim3(BLOCK), 0, s, m);
    return hipGetLastError();
}

/* T activation columns per weight read (x_stride / y_stride of d are the column strides). */
template <int FMT, int T>
__global__ __launch_bounds__(BLOCK) void k_gemv16_cols(DevMat d) {
    constexpr int R = Cols16<T>::R;
    const int lane = threadIdx.x & (WAVE - 1);
    const int64_t wave = (int64_t)blockIdx.x * WAVES_PER_BLOCK + wave_in_block();
    const int64_t r0 = wave * R;
    if (r0 >= d.M) return;
    rows16_cols<FMT, T>(d, r0, std::min<int64_t>(r0 + R, d.M), 0, lane);
}

template <int FMT>
static hipError_t launch_gemv16_cols(const DevMat& m, int T, hipStream_t s) {
    switch (T) {
        case 1: return launch_rows(k_gemv16_cols<FMT, 1>, m, Cols16<1>::R, s);
        case 2: return launch_rows(k_gemv16_cols<FMT, 2>, m, Cols16<2>::R, s);
        case 4: return launch_rows(k_gemv16_cols<FMT, 4>, m, Cols16<4>::R, s);
        case 8: return launch_rows(k_gemv16_cols<FMT, 8>, m, Cols16<8>::R, s);
        case 16: return launch_rows(k_gemv16_cols<FMT, 16>, m, Cols16<16>::R, s);
        default: return hipErrorInvalidValue;
    }
}

template <int T>
__global__ __launch_bounds__(BLOCK) void k_gemv_q4_cols(DevMat d) {
    constexpr int R = Cols4<T>::R;
    const int lane = threadIdx.x & (WAVE - 1);
    const int64_t wave = (int64_t)blockIdx.x * WAVES_PER_BLOCK + wave_in_block();
    const int64_t r0 = wave * R;
    if (r0 >= d.M) return;
    rows_q4_cols<T>(d, r0, std::min<int64_t>(r0 + R, d.M), 0, lane);
}

/* One group of R rows per wave.  The full and the partial group take separate branches rather than
   a clamp of the row end: the clamp's select was miscompiled (the pre-emit peephole dropped the
   instruction that set the select's condition, so the end became r0 + R past the last row). */
template <int T>
__global__ __launch_bounds__(BLOCK) void k_gemv_i8(DevMat d) {
    constexpr int R = GemvI8<T>::R;
    const int lane = threadIdx.x & (WAVE - 1);
    const int64_t wave = (int64_t)blockIdx.x * WAVES_PER_BLOCK + wave_in_block();
    const int64_t r0 = wave * R;
    if (r0 >= d.M) return;
    if (d.M - r0 >= R) rows_i8<T, R, GemvI8<T>::U>(d, r0, r0 + R, 0, lane);
    else rows_i8<T, 1, GemvI8<T>::U>(d, r0, d.M, 0, lane);
}

static hipError_t launch_gemv_i8(const DevMat& m, int T, hipStream_t s) {
    switch (T) {
        case 1: return launch_rows(k_gemv_i8<1>, m, GemvI8<1>::R, s);
        case 2: return launch_rows(k_gemv_i8<2>, m, GemvI8<2>::R, s);
        case 4: return launch_rows(k_gemv_i8<4>, m, GemvI8<4>::R, s);
        case 8: return launch_rows(k_gemv_i8<8>, m, GemvI8<8>::R, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_gemv_cols(const DevMat& m, int T, hipStream_t s) {
    if (m.M == 0) return hipSuccess;
    if (m.fmt == FMT_F16) return launch_gemv16_cols<FMT_F16>(m, T, s);
    if (m.fmt == FMT_BF16) return launch_gemv16_cols<FMT_BF16>(m, T, s);
    if (m.fmt == FMT_I8) return launch_gemv_i8(m, T, s);
    if (m.fmt == FMT_Q4) {
        switch (T) {
            case 1: return launch_rows(k_gemv_q4_cols<1>, m, Cols4<1>::R, s);
            case 2: return launch_rows(k_gemv_q4_cols<2>, m, Cols4<2>::R, s);
            case 4: return launch_rows(k_gemv_q4_cols<4>, m, Cols4<4>::R, s);
            case 8: return launch_rows(k_gemv_q4_cols<8>, m, Cols4<8>::R, s);
            default: return hipErrorInvalidValue;
        }
    }
    return hipErrorInvalidValue;
}

/* Rows of 128 KiB or more (K >= 65536 at 16 bits) go four to a wave when that still leaves a wave
   per SIMD: with one row per wave each row rereads the whole activation vector from L2, as many
   bytes as its weights.  Measured on 4096 rows: K = 65536 5.87 -> 6.47 TB/s, K = 140800 6.13 ->
   6.76 TB/s; at K <= 32768 four rows per wave were slower (the 1,024 waves cannot cover the
   latency), so shorter rows keep one per wave. */
static bool gemv16_long_rows(const DevMat& m) { return m.nc >= 8192 && m.M >= 4 * 1024; }

hipError_t launch_gemv(const DevMat& m, hipStream_t s) {
    if (m.M == 0) return hipSuccess;
    switch (m.fmt) {
        case FMT_F16:
            return gemv16_long_rows(m) ? launch_rows(k_gemv16<FMT_F16, 4, 8>, m, 4, s)
                                       : launch_rows(k_gemv16<FMT_F16, 1, 8>, m, 1, s);
        case FMT_BF16:
            return gemv16_long_rows(m) ? launch_rows(k_gemv16<FMT_BF16, 4, 8>, m, 4, s)
                                       : launch_rows(k_gemv16<FMT_BF16, 1, 8>, m, 1, s);
        case FMT_Q4:
            return m.nc >= 256 ? launch_rows(k_gemv_q4<2, 2>, m, 2, s)
                               : launch_rows(k_gemv_q4<4, 1>, m, 4, s);
        case FMT_I8:
            return launch_gemv_i8(m, 1, s);
        default:
            return hipErrorInvalidValue;
    }
}

/* ======================================= sweep ================================================ */

/* Matrices per table-upload launch.  The chunk travels as a by-value kernel argument (30.7 KB at
   320 entries; arguments of up to 32,000 bytes were checked to arrive intact on this stack), so one
   launch uploads the table of a 225-matrix model and the arguments are captured by value when a
   caller records the sweep into a graph. */
constexpr int TABLE_CHUNK = 320;
struct TableChunk {
    int32_t n;
    int32_t pad_[3];
    DevMat m[TABLE_CHUNK];
};
static_assert(sizeof(TableChunk) <= 31 * 1024, "table chunk must stay within the checked argument size");

__global__ __launch_bounds__(BLOCK) void k_put_table(DevMat* __restrict__ dst, int64_t* __restrict__ cost,
                                                     TableChunk c, unsigned* __restrict__ ctr) {
    for (int i = threadIdx.x; i < c.n; i += BLOCK) {
        dst[i] = c.m[i];
        cost[i] = c.m[i].cost0;
    }
    if (ctr && threadIdx.x < 2) ctr[threadIdx.x] = 0u;
}

hipError_t launch_put_table(DevMat* dst, int64_t* cost, const DevMat* src, int n, unsigned* ctr,
                            hipStream_t s) {
    for (int first = 0; first < n; first += TABLE_CHUNK) {
        TableChunk c{};
        c.n = std::min(TABLE_CHUNK, n - first);
        for (int i = 0; i < c.n; ++i) c.m[i] = src[first + i];
        hipLaunchKernelGGL(k_put_table, dim3(1), dim3(BLOCK), 0, s, dst + first, cost + first, c,
                           first == 0 ? ctr : nullptr);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

enum : int { SCHED_TILES = 0, SCHED_SPANS = 1, SCHED_HYBRID = 2 };

/* Tile size: about four tiles per wave, a power of two between 64 KiB and 2 MiB. */
int64_t sweep_tile(int64_t total, int64_t waves) {
    int64_t t = 64 << 10;
    while (t < (2 << 20) && t * waves * 4 < total) t <<= 1;
    return t;
}

/* The wave's index in the order of spans.  The hardware hands consecutive blocks to the 8 XCDs in
   turn, each with its own L2, so numbering spans by block index would have every XCD work on every
   part of the stream at once.  Block b, on XCD b % 8, instead takes place b / 8 among that XCD's
   blocks inside the XCD's own eighth of the spans: each L2 then holds one contiguous part of the
   stream, so the activations of a matrix are fetched into fewer L2s and the output lines that
   neighbouring waves share are written through one L2 (8B q4 token: 619 -> 612 us). */
constexpr unsigned XCDS = 8;
__device__ __forceinline__ int64_t span_wave() {
    const unsigned nb = gridDim.x, b = blockIdx.x, xcd = b % XCDS, per = nb / XCDS, rem = nb % XCDS;
    const unsigned place = xcd * per + (xcd < rem ? xcd : rem) + b / XCDS;
    return (int64_t)place * WAVES_PER_BLOCK + wave_in_block();
}

/* Wave w takes bytes [w span, (w + 1) span) of the stream, cut at its end; the launcher sets span to
   ceil(total / waves), so no division runs on the device. */
__device__ __forceinline__ void span_bounds(int64_t total, int64_t w, int64_t span, int64_t& lo, int64_t& hi) {
    lo = w * span;
    hi = std::min<int64_t>(total, lo + span);
}

/* Work distribution over the weight stream [0, total) of one token:
     SCHED_TILES   tiles of `tile` bytes, claimed in order from a counter;
     SCHED_SPANS   wave w takes [span w, span (w + 1)) (span = ceil(total / nw)); with many more blocks than the
                   chip holds at once, the hardware starts each block as an earlier one retires,
                   which balances the end of the token at no cost;
     SCHED_HYBRID  wave w first takes [span w, span (w + 1)), then the rest [span nw, total) goes out
                   in claimed tiles, so long uninterrupted runs carry most of the stream and the
                   waves that finish early share the remainder.
   The counters ctr[0] (next tile) and ctr[1] (waves done) start at zero and the last wave to
   finish puts them back to zero for the next launch. */
template <int FMT, int SCHED, int R16, int U16, int RQ, int UQ, int QNB = 2, int T = 1, int RC = Cols16<T>::R,
          int UC = Cols16<T>::U, int RQC = Cols4<(T <= 8 ? T : 8)>::R>
__global__ __launch_bounds__(BLOCK) void k_sweep(const DevMat* __restrict__ tab, const int64_t* __restrict__ cost,
                                                 int nmat, int64_t total, int64_t span, int64_t tile,
                                                 int32_t token, unsigned* __restrict__ ctr) {
    const int lane = threadIdx.x & (WAVE - 1);
    const unsigned nw = gridDim.x * WAVES_PER_BLOCK;
    const int64_t w = (int64_t)blockIdx.x * WAVES_PER_BLOCK + wave_in_block();
    int hint = 0;
    if constexpr (SCHED == SCHED_SPANS) {
        int64_t lo, hi;
        span_bounds(total, span_wave(), span, lo, hi);
        if (lo < hi) stream_range<FMT, R16, U16, RQ, UQ, QNB, T, RC, UC, RQC>(tab, cost, nmat, lo, hi, token, lane, hint);
    } else {
        int64_t base = 0;
        if constexpr (SCHED == SCHED_HYBRID) {
            base = span * nw;
            if (span > 0) stream_range<FMT, R16, U16, RQ, UQ, QNB, T, RC, UC, RQC>(tab, cost, nmat, span * w, span * (w + 1),
                                                                   token, lane, hint);
        }
        /* Each wave claims its next tile before working on the current one, so the round trip of
           the claim overlaps the current tile's loads. */
        const int64_t ntiles = ceil_div(total - base, tile);
        unsigned claim = 0;
        if (lane == 0) claim = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        for (;;) {
            const unsigned t = __builtin_amdgcn_readfirstlane(claim);
            if ((int64_t)t >= ntiles) break;
            if (lane == 0) claim = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            const int64_t lo = base + (int64_t)t * tile;
            stream_range<FMT, R16, U16, RQ, UQ, QNB, T, RC, UC, RQC>(tab, cost, nmat, lo, std::min<int64_t>(total, lo + tile),
                                                     token, lane, hint);
        }
        if (lane == 0) {
            const unsigned e = __hip_atomic_fetch_add(ctr + 1, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
            if (e == nw - 1) {
                __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(ctr + 1, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    }
}

/* A table of up to N matrices carried by value in the arguments of a span-scheduled sweep launch.
   The waves read their matrix records and stream offsets straight from the argument memory through
   the scalar cache, so such a sweep needs neither a workspace nor the table upload launch before
   it, whose kernel boundary measured about 4 us per call against a 1 GB pass of about 150 us.  Two
   sizes: 32 entries (3.3 KB, about 1 us per launch cheaper than the large block on a 32-matrix
   pass) and TABLE_ARG_MAX (29,952 bytes; arguments of up to 32,000 bytes were checked to arrive
   intact). */
constexpr int TABLE_ARG_SMALL = 32, TABLE_ARG_MAX = 288;
template <int N>
struct TableArg {
    DevMat m[N];
    int64_t cost[N];
};
static_assert(sizeof(TableArg<TABLE_ARG_MAX>) + 32 <= 32000, "the by-value table must stay within the checked argument size");

template <int FMT, int R16, int U16, int T, int N>
__global__ __launch_bounds__(BLOCK) void k_sweep_arg(TableArg<N> tb, int nmat, int64_t total, int64_t span,
                                                     int32_t token) {
    const int lane = threadIdx.x & (WAVE - 1);
    int hint = 0;
    int64_t lo, hi;
    span_bounds(total, span_wave(), span, lo, hi);
    if (lo < hi) stream_range<FMT, R16, U16, 8, 1, 2, T>(tb.m, tb.cost, nmat, lo, hi, token, lane, hint);
}

static int cu_count() {
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (cache[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        cache[dev] = n;
    }
    return cache[dev];
}

/* 16-bit weights: tiles, 4 rows x 4 KiB steps per wave, one block (4 waves) per CU (few, long
   streams).  q4: spans of about 48 KiB per wave, 8 rows x 1 block per lane per step (eight rows
   share each block's activation decode), two register sets in flight; the grid is sized so that
   blocks retire and are replaced throughout the token (21,500 blocks for 4.2 GB).  int8: spans of
   about SWEEP_SPAN_I8[T] bytes per wave with 8 rows x 1 chunk per lane per step and, for one
   column, three register sets in flight; tiles with one block per CU reach about half the rate
   (one wave per SIMD cannot cover the latency at each row group's start). */
constexpr int SWEEP_BLOCKS_PER_CU_16 = 1;
constexpr int64_t SWEEP_SPAN_Q4 = 48 << 10;
/* 16-bit streams shorter than four tiles of the largest size per wave (8 GiB with 1024 waves) go
   over spans of about 48 KiB per wave, two rows x 8 KiB steps, instead of claimed tiles: with few
   tiles per wave the end of the launch is uneven (the 1 GiB pass of 32 matrices of 4096 x 4096 fp16
   measured 4.47 TB/s over tiles and 6.8 TB/s over spans), while on long streams tiles keep the
   waves on one moving front (the 70B bf16 token measured 7.22 TB/s over tiles, 7.10 over spans). */
constexpr int64_t SWEEP_SPAN_16 = 48 << 10;
constexpr int64_t SWEEP16_TILES_FROM = int64_t{8} << 30;
constexpr int SPAN16_R = 2, SPAN16_U = 8;
constexpr int64_t SWEEP_SPAN_I8[4] = {32 << 10, 32 << 10, 128 << 10, 128 << 10};   /* T = 1, 2, 4, 8 */

/* Grid of a span-scheduled sweep: about `target` bytes per wave, at least one wave per SIMD; *span
   receives the bytes per wave, ceil(total / waves). */
static hipError_t span_grid(int64_t total, int64_t target, dim3& g, int64_t* span) {
    const int64_t waves = std::max<int64_t>((int64_t)cu_count() * WAVES_PER_BLOCK, (total + target - 1) / target);
    const int64_t blocks = (waves + WAVES_PER_BLOCK - 1) / WAVES_PER_BLOCK;
    if (blocks > INT32_MAX) return hipErrorInvalidValue;
    g = dim3((unsigned)blocks);
    const int64_t nw = blocks * WAVES_PER_BLOCK;
    *span = (total + nw - 1) / nw;
    return hipSuccess;
}

template <int N>
static void fill_table_arg(TableArg<N>& tb, const DevMat* htab, int nmat) {
    for (int i = 0; i < nmat; ++i) {
        tb.m[i] = htab[i];
        tb.cost[i] = htab[i].cost0;
    }
}

/* One span-scheduled launch: the table by value when the host table is given (nmat <= TABLE_ARG_MAX),
   else from the device table. */
template <int FMT, int T>
static void launch_sweep_spans(dim3 g, int64_t span, hipStream_t s, const DevMat* tab, const int64_t* cost,
                               const DevMat* htab, int nmat, int64_t total, int32_t token) {
    constexpr int R = (FMT == FMT_F16 || FMT == FMT_BF16) ? SPAN16_R : 4;
    constexpr int U = (FMT == FMT_F16 || FMT == FMT_BF16) ? SPAN16_U : 4;
    if (htab && nmat <= TABLE_ARG_SMALL) {
        TableArg<TABLE_ARG_SMALL> tb;
        fill_table_arg(tb, htab, nmat);
        hipLaunchKernelGGL((k_sweep_arg<FMT, R, U, T, TABLE_ARG_SMALL>), g, dim3(BLOCK), 0, s, tb, nmat, total, span,
                           token);
    } else if (htab) {
        TableArg<TABLE_ARG_MAX> tb;
        fill_table_arg(tb, htab, nmat);
        hipLaunchKernelGGL((k_sweep_arg<FMT, R, U, T, TABLE_ARG_MAX>), g, dim3(BLOCK), 0, s, tb, nmat, total, span,
                           token);
    } else {
        hipLaunchKernelGGL((k_sweep<FMT, SCHED_SPANS, R, U, 8, 1, 2, T>), g, dim3(BLOCK), 0, s, tab, cost, nmat,
                           total, span, (int64_t)0, token, nullptr);
    }
}

/* q4 and int8 sweeps (T <= 8) over spans. */
template <int FMT>
static hipError_t launch_sweep_quant(int T, hipStream_t s, const DevMat* tab, const int64_t* cost, const DevMat* htab,
                                     int nmat, int64_t total, int32_t token) {
    const int ti = T == 1 ? 0 : T == 2 ? 1 : T == 4 ? 2 : 3;
    dim3 g;
    int64_t span = 0;
    const hipError_t e = span_grid(total, FMT == FMT_Q4 ? SWEEP_SPAN_Q4 : SWEEP_SPAN_I8[ti], g, &span);
    if (e != hipSuccess) return e;
    switch (T) {
        case 1: launch_sweep_spans<FMT, 1>(g, span, s, tab, cost, htab, nmat, total, token); break;
        case 2: launch_sweep_spans<FMT, 2>(g, span, s, tab, cost, htab, nmat, total, token); break;
        case 4: launch_sweep_spans<FMT, 4>(g, span, s, tab, cost, htab, nmat, total, token); break;
        case 8: launch_sweep_spans<FMT, 8>(g, span, s, tab, cost, htab, nmat, total, token); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

/* Which launches run over spans (those may take their table by value). */
static bool sweep_spans(int64_t total, int fmt_all, int T) {
    return fmt_all == FMT_Q4 || fmt_all == FMT_I8 ||
           ((fmt_all == FMT_F16 || fmt_all == FMT_BF16) && T == 1 && total < SWEEP16_TILES_FROM);
}

bool sweep_table_by_value(int nmat, int64_t total, int fmt_all, int T) {
    return nmat <= TABLE_ARG_MAX && sweep_spans(total, fmt_all, T);
}

/* 16-bit (or mixed-format) sweep over tiles, tokens token .. token + T - 1 per weight pass. */
template <int FMT, int T>
static void launch_sweep_tiles(dim3 grid, hipStream_t s, const DevMat* tab, const int64_t* cost, int nmat,
                               int64_t total, int64_t tile, int32_t token, unsigned* ctr) {
    hipLaunchKernelGGL((k_sweep<FMT, SCHED_TILES, 4, 4, 8, 1, 2, T>), grid, dim3(BLOCK), 0, s, tab, cost, nmat,
                       total, (int64_t)0, tile, token, ctr);
}

template <int FMT>
static hipError_t launch_sweep_cols(dim3 grid, int T, hipStream_t s, const DevMat* tab, const int64_t* cost,
                                    int nmat, int64_t total, int64_t tile, int32_t token, unsigned* ctr) {
    switch (T) {
        case 1: launch_sweep_tiles<FMT, 1>(grid, s, tab, cost, nmat, total, tile, token, ctr); break;
        case 2: launch_sweep_tiles<FMT, 2>(grid, s, tab, cost, nmat, total, tile, token, ctr); break;
        case 4: launch_sweep_tiles<FMT, 4>(grid, s, tab, cost, nmat, total, tile, token, ctr); break;
        case 8: launch_sweep_tiles<FMT, 8>(grid, s, tab, cost, nmat, total, tile, token, ctr); break;
        case 16: launch_sweep_tiles<FMT, 16>(grid, s, tab, cost, nmat, total, tile, token, ctr); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_sweep(const DevMat* tab, const int64_t* cost, const DevMat* htab, int nmat, int64_t total,
                        int fmt_all, int32_t token, int T, unsigned* ctr, hipStream_t s) {
    if (nmat == 0 || total == 0) return hipSuccess;
    if (!sweep_table_by_value(nmat, total, fmt_all, T)) htab = nullptr;
    if (fmt_all == FMT_Q4) return launch_sweep_quant<FMT_Q4>(T, s, tab, cost, htab, nmat, total, token);
    if (fmt_all == FMT_I8) return launch_sweep_quant<FMT_I8>(T, s, tab, cost, htab, nmat, total, token);
    if (sweep_spans(total, fmt_all, T)) {
        dim3 g;
        int64_t span = 0;
        const hipError_t e = span_grid(total, SWEEP_SPAN_16, g, &span);
        if (e != hipSuccess) return e;
        if (fmt_all == FMT_F16) launch_sweep_spans<FMT_F16, 1>(g, span, s, tab, cost, htab, nmat, total, token);
        else launch_sweep_spans<FMT_BF16, 1>(g, span, s, tab, cost, htab, nmat, total, token);
        return hipGetLastError();
    }
    const dim3 grid((unsigned)(cu_count() * SWEEP_BLOCKS_PER_CU_16));
    const int64_t tile = sweep_tile(total, (int64_t)grid.x * WAVES_PER_BLOCK);
    switch (fmt_all) {
        case FMT_F16: return launch_sweep_cols<FMT_F16>(grid, T, s, tab, cost, nmat, total, tile, token, ctr);
        case FMT_BF16: return launch_sweep_cols<FMT_BF16>(grid, T, s, tab, cost, nmat, total, tile, token, ctr);
        default:   /* mixed formats; a table holding q4 or int8 comes with T <= 8 */
            return launch_sweep_cols<0>(grid, T, s, tab, cost, nmat, total, tile, token, ctr);
    }
}

/* ================================ allocation-free sweep scratch ================================ */

/* Each device holds its own copy of this array, at its own address, from the time the library's
   code is loaded on that device until the process ends.  Host code never passes the array's name
   to a kernel or a copy: that name is a host-side stand-in, not a device address.  It uses the
   address hipGetSymbolAddress reports for the current device, looked up once per device. */
static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

hipError_t noalloc_scratch(void** ptr) {
    static std::mutex mu;
    static void* addr[64] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

}  // namespace wsr
