/*
 * wsr_kernels.hip - HIP kernels of the weight-streaming read path for gfx950 and their launchers.
 *
 *  k_probe     pure-read reference: fp32 buffer -> fp64 sum (Sec. 3.1, 3.3 of the paper)
 *  k_gemv16    single-token GEMV, fp16 / bf16 weights and activations, fp32 accumulate (Sec. 3.1)
 *  k_gemv_q4   single-token GEMV over 4-bit block-quantised weights, decoded in registers
 *  k_sweep     one decode token: every matrix of the model in one persistent launch (Sec. 6.2)
 *  k_put_table writes the sweep's matrix table into the caller's workspace from kernel arguments,
 *              so a sweep needs no host-side copy or synchronisation (C3, Table 1)
 */
#include <hip/hip_runtime.h>

#include <algorithm>

#include "wsr_device.h"

namespace wsr {

/* ======================================= probe ================================================ */

constexpr int PROBE_BLOCK = 256;
constexpr int PROBE_UNROLL = 8;
constexpr int64_t PROBE_MAX_GRID = 2048;   /* 8 blocks per CU on a 256-CU part */
constexpr int64_t PROBE_PART_OFFSET = 64;  /* ws: [ticket | pad to 64 B][fp64 partial per block] */

int64_t probe_grid(int64_t n) {
    const int64_t n4 = n / 4;
    const int64_t per_block = (int64_t)PROBE_BLOCK * PROBE_UNROLL;
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

/* Sum of a block's values in thread order of waves: valid in thread 0. */
__device__ __forceinline__ double block_sum(double v, double* red) {
    v = wave_sum(v);
    const int w = threadIdx.x / WAVE;
    if ((threadIdx.x & (WAVE - 1)) == 0) red[w] = v;
    __syncthreads();
    double s = 0.0;
    if (threadIdx.x == 0)
        for (int i = 0; i < PROBE_BLOCK / WAVE; ++i) s += red[i];
    return s;
}

/* Grid-stride over 16-byte groups: thread t of block b reads groups b*256 + t + j*stride.  Each
   block publishes one fp64 partial; the last block to take a ticket adds the partials in index order
   (plus the n % 4 tail) and resets the ticket for the next call. */
__global__ __launch_bounds__(PROBE_BLOCK) void k_probe(const u32x4* __restrict__ buf, int64_t n4,
                                                       int ntail, double* __restrict__ part,
                                                       unsigned* __restrict__ ticket,
                                                       double* __restrict__ out) {
    __shared__ double red[PROBE_BLOCK / WAVE];
    __shared__ int last;
    const int64_t stride = (int64_t)gridDim.x * PROBE_BLOCK;
    int64_t i = (int64_t)blockIdx.x * PROBE_BLOCK + threadIdx.x;
    double acc = 0.0;
    for (; i + (PROBE_UNROLL - 1) * stride < n4; i += PROBE_UNROLL * stride) {
        u32x4 v[PROBE_UNROLL];
#pragma unroll
        for (int j = 0; j < PROBE_UNROLL; ++j) v[j] = load_once(buf + i + j * stride);
#pragma unroll
        for (int j = 0; j < PROBE_UNROLL; ++j) acc = sum4(v[j], acc);
    }
    for (; i < n4; i += stride) acc = sum4(load_once(buf + i), acc);

    const double b = block_sum(acc, red);
    if (threadIdx.x == 0) {
        __hip_atomic_store(part + blockIdx.x, b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __threadfence();
        const unsigned t = __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        last = (t == gridDim.x - 1);
    }
    __syncthreads();
    if (!last) return;
    __threadfence();
    double a = 0.0;
    for (int64_t j = threadIdx.x; j < (int64_t)gridDim.x; j += PROBE_BLOCK)
        a += __hip_atomic_load(part + j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();  /* red[] is reused */
    double s = block_sum(a, red);
    if (threadIdx.x == 0) {
        const float* tail = reinterpret_cast<const float*>(buf + n4);
        for (int j = 0; j < ntail; ++j) s += (double)tail[j];
        *out = s;
        __hip_atomic_store(ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

hipError_t launch_probe(const float* buf, int64_t n, double* sum_dev, void* ws, hipStream_t s) {
    const int64_t g = probe_grid(n);
    unsigned* ticket = static_cast<unsigned*>(ws);
    double* part = reinterpret_cast<double*>(static_cast<char*>(ws) + PROBE_PART_OFFSET);
    hipLaunchKernelGGL(k_probe, dim3((unsigned)g), dim3(PROBE_BLOCK), 0, s,
                       reinterpret_cast<const u32x4*>(buf), n / 4, (int)(n % 4), part, ticket, sum_dev);
    return hipGetLastError();
}

/* ======================================= GEMVs ================================================ */

constexpr int BLOCK = 256;
constexpr int WAVES_PER_BLOCK = BLOCK / WAVE;

/* One wave per R consecutive rows. */
template <int FMT, int R, int U>
__global__ __launch_bounds__(BLOCK) void k_gemv16(DevMat d) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int64_t wave = (int64_t)blockIdx.x * WAVES_PER_BLOCK + threadIdx.x / WAVE;
    const int64_t r0 = wave * R;
    if (r0 >= d.M) return;
    rows16<FMT, R, U>(d, r0, std::min<int64_t>(r0 + R, d.M), 0, lane);
}

template <int R, int U>
__global__ __launch_bounds__(BLOCK) void k_gemv_q4(DevMat d) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int64_t wave = (int64_t)blockIdx.x * WAVES_PER_BLOCK + threadIdx.x / WAVE;
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

hipError_t launch_gemv(const DevMat& m, hipStream_t s) {
    if (m.M == 0) return hipSuccess;
    switch (m.fmt) {
        case FMT_F16:
            return m.M >= 8192 ? launch_rows(k_gemv16<FMT_F16, 2, 8>, m, 2, s)
                               : launch_rows(k_gemv16<FMT_F16, 1, 8>, m, 1, s);
        case FMT_BF16:
            return m.M >= 8192 ? launch_rows(k_gemv16<FMT_BF16, 2, 8>, m, 2, s)
                               : launch_rows(k_gemv16<FMT_BF16, 1, 8>, m, 1, s);
        case FMT_Q4:
            return launch_rows(k_gemv_q4<4, 1>, m, 4, s);
        default:
            return hipErrorInvalidValue;
    }
}

/* ======================================= sweep ================================================ */

constexpr int TABLE_CHUNK = 16;
struct TableChunk {
    int32_t n;
    int32_t pad_[3];
    DevMat m[TABLE_CHUNK];
};

__global__ __launch_bounds__(WAVE) void k_put_table(DevMat* __restrict__ dst, TableChunk c) {
    const int i = threadIdx.x;
    if (i < c.n) dst[i] = c.m[i];
}

hipError_t launch_put_table(DevMat* dst, const DevMat* src, int n, hipStream_t s) {
    for (int first = 0; first < n; first += TABLE_CHUNK) {
        TableChunk c{};
        c.n = std::min(TABLE_CHUNK, n - first);
        for (int i = 0; i < c.n; ++i) c.m[i] = src[first + i];
        hipLaunchKernelGGL(k_put_table, dim3(1), dim3(WAVE), 0, s, dst + first, c);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

__device__ __forceinline__ int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

/* Rows of all matrices, in table order, form one weight stream of `total` bytes.  Wave w of nw owns
   the rows whose first byte lies in [w * total / nw, (w + 1) * total / nw), so every wave streams
   the same number of bytes and every row has exactly one owner. */
template <int FMTALL>
__global__ __launch_bounds__(BLOCK) void k_sweep(const DevMat* __restrict__ tab, int nmat,
                                                 int64_t total, int32_t token) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int64_t nw = (int64_t)gridDim.x * WAVES_PER_BLOCK;
    const int64_t w = (int64_t)blockIdx.x * WAVES_PER_BLOCK + threadIdx.x / WAVE;
    const int64_t lo = total * w / nw, hi = total * (w + 1) / nw;
    if (lo >= hi) return;
    int a = 0, b = nmat - 1;  /* last matrix whose stream starts at or before lo */
    while (a < b) {
        const int mid = (a + b + 1) >> 1;
        if (tab[mid].cost0 <= lo) a = mid; else b = mid - 1;
    }
    for (int m = a; m < nmat; ++m) {
        const DevMat d = tab[m];
        if (d.cost0 >= hi) break;
        const int64_t r0 = lo > d.cost0 ? ceil_div(lo - d.cost0, d.row_bytes) : 0;
        const int64_t r1 = std::min<int64_t>(d.M, ceil_div(hi - d.cost0, d.row_bytes));
        if (r0 >= r1) continue;
        const int fmt = FMTALL ? FMTALL : d.fmt;
        if ((FMTALL == 0 || FMTALL == FMT_F16) && fmt == FMT_F16)
            rows16<FMT_F16, 2, 4>(d, r0, r1, token, lane);
        else if ((FMTALL == 0 || FMTALL == FMT_BF16) && fmt == FMT_BF16)
            rows16<FMT_BF16, 2, 4>(d, r0, r1, token, lane);
        else if ((FMTALL == 0 || FMTALL == FMT_Q4) && fmt == FMT_Q4)
            rows_q4<4, 1>(d, r0, r1, token, lane);
    }
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

hipError_t launch_sweep(const DevMat* tab, int nmat, int64_t total, int fmt_all, int32_t token,
                        hipStream_t s) {
    if (nmat == 0 || total == 0) return hipSuccess;
    const unsigned blocks = (unsigned)cu_count() * 4;
    switch (fmt_all) {
        case FMT_F16:
            hipLaunchKernelGGL(k_sweep<FMT_F16>, dim3(blocks), dim3(BLOCK), 0, s, tab, nmat, total, token);
            break;
        case FMT_BF16:
            hipLaunchKernelGGL(k_sweep<FMT_BF16>, dim3(blocks), dim3(BLOCK), 0, s, tab, nmat, total, token);
            break;
        case FMT_Q4:
            hipLaunchKernelGGL(k_sweep<FMT_Q4>, dim3(blocks), dim3(BLOCK), 0, s, tab, nmat, total, token);
            break;
        default:
            hipLaunchKernelGGL(k_sweep<0>, dim3(blocks), dim3(BLOCK), 0, s, tab, nmat, total, token);
            break;
    }
    return hipGetLastError();
}

}  // namespace wsr
