/*
 * synth_dev.hip - the input generator on the GPU: the same draws and encoders as synth.c
 * (synth_core.h), written straight into device memory, so large synthetic models need no host
 * generation or upload.  Built without floating-point contraction so the one double expression
 * (uniform scaling) rounds exactly as on the host.  Input generation only.
 */
#include <hip/hip_runtime.h>

#include "synth_core.h"

namespace {

constexpr int BLOCK = 256;
constexpr int PER = 8;   /* elements per thread per step */

__global__ __launch_bounds__(BLOCK) void k_normal16(uint16_t* __restrict__ out, int64_t n, uint64_t seed,
                                                    uint64_t stream, uint64_t e0,
                                                    const uint64_t* __restrict__ q,
                                                    const uint16_t* __restrict__ alias) {
    const int64_t step = (int64_t)gridDim.x * BLOCK * PER;
    for (int64_t i = ((int64_t)blockIdx.x * BLOCK + threadIdx.x) * PER; i < n; i += step)
        for (int j = 0; j < PER && i + j < n; ++j)
            out[i + j] = synth_table_draw(q, alias, synth_draw(seed, stream, e0 + (uint64_t)(i + j)));
}

__global__ __launch_bounds__(BLOCK) void k_uniform16(uint16_t* __restrict__ out, int64_t n, uint64_t seed,
                                                     uint64_t stream, uint64_t e0, double lo, double hi,
                                                     int fmt) {
    const int64_t step = (int64_t)gridDim.x * BLOCK * PER;
    for (int64_t i = ((int64_t)blockIdx.x * BLOCK + threadIdx.x) * PER; i < n; i += step)
        for (int j = 0; j < PER && i + j < n; ++j)
            out[i + j] = synth_uniform16_value(synth_draw(seed, stream, e0 + (uint64_t)(i + j)), lo, hi, fmt);
}

__global__ __launch_bounds__(BLOCK) void k_q4(uint8_t* __restrict__ out, int64_t nbytes, uint64_t seed,
                                              uint64_t stream, uint64_t e0) {
    const int64_t step = (int64_t)gridDim.x * BLOCK * PER;
    for (int64_t i = ((int64_t)blockIdx.x * BLOCK + threadIdx.x) * PER; i < nbytes; i += step)
        for (int j = 0; j < PER && i + j < nbytes; ++j) out[i + j] = synth_q4_byte(seed, stream, e0, i + j);
}

__global__ __launch_bounds__(BLOCK) void k_i8(int8_t* __restrict__ out, int64_t n, uint64_t seed,
                                              uint64_t stream, uint64_t e0) {
    const int64_t step = (int64_t)gridDim.x * BLOCK * PER;
    for (int64_t i = ((int64_t)blockIdx.x * BLOCK + threadIdx.x) * PER; i < n; i += step)
        for (int j = 0; j < PER && i + j < n; ++j)
            out[i + j] = synth_int8_value(synth_draw(seed, stream, e0 + (uint64_t)(i + j)));
}

__global__ __launch_bounds__(BLOCK) void k_grid(float* __restrict__ out, int64_t n, uint64_t seed,
                                                uint64_t stream, uint64_t e0) {
    const int64_t step = (int64_t)gridDim.x * BLOCK * PER;
    for (int64_t i = ((int64_t)blockIdx.x * BLOCK + threadIdx.x) * PER; i < n; i += step)
        for (int j = 0; j < PER && i + j < n; ++j)
            out[i + j] = synth_grid_value(synth_draw(seed, stream, e0 + (uint64_t)(i + j)));
}

unsigned grid_for(int64_t n) {
    const int64_t g = (n + (int64_t)BLOCK * PER - 1) / ((int64_t)BLOCK * PER);
    return (unsigned)(g < 1 ? 1 : (g > 65536 ? 65536 : g));
}

}  // namespace

extern "C" {

int synth_dev_normal16(uint16_t* out, int64_t n, uint64_t seed, uint64_t stream, uint64_t e0,
                       const uint64_t* q, const uint16_t* alias, void* s) {
    if (n <= 0) return 0;
    hipLaunchKernelGGL(k_normal16, dim3(grid_for(n)), dim3(BLOCK), 0, (hipStream_t)s, out, n, seed,
                       stream, e0, q, alias);
    return (int)hipGetLastError();
}

int synth_dev_uniform16(uint16_t* out, int64_t n, uint64_t seed, uint64_t stream, uint64_t e0,
                        double lo, double hi, int fmt, void* s) {
    if (n <= 0) return 0;
    hipLaunchKernelGGL(k_uniform16, dim3(grid_for(n)), dim3(BLOCK), 0, (hipStream_t)s, out, n, seed,
                       stream, e0, lo, hi, fmt);
    return (int)hipGetLastError();
}

int synth_dev_q4(uint8_t* out, int64_t nbytes, uint64_t seed, uint64_t stream, uint64_t e0, void* s) {
    if (nbytes <= 0) return 0;
    hipLaunchKernelGGL(k_q4, dim3(grid_for(nbytes)), dim3(BLOCK), 0, (hipStream_t)s, out, nbytes, seed,
                       stream, e0);
    return (int)hipGetLastError();
}

int synth_dev_i8(int8_t* out, int64_t n, uint64_t seed, uint64_t stream, uint64_t e0, void* s) {
    if (n <= 0) return 0;
    hipLaunchKernelGGL(k_i8, dim3(grid_for(n)), dim3(BLOCK), 0, (hipStream_t)s, out, n, seed, stream, e0);
    return (int)hipGetLastError();
}

int synth_dev_grid_f32(float* out, int64_t n, uint64_t seed, uint64_t stream, uint64_t e0, void* s) {
    if (n <= 0) return 0;
    hipLaunchKernelGGL(k_grid, dim3(grid_for(n)), dim3(BLOCK), 0, (hipStream_t)s, out, n, seed, stream, e0);
    return (int)hipGetLastError();
}

}  // extern "C"
