/*
 * wsr_internal.h - what the host side of libwsr passes to the kernels.
 *
 * A matrix as the kernels see it (built by the host from a wsr_mat or a GEMV call).  Costs are in
 * bytes of weight stream (weights plus scales), the unit the work is balanced on.
 */
#ifndef WSR_INTERNAL_H
#define WSR_INTERNAL_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

namespace wsr {

enum : int32_t { FMT_F16 = 1, FMT_BF16 = 2, FMT_Q4 = 3, FMT_I8 = 4 };

struct alignas(16) DevMat {
    const void* w;          /* 16-bit weights, packed int4 codes or int8 codes              */
    const void* s;          /* q4 block scales or int8 row scales                           */
    const void* x;          /* activation of token 0                                        */
    float* y;               /* output of token 0                                            */
    int64_t M;              /* rows                                                         */
    int64_t nc;             /* per row: 16-byte chunks (16-bit, int8) or 32-weight blocks    */
    int64_t x_stride;       /* bytes between tokens                                         */
    int64_t y_stride;
    int64_t cost0;          /* weight-stream byte offset of row 0 within its launch         */
    int64_t row_bytes;      /* weight-stream bytes per row                                  */
    int32_t fmt;
    int32_t pad_[3];
};
static_assert(sizeof(DevMat) == 96, "DevMat layout");

/* Launchers (defined with the kernels).  All return the status of the launch. */
hipError_t launch_probe(const float* buf, int64_t n, double* sum_dev, void* ws, hipStream_t s);
int64_t probe_grid(int64_t n);

hipError_t launch_gemv(const DevMat& m, hipStream_t s);
/* T activation columns per weight read (1, 2, 4, 8 or 16 for 16-bit formats, up to 8 for q4 and
   int8).
   m.x_stride and m.y_stride are the column strides in bytes. */
hipError_t launch_gemv_cols(const DevMat& m, int T, hipStream_t s);
/* Writes the table and clears the two tile counters at ctr (ctr may be null). */
hipError_t launch_put_table(DevMat* dst, int64_t* cost, const DevMat* src, int n, unsigned* ctr,
                            hipStream_t s);
/* One pass over the table's weights for tokens token .. token + T - 1 (T = 1, 2, 4, 8, 16; at most
   8 when the table holds a q4 or int8 matrix).  tab / cost: the table in device memory (written by
   launch_put_table); htab: the same table on the host, or null.  A launch for which
   sweep_table_by_value() holds and htab is given carries the table in its arguments and reads
   neither tab, cost nor ctr. */
hipError_t launch_sweep(const DevMat* tab, const int64_t* cost, const DevMat* htab, int nmat, int64_t total_bytes,
                        int fmt_all, int32_t token, int T, unsigned* ctr, hipStream_t s);
bool sweep_table_by_value(int nmat, int64_t total_bytes, int fmt_all, int T);

/* Sweep workspace: tile counters in the first SWEEP_CTR_BYTES, then the table, then the matrices'
   stream offsets (DevMat::cost0) as a dense int64 array, each part padded to 256 bytes. */
constexpr size_t SWEEP_CTR_BYTES = 256;

/* The library's own sweep workspace for callers that cannot allocate device memory: a file-scope
   device array of NOALLOC_SCRATCH_BYTES per device (a table of up to about 5,000 matrices).
   noalloc_scratch returns its address on the current device; the first call on a device looks it
   up (hipGetSymbolAddress) and later calls reuse that address. */
constexpr size_t NOALLOC_SCRATCH_BYTES = 512 << 10;
hipError_t noalloc_scratch(void** ptr);

}  // namespace wsr

#endif
