/*
 * wsr_mma_launch.h - launcher of the batched decode sweep on the matrix cores (defined in wsr_mma.hip).
 */
#ifndef WSR_MMA_LAUNCH_H
#define WSR_MMA_LAUNCH_H

#include "wsr_internal.h"

namespace wsr {

/* The kernel format of a q4 table whose every matrix reads a step's eight block scales as one
   16-byte load: rows of a whole number of 8-block steps (nc % 8 == 0) and 16-byte aligned scales.
   Its kernel holds only that loop, which fits two waves per SIMD (255 registers, against 280 for
   the kernel with every q4 loop). */
constexpr int FMT_Q4_WHOLE = 8;

/* Tokens token0 .. token0 + ntok - 1 (ntok <= 16) of the sweep on the matrix cores, in row groups
   of 16 tiles rows (tiles 4 or 8, as mma_tiles chooses for the table's format, the pass's tokens
   and its longest row); max_group and max_tail_group are the largest row group's weight-stream
   bytes (16 tiles rows, and mma_tail_rows() rows for the tail of the stream, of any matrix in the
   table). */
int mma_tiles(int fmt_all, int ntok, int64_t max_row_bytes);
int64_t mma_tail_rows();
hipError_t launch_sweep_mma(const DevMat* tab, const int64_t* cost, int nmat, int64_t total, int tiles,
                            int64_t max_group, int64_t max_tail_group, int fmt_all, int32_t token0, int ntok,
                            hipStream_t s);

}  // namespace wsr

#endif
