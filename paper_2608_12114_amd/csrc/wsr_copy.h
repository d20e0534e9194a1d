/*
 * wsr_copy.h - the staged sweep's per-use copy of pinned host pages into device memory (defined in
 * wsr_copy.hip).
 */
#ifndef WSR_COPY_H
#define WSR_COPY_H

#include <hip/hip_runtime.h>

#include <cstddef>

namespace wsr {

/* dst[0, bytes) = src[0, bytes) on stream s, the source read by the shaders: src is the device view
   of pinned host memory (or device memory), dst device memory, both 16-byte aligned and bytes a
   multiple of 16; the caller has checked that the whole source range is mapped. */
hipError_t launch_copy16(const void* src, void* dst, size_t bytes, hipStream_t s);

}  // namespace wsr

#endif
