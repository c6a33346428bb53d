// Host-side launchers of the device kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace osm {

// Row kernels: team = lanes per row (4..64 inside a wavefront, 128..1024 one
// row per workgroup).  vec: x and y rows may be read / written as 16-byte
// vectors (x and y congruent modulo 16 bytes).
hipError_t launch_softmax_rows(const void* x, void* y, int64_t N, int64_t V, int dtype,
                               int mode, int team, bool vec, hipStream_t st);

// Split-V: S chunks of `chunk` elements per row; scratch holds N * S float2.
hipError_t launch_softmax_split(const void* x, void* y, void* scratch, int64_t N, int64_t V,
                                int dtype, int mode, int64_t S, int64_t chunk, bool vec,
                                hipStream_t st);

// Fused online softmax + top-k; waves_per_row = 1 (four rows per workgroup)
// or 4 (one row per workgroup).
hipError_t launch_topk_fused(const void* x, float* vals, int32_t* idx, int64_t N, int64_t V,
                             int K, int dtype, int waves_per_row, hipStream_t st);

}  // namespace osm
