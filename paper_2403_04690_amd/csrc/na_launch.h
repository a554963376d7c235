// na_launch.h -- host-side launchers of the HIP kernels (internal to libna.so).
#pragma once

#include <hip/hip_runtime.h>

#include "na_common.h"

namespace na {

// Forward: q, k, v, o in dtype (0 fp32, 1 fp16, 2 bf16); lse fp32.
hipError_t launch_forward(const Geo& g, int rank, int D, int dtype, int qm, const void* q,
                          const void* k, const void* v, void* o, float* lse, float scale,
                          hipStream_t s);

// Backward: one launch of dK/dV-role and dQ-role workgroups (Delta in-kernel).
hipError_t launch_backward(const Geo& g, int rank, int D, int dtype, int m, const void* q,
                           const void* k, const void* v, const void* o, const float* lse,
                           const void* dout, void* dq, void* dk, void* dv, float scale,
                           hipStream_t s);

// Per-axis window starts and inverse ranges (absolute coordinates), int32.
hipError_t launch_debug_windows(int rank, const int* L, const int* k, const int* d, const int* c,
                                int* start, int* inv_lo, int* inv_hi, hipStream_t s);

}  // namespace na
