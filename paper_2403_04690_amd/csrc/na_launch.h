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

// Geometry of the unfused operators (filled on the host).  A rank-r problem
// occupies the last r axes; the leading ones are inert (extent, window and
// dilation 1, token stride 0).
struct UGeo {
    int L[kMaxRank], k[kMaxRank], d[kMaxRank], causal[kMaxRank];
    int ts[kMaxRank];   // token stride of each axis (0 for inert axes)
    int kst[kMaxRank];  // stride of each axis's window offset in a weight row
    int N;              // tokens per (batch, head)
    int ell;            // weights per row: prod k
    int64_t rows;       // batch * heads * N
    FastDiv fd_L[kMaxRank], fd_d[kMaxRank], fd_k[kMaxRank];
};

// The unfused operators (na_unfused.hip): x, y, z are the op's operands.
enum {
    kUnfusedPN = 0,        // z[i, e] = scale * x_i . y_j(i,e)            (weights z)
    kUnfusedSoftmax = 1,   // z = softmax of each row of z in place; lse  (weights z)
    kUnfusedNN = 2,        // z_i = scale * sum_e x[i, e] y_j(i,e)        (weights x)
    kUnfusedIN = 3,        // z_j = scale * sum_i x[i, e(i,j)] y_i         (weights x)
    kUnfusedSoftmaxBwd = 4 // z = x * (z - rowsum(x * z)) in place          (probs x)
};
hipError_t launch_unfused(const UGeo& u, int D, int dtype, int op, const void* x, const void* y,
                          void* z, float* lse, float scale, hipStream_t s);

// Per-axis window starts and inverse ranges (absolute coordinates), int32.
hipError_t launch_debug_windows(int rank, const int* L, const int* k, const int* d, const int* c,
                                int* start, int* inv_lo, int* inv_hi, hipStream_t s);

}  // namespace na
