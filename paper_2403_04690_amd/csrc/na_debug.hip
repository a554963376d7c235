// na_debug.hip -- device evaluation of the per-axis neighbourhood summary with
// the same index functions the attention kernels use (window start of each
// query, first and last query of each key's inverse neighbourhood), causal
// axes included.
#include "na_launch.h"

namespace na {

__global__ void na_debug_windows_kernel(int rank, int L0, int L1, int L2, int k0, int k1, int k2,
                                        int d0, int d1, int d2, int c0, int c1, int c2, int* start,
                                        int* ilo, int* ihi) {
    const int Ls[3] = {L0, L1, L2}, ks[3] = {k0, k1, k2}, ds[3] = {d0, d1, d2};
    const bool cs[3] = {c0 != 0, c1 != 0, c2 != 0};
    int x = blockIdx.x * blockDim.x + threadIdx.x;
    int off = 0;
    for (int a = 0; a < rank; ++a) {
        if (x < Ls[a]) {
            const int d = ds[a], k = ks[a];
            const int gidx = x % d, p = x / d;
            const int n = group_len(Ls[a], d, gidx);
            start[off + x] = gidx + d * win_start(p, n, k, cs[a]);
            ilo[off + x] = gidx + d * inv_lo(p, n, k, cs[a]);
            ihi[off + x] = gidx + d * inv_hi(p, n, k, cs[a]);
            return;
        }
        x -= Ls[a];
        off += Ls[a];
    }
}

hipError_t launch_debug_windows(int rank, const int* L, const int* k, const int* d, const int* c,
                                int* start, int* inv_lo_out, int* inv_hi_out, hipStream_t s) {
    int total = 0;
    int Ls[3] = {1, 1, 1}, ks[3] = {1, 1, 1}, ds[3] = {1, 1, 1}, cs[3] = {0, 0, 0};
    for (int a = 0; a < rank; ++a) {
        total += L[a];
        Ls[a] = L[a];
        ks[a] = k[a];
        ds[a] = d[a];
        cs[a] = c[a];
    }
    const int blocks = (total + 255) / 256;
    hipLaunchKernelGGL(na_debug_windows_kernel, dim3(blocks), dim3(256), 0, s, rank, Ls[0], Ls[1],
                       Ls[2], ks[0], ks[1], ks[2], ds[0], ds[1], ds[2], cs[0], cs[1], cs[2], start,
                       inv_lo_out, inv_hi_out);
    return hipGetLastError();
}

}  // namespace na
