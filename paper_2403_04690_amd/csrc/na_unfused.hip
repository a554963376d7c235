// na_unfused.hip -- the unfused neighborhood-attention operators for gfx950:
// the baseline the fused kernels are measured against.
//
// Sec. 3.1 of the paper splits NA into operators that each read or write the
// l-wide attention weights (l = prod_a k_a per query) in global memory:
//   PN  w[i, e]  = scale * a_i . b_{j(i,e)}                (QK^T; dO V^T)
//   NN  out_i    = scale * sum_e w[i, e] b_{j(i,e)}        (AV; dA K)
//   IN  out_j    = scale * sum_{i : j in N(i)} w[i, e(i,j)] b_i   (dA^T Q; P^T dO)
// with the softmax between PN and NN (and its backward, dA = P (dP - Delta),
// Delta_i = sum_e P_ie dP_ie) as kernels of their own.  Each operator is one
// launch; nothing is fused across them, so a forward writes and re-reads the
// weights twice and a backward four times more (Sec. 3.2 names that traffic
// as what bounds such implementations).
//
// Weight layout: [B, H, N, l] in the inputs' type, row i holding query i's
// neighbours in the row-major order of the per-axis window offsets t_a
// (axis 0 outermost): e = sum_a t_a * prod_{b > a} k_b, neighbour
// coordinate g_a + d_a (s_a + t_a) with s_a the window start of the query's
// group position.  Along a causal axis the window of position p holds only
// min(k, p + 1) positions; offsets beyond them are not neighbours (PN writes
// -inf there, the softmax turns that into 0, NN and IN skip them).
//
// Mapping: one wave per weight row in PN (lanes over e, each lane a full dot
// product from its key row) and in the softmax kernels (lanes over e); in NN
// and IN each query (key) row of D elements is spread over D/2 lanes, two
// elements per lane, so the rows of b are read coalesced, and the loop over
// neighbours is a nest over the per-axis windows.  Rows are visited by a
// grid-stride loop.
#include <type_traits>

#include "na_launch.h"

namespace na {

namespace {

constexpr int kUThreads = 256;
constexpr int kUWaves = kUThreads / kWave;
constexpr int kUMaxBlocks = 1 << 18;

// Per-axis position of a token in its dilation group and its window there.
struct AxisPos {
    int g, p, n;  // group, position in the group, group length
};

__device__ __forceinline__ void token_axes(const UGeo& u, int tok, AxisPos* ax) {
#pragma unroll
    for (int a = kMaxRank - 1; a >= 0; --a) {
        const int rest = u.fd_L[a].div(tok);
        const int x = tok - rest * u.L[a];
        tok = rest;
        const int p = u.fd_d[a].div(x);
        ax[a].g = x - p * u.d[a];
        ax[a].p = p;
        ax[a].n = u.fd_d[a].div(u.L[a] - ax[a].g + u.d[a] - 1);
    }
}

template <typename T>
__device__ __forceinline__ float to_f(T x) {
    return (float)x;
}

// ---- PN: w[i, e] = scale * a_i . b_j(i,e) (or -inf where e is not a neighbour) ----
template <typename T, int D>
__global__ __launch_bounds__(kUThreads) void pn_kernel(UGeo u, const T* __restrict__ ag,
                                                       const T* __restrict__ bg,
                                                       T* __restrict__ wg, float scale) {
    using x8 = typename Tr<T>::x8;
    const int lane = threadIdx.x & 63;
    const int64_t nw = (int64_t)gridDim.x * kUWaves;
    for (int64_t row = (int64_t)blockIdx.x * kUWaves + (threadIdx.x >> 6); row < u.rows;
         row += nw) {
        const int64_t slice = row / u.N;
        const int tok = (int)(row - slice * u.N);
        const T* arow = ag + row * D;
        const T* bs = bg + slice * u.N * (int64_t)D;
        T* wrow = wg + row * u.ell;
        AxisPos ax[kMaxRank];
        token_axes(u, tok, ax);
        int s[kMaxRank], c[kMaxRank];
#pragma unroll
        for (int a = 0; a < kMaxRank; ++a) {
            s[a] = win_start(ax[a].p, ax[a].n, u.k[a], u.causal[a] != 0);
            c[a] = u.causal[a] ? ax[a].p - s[a] + 1 : u.k[a];
        }
        x8 af[D / 8];
#pragma unroll
        for (int i = 0; i < D / 8; ++i) af[i] = ld_x8<T>(arow + 8 * i);
        for (int e = lane; e < u.ell; e += kWave) {
            int rem = e, j = 0;
            bool valid = true;
#pragma unroll
            for (int a = kMaxRank - 1; a >= 0; --a) {
                const int q = u.fd_k[a].div(rem);
                const int t = rem - q * u.k[a];
                rem = q;
                valid = valid && t < c[a];
                j += (ax[a].g + u.d[a] * (s[a] + t)) * u.ts[a];
            }
            float acc = -INFINITY;
            if (valid) {
                const T* brow = bs + (int64_t)j * D;
                float dot = 0.f;
#pragma unroll
                for (int i = 0; i < D / 8; ++i) {
                    dot = dot8<T>(af[i], ld_x8<T>(brow + 8 * i), dot);
                }
                acc = dot * scale;
            }
            wrow[e] = Tr<T>::cvt(acc);
        }
    }
}

// Wave-wide combination of per-lane (max, sum of exp(x - max)) pairs.
__device__ __forceinline__ void wave_lse(float& m, float& z) {
#pragma unroll
    for (int w = 32; w >= 1; w >>= 1) {
        const float m2 = __shfl_xor(m, w, kWave);
        const float z2 = __shfl_xor(z, w, kWave);
        const float mn = fmaxf(m, m2);
        if (mn == -INFINITY) continue;  // both empty
        z = z * __expf(m - mn) + z2 * __expf(m2 - mn);
        m = mn;
    }
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int w = 32; w >= 1; w >>= 1) x += __shfl_xor(x, w, kWave);
    return x;
}

// ---- softmax over each weight row, in place; logsumexp (natural log) per row ----
template <typename T>
__global__ __launch_bounds__(kUThreads) void softmax_kernel(UGeo u, T* __restrict__ wg,
                                                            float* __restrict__ lseg) {
    const int lane = threadIdx.x & 63;
    const int64_t nw = (int64_t)gridDim.x * kUWaves;
    for (int64_t row = (int64_t)blockIdx.x * kUWaves + (threadIdx.x >> 6); row < u.rows;
         row += nw) {
        T* wrow = wg + row * u.ell;
        float m = -INFINITY, z = 0.f;
        for (int e = lane; e < u.ell; e += kWave) {
            const float x = to_f(wrow[e]);
            if (x == -INFINITY) continue;
            const float mn = fmaxf(m, x);
            z = z * __expf(m - mn) + __expf(x - mn);
            m = mn;
        }
        wave_lse(m, z);
        const float lse = m + __logf(z);
        for (int e = lane; e < u.ell; e += kWave) wrow[e] = Tr<T>::cvt(__expf(to_f(wrow[e]) - lse));
        if (lane == 0) lseg[row] = lse;
    }
}

// ---- softmax backward, in place on the gradient: dA = P (dP - sum_e P dP) ----
template <typename T>
__global__ __launch_bounds__(kUThreads) void softmax_bwd_kernel(UGeo u, const T* __restrict__ pg,
                                                                T* __restrict__ gg) {
    const int lane = threadIdx.x & 63;
    const int64_t nw = (int64_t)gridDim.x * kUWaves;
    for (int64_t row = (int64_t)blockIdx.x * kUWaves + (threadIdx.x >> 6); row < u.rows;
         row += nw) {
        const T* prow = pg + row * u.ell;
        T* grow = gg + row * u.ell;
        float part = 0.f;
        for (int e = lane; e < u.ell; e += kWave) {
            const float p = to_f(prow[e]);
            if (p != 0.f) part += p * to_f(grow[e]);  // (masked entries: P = 0, dP = -inf)
        }
        const float delta = wave_sum(part);
        for (int e = lane; e < u.ell; e += kWave) {
            const float p = to_f(prow[e]);
            grow[e] = Tr<T>::cvt(p != 0.f ? p * (to_f(grow[e]) - delta) : 0.f);
        }
    }
}

// Two consecutive elements of a row (a 4-byte load for 16-bit types).
template <typename T>
__device__ __forceinline__ void ld2(const T* p, float& x, float& y) {
    if constexpr (sizeof(T) == 2) {
        typedef T t2 __attribute__((ext_vector_type(2)));
        const t2 v = *reinterpret_cast<const t2*>(p);
        x = (float)v[0];
        y = (float)v[1];
    } else {
        const float2 v = *reinterpret_cast<const float2*>(p);
        x = v.x;
        y = v.y;
    }
}
template <typename T>
__device__ __forceinline__ void st2(T* p, float x, float y) {
    if constexpr (sizeof(T) == 2) {
        typedef T t2 __attribute__((ext_vector_type(2)));
        *reinterpret_cast<t2*>(p) = t2{Tr<T>::cvt(x), Tr<T>::cvt(y)};
    } else {
        *reinterpret_cast<float2*>(p) = float2{x, y};
    }
}

// ---- NN: out_i = scale * sum_e w[i, e] b_j(i,e) ----
template <typename T, int D>
__global__ __launch_bounds__(kUThreads) void nn_kernel(UGeo u, const T* __restrict__ wg,
                                                       const T* __restrict__ bg,
                                                       T* __restrict__ og, float scale) {
    constexpr int kTpr = D / 2;             // lanes per row
    constexpr int kRpb = kUThreads / kTpr;  // rows per workgroup pass
    const int sub = threadIdx.x % kTpr;
    const int64_t step = (int64_t)gridDim.x * kRpb;
    for (int64_t row = (int64_t)blockIdx.x * kRpb + threadIdx.x / kTpr; row < u.rows;
         row += step) {
        const int64_t slice = row / u.N;
        const int tok = (int)(row - slice * u.N);
        const T* bs = bg + slice * u.N * (int64_t)D + 2 * sub;
        const T* wrow = wg + row * u.ell;
        AxisPos ax[kMaxRank];
        token_axes(u, tok, ax);
        int s[kMaxRank], c[kMaxRank];
#pragma unroll
        for (int a = 0; a < kMaxRank; ++a) {
            s[a] = win_start(ax[a].p, ax[a].n, u.k[a], u.causal[a] != 0);
            c[a] = u.causal[a] ? ax[a].p - s[a] + 1 : u.k[a];
        }
        float acc0 = 0.f, acc1 = 0.f;
        for (int t0 = 0; t0 < c[0]; ++t0) {
            const int j0 = (ax[0].g + u.d[0] * (s[0] + t0)) * u.ts[0];
            for (int t1 = 0; t1 < c[1]; ++t1) {
                const int j1 = j0 + (ax[1].g + u.d[1] * (s[1] + t1)) * u.ts[1];
                const int e1 = t0 * u.kst[0] + t1 * u.kst[1];
#pragma unroll 8
                for (int t2 = 0; t2 < c[2]; ++t2) {
                    const int j = j1 + (ax[2].g + u.d[2] * (s[2] + t2)) * u.ts[2];
                    const float w = to_f(wrow[e1 + t2]);
                    float x, y;
                    ld2<T>(bs + (int64_t)j * D, x, y);
                    acc0 = fmaf(w, x, acc0);
                    acc1 = fmaf(w, y, acc1);
                }
            }
        }
        st2<T>(og + row * D + 2 * sub, acc0 * scale, acc1 * scale);
    }
}

// ---- IN: out_j = scale * sum over the queries i whose window holds j of w[i, e(i,j)] b_i ----
template <typename T, int D>
__global__ __launch_bounds__(kUThreads) void in_kernel(UGeo u, const T* __restrict__ wg,
                                                       const T* __restrict__ bg,
                                                       T* __restrict__ og, float scale) {
    constexpr int kTpr = D / 2;
    constexpr int kRpb = kUThreads / kTpr;
    const int sub = threadIdx.x % kTpr;
    const int64_t step = (int64_t)gridDim.x * kRpb;
    for (int64_t row = (int64_t)blockIdx.x * kRpb + threadIdx.x / kTpr; row < u.rows;
         row += step) {
        const int64_t slice = row / u.N;
        const int tok = (int)(row - slice * u.N);
        const int64_t base = slice * u.N;
        AxisPos ax[kMaxRank];
        token_axes(u, tok, ax);
        int lo[kMaxRank], hi[kMaxRank];
#pragma unroll
        for (int a = 0; a < kMaxRank; ++a) {
            const bool ca = u.causal[a] != 0;
            lo[a] = inv_lo(ax[a].p, ax[a].n, u.k[a], ca);
            hi[a] = inv_hi(ax[a].p, ax[a].n, u.k[a], ca);
        }
        float acc0 = 0.f, acc1 = 0.f;
        for (int p0 = lo[0]; p0 <= hi[0]; ++p0) {
            const int i0 = (ax[0].g + u.d[0] * p0) * u.ts[0];
            const int e0 = (ax[0].p - win_start(p0, ax[0].n, u.k[0], u.causal[0] != 0)) * u.kst[0];
            for (int p1 = lo[1]; p1 <= hi[1]; ++p1) {
                const int i1 = i0 + (ax[1].g + u.d[1] * p1) * u.ts[1];
                const int e1 =
                    e0 + (ax[1].p - win_start(p1, ax[1].n, u.k[1], u.causal[1] != 0)) * u.kst[1];
#pragma unroll 8
                for (int p2 = lo[2]; p2 <= hi[2]; ++p2) {
                    const int i = i1 + (ax[2].g + u.d[2] * p2) * u.ts[2];
                    const int e =
                        e1 + (ax[2].p - win_start(p2, ax[2].n, u.k[2], u.causal[2] != 0));
                    const float w = to_f(wg[(base + i) * u.ell + e]);
                    float x, y;
                    ld2<T>(bg + (base + i) * D + 2 * sub, x, y);
                    acc0 = fmaf(w, x, acc0);
                    acc1 = fmaf(w, y, acc1);
                }
            }
        }
        st2<T>(og + row * D + 2 * sub, acc0 * scale, acc1 * scale);
    }
}

int blocks_for(int64_t rows, int rows_per_block) {
    const int64_t b = (rows + rows_per_block - 1) / rows_per_block;
    return (int)(b < kUMaxBlocks ? b : kUMaxBlocks);
}

template <typename T, int D>
hipError_t launch_unfused_t(const UGeo& u, int op, const void* x, const void* y, void* z,
                            float* lse, float scale, hipStream_t s) {
    switch (op) {
        case kUnfusedPN:
            hipLaunchKernelGGL((pn_kernel<T, D>), dim3(blocks_for(u.rows, kUWaves)),
                               dim3(kUThreads), 0, s, u, static_cast<const T*>(x),
                               static_cast<const T*>(y), static_cast<T*>(z), scale);
            break;
        case kUnfusedNN:
            hipLaunchKernelGGL((nn_kernel<T, D>), dim3(blocks_for(u.rows, kUThreads / (D / 2))),
                               dim3(kUThreads), 0, s, u, static_cast<const T*>(x),
                               static_cast<const T*>(y), static_cast<T*>(z), scale);
            break;
        case kUnfusedIN:
            hipLaunchKernelGGL((in_kernel<T, D>), dim3(blocks_for(u.rows, kUThreads / (D / 2))),
                               dim3(kUThreads), 0, s, u, static_cast<const T*>(x),
                               static_cast<const T*>(y), static_cast<T*>(z), scale);
            break;
        case kUnfusedSoftmax:
            hipLaunchKernelGGL((softmax_kernel<T>), dim3(blocks_for(u.rows, kUWaves)),
                               dim3(kUThreads), 0, s, u, static_cast<T*>(z), lse);
            break;
        case kUnfusedSoftmaxBwd:
            hipLaunchKernelGGL((softmax_bwd_kernel<T>), dim3(blocks_for(u.rows, kUWaves)),
                               dim3(kUThreads), 0, s, u, static_cast<const T*>(x),
                               static_cast<T*>(z));
            break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename T>
hipError_t launch_unfused_d(const UGeo& u, int D, int op, const void* x, const void* y, void* z,
                            float* lse, float scale, hipStream_t s) {
    switch (D) {
        case 32: return launch_unfused_t<T, 32>(u, op, x, y, z, lse, scale, s);
        case 64: return launch_unfused_t<T, 64>(u, op, x, y, z, lse, scale, s);
        case 128: return launch_unfused_t<T, 128>(u, op, x, y, z, lse, scale, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_unfused(const UGeo& u, int D, int dtype, int op, const void* x, const void* y,
                          void* z, float* lse, float scale, hipStream_t s) {
    switch (dtype) {
        case 0: return launch_unfused_d<float>(u, D, op, x, y, z, lse, scale, s);
        case 1: return launch_unfused_d<_Float16>(u, D, op, x, y, z, lse, scale, s);
        case 2: return launch_unfused_d<__bf16>(u, D, op, x, y, z, lse, scale, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace na
