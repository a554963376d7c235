// na_common.h -- shared device infrastructure of the fused NA kernels (gfx950).
//
// Matrix-core convention used throughout (v_mfma_f32_16x16x32_{f16,bf16}):
//   operand A (16 x 32): lane l holds row (l % 16), contraction slots
//                        8*(l/16) .. 8*(l/16)+7
//   operand B (32 x 16): lane l holds column (l % 16), the same 8 slots
//   result  C (16 x 16): lane l holds column (l % 16), rows 4*(l/16) .. +3
// The contraction only needs A and B to agree on which real index sits in
// each slot, so the kernels freely permute slots.  fp32 runs the same 16x16x32
// step as eight v_mfma_f32_16x16x4_f32 instructions (one slot each).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "na_fastdiv.h"
#include "na_index.h"

namespace na {

constexpr int kWave = 64;
constexpr int kMaxRank = 3;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

// Element traits: 8-slot fragments, the 16x16x32 matrix step, rounding.
template <typename T>
struct Tr;

template <>
struct Tr<_Float16> {
    using x8 = f16x8;
    using x4 = f16x4;
    static constexpr int kVec = 8;  // elements per 16-byte access
    __device__ static f32x4 mma(x8 a, x8 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
    __device__ static _Float16 cvt(float x) { return (_Float16)x; }
};

template <>
struct Tr<__bf16> {
    using x8 = bf16x8;
    using x4 = bf16x4;
    static constexpr int kVec = 8;
    __device__ static f32x4 mma(x8 a, x8 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    __device__ static __bf16 cvt(float x) { return (__bf16)x; }
};

template <>
struct Tr<float> {
    using x8 = f32x8;
    using x4 = f32x4;
    static constexpr int kVec = 4;
    __device__ static f32x4 mma(x8 a, x8 b, f32x4 c) {
#pragma unroll
        for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[j], c, 0, 0, 0);
        return c;
    }
    __device__ static float cvt(float x) { return x; }
};

// 16-byte vector moves (global or LDS); the element type is reinterpreted.
template <typename V>
__device__ __forceinline__ V ld16(const void* p) {
    static_assert(sizeof(V) == 16, "16-byte access");
    return *reinterpret_cast<const V*>(p);
}
template <typename V>
__device__ __forceinline__ void st16(void* p, V v) {
    static_assert(sizeof(V) == 16, "16-byte access");
    *reinterpret_cast<V*>(p) = v;
}

// Eight consecutive elements at p (16-byte aligned) as an A/B fragment.
template <typename T>
__device__ __forceinline__ typename Tr<T>::x8 ld_x8(const T* p) {
    using x8 = typename Tr<T>::x8;
    if constexpr (sizeof(T) == 2) {
        return __builtin_bit_cast(x8, ld16<i32x4>(p));
    } else {
        f32x4 a = ld16<f32x4>(p), b = ld16<f32x4>(p + 4);
        return x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    }
}

// Four consecutive elements at p (8-byte aligned for 16-bit, 16 for fp32).
template <typename T>
__device__ __forceinline__ typename Tr<T>::x4 ld_x4(const T* p) {
    using x4 = typename Tr<T>::x4;
    if constexpr (sizeof(T) == 2) {
        return __builtin_bit_cast(x4, *reinterpret_cast<const i32x2*>(p));
    } else {
        return ld16<f32x4>(p);
    }
}

template <typename T>
__device__ __forceinline__ typename Tr<T>::x8 cat_x4(typename Tr<T>::x4 a, typename Tr<T>::x4 b) {
    return typename Tr<T>::x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

template <typename T>
__device__ __forceinline__ typename Tr<T>::x8 zero_x8() {
    return typename Tr<T>::x8{};
}

// Store four fp32 values rounded to T at p (8 or 16 bytes).
template <typename T>
__device__ __forceinline__ void st_x4(T* p, f32x4 v) {
    if constexpr (sizeof(T) == 2) {
        typename Tr<T>::x4 h = {Tr<T>::cvt(v[0]), Tr<T>::cvt(v[1]), Tr<T>::cvt(v[2]),
                                Tr<T>::cvt(v[3])};
        *reinterpret_cast<i32x2*>(p) = __builtin_bit_cast(i32x2, h);
    } else {
        st16<f32x4>(p, v);
    }
}

// Reductions over the four 16-lane groups holding the same column, with the
// gfx950 lane-swap instructions (VALU, no LDS traffic): permlane16_swap pairs
// groups (0,1) and (2,3), permlane32_swap pairs (0,2) and (1,3).
__device__ __forceinline__ float group_max4(float x) {
    const unsigned u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const unsigned v = __float_as_uint(x);
    const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float group_sum4(float x) {
    const unsigned u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const unsigned v = __float_as_uint(x);
    const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// acc + sum of the 8 probabilities of a P fragment.  16-bit types sum the
// rounded values the matrix product uses, two at a time (v_dot2 with 1.0);
// fp32 sums the values themselves.
template <typename T>
__device__ __forceinline__ float row_sum8(typename Tr<T>::x8 pf, const float (&p)[2][4],
                                          float acc) {
    if constexpr (sizeof(T) == 4) {
        return acc + ((p[0][0] + p[0][1]) + (p[0][2] + p[0][3])) +
               ((p[1][0] + p[1][1]) + (p[1][2] + p[1][3]));
    } else {
        typedef T t2 __attribute__((ext_vector_type(2)));
        const t2 one = {(T)1.0f, (T)1.0f};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const t2 pr = {pf[2 * j], pf[2 * j + 1]};
            if constexpr (std::is_same<T, _Float16>::value)
                acc = __builtin_amdgcn_fdot2(pr, one, acc, false);
            else
                acc = __builtin_amdgcn_fdot2_f32_bf16(pr, one, acc, false);
        }
        return acc;
    }
}

// acc + sum_j a[j] * b[j] over one 8-slot fragment, accumulated in fp32
// (16-bit types: four v_dot2 steps, the products are exact in fp32).
template <typename T>
__device__ __forceinline__ float dot8(typename Tr<T>::x8 a, typename Tr<T>::x8 b, float acc) {
    if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc = fmaf(a[j], b[j], acc);
        return acc;
    } else {
        typedef T t2 __attribute__((ext_vector_type(2)));
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const t2 x = {a[2 * j], a[2 * j + 1]}, y = {b[2 * j], b[2 * j + 1]};
            if constexpr (std::is_same<T, _Float16>::value)
                acc = __builtin_amdgcn_fdot2(x, y, acc, false);
            else
                acc = __builtin_amdgcn_fdot2_f32_bf16(x, y, acc, false);
        }
        return acc;
    }
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Problem geometry shared by all kernels (filled on the host).  Axes beyond
// the problem's rank are inert (extent 1, window 1, dilation 1).
struct Geo {
    int L[kMaxRank], k[kMaxRank], d[kMaxRank];
    int causal[kMaxRank];  // 1: causal axis (window [max(0, p - k + 1), p])
    int ts[kMaxRank];    // token stride of each axis
    int N;               // tokens per (batch, head)
    int BH;              // batch * heads
    int ngroups;         // prod d
    int T[kMaxRank];     // workgroup tile (group coordinates)
    int WT[kMaxRank];    // wave tile
    int WGd[kMaxRank];   // waves per axis (T = WT * WGd)
    int nt[kMaxRank];    // tiles per axis (sized for the longest group)
    int ntiles;          // prod nt
    int nwg;             // workgroups in the grid
    int lgWT[kMaxRank];  // log2 WT (wave tiles are powers of two)
    int lgWGd[kMaxRank]; // log2 WGd
    FastDiv fd_ntiles, fd_ngroups, fd_d[kMaxRank], fd_nt[kMaxRank];
    int bwd_split;       // backward only: run as the split form (chosen on the host)
};

// Brings the Geo fields of the problem's R axes into scalar registers in one
// batch of loads: without it the compiler issues the kernel-argument loads
// lazily, behind the early-exit branches, and the prologue pays one memory
// round trip per group of fields.  The empty asm statement only consumes the
// values (one statement: each volatile asm is a scheduling boundary).
template <int R>
__device__ __forceinline__ void fetch_geo(const Geo& g) {
    constexpr int r1 = R > 1 ? 1 : 0, r2 = R > 2 ? 2 : 0;
    asm volatile("" ::"s"(g.N), "s"(g.ngroups), "s"(g.ntiles), "s"(g.nwg),
                 "s"(g.fd_ntiles.mul), "s"(g.fd_ntiles.shr), "s"(g.fd_ngroups.mul),
                 "s"(g.fd_ngroups.shr),
                 "s"(g.L[0]), "s"(g.k[0]), "s"(g.d[0]), "s"(g.ts[0]), "s"(g.T[0]), "s"(g.nt[0]),
                 "s"(g.lgWT[0]), "s"(g.lgWGd[0]), "s"(g.fd_d[0].mul), "s"(g.fd_d[0].shr),
                 "s"(g.fd_nt[0].mul), "s"(g.fd_nt[0].shr), "s"(g.causal[0]), "s"(g.causal[r1]),
                 "s"(g.causal[r2]),
                 "s"(g.L[r1]), "s"(g.k[r1]), "s"(g.d[r1]), "s"(g.ts[r1]), "s"(g.T[r1]),
                 "s"(g.nt[r1]), "s"(g.lgWT[r1]), "s"(g.lgWGd[r1]), "s"(g.fd_d[r1].mul),
                 "s"(g.fd_d[r1].shr), "s"(g.fd_nt[r1].mul), "s"(g.fd_nt[r1].shr),
                 "s"(g.L[r2]), "s"(g.k[r2]), "s"(g.d[r2]), "s"(g.ts[r2]), "s"(g.T[r2]),
                 "s"(g.nt[r2]), "s"(g.lgWT[r2]), "s"(g.lgWGd[r2]), "s"(g.fd_d[r2].mul),
                 "s"(g.fd_d[r2].shr), "s"(g.fd_nt[r2].mul), "s"(g.fd_nt[r2].shr));
}

// Workgroup -> (batch*head, dilation group coordinates, tile coordinates) and
// the length of this group along every axis.
template <int R>
__device__ __forceinline__ void decode_workgroup(const Geo& g, int bid, int& bh, int* gc, int* tc,
                                                 int* n) {
    const int rest = g.fd_ntiles.div(bid);
    int tile = bid - rest * g.ntiles;
    bh = g.fd_ngroups.div(rest);
    int gidx = rest - bh * g.ngroups;
#pragma unroll
    for (int a = R - 1; a >= 0; --a) {
        const int gq = g.fd_d[a].div(gidx);
        gc[a] = gidx - gq * g.d[a];
        gidx = gq;
        const int tq = g.fd_nt[a].div(tile);
        tc[a] = tile - tq * g.nt[a];
        tile = tq;
        n[a] = g.fd_d[a].div(g.L[a] - gc[a] + g.d[a] - 1);
    }
}

// Row-major unravel of idx over power-of-two extents 2^lg[a].
template <int R>
__device__ __forceinline__ void unravel_pow2(int idx, const int* lg, int* c) {
#pragma unroll
    for (int a = R - 1; a >= 0; --a) {
        c[a] = idx & ((1 << lg[a]) - 1);
        idx >>= lg[a];
    }
}

// Workgroups are dispatched round-robin over the 8 XCDs; renumber them so
// that each XCD receives a contiguous run of logical tiles (neighbouring tiles
// share halo rows in that XCD's L2).
__device__ __forceinline__ int xcd_remap(int bid, int nwg) {
    const int q = nwg >> 3, r = nwg & 7;
    const int x = bid & 7, slot = bid >> 3;
    return x * q + (x < r ? x : r) + slot;
}

template <int R>
__device__ __forceinline__ void unravel(int idx, const int* ext, int* c) {
#pragma unroll
    for (int a = R - 1; a >= 0; --a) {
        c[a] = idx % ext[a];
        idx /= ext[a];
    }
}

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

}  // namespace na
