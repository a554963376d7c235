// na_stage.h -- global -> register -> LDS staging of token rows, and the
// halo geometry those rows come from.
#pragma once

#include "na_common.h"

namespace na {

// A box of tokens in group coordinates, [lo, lo + E) per axis, cut into rows
// along the innermost axis and each row into 16-token blocks (rows are padded
// to a multiple of 16; padding tokens are zero-filled and always masked).
template <int R>
struct Box {
    int lo[kMaxRank];
    int E[kMaxRank];
    int nbr;  // blocks per row
    int nb;   // total blocks
    FastDiv fd_nbr;
    FastDiv fd_E[kMaxRank];

    __device__ __forceinline__ void finish() {
        nbr = (E[R - 1] + 15) >> 4;
        nb = nbr;
#pragma unroll
        for (int a = 0; a < R - 1; ++a) nb *= E[a];
        fd_nbr.init(nbr);
#pragma unroll
        for (int a = 1; a < R - 1; ++a) fd_E[a].init(E[a]);
    }

    // Outer coordinates (relative to lo) and first inner coordinate of block b.
    __device__ __forceinline__ void block_coords(int b, int* oc, int& inner0) const {
        int row = fd_nbr.div(b);
        inner0 = (b - row * nbr) * 16;
#pragma unroll
        for (int a = R - 2; a >= 1; --a) {
            const int nx = fd_E[a].div(row);
            oc[a] = row - nx * E[a];
            row = nx;
        }
        if (R >= 2) oc[0] = row;
    }

    // Token (within the (batch, head) slice) of token j0 of block b, and how
    // many of the tokens j0 .. j0+3 exist (0 for blocks past the end).
    // Consecutive tokens of a block are g.d[R-1] tokens apart.
    __device__ __forceinline__ int quad_token(const Geo& g, const int* gc, int b, int j0,
                                              int& cnt) const {
        int oc[kMaxRank];
        int inner0;
        block_coords(b, oc, inner0);
        oc[R - 1] = inner0 + j0;
        const int left = E[R - 1] - oc[R - 1];
        cnt = b < nb ? (left < 0 ? 0 : (left > 4 ? 4 : left)) : 0;
        int tok = 0;
#pragma unroll
        for (int a = 0; a < R; ++a) tok += (gc[a] + g.d[a] * (lo[a] + oc[a])) * g.ts[a];
        return tok;
    }
};

// Per-wave block tests against a box of the other side: a block is relevant
// when it intersects [lo, hi) on every axis, and full when it lies inside
// [flo, fhi) on every axis (all its pairs with the wave's tokens are valid).
template <int R>
struct WaveRange {
    int lo[kMaxRank], hi[kMaxRank], flo[kMaxRank], fhi[kMaxRank];

    __device__ __forceinline__ void test(const Box<R>& box, int b, int* oc, int& inner0, bool& rel,
                                         bool& full) const {
        box.block_coords(b, oc, inner0);
        bool r_ = b < box.nb, f_ = b < box.nb;
#pragma unroll
        for (int a = 0; a < R - 1; ++a) {
            r_ = r_ && oc[a] >= lo[a] && oc[a] < hi[a];
            f_ = f_ && oc[a] >= flo[a] && oc[a] < fhi[a];
        }
        r_ = r_ && inner0 < hi[R - 1] && inner0 + 16 > lo[R - 1];
        f_ = f_ && inner0 >= flo[R - 1] && inner0 + 16 <= fhi[R - 1];
        rel = r_;
        full = f_;
    }
};

// Stages ROWS token rows of D elements.  Each thread item is 4 consecutive
// rows (of one 16-row block) x one 16-byte segment, loaded with 16-byte
// global loads; rows can then be written row-major (dst[row][d]) and/or
// transposed (dst[d][row]).  Several stagers of the same shape share one
// set of item addresses (QuadAddr).
template <int ROWS, int SEGS, int NT>
struct QuadAddr {
    static constexpr int kQuads = ROWS / 4;
    static constexpr int kItems = (kQuads * SEGS + NT - 1) / NT;
    int tok[kItems];  // token of the item's first row
    int cnt[kItems];  // rows of the item that exist (0..4)

    template <class QuadTok>
    __device__ __forceinline__ void compute(int tid, QuadTok quad_tok) {
#pragma unroll
        for (int it = 0; it < kItems; ++it) {
            const int i = tid + it * NT;
            cnt[it] = 0;
            tok[it] = 0;
            if (i < kQuads * SEGS) {
                const int quad = i / SEGS;
                const int t = quad_tok(quad, cnt[it]);
                tok[it] = cnt[it] > 0 ? t : 0;  // token 0 is a safe dummy address
            }
        }
    }
};

template <typename T, int D, int ROWS, int NT>
struct Stager {
    static constexpr int kVec = Tr<T>::kVec;
    static constexpr int kSegs = D / kVec;
    static constexpr int kQuads = ROWS / 4;
    using Addr = QuadAddr<ROWS, kSegs, NT>;
    static constexpr int kItems = Addr::kItems;
    i32x4 r[kItems][4];

    // tstep: token distance between consecutive rows of a quad
    __device__ __forceinline__ void load(const T* base, int tid, const Addr& ad, int tstep) {
#pragma unroll
        for (int it = 0; it < kItems; ++it) {
            const int i = tid + it * NT;
            const int seg = i % kSegs;
            const T* p = base + (size_t)ad.tok[it] * D + seg * kVec;
            // branch-free: absent rows re-read the first row and are zeroed
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                const bool ok = rr < ad.cnt[it];
                const i32x4 v = ld16<i32x4>(p + (ok ? (size_t)(rr * tstep) * D : 0));
                r[it][rr] = ok ? v : i32x4{0, 0, 0, 0};
            }
        }
    }

    __device__ __forceinline__ void store_rows(T* dst, int row_stride, int tid) const {
#pragma unroll
        for (int it = 0; it < kItems; ++it) {
            const int i = tid + it * NT;
            if (i < kQuads * kSegs) {
                const int quad = i / kSegs, seg = i - quad * kSegs;
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    st16<i32x4>(dst + (quad * 4 + rr) * row_stride + seg * kVec, r[it][rr]);
            }
        }
    }

    __device__ __forceinline__ void store_cols(T* dst, int col_stride, int tid) const {
#pragma unroll
        for (int it = 0; it < kItems; ++it) {
            const int i = tid + it * NT;
            if (i < kQuads * kSegs) {
                const int quad = i / kSegs, seg = i - quad * kSegs;
                T* d0 = dst + (seg * kVec) * col_stride + quad * 4;
                if constexpr (sizeof(T) == 2) {
                    // 4 rows x 8 elements -> 8 lines of 4 rows (16-bit pair transpose)
#pragma unroll
                    for (int w = 0; w < 4; ++w) {
                        const uint32_t a0 = r[it][0][w], a1 = r[it][1][w];
                        const uint32_t a2 = r[it][2][w], a3 = r[it][3][w];
                        const i32x2 lo = {(int)((a0 & 0xffffu) | (a1 << 16)),
                                          (int)((a2 & 0xffffu) | (a3 << 16))};
                        const i32x2 hi = {(int)((a0 >> 16) | (a1 & 0xffff0000u)),
                                          (int)((a2 >> 16) | (a3 & 0xffff0000u))};
                        *reinterpret_cast<i32x2*>(d0 + (2 * w) * col_stride) = lo;
                        *reinterpret_cast<i32x2*>(d0 + (2 * w + 1) * col_stride) = hi;
                    }
                } else {
#pragma unroll
                    for (int w = 0; w < 4; ++w) {
                        const i32x4 t = {r[it][0][w], r[it][1][w], r[it][2][w], r[it][3][w]};
                        st16<i32x4>(d0 + w * col_stride, t);
                    }
                }
            }
        }
    }
};

// Row-wise dot products of two stagers loaded from the same addresses, in
// fp32: the kSegs lanes that hold one quad's segments reduce their partial
// sums with lane shuffles (a fixed order, so the result is deterministic)
// and the lane of segment 0 writes the quad's 4 sums to dst[4 * quad ...].
// Absent rows were zero-filled by load() and give 0.
template <typename T, int D, int ROWS, int NT>
__device__ __forceinline__ void store_row_dots(const Stager<T, D, ROWS, NT>& a,
                                               const Stager<T, D, ROWS, NT>& b, float* dst,
                                               int tid) {
    using S = Stager<T, D, ROWS, NT>;
    using x8 = typename Tr<T>::x8;
    static_assert(kWave % S::kSegs == 0 && NT % S::kSegs == 0, "a quad's segments share a wave");
#pragma unroll
    for (int it = 0; it < S::kItems; ++it) {
        const int i = tid + it * NT;
        float s[4];
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
            if constexpr (sizeof(T) == 2) {
                s[rr] = dot8<T>(__builtin_bit_cast(x8, a.r[it][rr]),
                                __builtin_bit_cast(x8, b.r[it][rr]), 0.f);
            } else {
                const f32x4 x = __builtin_bit_cast(f32x4, a.r[it][rr]);
                const f32x4 y = __builtin_bit_cast(f32x4, b.r[it][rr]);
                s[rr] = fmaf(x[3], y[3], fmaf(x[2], y[2], fmaf(x[1], y[1], x[0] * y[0])));
            }
        }
#pragma unroll
        for (int w = 1; w < S::kSegs; w <<= 1)
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) s[rr] += __shfl_xor(s[rr], w, kWave);
        if (i < S::kQuads * S::kSegs && i % S::kSegs == 0)
            st16<f32x4>(dst + (i / S::kSegs) * 4, f32x4{s[0], s[1], s[2], s[3]});
    }
}

// LDS row strides: row-major rows get a 16-byte pad, transposed lines a
// 4-element pad (keeps 16-byte alignment for fp32 and 8-byte for 16-bit).
template <typename T, int D>
struct RowLayout {
    static constexpr int kRow = D + Tr<T>::kVec;
};
template <int ROWS>
struct ColLayout {
    static constexpr int kCol = ROWS + 4;
};

}  // namespace na
