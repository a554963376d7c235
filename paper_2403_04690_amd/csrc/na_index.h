// na_index.h -- neighbourhood index math used by every kernel of the library.
//
// Neighborhood attention (Sec. 1-2 of Faster Neighborhood Attention) gives each
// query the k nearest tokens of its own dilation group along an axis; the
// window is centred where possible and shifted at borders so its size never
// changes.  Dilation d partitions an axis of length L into d groups
// (x mod d), each an independent problem over n = ceil((L - g) / d) tokens
// (Sec. 3.4).  All functions below work in group coordinates p = x / d.
#pragma once

#if defined(__HIPCC__)
#define NA_HD __host__ __device__ __forceinline__
#else
#define NA_HD inline
#endif

namespace na {

// Tokens in dilation group g of an axis of length L.
NA_HD int group_len(int L, int d, int g) { return (L - g + d - 1) / d; }

// First window position of the query at group position p (group of n tokens,
// window k): the window is [win_start, win_start + k).
NA_HD int win_start(int p, int n, int k) {
    int s = p - k / 2;
    s = s < 0 ? 0 : s;
    return s > n - k ? n - k : s;
}

// Inverse neighbourhood of key position j (Sec. 3.1, operator IN): the
// queries whose window contains j form the contiguous range [inv_lo, inv_hi],
// because win_start is non-decreasing in p.
NA_HD int inv_lo(int j, int n, int k) { return j <= k - 1 ? 0 : j - k + 1 + k / 2; }
NA_HD int inv_hi(int j, int n, int k) { return j >= n - k ? n - 1 : j + k / 2; }

}  // namespace na
