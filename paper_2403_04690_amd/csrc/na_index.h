// na_index.h -- neighbourhood index math used by every kernel of the library.
//
// Neighborhood attention (Sec. 1-2 of Faster Neighborhood Attention) gives each
// query the k nearest tokens of its own dilation group along an axis; the
// window is centred where possible and shifted at borders so its size never
// changes.  Dilation d partitions an axis of length L into d groups
// (x mod d), each an independent problem over n = ceil((L - g) / d) tokens
// (Sec. 3.4).  Along a causal axis (Sec. 3.4) a query never attends to a token
// of larger coordinate: its window is the k nearest positions not after it,
// [max(0, p - k + 1), p], shorter than k for the first k - 1 positions.  All
// functions below work in group coordinates p = x / d.
#pragma once

#if defined(__HIPCC__)
#define NA_HD __host__ __device__ __forceinline__
#else
#define NA_HD inline
#endif

namespace na {

// Tokens in dilation group g of an axis of length L.
NA_HD int group_len(int L, int d, int g) { return (L - g + d - 1) / d; }

// First and last (inclusive) window positions of the query at group position
// p (group of n tokens, window k, causal axis or not).
// Both forms are one clamp, min(max(p - h, 0), n - k), with h = k - 1 on a
// causal axis and k / 2 otherwise (a causal start p - k + 1 never exceeds
// n - k, as p <= n - 1); written without branches.
NA_HD int win_half(int k, bool causal) { return causal ? k - 1 : k >> 1; }
NA_HD int win_start(int p, int n, int k, bool causal) {
    const int s = p - win_half(k, causal);
    const int c = s < 0 ? 0 : s;
    return c > n - k ? n - k : c;
}
NA_HD int win_last(int p, int n, int k, bool causal) {
    const int e = win_start(p, n, k, causal) + k - 1;
    return causal ? p : e;
}

// Start of the window as the kernels' mask tests use it, (unsigned)(j - s) < k:
// along a causal axis the unclamped p - k + 1, which with j >= 0 admits exactly
// the positions max(0, p - k + 1) .. p.
NA_HD int mask_start(int p, int n, int k, bool causal) {
    const int s = p - win_half(k, causal);
    const int c = s < 0 && !causal ? 0 : s;
    return c > n - k ? n - k : c;
}

// Inverse neighbourhood of key position j (Sec. 3.1, operator IN): the
// queries whose window contains j form the contiguous range [inv_lo, inv_hi],
// because window starts and ends are non-decreasing in p.
NA_HD int inv_lo(int j, int n, int k, bool causal) {
    if (causal) return j;
    return j <= k - 1 ? 0 : j - k + 1 + k / 2;
}
NA_HD int inv_hi(int j, int n, int k, bool causal) {
    if (causal) return j + k - 1 < n - 1 ? j + k - 1 : n - 1;
    return j >= n - k ? n - 1 : j + k / 2;
}

}  // namespace na
