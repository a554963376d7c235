// na_api.cpp -- the C ABI of libna.so: problem validation, tile selection and
// kernel dispatch.  Everything before the launch is plain host code; no entry
// point allocates, frees or synchronises.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>

#include "na.h"
#include "na_launch.h"

namespace {

constexpr int kVersion = 200;  // 0.2.0

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int ilog2(int x) {  // x is a power of two
    int l = 0;
    while ((1 << l) < x) ++l;
    return l;
}

int pow2ceil(int x) {
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}

// Tokens per (batch, head), or -1 if it does not fit the 32-bit token index.
int64_t token_count(int rank, const int64_t* extents) {
    int64_t n = 1;
    for (int a = 0; a < rank; ++a) {
        n *= extents[a];
        if (n >= (int64_t(1) << 31)) return -1;
    }
    return n;
}

// Wave tile (queries or keys owned by one wave, 16 * m of them) along each
// axis, sized from the innermost axis outwards and never longer than the
// longest dilation group of an axis (rounded up to a power of two).
void wave_tile(int rank, const int* glen, int m, int waves, int* wt, int* wgd) {
    const int q = 16 * m;
    for (int a = 0; a < 3; ++a) wt[a] = wgd[a] = 1;
    if (rank == 1) {
        wt[0] = q;
        wgd[0] = waves;
        return;
    }
    const int inner = rank - 1;
    const int cap = rank == 2 ? (m == 1 ? 8 : 16) : 8;
    wt[inner] = std::min(cap, pow2ceil(glen[inner]));
    int rem = q / wt[inner];
    // hand out the remaining factor 2 at a time over the outer axes, outermost first
    int a = 0;
    while (rem > 1) {
        bool placed = false;
        for (int t = 0; t < inner && rem > 1; ++t) {
            const int ax = (a + t) % inner;
            if (wt[ax] < pow2ceil(glen[ax]) || t == inner - 1) {
                wt[ax] *= 2;
                rem /= 2;
                a = (ax + 1) % inner;
                placed = true;
                break;
            }
        }
        if (!placed) {
            wt[0] *= rem;
            rem = 1;
        }
    }
    if (rank == 2) {
        wgd[0] = 4;
    } else {
        wgd[0] = 2;
        wgd[1] = 2;
    }
}

// Fills the geometry of a problem for wave tiles of 16 * m tokens.
bool make_geo(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
              const int32_t* causal, int64_t BH, int m, na::Geo& g, int waves = 4) {
    std::memset(&g, 0, sizeof(g));
    int glen[3] = {1, 1, 1};
    for (int a = 0; a < 3; ++a) {
        g.L[a] = a < rank ? (int)extents[a] : 1;
        g.k[a] = a < rank ? ks[a] : 1;
        g.d[a] = a < rank ? ds[a] : 1;
        g.causal[a] = a < rank && causal && causal[a] ? 1 : 0;
        glen[a] = na::group_len(g.L[a], g.d[a], 0);
    }
    {
        int s = 1;  // token strides of the problem's own axes (row-major)
        for (int a = rank - 1; a >= 0; --a) {
            g.ts[a] = s;
            s *= g.L[a];
        }
        for (int a = rank; a < 3; ++a) g.ts[a] = 0;
    }
    g.N = (int)token_count(rank, extents);
    g.BH = (int)BH;
    g.ngroups = 1;
    for (int a = 0; a < rank; ++a) g.ngroups *= g.d[a];
    wave_tile(rank, glen, m, rank == 1 ? waves : 4, g.WT, g.WGd);
    int64_t ntiles = 1;
    for (int a = 0; a < 3; ++a) {
        g.T[a] = g.WT[a] * g.WGd[a];
        g.nt[a] = a < rank ? (glen[a] + g.T[a] - 1) / g.T[a] : 1;
        ntiles *= g.nt[a];
    }
    const int64_t nwg = ntiles * g.ngroups * BH;
    if (nwg >= (int64_t(1) << 31)) return false;
    g.ntiles = (int)ntiles;
    g.nwg = (int)nwg;
    for (int a = 0; a < 3; ++a) {
        g.lgWT[a] = ilog2(g.WT[a]);
        g.lgWGd[a] = ilog2(g.WGd[a]);
        g.fd_d[a].init(g.d[a]);
        g.fd_nt[a].init(g.nt[a]);
    }
    g.fd_ntiles.init(g.ntiles);
    g.fd_ngroups.init(g.ngroups);
    return true;
}

// Wave size multiplier: two 16-token blocks per wave unless that leaves the
// GPU (256 CUs) with too few workgroups.  NA_WAVE_BLOCKS=1|2 overrides.
int choose_m(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds, int64_t BH) {
    if (const char* env = std::getenv("NA_WAVE_BLOCKS")) {
        const int v = std::atoi(env);
        if (v == 1 || v == 2) return v;
    }
    na::Geo g;
    if (!make_geo(rank, extents, ks, ds, nullptr, BH, 2, g)) return 1;
    return g.nwg < 1024 ? 1 : 2;
}

// Forward workgroup size: 1-D problems of 16-bit types with plenty of
// 4-wave workgroups run 8-wave ones instead (each stage of K/V rows then
// serves twice the queries).  NA_FWD_WAVES=4|8 overrides.
int forward_waves(int rank, na_dtype dtype, const na::Geo& g4) {
    if (rank != 1 || dtype == NA_FP32) return 4;
    if (const char* env = std::getenv("NA_FWD_WAVES")) {
        const int v = std::atoi(env);
        if (v == 4 || v == 8) return v;
    }
    return g4.nwg >= 2048 ? 8 : 4;
}

na_status check_problem(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
                        int64_t batch, int64_t heads, int64_t head_dim, na_dtype dtype,
                        float scale) {
    if (rank < 1 || rank > 3) return NA_ERR_RANK;
    if (!extents || !ks || !ds) return NA_ERR_NULL;
    for (int a = 0; a < rank; ++a) {
        if (extents[a] < 1) return NA_ERR_SHAPE;
        if (ks[a] < 1) return NA_ERR_KERNEL_SIZE;
        if (ds[a] < 1) return NA_ERR_DILATION;
        if ((int64_t)ks[a] * (int64_t)ds[a] > extents[a]) return NA_ERR_WINDOW_EXCEEDS_EXTENT;
    }
    if (batch < 0 || heads < 0) return NA_ERR_SHAPE;
    if (head_dim != 32 && head_dim != 64 && head_dim != 128) return NA_ERR_HEAD_DIM;
    if (dtype != NA_FP32 && dtype != NA_FP16 && dtype != NA_BF16) return NA_ERR_DTYPE;
    if (!std::isfinite(scale)) return NA_ERR_SCALE;
    const int64_t N = token_count(rank, extents);
    if (N < 0 || N * head_dim >= (int64_t(1) << 31)) return NA_ERR_SHAPE;
    if (batch * heads >= (int64_t(1) << 31)) return NA_ERR_SHAPE;
    return NA_OK;
}

bool empty_problem(int rank, const int64_t* extents, int64_t batch, int64_t heads) {
    return batch == 0 || heads == 0 || token_count(rank, extents) == 0;
}

}  // namespace

extern "C" {

const char* na_status_string(na_status status) {
    switch (status) {
        case NA_OK: return "ok";
        case NA_ERR_NULL: return "a required pointer is NULL";
        case NA_ERR_RANK: return "rank must be 1, 2 or 3";
        case NA_ERR_SHAPE: return "invalid extents, batch or heads, or problem too large";
        case NA_ERR_KERNEL_SIZE: return "kernel_size must be >= 1 on every axis";
        case NA_ERR_DILATION: return "dilation must be >= 1 on every axis";
        case NA_ERR_WINDOW_EXCEEDS_EXTENT: return "kernel_size * dilation exceeds the extent";
        case NA_ERR_HEAD_DIM: return "head_dim must be 32, 64 or 128";
        case NA_ERR_DTYPE: return "unknown dtype";
        case NA_ERR_ALIGNMENT: return "device pointers must be 16-byte aligned";
        case NA_ERR_HIP: return "HIP launch failed";
        case NA_ERR_SCALE: return "scale must be finite";
    }
    return "unknown status";
}

int na_version(void) { return kVersion; }

na_status na_validate(int rank, const int64_t* extents, const int32_t* kernel_size,
                      const int32_t* dilation, const int32_t* causal, int64_t batch, int64_t heads,
                      int64_t head_dim, na_dtype dtype, float scale) {
    (void)causal;  // any value is legal (NULL: no causal axis)
    return check_problem(rank, extents, kernel_size, dilation, batch, heads, head_dim, dtype,
                         scale);
}

na_status na_forward(int rank, const int64_t* extents, const int32_t* kernel_size,
                     const int32_t* dilation, const int32_t* causal, int64_t batch, int64_t heads,
                     int64_t head_dim, na_dtype dtype, float scale, const void* q, const void* k,
                     const void* v, void* out, float* logsumexp, na_stream_t stream) {
    na_status st = check_problem(rank, extents, kernel_size, dilation, batch, heads, head_dim,
                                 dtype, scale);
    if (st != NA_OK) return st;
    if (empty_problem(rank, extents, batch, heads)) return NA_OK;
    if (!q || !k || !v || !out || !logsumexp) return NA_ERR_NULL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) ||
        !aligned16(logsumexp))
        return NA_ERR_ALIGNMENT;
    const int64_t BH = batch * heads;
    const int m = choose_m(rank, extents, kernel_size, dilation, BH);
    na::Geo g;
    if (!make_geo(rank, extents, kernel_size, dilation, causal, BH, m, g)) return NA_ERR_SHAPE;
    if (forward_waves(rank, dtype, g) == 8 &&
        !make_geo(rank, extents, kernel_size, dilation, causal, BH, m, g, 8))
        return NA_ERR_SHAPE;
    hipError_t e = na::launch_forward(g, rank, (int)head_dim, (int)dtype, m, q, k, v, out,
                                      logsumexp, scale, reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? NA_OK : NA_ERR_HIP;
}

na_status na_backward(int rank, const int64_t* extents, const int32_t* kernel_size,
                      const int32_t* dilation, const int32_t* causal, int64_t batch, int64_t heads,
                      int64_t head_dim, na_dtype dtype, float scale, const void* q, const void* k,
                      const void* v, const void* out, const float* logsumexp, const void* dout,
                      void* dq, void* dk, void* dv, na_stream_t stream) {
    na_status st = check_problem(rank, extents, kernel_size, dilation, batch, heads, head_dim,
                                 dtype, scale);
    if (st != NA_OK) return st;
    if (empty_problem(rank, extents, batch, heads)) return NA_OK;
    if (!q || !k || !v || !out || !logsumexp || !dout || !dq || !dk || !dv) return NA_ERR_NULL;
    const void* ptrs[] = {q, k, v, out, logsumexp, dout, dq, dk, dv};
    for (const void* p : ptrs)
        if (!aligned16(p)) return NA_ERR_ALIGNMENT;
    const int64_t BH = batch * heads;
    const int m = choose_m(rank, extents, kernel_size, dilation, BH);
    na::Geo g;
    if (!make_geo(rank, extents, kernel_size, dilation, causal, BH, m, g)) return NA_ERR_SHAPE;
    hipError_t e = na::launch_backward(g, rank, (int)head_dim, (int)dtype, m, q, k, v, out,
                                       logsumexp, dout, dq, dk, dv, scale,
                                       reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? NA_OK : NA_ERR_HIP;
}

na_status na_debug_windows(int rank, const int64_t* extents, const int32_t* kernel_size,
                           const int32_t* dilation, const int32_t* causal, int32_t* start,
                           int32_t* inv_lo, int32_t* inv_hi, na_stream_t stream) {
    na_status st = check_problem(rank, extents, kernel_size, dilation, 1, 1, 32, NA_FP16, 1.0f);
    if (st != NA_OK) return st;
    if (!start || !inv_lo || !inv_hi) return NA_ERR_NULL;
    int L[3], ks[3], ds[3], cs[3];
    for (int a = 0; a < rank; ++a) {
        L[a] = (int)extents[a];
        ks[a] = kernel_size[a];
        ds[a] = dilation[a];
        cs[a] = causal && causal[a] ? 1 : 0;
    }
    hipError_t e = na::launch_debug_windows(rank, L, ks, ds, cs, start, inv_lo, inv_hi,
                                            reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? NA_OK : NA_ERR_HIP;
}

}  // extern "C"
