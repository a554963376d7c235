// na_api.cpp -- the C ABI of libna.so: problem validation, tile selection,
// the tiling tuner and kernel dispatch.  Everything before the launch is plain
// host code; no entry point allocates or frees device memory, and only
// na_tune synchronises.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <atomic>
#include <map>
#include <mutex>
#include <vector>

#include "na.h"
#include "na_launch.h"

namespace {

constexpr int kVersion = 400;  // 0.4.0

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// A C caller may pass any int where the interface declares an enum, while C++
// allows an enum object only the values of its enumerators' bit range.  Enum
// arguments are therefore handed on by reference until they are validated, and
// read through their bytes, so that an out-of-range value is rejected as such.
template <class E>
int enum_bits(const E& e) {
    static_assert(sizeof(E) == sizeof(int), "C enums are int-sized here");
    int v;
    std::memcpy(&v, &e, sizeof v);
    return v;
}

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

// Longest dilation group along each axis (inert axes: 1).
void group_lengths(int rank, const int64_t* extents, const int32_t* ds, int* glen) {
    for (int a = 0; a < 3; ++a)
        glen[a] = a < rank ? na::group_len((int)extents[a], ds[a], 0) : 1;
}

// Threads in the x dimension of a launch must stay below 2^32.  The forward
// runs nwg workgroups of 64 * (waves per workgroup) threads; the backward runs
// nwk + nwg workgroups of 256 threads, nwk being nwg rounded up to a multiple
// of the 8 XCDs.
bool grid_fits(int64_t nwg, const na_tiling& t, bool forward) {
    const int64_t limit = int64_t(1) << 32;
    if (forward) {
        const int64_t waves = int64_t(t.waves[0]) * t.waves[1] * t.waves[2];
        return nwg * waves * 64 < limit;
    }
    return (((nwg + 7) & ~int64_t(7)) + nwg) * 256 < limit;
}

// Fills the geometry of a problem for a tiling (validated by the caller);
// false if the launch it needs would be too large (grid_fits).
bool geo_from_tiling(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
                     const int32_t* causal, int64_t BH, const na_tiling& t, na::Geo& g,
                     bool forward) {
    std::memset(&g, 0, sizeof(g));
    int glen[3];
    group_lengths(rank, extents, ds, glen);
    for (int a = 0; a < 3; ++a) {
        g.L[a] = a < rank ? (int)extents[a] : 1;
        g.k[a] = a < rank ? ks[a] : 1;
        g.d[a] = a < rank ? ds[a] : 1;
        g.causal[a] = a < rank && causal && causal[a] ? 1 : 0;
        g.WT[a] = t.wave_tile[a];
        g.WGd[a] = t.waves[a];
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
    int64_t ntiles = 1;
    for (int a = 0; a < 3; ++a) {
        g.T[a] = g.WT[a] * g.WGd[a];
        g.nt[a] = a < rank ? (glen[a] + g.T[a] - 1) / g.T[a] : 1;
        ntiles *= g.nt[a];
    }
    const int64_t nwg = ntiles * g.ngroups * BH;
    if (!grid_fits(nwg, t, forward)) return false;
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

na_status check_problem(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
                        int64_t batch, int64_t heads, int64_t head_dim, const na_dtype& dtype,
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
    const int dt = enum_bits(dtype);
    if (dt != NA_FP32 && dt != NA_FP16 && dt != NA_BF16) return NA_ERR_DTYPE;
    if (!std::isfinite(scale)) return NA_ERR_SCALE;
    const int64_t N = token_count(rank, extents);
    if (N < 0 || N * head_dim >= (int64_t(1) << 31)) return NA_ERR_SHAPE;
    if (batch * heads >= (int64_t(1) << 31)) return NA_ERR_SHAPE;
    return NA_OK;
}

bool empty_problem(int rank, const int64_t* extents, int64_t batch, int64_t heads) {
    return batch == 0 || heads == 0 || token_count(rank, extents) == 0;
}

bool is_pow2(int x) { return x >= 1 && (x & (x - 1)) == 0; }

// A tiling the kernels accept for this problem (see na_tiling).
bool valid_tiling(int rank, na_dtype dtype, bool forward, const na_tiling& t) {
    if (t.blocks_per_wave != 1 && t.blocks_per_wave != 2) return false;
    int64_t pw = 1, pg = 1;
    for (int a = 0; a < 3; ++a) {
        const int wt = t.wave_tile[a], wg = t.waves[a];
        if (!is_pow2(wt) || !is_pow2(wg) || wt > 4096) return false;
        if (a >= rank && (wt != 1 || wg != 1)) return false;
        pw *= wt;
        pg *= wg;
    }
    if (pw != 16 * t.blocks_per_wave) return false;
    if (pg == 4) return true;
    // 8 waves: the 1-D forward of 16-bit types only
    return pg == 8 && forward && rank == 1 && dtype != NA_FP32;
}

int env_choice(const char* name, int a, int b) {
    if (const char* env = std::getenv(name)) {
        const int v = std::atoi(env);
        if (v == a || v == b) return v;
    }
    return 0;
}

// The heuristic tiling: the wave tile of 16 * m queries that multiplies each
// query with the fewest keys.  Along each outer axis a wave visits
// h + k - 1 halo rows, and along the inner axis ceil((w + k - 1) / 16)
// 16-key blocks (group coordinates, clipped to the group).  Two weights for
// what else a key costs: two blocks per wave share every K/V fragment read
// (x 0.85, and x 0.8 in 1-D), and a 4-wide inner tile spreads a 16-query
// block over four rows (x 1.25).  Partly filled waves count per useful query.
//
// m = 2 only where that still leaves 1024 workgroups, and neither for fp32
// nor in the backward at head dim 128: those two-block kernels hold half the
// waves per SIMD of the one-block ones, or fewer (one-block tilings were
// 18-31 % faster wherever measured).
// Workgroups are 4 waves along the outermost axis (1-D, 2-D) or 2 x 2 over
// the two outer axes (3-D).  The 1-D forward of a 16-bit type with a window
// of at least 512 keys and 2048 such workgroups runs 8-wave workgroups
// instead: each stage of K/V rows then serves twice the queries.  With
// smaller windows the larger halo stage costs more than it saves (up to
// +38 % at 63 keys).  NA_WAVE_BLOCKS=1|2 and NA_FWD_WAVES=4|8 force m and
// the workgroup size.
//
// The weights come from timing every candidate tiling (na_tune, or all five
// 2-D wave tiles of both m) on 1-D windows of 7 to 1023 keys, 2-D windows
// of 5 to 31 and 3-D windows of 3 x 7 x 7 to 7 x 7 x 7.  In the forward the
// choice is the fastest measured, or within 2 % of it, in every case.
na_tiling model_tiling(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
                       int64_t BH, int64_t head_dim, na_dtype dtype, bool forward) {
    int glen[3];
    group_lengths(rank, extents, ds, glen);
    const int inner = rank - 1;
    const int forced = env_choice("NA_WAVE_BLOCKS", 1, 2);
    na_tiling best{};
    double best_cost = 0.0;
    bool have = false;
    for (int m = 1; m <= 2; ++m) {
        if (forced && m != forced) continue;
        if (!forced && m == 2 && (dtype == NA_FP32 || (!forward && head_dim == 128))) continue;
        for (int w = rank == 1 ? 16 * m : 4; w <= (rank == 1 ? 16 * m : 16); w *= 2) {
            const int outer = 16 * m / w;  // product of the outer wave-tile lengths
            for (int t0 = 1; t0 <= (rank == 3 ? outer : 1); t0 *= 2) {
                na_tiling t;
                t.blocks_per_wave = m;
                for (int a = 0; a < 3; ++a) t.wave_tile[a] = t.waves[a] = 1;
                t.wave_tile[inner] = w;
                if (rank == 2) {
                    t.wave_tile[0] = outer;
                } else if (rank == 3) {
                    t.wave_tile[0] = t0;
                    t.wave_tile[1] = outer / t0;
                }
                if (rank == 3)
                    t.waves[0] = t.waves[1] = 2;
                else
                    t.waves[0] = 4;
                bool fits = rank == 1 || w == 4 || w <= pow2ceil(glen[inner]);
                for (int a = 0; a < inner; ++a) fits = fits && t.wave_tile[a] <= pow2ceil(glen[a]);
                if (!fits) continue;
                if (m == 2 && !forced) {
                    na::Geo g;
                    if (!geo_from_tiling(rank, extents, ks, ds, nullptr, BH, t, g, forward) ||
                        g.nwg < 1024)
                        continue;
                }
                double keys = 16.0 * ((std::min(w + ks[inner] - 1, glen[inner]) + 15) / 16);
                double useful = std::min(w, glen[inner]);
                for (int a = 0; a < inner; ++a) {
                    keys *= std::min(t.wave_tile[a] + ks[a] - 1, glen[a]);
                    useful *= std::min(t.wave_tile[a], glen[a]);
                }
                const double share = rank == 1 ? 0.8 : 0.85;
                const double cost = keys * (m == 2 ? share : 1.0) *
                                    (rank > 1 && w == 4 ? 1.25 : 1.0) * (16.0 * m / useful);
                if (!have || cost < best_cost) {
                    best = t;
                    best_cost = cost;
                    have = true;
                }
            }
        }
    }
    if (!have) {  // no wave tile fits the groups: one block per wave along the inner axis
        for (int a = 0; a < 3; ++a) best.wave_tile[a] = best.waves[a] = 1;
        best.blocks_per_wave = 1;
        best.wave_tile[inner] = 16;
        if (rank == 3) best.waves[0] = best.waves[1] = 2;
        else best.waves[0] = 4;
    }
    if (forward && rank == 1 && dtype != NA_FP32) {
        const int fw = env_choice("NA_FWD_WAVES", 4, 8);
        na::Geo g4;
        if (fw == 8 || (fw == 0 && ks[0] >= 512 &&
                        geo_from_tiling(1, extents, ks, ds, nullptr, BH, best, g4, true) &&
                        g4.nwg >= 2048))
            best.waves[0] = 8;
    }
    return best;
}

// Heuristic tilings of na_forward / na_backward.
na_tiling default_forward_tiling(int rank, const int64_t* extents, const int32_t* ks,
                                 const int32_t* ds, int64_t BH, int64_t head_dim, na_dtype dtype) {
    return model_tiling(rank, extents, ks, ds, BH, head_dim, dtype, true);
}

na_tiling default_backward_tiling(int rank, const int64_t* extents, const int32_t* ks,
                                  const int32_t* ds, int64_t BH, int64_t head_dim, na_dtype dtype) {
    return model_tiling(rank, extents, ks, ds, BH, head_dim, dtype, false);
}

// ---- tiling cache (filled by na_tune) ----
struct Tuned {
    bool has_fwd = false, has_bwd = false;
    na_tiling fwd{}, bwd{};
};
std::mutex g_cache_mu;
std::map<std::vector<int64_t>, Tuned>& tiling_cache() {
    static std::map<std::vector<int64_t>, Tuned> cache;
    return cache;
}

std::vector<int64_t> problem_key(int rank, const int64_t* extents, const int32_t* ks,
                                 const int32_t* ds, const int32_t* causal, int64_t BH,
                                 int64_t head_dim, na_dtype dtype) {
    std::vector<int64_t> key = {rank, BH, head_dim, (int64_t)dtype};
    for (int a = 0; a < rank; ++a) {
        key.push_back(extents[a]);
        key.push_back(ks[a]);
        key.push_back(ds[a]);
        key.push_back(causal && causal[a] ? 1 : 0);
    }
    return key;
}

na_tiling current_tiling(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
                         const int32_t* causal, int64_t BH, int64_t head_dim, na_dtype dtype,
                         bool forward) {
    {
        std::lock_guard<std::mutex> lock(g_cache_mu);
        auto& cache = tiling_cache();
        auto it = cache.find(problem_key(rank, extents, ks, ds, causal, BH, head_dim, dtype));
        if (it != cache.end()) {
            if (forward && it->second.has_fwd) return it->second.fwd;
            if (!forward && it->second.has_bwd) return it->second.bwd;
        }
    }
    return forward ? default_forward_tiling(rank, extents, ks, ds, BH, head_dim, dtype)
                   : default_backward_tiling(rank, extents, ks, ds, BH, head_dim, dtype);
}

bool same_tiling(const na_tiling& a, const na_tiling& b) {
    if (a.blocks_per_wave != b.blocks_per_wave) return false;
    for (int i = 0; i < 3; ++i)
        if (a.wave_tile[i] != b.wave_tile[i] || a.waves[i] != b.waves[i]) return false;
    return true;
}

// Candidate tilings: the heuristic one, then every valid factorisation
// whose workgroup tile is no longer than twice an axis's longest group
// (rounded up to a power of two), whose wave tile along the innermost axis is
// at least 4 (2-D, 3-D) and whose launch fits (grid_fits).
std::vector<na_tiling> candidates(int rank, const int64_t* extents, const int32_t* ks,
                                  const int32_t* ds, int64_t BH, int64_t head_dim, na_dtype dtype,
                                  bool forward) {
    std::vector<na_tiling> out;
    out.push_back(forward ? default_forward_tiling(rank, extents, ks, ds, BH, head_dim, dtype)
                          : default_backward_tiling(rank, extents, ks, ds, BH, head_dim, dtype));
    int glen[3];
    group_lengths(rank, extents, ds, glen);
    const int maxwg = forward && rank == 1 && dtype != NA_FP32 ? 8 : 4;
    for (int m = 1; m <= 2; ++m) {
        const int q = 16 * m;
        for (int w0 = 1; w0 <= q; w0 *= 2)
            for (int w1 = 1; w1 <= (rank > 1 ? q : 1); w1 *= 2)
                for (int w2 = 1; w2 <= (rank > 2 ? q : 1); w2 *= 2) {
                    if (w0 * w1 * w2 != q) continue;
                    const int wt[3] = {w0, w1, w2};
                    if (rank > 1 && wt[rank - 1] < 4) continue;
                    for (int p = 4; p <= maxwg; p *= 2)
                        for (int g0 = 1; g0 <= p; g0 *= 2)
                            for (int g1 = 1; g1 <= (rank > 1 ? p : 1); g1 *= 2)
                                for (int g2 = 1; g2 <= (rank > 2 ? p : 1); g2 *= 2) {
                                    if (g0 * g1 * g2 != p) continue;
                                    const int wg[3] = {g0, g1, g2};
                                    na_tiling t;
                                    t.blocks_per_wave = m;
                                    bool ok = true;
                                    for (int a = 0; a < 3; ++a) {
                                        t.wave_tile[a] = wt[a];
                                        t.waves[a] = wg[a];
                                        if (a < rank && wt[a] * wg[a] > 2 * pow2ceil(glen[a]) &&
                                            !(rank == 1 && wg[a] == 4))
                                            ok = false;
                                    }
                                    if (!ok || !valid_tiling(rank, dtype, forward, t)) continue;
                                    na::Geo g;
                                    if (!geo_from_tiling(rank, extents, ks, ds, nullptr, BH, t, g,
                                                         forward))
                                        continue;
                                    bool dup = false;
                                    for (const auto& c : out) dup = dup || same_tiling(c, t);
                                    if (!dup) out.push_back(t);
                                }
                }
    }
    return out;
}

// The heuristic forward and backward launches of a valid problem fit
// (grid_fits); NA_ERR_SHAPE otherwise.
na_status check_launchable(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
                           int64_t batch, int64_t heads, int64_t head_dim, na_dtype dtype) {
    const int64_t BH = batch * heads;
    na::Geo g;
    if (!geo_from_tiling(rank, extents, ks, ds, nullptr, BH,
                         default_forward_tiling(rank, extents, ks, ds, BH, head_dim, dtype), g,
                         true) ||
        !geo_from_tiling(rank, extents, ks, ds, nullptr, BH,
                         default_backward_tiling(rank, extents, ks, ds, BH, head_dim, dtype), g,
                         false))
        return NA_ERR_SHAPE;
    return NA_OK;
}

na_status check_all(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
                    int64_t batch, int64_t heads, int64_t head_dim, const na_dtype& dtype,
                    float scale) {
    na_status st = check_problem(rank, extents, ks, ds, batch, heads, head_dim, dtype, scale);
    if (st != NA_OK) return st;
    return check_launchable(rank, extents, ks, ds, batch, heads, head_dim, dtype);
}

// Launchers for a validated, non-empty problem with checked pointers.
na_status run_forward(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
                      const int32_t* causal, int64_t BH, int64_t head_dim, na_dtype dtype,
                      float scale, const na_tiling& t, const void* q, const void* k,
                      const void* v, void* out, float* lse, hipStream_t s) {
    na::Geo g;
    if (!geo_from_tiling(rank, extents, ks, ds, causal, BH, t, g, true)) return NA_ERR_SHAPE;
    hipError_t e = na::launch_forward(g, rank, (int)head_dim, (int)dtype, t.blocks_per_wave, q, k,
                                      v, out, lse, scale, s);
    return e == hipSuccess ? NA_OK : NA_ERR_HIP;
}

// Whether a backward runs as the split form (a Delta pre-pass, then the dK/dV
// and the dQ workgroups as two launches; 16-bit types at D <= 64, ignored
// elsewhere): large 3-D problems with two blocks per wave, whose dK/dV role
// otherwise holds the dQ role to its own occupancy, and 1-D windows of 512
// keys or more, where each launch's smaller working set (Q and dO, or K and V,
// of the slices in flight) stays in L2 (C4: 650 -> 628 us; 2-D problems lose
// 14-47 %).  NA_BWD_SPLIT=0|1 forces the choice.
int bwd_split(int rank, const int32_t* ks, const na_tiling& t) {
    if (const char* env = std::getenv("NA_BWD_SPLIT")) {
        if (env[0] == '0') return 0;
        if (env[0] == '1') return 1;
    }
    if (rank == 3 && t.blocks_per_wave == 2) return 1;
    return rank == 1 && ks[0] >= 512 ? 1 : 0;
}

na_status run_backward(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
                       const int32_t* causal, int64_t BH, int64_t head_dim, na_dtype dtype,
                       float scale, const na_tiling& t, const void* q, const void* k,
                       const void* v, const void* out, const float* lse, const void* dout,
                       void* dq, void* dk, void* dv, hipStream_t s) {
    na::Geo g;
    if (!geo_from_tiling(rank, extents, ks, ds, causal, BH, t, g, false)) return NA_ERR_SHAPE;
    g.bwd_split = bwd_split(rank, ks, t);
    hipError_t e = na::launch_backward(g, rank, (int)head_dim, (int)dtype, t.blocks_per_wave, q,
                                       k, v, out, lse, dout, dq, dk, dv, scale, s);
    return e == hipSuccess ? NA_OK : NA_ERR_HIP;
}

na_status forward_pointers(const void* q, const void* k, const void* v, const void* out,
                           const float* lse) {
    if (!q || !k || !v || !out || !lse) return NA_ERR_NULL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) || !aligned16(lse))
        return NA_ERR_ALIGNMENT;
    return NA_OK;
}

na_status backward_pointers(const void* q, const void* k, const void* v, const void* out,
                            const float* lse, const void* dout, const void* dq, const void* dk,
                            const void* dv) {
    if (!q || !k || !v || !out || !lse || !dout || !dq || !dk || !dv) return NA_ERR_NULL;
    const void* ptrs[] = {q, k, v, out, lse, dout, dq, dk, dv};
    for (const void* p : ptrs)
        if (!aligned16(p)) return NA_ERR_ALIGNMENT;
    return NA_OK;
}

// ---- the auto-tuner (App. A): time candidate tilings on the caller's buffers ----
// Candidates timed by default (the heuristic one and the next ones in
// enumeration order); NA_TUNE_THOROUGH times every candidate.
constexpr int kDefaultCandidates = 64;
constexpr int kFinalRounds = 5;  // interleaved timings of each finalist

// Times launches of a candidate list on one stream and picks one: after a
// warm-up of the heuristic (candidate 0), every candidate is timed once over
// `reps` launches (after one launch of its own); the three fastest and the
// heuristic are then timed again in kFinalRounds rounds, interleaved, the
// order reversed every other round, and compared by their medians (one
// timing of a few launches varies by a few percent from run to run, more
// than the margin); the heuristic stays unless another finalist beats it by
// more than 2 %.
class Tuner {
  public:
    Tuner(hipStream_t s, int reps) : s_(s), reps_(reps < 1 ? 1 : reps) {
        ok_ = hipEventCreate(&e0_) == hipSuccess && hipEventCreate(&e1_) == hipSuccess;
    }
    ~Tuner() {
        if (e0_) (void)hipEventDestroy(e0_);
        if (e1_) (void)hipEventDestroy(e1_);
    }
    bool ok() const { return ok_; }

    template <class Launch>
    na_status pick(std::vector<na_tiling> c, bool thorough, Launch launch, na_tiling& chosen,
                   float& t_best, float& t_heur) {
        if (!thorough && (int)c.size() > kDefaultCandidates) c.resize(kDefaultCandidates);
        for (int r = 0; r < 3 * reps_; ++r)
            if (launch(c[0]) != NA_OK) return NA_ERR_HIP;
        std::vector<float> t1(c.size());
        for (size_t i = 0; i < c.size(); ++i) {
            t1[i] = time_it([&] { return launch(c[i]); });
            if (t1[i] < 0.f) return NA_ERR_HIP;
        }
        std::vector<size_t> order(c.size());
        for (size_t i = 0; i < c.size(); ++i) order[i] = i;
        std::sort(order.begin(), order.end(), [&](size_t a, size_t b) { return t1[a] < t1[b]; });
        std::vector<size_t> fin = {0};
        for (size_t j = 0; j < order.size() && fin.size() < 4; ++j)
            if (order[j] != 0) fin.push_back(order[j]);
        std::vector<std::vector<float>> tf(fin.size());
        for (int r = 0; r < kFinalRounds; ++r)
            for (size_t jj = 0; jj < fin.size(); ++jj) {
                const size_t j = (r & 1) ? fin.size() - 1 - jj : jj;
                const float t = time_it([&] { return launch(c[fin[j]]); });
                if (t < 0.f) return NA_ERR_HIP;
                tf[j].push_back(t);
            }
        size_t best = 0;
        float tb = -1.f;
        for (size_t j = 0; j < fin.size(); ++j) {
            std::sort(tf[j].begin(), tf[j].end());
            const float t = tf[j][tf[j].size() / 2];
            if (fin[j] == 0) t_heur = t;
            if (tb < 0.f || t < tb) {
                tb = t;
                best = fin[j];
            }
        }
        if (best != 0 && tb > 0.98f * t_heur) {
            best = 0;
            tb = t_heur;
        }
        chosen = c[best];
        t_best = tb;
        return NA_OK;
    }

  private:
    // ms per launch of `launch` (one launch first, untimed), or < 0 on failure
    template <class Launch>
    float time_it(Launch launch) {
        if (launch() != NA_OK) return -1.f;
        if (hipEventRecord(e0_, s_) != hipSuccess) return -1.f;
        for (int r = 0; r < reps_; ++r)
            if (launch() != NA_OK) return -1.f;
        float ms = 0.f;
        if (hipEventRecord(e1_, s_) != hipSuccess || hipEventSynchronize(e1_) != hipSuccess ||
            hipEventElapsedTime(&ms, e0_, e1_) != hipSuccess)
            return -1.f;
        return ms / reps_;
    }
    hipStream_t s_;
    int reps_;
    bool ok_ = false;
    hipEvent_t e0_ = nullptr, e1_ = nullptr;
};

// Tunes the forward tiling of a valid, non-empty problem; the buffers end up
// holding the result of the chosen tiling.
na_status tune_forward(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
                       const int32_t* causal, int64_t BH, int64_t head_dim, na_dtype dtype,
                       float scale, const void* q, const void* k, const void* v, void* out,
                       float* lse, int reps, bool thorough, hipStream_t s, na_tiling& chosen,
                       float& t_best, float& t_heur) {
    Tuner tuner(s, reps);
    if (!tuner.ok()) return NA_ERR_HIP;
    na_status st = tuner.pick(
        candidates(rank, extents, ks, ds, BH, head_dim, dtype, true), thorough,
        [&](const na_tiling& t) {
            return run_forward(rank, extents, ks, ds, causal, BH, head_dim, dtype, scale, t, q, k,
                               v, out, lse, s);
        },
        chosen, t_best, t_heur);
    if (st != NA_OK) return st;
    return run_forward(rank, extents, ks, ds, causal, BH, head_dim, dtype, scale, chosen, q, k, v,
                       out, lse, s);
}

na_status tune_backward(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
                        const int32_t* causal, int64_t BH, int64_t head_dim, na_dtype dtype,
                        float scale, const void* q, const void* k, const void* v, const void* out,
                        const float* lse, const void* dout, void* dq, void* dk, void* dv,
                        int reps, bool thorough, hipStream_t s, na_tiling& chosen, float& t_best,
                        float& t_heur) {
    Tuner tuner(s, reps);
    if (!tuner.ok()) return NA_ERR_HIP;
    na_status st = tuner.pick(
        candidates(rank, extents, ks, ds, BH, head_dim, dtype, false), thorough,
        [&](const na_tiling& t) {
            return run_backward(rank, extents, ks, ds, causal, BH, head_dim, dtype, scale, t, q, k,
                                v, out, lse, dout, dq, dk, dv, s);
        },
        chosen, t_best, t_heur);
    if (st != NA_OK) return st;
    return run_backward(rank, extents, ks, ds, causal, BH, head_dim, dtype, scale, chosen, q, k, v,
                        out, lse, dout, dq, dk, dv, s);
}

// ---- per-thread plans ----
// A problem's validation, tiling and launch geometry depend only on its shape,
// the tuner's cache, the autotune mode and the forcing variables (NA_WAVE_BLOCKS,
// NA_FWD_WAVES, NA_BWD_SPLIT), so each thread keeps the last few it made and
// launches from them directly.  A plan belongs to the generation it was made
// in; storing a tuned tiling, na_tune_clear and na_set_autotune start a new
// one (na_tune_clear is also how a changed forcing variable takes effect).
std::atomic<unsigned> g_generation{1};

void new_generation() { g_generation.fetch_add(1, std::memory_order_acq_rel); }

struct PlanKey {
    int32_t rank, dtype, forward, causal[3], k[3], d[3];
    int64_t L[3], batch, heads, head_dim;
};
struct Plan {
    PlanKey key;
    unsigned gen;  // 0: never filled
    na_tiling t;
    na::Geo g;
};
constexpr int kPlans = 8;
thread_local Plan t_plans[kPlans];
thread_local int t_plan_next = 0;

// The key of a problem whose arrays can be read (false: the full validation
// reports the problem).
bool plan_key(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
              const int32_t* causal, int64_t batch, int64_t heads, int64_t head_dim,
              const na_dtype& dtype, bool forward, PlanKey& key) {
    if (rank < 1 || rank > 3 || !extents || !ks || !ds) return false;
    std::memset(&key, 0, sizeof(key));
    key.rank = rank;
    key.dtype = enum_bits(dtype);
    key.forward = forward ? 1 : 0;
    for (int a = 0; a < rank; ++a) {
        key.L[a] = extents[a];
        key.k[a] = ks[a];
        key.d[a] = ds[a];
        key.causal[a] = causal && causal[a] ? 1 : 0;
    }
    key.batch = batch;
    key.heads = heads;
    key.head_dim = head_dim;
    return true;
}

const Plan* find_plan(const PlanKey& key) {
    const unsigned gen = g_generation.load(std::memory_order_acquire);
    for (const Plan& p : t_plans)
        if (p.gen == gen && std::memcmp(&p.key, &key, sizeof(key)) == 0) return &p;
    return nullptr;
}

// gen: the generation read before the plan's tiling was chosen (a plan made
// across a change of generation is never found again)
void store_plan(const PlanKey& key, unsigned gen, const na_tiling& t, const na::Geo& g) {
    Plan& p = t_plans[t_plan_next];
    t_plan_next = (t_plan_next + 1) % kPlans;
    p.key = key;
    p.gen = gen;
    p.t = t;
    p.g = g;
}

void cache_store(const std::vector<int64_t>& key, const na_tiling* fwd, const na_tiling* bwd) {
    new_generation();
    std::lock_guard<std::mutex> lock(g_cache_mu);
    Tuned& e = tiling_cache()[key];
    if (fwd) {
        e.has_fwd = true;
        e.fwd = *fwd;
    }
    if (bwd) {
        e.has_bwd = true;
        e.bwd = *bwd;
    }
}

bool cache_has(const std::vector<int64_t>& key, bool forward) {
    std::lock_guard<std::mutex> lock(g_cache_mu);
    auto& cache = tiling_cache();
    auto it = cache.find(key);
    return it != cache.end() && (forward ? it->second.has_fwd : it->second.has_bwd);
}

// Tune-on-miss mode: -1 until first read (then from NA_AUTOTUNE: 0 off,
// 1 on, 2 on and thorough), or as set by na_set_autotune.
std::atomic<int> g_autotune{-1};

int autotune_mode() {
    int m = g_autotune.load();
    if (m < 0) {
        const char* env = std::getenv("NA_AUTOTUNE");
        const int v = env ? std::atoi(env) : 0;
        m = (v == 1 || v == 2) ? v : 0;
        int expected = -1;
        g_autotune.compare_exchange_strong(expected, m);
        m = g_autotune.load();
    }
    return m;
}

// Tuning synchronises the stream, which a stream being captured into a graph
// does not allow: such calls use the cached or heuristic tiling.
bool stream_capturing(hipStream_t s) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cs) != hipSuccess) return true;
    return cs != hipStreamCaptureStatusNone;
}

constexpr int kAutotuneRepeats = 3;

// ---- the unfused operators (Sec. 3.1) ----
// Geometry of a valid problem; false if its weight tensor cannot be indexed
// (more than 2^31 - 1 weights per row or 2^62 in all).
bool ugeo_from_problem(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
                       const int32_t* causal, int64_t BH, na::UGeo& u) {
    std::memset(&u, 0, sizeof(u));
    // the problem's axes are the last `rank` of the three, so that the
    // kernels' innermost neighbour loop runs along its innermost axis
    const int off = 3 - rank;
    int64_t ell = 1;
    for (int a = 0; a < 3; ++a) {
        const bool real = a >= off;
        u.L[a] = real ? (int)extents[a - off] : 1;
        u.k[a] = real ? ks[a - off] : 1;
        u.d[a] = real ? ds[a - off] : 1;
        u.causal[a] = real && causal && causal[a - off] ? 1 : 0;
        ell *= u.k[a];
    }
    if (ell >= (int64_t(1) << 31)) return false;
    int s = 1, ks_ = 1;
    for (int a = 2; a >= 0; --a) {
        u.ts[a] = a >= off ? s : 0;
        s *= u.L[a];
        u.kst[a] = ks_;
        ks_ *= u.k[a];
    }
    u.N = (int)token_count(rank, extents);
    u.ell = (int)ell;
    u.rows = BH * u.N;
    if (u.rows > 0 && ell > (int64_t(1) << 62) / u.rows) return false;
    for (int a = 0; a < 3; ++a) {
        u.fd_L[a].init(u.L[a]);
        u.fd_d[a].init(u.d[a]);
        u.fd_k[a].init(u.k[a]);
    }
    return true;
}

// Validation, pointer checks and launch of one unfused operator.  need[] marks
// which of x, y, z (and lse) the operator reads or writes.
na_status run_unfused(int rank, const int64_t* extents, const int32_t* ks, const int32_t* ds,
                      const int32_t* causal, int64_t batch, int64_t heads, int64_t head_dim,
                      const na_dtype& dtype, float scale, int op, const void* x, const void* y,
                      void* z, float* lse, na_stream_t stream) {
    na_status st = check_problem(rank, extents, ks, ds, batch, heads, head_dim, dtype, scale);
    if (st != NA_OK) return st;
    if (empty_problem(rank, extents, batch, heads)) return NA_OK;
    const bool use_x = op != na::kUnfusedSoftmax;
    const bool use_y = op == na::kUnfusedPN || op == na::kUnfusedNN || op == na::kUnfusedIN;
    const bool use_lse = op == na::kUnfusedSoftmax;
    if ((use_x && !x) || (use_y && !y) || !z || (use_lse && !lse)) return NA_ERR_NULL;
    if ((use_x && !aligned16(x)) || (use_y && !aligned16(y)) || !aligned16(z) ||
        (use_lse && !aligned16(lse)))
        return NA_ERR_ALIGNMENT;
    na::UGeo u;
    if (!ugeo_from_problem(rank, extents, ks, ds, causal, batch * heads, u)) return NA_ERR_SHAPE;
    hipError_t e = na::launch_unfused(u, (int)head_dim, (int)dtype, op, x, y, z, lse, scale,
                                      reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? NA_OK : NA_ERR_HIP;
}

}  // namespace

extern "C" {

const char* na_status_string(na_status status) {
    switch (enum_bits(status)) {
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
        case NA_ERR_TILING: return "the tiling is not valid for this problem";
    }
    return "unknown status";
}

int na_version(void) { return kVersion; }

na_status na_validate(int rank, const int64_t* extents, const int32_t* kernel_size,
                      const int32_t* dilation, const int32_t* causal, int64_t batch, int64_t heads,
                      int64_t head_dim, na_dtype dtype, float scale) {
    (void)causal;  // any value is legal (NULL: no causal axis)
    return check_all(rank, extents, kernel_size, dilation, batch, heads, head_dim, dtype, scale);
}

na_status na_forward(int rank, const int64_t* extents, const int32_t* kernel_size,
                     const int32_t* dilation, const int32_t* causal, int64_t batch, int64_t heads,
                     int64_t head_dim, na_dtype dtype, float scale, const void* q, const void* k,
                     const void* v, void* out, float* logsumexp, na_stream_t stream) {
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    PlanKey pk;
    const bool keyed = plan_key(rank, extents, kernel_size, dilation, causal, batch, heads,
                                head_dim, dtype, true, pk);
    if (keyed) {
        if (const Plan* p = find_plan(pk)) {
            if (!std::isfinite(scale)) return NA_ERR_SCALE;
            const na_status st = forward_pointers(q, k, v, out, logsumexp);
            if (st != NA_OK) return st;
            const hipError_t e = na::launch_forward(p->g, rank, (int)head_dim, (int)dtype,
                                                    p->t.blocks_per_wave, q, k, v, out, logsumexp,
                                                    scale, s);
            return e == hipSuccess ? NA_OK : NA_ERR_HIP;
        }
    }
    const unsigned gen = g_generation.load(std::memory_order_acquire);
    na_status st = check_all(rank, extents, kernel_size, dilation, batch, heads, head_dim, dtype,
                             scale);
    if (st != NA_OK) return st;
    if (empty_problem(rank, extents, batch, heads)) return NA_OK;
    st = forward_pointers(q, k, v, out, logsumexp);
    if (st != NA_OK) return st;
    const int64_t BH = batch * heads;
    bool planned = keyed;
    const int mode = autotune_mode();
    if (mode) {
        const auto key = problem_key(rank, extents, kernel_size, dilation, causal, BH, head_dim,
                                     dtype);
        if (!cache_has(key, true)) {
            if (!stream_capturing(s)) {
                na_tiling t;
                float tb = 0.f, th = 0.f;
                st = tune_forward(rank, extents, kernel_size, dilation, causal, BH, head_dim,
                                  dtype, scale, q, k, v, out, logsumexp, kAutotuneRepeats,
                                  mode == 2, s, t, tb, th);
                if (st == NA_OK) cache_store(key, &t, nullptr);
                return st;
            }
            planned = false;  // tuned by a later call, outside the capture
        }
    }
    const na_tiling t = current_tiling(rank, extents, kernel_size, dilation, causal, BH, head_dim,
                                       dtype, true);
    na::Geo g;
    if (!geo_from_tiling(rank, extents, kernel_size, dilation, causal, BH, t, g, true))
        return NA_ERR_SHAPE;
    if (planned) store_plan(pk, gen, t, g);
    const hipError_t e = na::launch_forward(g, rank, (int)head_dim, (int)dtype, t.blocks_per_wave,
                                            q, k, v, out, logsumexp, scale, s);
    return e == hipSuccess ? NA_OK : NA_ERR_HIP;
}

na_status na_backward(int rank, const int64_t* extents, const int32_t* kernel_size,
                      const int32_t* dilation, const int32_t* causal, int64_t batch, int64_t heads,
                      int64_t head_dim, na_dtype dtype, float scale, const void* q, const void* k,
                      const void* v, const void* out, const float* logsumexp, const void* dout,
                      void* dq, void* dk, void* dv, na_stream_t stream) {
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    PlanKey pk;
    const bool keyed = plan_key(rank, extents, kernel_size, dilation, causal, batch, heads,
                                head_dim, dtype, false, pk);
    if (keyed) {
        if (const Plan* p = find_plan(pk)) {
            if (!std::isfinite(scale)) return NA_ERR_SCALE;
            const na_status st = backward_pointers(q, k, v, out, logsumexp, dout, dq, dk, dv);
            if (st != NA_OK) return st;
            const hipError_t e = na::launch_backward(p->g, rank, (int)head_dim, (int)dtype,
                                                     p->t.blocks_per_wave, q, k, v, out, logsumexp,
                                                     dout, dq, dk, dv, scale, s);
            return e == hipSuccess ? NA_OK : NA_ERR_HIP;
        }
    }
    const unsigned gen = g_generation.load(std::memory_order_acquire);
    na_status st = check_all(rank, extents, kernel_size, dilation, batch, heads, head_dim, dtype,
                             scale);
    if (st != NA_OK) return st;
    if (empty_problem(rank, extents, batch, heads)) return NA_OK;
    st = backward_pointers(q, k, v, out, logsumexp, dout, dq, dk, dv);
    if (st != NA_OK) return st;
    const int64_t BH = batch * heads;
    bool planned = keyed;
    const int mode = autotune_mode();
    if (mode) {
        const auto key = problem_key(rank, extents, kernel_size, dilation, causal, BH, head_dim,
                                     dtype);
        if (!cache_has(key, false)) {
            if (!stream_capturing(s)) {
                na_tiling t;
                float tb = 0.f, th = 0.f;
                st = tune_backward(rank, extents, kernel_size, dilation, causal, BH, head_dim,
                                   dtype, scale, q, k, v, out, logsumexp, dout, dq, dk, dv,
                                   kAutotuneRepeats, mode == 2, s, t, tb, th);
                if (st == NA_OK) cache_store(key, nullptr, &t);
                return st;
            }
            planned = false;  // tuned by a later call, outside the capture
        }
    }
    const na_tiling t = current_tiling(rank, extents, kernel_size, dilation, causal, BH, head_dim,
                                       dtype, false);
    na::Geo g;
    if (!geo_from_tiling(rank, extents, kernel_size, dilation, causal, BH, t, g, false))
        return NA_ERR_SHAPE;
    g.bwd_split = bwd_split(rank, kernel_size, t);
    if (planned) store_plan(pk, gen, t, g);
    const hipError_t e = na::launch_backward(g, rank, (int)head_dim, (int)dtype,
                                             t.blocks_per_wave, q, k, v, out, logsumexp, dout, dq,
                                             dk, dv, scale, s);
    return e == hipSuccess ? NA_OK : NA_ERR_HIP;
}

int na_candidate_tilings(int rank, const int64_t* extents, const int32_t* kernel_size,
                         const int32_t* dilation, int64_t batch, int64_t heads, int64_t head_dim,
                         na_dtype dtype, int forward, na_tiling* out, int max) {
    na_status st = check_all(rank, extents, kernel_size, dilation, batch, heads, head_dim, dtype,
                             1.0f);
    if (st != NA_OK) return -(int)st;
    const auto c = candidates(rank, extents, kernel_size, dilation, batch * heads, head_dim, dtype,
                              forward != 0);
    for (int i = 0; i < (int)c.size() && i < max && out; ++i) out[i] = c[i];
    return (int)c.size();
}

na_status na_current_tiling(int rank, const int64_t* extents, const int32_t* kernel_size,
                            const int32_t* dilation, const int32_t* causal, int64_t batch,
                            int64_t heads, int64_t head_dim, na_dtype dtype, int forward,
                            na_tiling* out) {
    na_status st = check_all(rank, extents, kernel_size, dilation, batch, heads, head_dim, dtype,
                             1.0f);
    if (st != NA_OK) return st;
    if (!out) return NA_ERR_NULL;
    *out = current_tiling(rank, extents, kernel_size, dilation, causal, batch * heads, head_dim,
                          dtype, forward != 0);
    return NA_OK;
}

na_status na_forward_tiled(int rank, const int64_t* extents, const int32_t* kernel_size,
                           const int32_t* dilation, const int32_t* causal, int64_t batch,
                           int64_t heads, int64_t head_dim, na_dtype dtype, float scale,
                           const na_tiling* tiling, const void* q, const void* k, const void* v,
                           void* out, float* logsumexp, na_stream_t stream) {
    na_status st = check_all(rank, extents, kernel_size, dilation, batch, heads, head_dim, dtype,
                             scale);
    if (st != NA_OK) return st;
    if (!tiling) return NA_ERR_NULL;
    if (!valid_tiling(rank, dtype, true, *tiling)) return NA_ERR_TILING;
    if (empty_problem(rank, extents, batch, heads)) return NA_OK;
    st = forward_pointers(q, k, v, out, logsumexp);
    if (st != NA_OK) return st;
    return run_forward(rank, extents, kernel_size, dilation, causal, batch * heads, head_dim,
                       dtype, scale, *tiling, q, k, v, out, logsumexp,
                       reinterpret_cast<hipStream_t>(stream));
}

na_status na_backward_tiled(int rank, const int64_t* extents, const int32_t* kernel_size,
                            const int32_t* dilation, const int32_t* causal, int64_t batch,
                            int64_t heads, int64_t head_dim, na_dtype dtype, float scale,
                            const na_tiling* tiling, const void* q, const void* k, const void* v,
                            const void* out, const float* logsumexp, const void* dout, void* dq,
                            void* dk, void* dv, na_stream_t stream) {
    na_status st = check_all(rank, extents, kernel_size, dilation, batch, heads, head_dim, dtype,
                             scale);
    if (st != NA_OK) return st;
    if (!tiling) return NA_ERR_NULL;
    if (!valid_tiling(rank, dtype, false, *tiling)) return NA_ERR_TILING;
    if (empty_problem(rank, extents, batch, heads)) return NA_OK;
    st = backward_pointers(q, k, v, out, logsumexp, dout, dq, dk, dv);
    if (st != NA_OK) return st;
    return run_backward(rank, extents, kernel_size, dilation, causal, batch * heads, head_dim,
                        dtype, scale, *tiling, q, k, v, out, logsumexp, dout, dq, dk, dv,
                        reinterpret_cast<hipStream_t>(stream));
}

na_status na_tune(int rank, const int64_t* extents, const int32_t* kernel_size,
                  const int32_t* dilation, const int32_t* causal, int64_t batch, int64_t heads,
                  int64_t head_dim, na_dtype dtype, float scale, const void* q, const void* k,
                  const void* v, void* out, float* logsumexp, const void* dout, void* dq, void* dk,
                  void* dv, int repeats, int flags, na_stream_t stream, na_tiling* best_forward,
                  na_tiling* best_backward, float* times_ms) {
    na_status st = check_all(rank, extents, kernel_size, dilation, batch, heads, head_dim, dtype,
                             scale);
    if (st != NA_OK) return st;
    if (flags & ~NA_TUNE_THOROUGH) return NA_ERR_TILING;
    const bool thorough = (flags & NA_TUNE_THOROUGH) != 0;
    const int64_t BH = batch * heads;
    na_tiling bf = default_forward_tiling(rank, extents, kernel_size, dilation, BH, head_dim, dtype);
    na_tiling bb = default_backward_tiling(rank, extents, kernel_size, dilation, BH, head_dim, dtype);
    float tm[4] = {0.f, 0.f, 0.f, 0.f};
    if (!empty_problem(rank, extents, batch, heads)) {
        st = backward_pointers(q, k, v, out, logsumexp, dout, dq, dk, dv);
        if (st != NA_OK) return st;
        hipStream_t s = reinterpret_cast<hipStream_t>(stream);
        // out and logsumexp from the chosen forward feed the backward's tuning
        st = tune_forward(rank, extents, kernel_size, dilation, causal, BH, head_dim, dtype, scale,
                          q, k, v, out, logsumexp, repeats, thorough, s, bf, tm[0], tm[2]);
        if (st == NA_OK)
            st = tune_backward(rank, extents, kernel_size, dilation, causal, BH, head_dim, dtype,
                               scale, q, k, v, out, logsumexp, dout, dq, dk, dv, repeats, thorough,
                               s, bb, tm[1], tm[3]);
        if (st == NA_OK && hipStreamSynchronize(s) != hipSuccess) st = NA_ERR_HIP;
        if (st != NA_OK) return st;
        cache_store(problem_key(rank, extents, kernel_size, dilation, causal, BH, head_dim, dtype),
                    &bf, &bb);
    }
    if (best_forward) *best_forward = bf;
    if (best_backward) *best_backward = bb;
    if (times_ms)
        for (int i = 0; i < 4; ++i) times_ms[i] = tm[i];
    return NA_OK;
}

void na_tune_clear(void) {
    new_generation();
    std::lock_guard<std::mutex> lock(g_cache_mu);
    tiling_cache().clear();
}

na_status na_unfused_pn(int rank, const int64_t* extents, const int32_t* kernel_size,
                        const int32_t* dilation, const int32_t* causal, int64_t batch,
                        int64_t heads, int64_t head_dim, na_dtype dtype, float scale,
                        const void* a, const void* b, void* weights, na_stream_t stream) {
    return run_unfused(rank, extents, kernel_size, dilation, causal, batch, heads, head_dim, dtype,
                       scale, na::kUnfusedPN, a, b, weights, nullptr, stream);
}

na_status na_unfused_softmax(int rank, const int64_t* extents, const int32_t* kernel_size,
                             const int32_t* dilation, const int32_t* causal, int64_t batch,
                             int64_t heads, int64_t head_dim, na_dtype dtype, void* weights,
                             float* logsumexp, na_stream_t stream) {
    return run_unfused(rank, extents, kernel_size, dilation, causal, batch, heads, head_dim, dtype,
                       1.0f, na::kUnfusedSoftmax, nullptr, nullptr, weights, logsumexp, stream);
}

na_status na_unfused_nn(int rank, const int64_t* extents, const int32_t* kernel_size,
                        const int32_t* dilation, const int32_t* causal, int64_t batch,
                        int64_t heads, int64_t head_dim, na_dtype dtype, float scale,
                        const void* weights, const void* b, void* out, na_stream_t stream) {
    return run_unfused(rank, extents, kernel_size, dilation, causal, batch, heads, head_dim, dtype,
                       scale, na::kUnfusedNN, weights, b, out, nullptr, stream);
}

na_status na_unfused_in(int rank, const int64_t* extents, const int32_t* kernel_size,
                        const int32_t* dilation, const int32_t* causal, int64_t batch,
                        int64_t heads, int64_t head_dim, na_dtype dtype, float scale,
                        const void* weights, const void* b, void* out, na_stream_t stream) {
    return run_unfused(rank, extents, kernel_size, dilation, causal, batch, heads, head_dim, dtype,
                       scale, na::kUnfusedIN, weights, b, out, nullptr, stream);
}

na_status na_unfused_softmax_backward(int rank, const int64_t* extents,
                                      const int32_t* kernel_size, const int32_t* dilation,
                                      const int32_t* causal, int64_t batch, int64_t heads,
                                      int64_t head_dim, na_dtype dtype, const void* probs,
                                      void* grad, na_stream_t stream) {
    return run_unfused(rank, extents, kernel_size, dilation, causal, batch, heads, head_dim, dtype,
                       1.0f, na::kUnfusedSoftmaxBwd, probs, nullptr, grad, nullptr, stream);
}

void na_set_autotune(int mode) {
    g_autotune.store(mode == 1 || mode == 2 ? mode : 0);
    new_generation();
}

int na_autotune(void) { return autotune_mode(); }

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
