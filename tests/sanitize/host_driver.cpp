// Sanitizer driver for the library's host code (na_api.cpp), built by
// tests/test_sanitizers.py with AddressSanitizer and UndefinedBehaviorSanitizer
// on the host pass only (no device code is compiled).  The kernel launchers and
// the few HIP runtime calls the host code makes are replaced by stubs:
//   * each launcher checks the geometry it is handed against what the kernels
//     assume (tile counts cover every dilation group, grid sizes, token and
//     weight strides, and every FastDiv divisor divides exactly) and counts
//     launches; it touches no buffer, so the device pointers are fake;
//   * events read a modelled clock that every launch advances by a cost fixed
//     per tiling, so the tuner's choice can be predicted and checked;
//   * stream capture and launch failure can be forced.
// Every public entry point is driven through valid, invalid and empty problems.
// Out-of-range enum values come from c_caller.c, compiled as C.
// Prints "ok host <checks> <launches>" and exits 0 on success.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "na.h"
#include "na_launch.h"

// c_caller.c: entry points called from C with an int where an enum is declared
extern "C" {
int c_validate(int rank, const int64_t* L, const int32_t* k, const int32_t* d, int64_t B,
               int64_t H, int64_t D, int dtype);
int c_forward(int rank, const int64_t* L, const int32_t* k, const int32_t* d, int64_t B,
              int64_t H, int64_t D, int dtype, void* buf);
int c_candidates(int rank, const int64_t* L, const int32_t* k, const int32_t* d, int64_t B,
                 int64_t H, int64_t D, int dtype);
int c_unfused_softmax(int rank, const int64_t* L, const int32_t* k, const int32_t* d, int64_t B,
                      int64_t H, int64_t D, int dtype, void* buf);
const char* c_status_string(int status);
}

namespace {

long g_checks = 0, g_launches = 0;
na_tiling g_last{};  // tiling of the last fused launch
bool g_fail_launch = false;
bool g_capturing = false;
double g_clock = 0.0;  // modelled device time, ms

[[noreturn]] void fail(const char* what, int line) {
    std::printf("FAIL line %d: %s\n", line, what);
    std::fflush(stdout);
    std::exit(1);
}
#define CHECK(c)                                \
    do {                                        \
        ++g_checks;                             \
        if (!(c)) fail(#c, __LINE__);           \
    } while (0)

// The problem the next launch belongs to (set by the driver before each call).
struct Problem {
    int rank;
    int64_t L[3];
    int32_t k[3], d[3], c[3];
    int64_t B, H, D;
    na_dtype dt;
    bool causal;  // c is passed (else NULL)
} g_prob;

const int32_t* causal_of(const Problem& p) { return p.causal ? p.c : nullptr; }

// Modelled cost of a launch with this tiling: distinct, deterministic values.
double tiling_cost(int m, const int* wt, const int* wg) {
    uint32_t h = 2166136261u;
    const int v[7] = {m, wt[0], wt[1], wt[2], wg[0], wg[1], wg[2]};
    for (int x : v) h = (h ^ (uint32_t)x) * 16777619u;
    return 1.0 + (h % 1000) / 250.0;
}

// FastDiv must divide every numerator the kernels use exactly (they stay below 2^31).
void check_fastdiv(const na::FastDiv& f, int d, int64_t hi) {
    CHECK(d >= 1);
    if (hi > (int64_t(1) << 31) - 1) hi = (int64_t(1) << 31) - 1;
    const int64_t probes[] = {0, 1, d - 1, d, d + 1, 2 * int64_t(d) - 1, 2 * int64_t(d), hi / 2,
                              hi - 1, hi};
    for (int64_t n : probes) {
        if (n < 0 || n > hi) continue;
        CHECK(na::FastDiv::divide((int)n, f.mul, f.shr) == (int)(n / d));
    }
    for (int i = 0; i < 64; ++i) {
        const int64_t n = (int64_t)((1103515245ull * (uint64_t)(i + 1) + 12345ull) % (uint64_t)(hi + 1));
        CHECK(na::FastDiv::divide((int)n, f.mul, f.shr) == (int)(n / d));
    }
}

int group_len(int64_t L, int d) { return (int)((L + d - 1) / d); }

void check_geo(const na::Geo& g, bool forward, int qm) {
    const Problem& p = g_prob;
    int64_t N = 1, ngroups = 1, ntiles = 1;
    for (int a = 0; a < 3; ++a) {
        const bool real = a < p.rank;
        CHECK(g.L[a] == (real ? p.L[a] : 1));
        CHECK(g.k[a] == (real ? p.k[a] : 1));
        CHECK(g.d[a] == (real ? p.d[a] : 1));
        CHECK(g.causal[a] == (real && p.causal && p.c[a] ? 1 : 0));
        CHECK(g.T[a] == g.WT[a] * g.WGd[a]);
        CHECK((1 << g.lgWT[a]) == g.WT[a] && (1 << g.lgWGd[a]) == g.WGd[a]);
        const int glen = real ? group_len(p.L[a], p.d[a]) : 1;
        CHECK(int64_t(g.nt[a]) * g.T[a] >= glen);             // every query is covered
        CHECK(int64_t(g.nt[a] - 1) * g.T[a] < glen);          // no tile row is empty
        if (!real) CHECK(g.WT[a] == 1 && g.WGd[a] == 1 && g.ts[a] == 0);
        N *= g.L[a];
        ngroups *= g.d[a];
        ntiles *= g.nt[a];
    }
    int64_t s = 1;
    for (int a = p.rank - 1; a >= 0; --a) {
        CHECK(g.ts[a] == s);
        s *= g.L[a];
    }
    int wt = 1, wg = 1;
    for (int a = 0; a < 3; ++a) {
        wt *= g.WT[a];
        wg *= g.WGd[a];
    }
    CHECK(wt == 16 * qm);
    CHECK(wg == 4 || (wg == 8 && forward && p.rank == 1 && p.dt != NA_FP32));
    CHECK(g.N == N && g.ngroups == ngroups && g.ntiles == ntiles);
    CHECK(g.BH == p.B * p.H);
    CHECK(int64_t(g.nwg) == ntiles * ngroups * p.B * p.H);
    const int64_t threads = forward ? int64_t(g.nwg) * wg * 64
                                    : (((int64_t(g.nwg) + 7) & ~int64_t(7)) + g.nwg) * 256;
    CHECK(threads < (int64_t(1) << 32));
    for (int a = 0; a < 3; ++a) {
        check_fastdiv(g.fd_d[a], g.d[a], N);
        check_fastdiv(g.fd_nt[a], g.nt[a], g.nwg);
    }
    check_fastdiv(g.fd_ntiles, g.ntiles, g.nwg);
    check_fastdiv(g.fd_ngroups, g.ngroups, g.nwg);
    // the split form: 3-D backwards with two blocks per wave, 1-D windows of 512 or more
    if (!forward)
        CHECK(g.bwd_split == ((p.rank == 3 && qm == 2) || (p.rank == 1 && p.k[0] >= 512) ? 1 : 0));
    const int wta[3] = {g.WT[0], g.WT[1], g.WT[2]}, wga[3] = {g.WGd[0], g.WGd[1], g.WGd[2]};
    g_last.blocks_per_wave = qm;
    for (int a = 0; a < 3; ++a) {
        g_last.wave_tile[a] = wta[a];
        g_last.waves[a] = wga[a];
    }
    g_clock += tiling_cost(qm, wta, wga);
}

void check_ugeo(const na::UGeo& u) {
    const Problem& p = g_prob;
    const int off = 3 - p.rank;
    int64_t N = 1, ell = 1;
    for (int a = 0; a < 3; ++a) {
        const bool real = a >= off;
        CHECK(u.L[a] == (real ? p.L[a - off] : 1));
        CHECK(u.k[a] == (real ? p.k[a - off] : 1));
        CHECK(u.d[a] == (real ? p.d[a - off] : 1));
        CHECK(u.causal[a] == (real && p.causal && p.c[a - off] ? 1 : 0));
        N *= u.L[a];
        ell *= u.k[a];
    }
    int64_t ts = 1, ks = 1;
    for (int a = 2; a >= 0; --a) {
        CHECK(u.ts[a] == (a >= off ? ts : 0));
        CHECK(u.kst[a] == ks);
        ts *= u.L[a];
        ks *= u.k[a];
    }
    CHECK(u.N == N && u.ell == ell && u.rows == p.B * p.H * N);
    for (int a = 0; a < 3; ++a) {
        check_fastdiv(u.fd_L[a], u.L[a], N);
        check_fastdiv(u.fd_d[a], u.d[a], N);
        check_fastdiv(u.fd_k[a], u.k[a], ell);
    }
    g_clock += 1.0;
}

}  // namespace

// ---- stubs of the kernel launchers ----
namespace na {

hipError_t launch_forward(const Geo& g, int rank, int D, int dtype, int qm, const void* q,
                          const void* k, const void* v, void* o, float* lse, float scale,
                          hipStream_t) {
    CHECK(rank == g_prob.rank && D == g_prob.D && dtype == (int)g_prob.dt);
    CHECK(qm == 1 || qm == 2);
    CHECK(q && k && v && o && lse && std::isfinite(scale));
    check_geo(g, true, qm);
    ++g_launches;
    return g_fail_launch ? hipErrorInvalidValue : hipSuccess;
}

hipError_t launch_backward(const Geo& g, int rank, int D, int dtype, int m, const void* q,
                           const void* k, const void* v, const void* o, const float* lse,
                           const void* dout, void* dq, void* dk, void* dv, float scale,
                           hipStream_t) {
    CHECK(rank == g_prob.rank && D == g_prob.D && dtype == (int)g_prob.dt);
    CHECK(m == 1 || m == 2);
    CHECK(q && k && v && o && lse && dout && dq && dk && dv && std::isfinite(scale));
    check_geo(g, false, m);
    ++g_launches;
    return g_fail_launch ? hipErrorInvalidValue : hipSuccess;
}

hipError_t launch_unfused(const UGeo& u, int D, int dtype, int op, const void* x, const void* y,
                          void* z, float* lse, float scale, hipStream_t) {
    CHECK(D == g_prob.D && dtype == (int)g_prob.dt && op >= 0 && op <= 4);
    CHECK(z && std::isfinite(scale));
    CHECK((op == kUnfusedSoftmax) == (lse != nullptr));
    CHECK((op == kUnfusedSoftmax) == (x == nullptr));
    CHECK((op == kUnfusedPN || op == kUnfusedNN || op == kUnfusedIN) == (y != nullptr));
    check_ugeo(u);
    ++g_launches;
    return g_fail_launch ? hipErrorInvalidValue : hipSuccess;
}

hipError_t launch_debug_windows(int rank, const int* L, const int* k, const int* d, const int* c,
                                int* start, int* inv_lo, int* inv_hi, hipStream_t) {
    CHECK(rank == g_prob.rank);
    for (int a = 0; a < rank; ++a) {
        CHECK(L[a] == g_prob.L[a] && k[a] == g_prob.k[a] && d[a] == g_prob.d[a]);
        CHECK(c[a] == (g_prob.causal && g_prob.c[a] ? 1 : 0));
    }
    // the buffers are host arrays of sum(L) entries here: write them all
    int64_t n = 0;
    for (int a = 0; a < rank; ++a) n += L[a];
    for (int64_t i = 0; i < n; ++i) start[i] = inv_lo[i] = inv_hi[i] = -1;
    ++g_launches;
    return g_fail_launch ? hipErrorInvalidValue : hipSuccess;
}

}  // namespace na

// ---- stubs of the HIP runtime calls the host code makes ----
hipError_t hipEventCreate(hipEvent_t* e) {
    *e = reinterpret_cast<hipEvent_t>(new double(0.0));
    return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t e) {
    delete reinterpret_cast<double*>(e);
    return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t e, hipStream_t) {
    *reinterpret_cast<double*>(e) = g_clock;
    return hipSuccess;
}
hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t a, hipEvent_t b) {
    *ms = (float)(*reinterpret_cast<double*>(b) - *reinterpret_cast<double*>(a));
    return hipSuccess;
}
hipError_t hipStreamIsCapturing(hipStream_t, hipStreamCaptureStatus* cs) {
    *cs = g_capturing ? hipStreamCaptureStatusActive : hipStreamCaptureStatusNone;
    return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }

// ---- the driver ----
namespace {

// Fake, 16-byte aligned device pointers: the stubs never dereference them.
void* fake(int i) { return reinterpret_cast<void*>(uintptr_t(0x100000) * (i + 1)); }

na_status validate(const Problem& p) {
    return na_validate(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f);
}

na_status fwd(const Problem& p) {
    return na_forward(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f, fake(0),
                      fake(1), fake(2), fake(3), (float*)fake(4), nullptr);
}

na_status bwd(const Problem& p) {
    return na_backward(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f, fake(0),
                       fake(1), fake(2), fake(3), (float*)fake(4), fake(5), fake(6), fake(7),
                       fake(8), nullptr);
}

na_status tune(const Problem& p, int flags, na_tiling* bf, na_tiling* bb, float* tm) {
    return na_tune(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f, fake(0),
                   fake(1), fake(2), fake(3), (float*)fake(4), fake(5), fake(6), fake(7), fake(8),
                   2, flags, nullptr, bf, bb, tm);
}

std::vector<na_tiling> cands(const Problem& p, bool forward) {
    const int n = na_candidate_tilings(p.rank, p.L, p.k, p.d, p.B, p.H, p.D, p.dt, forward ? 1 : 0,
                                       nullptr, 0);
    CHECK(n >= 1);
    // exactly n entries: a write past the end would be a heap overflow
    std::vector<na_tiling> v(n);
    CHECK(na_candidate_tilings(p.rank, p.L, p.k, p.d, p.B, p.H, p.D, p.dt, forward ? 1 : 0,
                               v.data(), n) == n);
    if (n > 1) {  // a short buffer gets the first entries only
        std::vector<na_tiling> s(n - 1);
        CHECK(na_candidate_tilings(p.rank, p.L, p.k, p.d, p.B, p.H, p.D, p.dt, forward ? 1 : 0,
                                   s.data(), n - 1) == n);
        CHECK(std::memcmp(s.data(), v.data(), sizeof(na_tiling) * (n - 1)) == 0);
    }
    return v;
}

bool same(const na_tiling& a, const na_tiling& b) { return std::memcmp(&a, &b, sizeof(a)) == 0; }

double cost_of(const na_tiling& t) { return tiling_cost(t.blocks_per_wave, t.wave_tile, t.waves); }

// What the tuner picks under the modelled clock: the cheapest of the timed
// candidates, unless it is within 2 % of the heuristic (candidate 0).
na_tiling expected_choice(const std::vector<na_tiling>& c, bool thorough) {
    const size_t n = thorough ? c.size() : std::min<size_t>(c.size(), NA_TUNE_DEFAULT_CANDIDATES);
    size_t best = 0;
    for (size_t i = 1; i < n; ++i)
        if (cost_of(c[i]) < cost_of(c[best])) best = i;
    if (best != 0 && (float)cost_of(c[best]) > 0.98f * (float)cost_of(c[0])) best = 0;
    return c[best];
}

void drive_valid(const Problem& p) {
    g_prob = p;
    CHECK(validate(p) == NA_OK);
    for (int forward = 0; forward <= 1; ++forward) {
        const auto c = cands(p, forward);
        na_tiling cur;
        CHECK(na_current_tiling(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, forward,
                                &cur) == NA_OK);
        CHECK(same(cur, c[0]));
        for (const auto& t : c) {
            const long before = g_launches;
            const na_status st =
                forward ? na_forward_tiled(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D,
                                           p.dt, 0.5f, &t, fake(0), fake(1), fake(2), fake(3),
                                           (float*)fake(4), nullptr)
                        : na_backward_tiled(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D,
                                            p.dt, 0.5f, &t, fake(0), fake(1), fake(2), fake(3),
                                            (float*)fake(4), fake(5), fake(6), fake(7), fake(8),
                                            nullptr);
            CHECK(st == NA_OK && g_launches == before + 1);
        }
        // tilings the kernels do not accept are refused before any launch
        na_tiling bad = c[0];
        bad.blocks_per_wave = 3;
        const long before = g_launches;
        CHECK(na_forward_tiled(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f,
                               &bad, fake(0), fake(1), fake(2), fake(3), (float*)fake(4),
                               nullptr) == NA_ERR_TILING);
        bad = c[0];
        bad.waves[0] *= 2;  // 8 or 16 waves: never valid in the backward
        CHECK(na_backward_tiled(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f,
                                &bad, fake(0), fake(1), fake(2), fake(3), (float*)fake(4),
                                fake(5), fake(6), fake(7), fake(8), nullptr) == NA_ERR_TILING);
        bad = c[0];
        bad.wave_tile[2] = p.rank < 3 ? 2 : 3;  // beyond the rank, or not a power of two
        CHECK(na_forward_tiled(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f,
                               &bad, fake(0), fake(1), fake(2), fake(3), (float*)fake(4),
                               nullptr) == NA_ERR_TILING);
        CHECK(na_forward_tiled(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f,
                               nullptr, fake(0), fake(1), fake(2), fake(3), (float*)fake(4),
                               nullptr) == NA_ERR_NULL);
        CHECK(g_launches == before);
    }
    // default entry points: one launch each, NULL and misaligned pointers refused
    // (the second calls take the per-thread plan the first made)
    na_set_autotune(0);
    long before = g_launches;
    CHECK(fwd(p) == NA_OK && bwd(p) == NA_OK && g_launches == before + 2);
    CHECK(fwd(p) == NA_OK && bwd(p) == NA_OK && g_launches == before + 4);
    before = g_launches;
    CHECK(na_forward(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, INFINITY, fake(0),
                     fake(1), fake(2), fake(3), (float*)fake(4), nullptr) == NA_ERR_SCALE);
    CHECK(na_backward(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, NAN, fake(0),
                      fake(1), fake(2), fake(3), (float*)fake(4), fake(5), fake(6), fake(7),
                      fake(8), nullptr) == NA_ERR_SCALE);
    CHECK(na_forward(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f, fake(0),
                     nullptr, fake(2), fake(3), (float*)fake(4), nullptr) == NA_ERR_NULL);
    CHECK(na_backward(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f, fake(0),
                      fake(1), fake(2), fake(3), (float*)fake(4), fake(5), fake(6),
                      (char*)fake(7) + 8, fake(8), nullptr) == NA_ERR_ALIGNMENT);
    CHECK(g_launches == before);
    // a failed launch is reported, also from inside the tuner
    g_fail_launch = true;
    CHECK(fwd(p) == NA_ERR_HIP && bwd(p) == NA_ERR_HIP);
    CHECK(tune(p, 0, nullptr, nullptr, nullptr) == NA_ERR_HIP);
    g_fail_launch = false;
    // the tuner's choice under the modelled clock, default and thorough
    for (int flags = 0; flags <= NA_TUNE_THOROUGH; ++flags) {
        na_tune_clear();
        CHECK(fwd(p) == NA_OK && bwd(p) == NA_OK);  // plans with the heuristic tilings
        na_tiling bf, bb;
        float tm[4] = {-1.f, -1.f, -1.f, -1.f};
        CHECK(tune(p, flags, &bf, &bb, tm) == NA_OK);
        // storing the tuned tilings retires those plans
        CHECK(fwd(p) == NA_OK && same(g_last, bf));
        CHECK(bwd(p) == NA_OK && same(g_last, bb));
        CHECK(fwd(p) == NA_OK && same(g_last, bf));
        CHECK(same(bf, expected_choice(cands(p, true), flags != 0)));
        CHECK(same(bb, expected_choice(cands(p, false), flags != 0)));
        for (float t : tm) CHECK(t > 0.f);
        CHECK(std::fabs(tm[0] - (float)cost_of(bf)) < 1e-3f);
        na_tiling cur;
        CHECK(na_current_tiling(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 1,
                                &cur) == NA_OK && same(cur, bf));
        CHECK(na_current_tiling(p.rank, p.L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0,
                                &cur) == NA_OK && same(cur, bb));
    }
    CHECK(tune(p, 4, nullptr, nullptr, nullptr) == NA_ERR_TILING);
    // tune on first use: one tuning per direction, then the cached tiling;
    // a stream being captured is never tuned
    na_tune_clear();
    na_set_autotune(1);
    CHECK(na_autotune() == 1);
    g_capturing = true;
    before = g_launches;
    CHECK(fwd(p) == NA_OK && g_launches == before + 1);
    g_capturing = false;
    before = g_launches;
    CHECK(fwd(p) == NA_OK && g_launches > before + 1);
    before = g_launches;
    CHECK(fwd(p) == NA_OK && g_launches == before + 1);
    CHECK(bwd(p) == NA_OK && g_launches > before + 2);
    before = g_launches;
    CHECK(bwd(p) == NA_OK && g_launches == before + 1);
    na_set_autotune(0);
    na_tune_clear();
    // the unfused operators
    const int64_t* L = p.L;
    before = g_launches;
    CHECK(na_unfused_pn(p.rank, L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f, fake(0),
                        fake(1), fake(2), nullptr) == NA_OK);
    CHECK(na_unfused_softmax(p.rank, L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, fake(2),
                             (float*)fake(3), nullptr) == NA_OK);
    CHECK(na_unfused_nn(p.rank, L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f, fake(2),
                        fake(1), fake(4), nullptr) == NA_OK);
    CHECK(na_unfused_in(p.rank, L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f, fake(2),
                        fake(1), fake(4), nullptr) == NA_OK);
    CHECK(na_unfused_softmax_backward(p.rank, L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt,
                                      fake(2), fake(5), nullptr) == NA_OK);
    CHECK(g_launches == before + 5);
    CHECK(na_unfused_softmax(p.rank, L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, fake(2),
                             nullptr, nullptr) == NA_ERR_NULL);
    CHECK(na_unfused_nn(p.rank, L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f, fake(2),
                        (char*)fake(1) + 4, fake(4), nullptr) == NA_ERR_ALIGNMENT);
    CHECK(na_unfused_pn(p.rank, L, p.k, p.d, causal_of(p), p.B, p.H, p.D, p.dt, 0.5f, fake(0),
                        nullptr, fake(2), nullptr) == NA_ERR_NULL);
    CHECK(g_launches == before + 5);
    // the window tables, on host arrays of the exact size
    int64_t n = 0;
    for (int a = 0; a < p.rank; ++a) n += p.L[a];
    std::vector<int32_t> st(n), lo(n), hi(n);
    CHECK(na_debug_windows(p.rank, p.L, p.k, p.d, causal_of(p), st.data(), lo.data(), hi.data(),
                           nullptr) == NA_OK);
    CHECK(na_debug_windows(p.rank, p.L, p.k, p.d, causal_of(p), st.data(), nullptr, hi.data(),
                           nullptr) == NA_ERR_NULL);
}

void drive_invalid() {
    Problem p{2, {16, 16, 1}, {3, 5, 1}, {1, 2, 1}, {0, 0, 0}, 2, 3, 64, NA_FP16, false};
    g_prob = p;
    CHECK(validate(p) == NA_OK);
    // unfused: false where only the fused launches are too large
    auto expect = [&](Problem q, na_status want, bool unfused = true) {
        const long before = g_launches;
        CHECK(validate(q) == want);
        CHECK(fwd(q) == want && bwd(q) == want);
        CHECK(tune(q, 0, nullptr, nullptr, nullptr) == want);
        if (unfused)
            CHECK(na_unfused_pn(q.rank, q.L, q.k, q.d, nullptr, q.B, q.H, q.D, q.dt, 0.5f, fake(0),
                                fake(1), fake(2), nullptr) == want);
        CHECK(na_candidate_tilings(q.rank, q.L, q.k, q.d, q.B, q.H, q.D, q.dt, 1, nullptr, 0) ==
              -(int)want);
        CHECK(g_launches == before);
    };
    Problem q = p;
    q.rank = 0;
    expect(q, NA_ERR_RANK);
    q.rank = 4;
    expect(q, NA_ERR_RANK);
    q = p;
    q.L[1] = 0;
    expect(q, NA_ERR_SHAPE);
    q = p;
    q.k[0] = 0;
    expect(q, NA_ERR_KERNEL_SIZE);
    q = p;
    q.d[1] = 0;
    expect(q, NA_ERR_DILATION);
    q = p;
    q.k[1] = 9;  // 9 * 2 > 16
    expect(q, NA_ERR_WINDOW_EXCEEDS_EXTENT);
    q = p;
    q.H = -1;
    expect(q, NA_ERR_SHAPE);
    q = p;
    q.D = 48;
    expect(q, NA_ERR_HEAD_DIM);
    for (int bad : {3, 99, -1}) {  // any int may come through the C interface
        const long before = g_launches;
        CHECK(c_validate(p.rank, p.L, p.k, p.d, p.B, p.H, p.D, bad) == NA_ERR_DTYPE);
        CHECK(c_forward(p.rank, p.L, p.k, p.d, p.B, p.H, p.D, bad, fake(0)) == NA_ERR_DTYPE);
        CHECK(c_candidates(p.rank, p.L, p.k, p.d, p.B, p.H, p.D, bad) == -NA_ERR_DTYPE);
        CHECK(c_unfused_softmax(p.rank, p.L, p.k, p.d, p.B, p.H, p.D, bad, fake(0)) ==
              NA_ERR_DTYPE);
        CHECK(g_launches == before);
    }
    q = p;
    q.rank = 1;
    q.L[0] = int64_t(1) << 25;  // N * D = 2^31
    q.k[0] = 3;
    q.d[0] = 1;
    expect(q, NA_ERR_SHAPE);
    q = p;
    q.B = int64_t(1) << 16;
    q.H = int64_t(1) << 15;  // B * H >= 2^31
    expect(q, NA_ERR_SHAPE);
    q = p;
    q.rank = 1;
    q.L[0] = 64;
    q.k[0] = 3;
    q.d[0] = 1;
    q.B = int64_t(1) << 23;  // the backward grid would reach 2^32 threads
    q.H = 1;
    expect(q, NA_ERR_SHAPE, false);
    CHECK(na_validate(2, p.L, p.k, p.d, nullptr, 1, 1, 64, NA_FP16, INFINITY) == NA_ERR_SCALE);
    CHECK(na_validate(2, p.L, p.k, p.d, nullptr, 1, 1, 64, NA_FP16, NAN) == NA_ERR_SCALE);
    CHECK(na_validate(2, nullptr, p.k, p.d, nullptr, 1, 1, 64, NA_FP16, 1.f) == NA_ERR_NULL);
    CHECK(na_validate(2, p.L, nullptr, p.d, nullptr, 1, 1, 64, NA_FP16, 1.f) == NA_ERR_NULL);
    CHECK(na_validate(2, p.L, p.k, nullptr, nullptr, 1, 1, 64, NA_FP16, 1.f) == NA_ERR_NULL);
    // empty problems launch nothing and succeed, with NULL buffers
    q = p;
    q.B = 0;
    g_prob = q;
    const long before = g_launches;
    CHECK(na_forward(q.rank, q.L, q.k, q.d, nullptr, q.B, q.H, q.D, q.dt, 0.5f, nullptr, nullptr,
                     nullptr, nullptr, nullptr, nullptr) == NA_OK);
    CHECK(na_backward(q.rank, q.L, q.k, q.d, nullptr, q.B, q.H, q.D, q.dt, 0.5f, nullptr, nullptr,
                      nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                      nullptr) == NA_OK);
    na_tiling bf, bb;
    float tm[4];
    CHECK(na_tune(q.rank, q.L, q.k, q.d, nullptr, q.B, q.H, q.D, q.dt, 0.5f, nullptr, nullptr,
                  nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 3, 0, nullptr,
                  &bf, &bb, tm) == NA_OK);
    CHECK(tm[0] == 0.f && tm[3] == 0.f);
    CHECK(na_unfused_in(q.rank, q.L, q.k, q.d, nullptr, q.B, q.H, q.D, q.dt, 0.5f, nullptr,
                        nullptr, nullptr, nullptr) == NA_OK);
    CHECK(g_launches == before);
    for (int s = 0; s <= 13; ++s) CHECK(na_status_string((na_status)s) != nullptr);
    for (int bad : {14, 99, -1}) CHECK(std::strcmp(c_status_string(bad), "unknown status") == 0);
    CHECK(na_version() > 0);
}

}  // namespace

int main() {
    drive_invalid();
    const Problem cases[] = {
        {1, {1000, 1, 1}, {13, 1, 1}, {1, 1, 1}, {0, 0, 0}, 2, 2, 64, NA_FP16, false},
        {1, {4096, 1, 1}, {1023, 1, 1}, {2, 1, 1}, {1, 0, 0}, 1, 3, 32, NA_BF16, true},
        {1, {300, 1, 1}, {300, 1, 1}, {1, 1, 1}, {0, 0, 0}, 1, 1, 128, NA_FP32, false},
        {2, {56, 56, 1}, {7, 7, 1}, {1, 1, 1}, {0, 0, 0}, 2, 4, 32, NA_FP16, false},
        {2, {37, 45, 1}, {4, 6, 1}, {3, 2, 1}, {1, 0, 0}, 1, 2, 64, NA_BF16, true},
        {2, {9, 200, 1}, {9, 5, 1}, {1, 7, 1}, {0, 1, 0}, 3, 1, 128, NA_FP32, true},
        {3, {16, 32, 32}, {7, 7, 7}, {1, 1, 1}, {0, 0, 0}, 1, 2, 64, NA_FP16, false},
        {3, {8, 15, 17}, {3, 5, 4}, {2, 1, 3}, {1, 0, 1}, 2, 1, 32, NA_BF16, true},
        {3, {5, 6, 7}, {5, 6, 7}, {1, 1, 1}, {0, 1, 0}, 1, 1, 128, NA_FP32, true},
    };
    for (const auto& p : cases) drive_valid(p);
    std::printf("ok host %ld %ld\n", g_checks, g_launches);
    return 0;
}
