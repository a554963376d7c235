/*
 * na_ref.c -- plain fp64 CPU oracle for neighborhood attention (NA).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file or the library built from it; only the test-suite, the smoke
 * check and the CPU-baseline leg of the benchmark use it.  It shares no code
 * with the HIP library: every index rule and every arithmetic step is written
 * out again here, deliberately slowly and literally.
 *
 * What it computes (Faster Neighborhood Attention, arXiv 2403.04690):
 *   - Neighborhood attention (Sec. 1, Fig. "neighborhoodattention" caption,
 *     Sec. 2 "Related works"): every query attends to its k nearest context
 *     tokens along each axis; the window is centred on the query where it can
 *     be and shifted (never truncated) at the borders, so every query has
 *     exactly prod_a k_a neighbours.
 *   - Dilation (Sec. 3.4): a dilated problem is a set of independent
 *     non-dilated problems on the sub-lattices x = g (mod d) of each axis.
 *   - Scaled dot-product attention restricted to that neighbourhood (Eq. 1):
 *     P = softmax(scale * q.k), O = sum_j P_j v_j, plus the natural-log
 *     logsumexp LSE = log sum_j exp(scale * q.k_j).
 *   - The backward pass in terms of the PN / NN / IN operators (Sec. 3.1):
 *     dP = PN(dO, V), dA = P * (dP - Delta), dQ = NN(dA, K) * scale,
 *     dK = IN(dA, Q) * scale, dV = IN(P, dO).
 *
 *   - Causal masking per axis (Fig. "neighborhoodattention" caption, Sec. 3.4
 *     "Dilation and causal masking"): along a causal axis a query never
 *     interacts with context tokens of larger coordinate.
 *
 * Readings where the paper is silent (listed in the design notes too):
 *   - window start in group coordinates is clamp(p - floor(k/2), 0, n - k);
 *     for odd k this is exactly "the k nearest same-group coordinates"; for
 *     even k it puts one more neighbour before the query than after it.
 *   - along a causal axis the window is the k nearest same-group positions
 *     not after the query: [max(0, p - k + 1), p], so queries with p < k - 1
 *     have only p + 1 neighbours on that axis (a variable window).
 *   - legal parameters: 1 <= rank <= 3, k >= 1, d >= 1, k * d <= extent.
 *   - layout [B, H, X_1 .. X_r, D] row-major, axis 1 outermost.
 *
 * Parity status: every function here is pinned by CPU tests against closed
 * forms and brute force (see tests/test_oracle_*.py); none is unpinned.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define NA_REF_MAX_RANK 3

enum {
    REF_OK = 0,
    REF_ERR_RANK = 2,
    REF_ERR_SHAPE = 3,
    REF_ERR_KERNEL_SIZE = 4,
    REF_ERR_DILATION = 5,
    REF_ERR_WINDOW_EXCEEDS_EXTENT = 6,
    REF_ERR_ALLOC = 13
};

int na_ref_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads for later calls (n >= 1); each thread still owns whole (b, h)
 * slices, so the results do not depend on n. */
void na_ref_set_num_threads(int n) {
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

static int check_problem(int rank, const int64_t* L, const int32_t* k, const int32_t* d) {
    if (rank < 1 || rank > NA_REF_MAX_RANK) return REF_ERR_RANK;
    for (int a = 0; a < rank; ++a) {
        if (L[a] < 1) return REF_ERR_SHAPE;
        if (k[a] < 1) return REF_ERR_KERNEL_SIZE;
        if (d[a] < 1) return REF_ERR_DILATION;
        if ((int64_t)k[a] * (int64_t)d[a] > L[a]) return REF_ERR_WINDOW_EXCEEDS_EXTENT;
    }
    return REF_OK;
}

/*
 * The neighbours of coordinate x along one axis of length L at dilation d;
 * returns how many there are.  The axis splits into d groups (x mod d);
 * inside its group, x sits at position p = x / d of a line of
 * n = ceil((L - g) / d) tokens.  Its window is the k consecutive group
 * positions starting at clamp(p - k/2, 0, n - k), or, along a causal axis,
 * the positions max(0, p - k + 1) .. p.
 */
static int32_t axis_window(int64_t x, int64_t L, int32_t k, int32_t d, int causal, int64_t* out) {
    int64_t g = x % d;
    int64_t p = x / d;
    int64_t n = (L - g + d - 1) / d;
    int64_t s, cnt;
    if (causal) {
        s = p - k + 1;
        if (s < 0) s = 0;
        cnt = p - s + 1;
    } else {
        s = p - k / 2;
        if (s < 0) s = 0;
        if (s > n - k) s = n - k;
        cnt = k;
    }
    for (int64_t t = 0; t < cnt; ++t) out[t] = g + (int64_t)d * (s + t);
    return (int32_t)cnt;
}

static int is_causal(const int32_t* causal, int a) { return causal != NULL && causal[a] != 0; }

static int64_t tokens_of(int rank, const int64_t* L) {
    int64_t n = 1;
    for (int a = 0; a < rank; ++a) n *= L[a];
    return n;
}

static int64_t window_size(int rank, const int32_t* k) {
    int64_t l = 1;
    for (int a = 0; a < rank; ++a) l *= k[a];
    return l;
}

/* Unravel a row-major token index into coordinates (axis 0 outermost). */
static void unravel(int rank, const int64_t* L, int64_t t, int64_t* x) {
    for (int a = rank - 1; a >= 0; --a) {
        x[a] = t % L[a];
        t /= L[a];
    }
}

/*
 * Full neighbour list of token t: the Cartesian product of the per-axis
 * windows, in row-major order (axis 0 outermost).  Writes the token indices
 * into nb and returns how many there are (prod k_a without causal axes).
 */
static int64_t neighbours_of(int rank, const int64_t* L, const int32_t* k, const int32_t* d,
                             const int32_t* causal, int64_t t, int64_t* nb) {
    int64_t x[NA_REF_MAX_RANK];
    int64_t w[NA_REF_MAX_RANK][4096];
    int32_t cnt[NA_REF_MAX_RANK];
    unravel(rank, L, t, x);
    int64_t ell = 1;
    for (int a = 0; a < rank; ++a) {
        cnt[a] = axis_window(x[a], L[a], k[a], d[a], is_causal(causal, a), w[a]);
        ell *= cnt[a];
    }
    for (int64_t e = 0; e < ell; ++e) {
        int64_t rem = e, tok = 0;
        int64_t pick[NA_REF_MAX_RANK];
        for (int a = rank - 1; a >= 0; --a) {
            pick[a] = rem % cnt[a];
            rem /= cnt[a];
        }
        for (int a = 0; a < rank; ++a) tok = tok * L[a] + w[a][pick[a]];
        nb[e] = tok;
    }
    return ell;
}

/* Neighbour lists for every token: idx is [N][prod k], rows padded with -1. */
int na_ref_neighbors(int rank, const int64_t* L, const int32_t* k, const int32_t* d,
                     const int32_t* causal, int64_t* idx) {
    int st = check_problem(rank, L, k, d);
    if (st) return st;
    for (int a = 0; a < rank; ++a)
        if (k[a] > 4096) return REF_ERR_KERNEL_SIZE;
    int64_t N = tokens_of(rank, L), ell = window_size(rank, k);
    for (int64_t t = 0; t < N; ++t) {
        int64_t c = neighbours_of(rank, L, k, d, causal, t, idx + t * ell);
        for (int64_t e = c; e < ell; ++e) idx[t * ell + e] = -1;
    }
    return REF_OK;
}

/*
 * Per-axis summary of the neighbour relation, by brute force over the axis:
 *   first[x]  = smallest neighbour coordinate of query x,
 *   inv_lo[j] = smallest query coordinate whose window contains j,
 *   inv_hi[j] = largest such query coordinate,
 *   inv_cnt[j] = number of such queries.
 */
int na_ref_axis_relation(int64_t L, int32_t k, int32_t d, int32_t causal, int64_t* first,
                         int64_t* inv_lo, int64_t* inv_hi, int64_t* inv_cnt) {
    int32_t kk[1] = {k}, dd[1] = {d};
    int64_t LL[1] = {L};
    int st = check_problem(1, LL, kk, dd);
    if (st) return st;
    int64_t* w = (int64_t*)malloc(sizeof(int64_t) * (size_t)k);
    if (!w) return REF_ERR_ALLOC;
    for (int64_t j = 0; j < L; ++j) {
        inv_lo[j] = -1;
        inv_hi[j] = -1;
        inv_cnt[j] = 0;
    }
    for (int64_t x = 0; x < L; ++x) {
        const int32_t c = axis_window(x, L, k, d, causal != 0, w);
        int64_t mn = w[0];
        for (int32_t t = 0; t < c; ++t) {
            if (w[t] < mn) mn = w[t];
            int64_t j = w[t];
            if (inv_lo[j] < 0 || x < inv_lo[j]) inv_lo[j] = x;
            if (x > inv_hi[j]) inv_hi[j] = x;
            inv_cnt[j] += 1;
        }
        first[x] = mn;
    }
    free(w);
    return REF_OK;
}

/*
 * Attention of one query row against its explicit neighbour list (Eq. 1):
 * scores, max-shifted exponentials, normalised probabilities, output row and
 * logsumexp.  p receives the ell probabilities.
 */
static void attend_row(int64_t D, double scale, const double* qrow, const double* kbase,
                       const double* vbase, const int64_t* nb, int64_t ell, double* p,
                       double* orow, double* lse) {
    double m = -INFINITY;
    for (int64_t e = 0; e < ell; ++e) {
        const double* krow = kbase + nb[e] * D;
        double s = 0.0;
        for (int64_t c = 0; c < D; ++c) s += qrow[c] * krow[c];
        s *= scale;
        p[e] = s;
        if (s > m) m = s;
    }
    double z = 0.0;
    for (int64_t e = 0; e < ell; ++e) {
        p[e] = exp(p[e] - m);
        z += p[e];
    }
    for (int64_t e = 0; e < ell; ++e) p[e] /= z;
    for (int64_t c = 0; c < D; ++c) orow[c] = 0.0;
    for (int64_t e = 0; e < ell; ++e) {
        const double* vrow = vbase + nb[e] * D;
        for (int64_t c = 0; c < D; ++c) orow[c] += p[e] * vrow[c];
    }
    *lse = m + log(z);
}

/*
 * Forward pass.  q, k, v, out are [B, H, N, D]; lse is [B, H, N].
 */
int na_ref_forward(int rank, const int64_t* L, const int32_t* ks, const int32_t* dil,
                   const int32_t* causal, int64_t B, int64_t H, int64_t D, double scale,
                   const double* q, const double* k, const double* v, double* out, double* lse) {
    int st = check_problem(rank, L, ks, dil);
    if (st) return st;
    for (int a = 0; a < rank; ++a)
        if (ks[a] > 4096) return REF_ERR_KERNEL_SIZE;
    int64_t N = tokens_of(rank, L), ell = window_size(rank, ks);
    int64_t rows = B * H * N;
    int fail = 0;
#pragma omp parallel
    {
        int64_t* nb = (int64_t*)malloc(sizeof(int64_t) * (size_t)ell);
        double* p = (double*)malloc(sizeof(double) * (size_t)ell);
        if (!nb || !p) {
#pragma omp atomic write
            fail = 1;
        } else {
#pragma omp for schedule(dynamic, 64)
            for (int64_t r = 0; r < rows; ++r) {
                int64_t slice = r / N, t = r % N;
                int64_t c = neighbours_of(rank, L, ks, dil, causal, t, nb);
                attend_row(D, scale, q + r * D, k + slice * N * D, v + slice * N * D, nb, c, p,
                           out + r * D, lse + r);
            }
        }
        free(nb);
        free(p);
    }
    return fail ? REF_ERR_ALLOC : REF_OK;
}

/*
 * Forward pass for a subset of query rows only (rows are flat indices into
 * [B*H*N]); out_rows is [nrows, D], lse_rows is [nrows].
 */
int na_ref_forward_rows(int rank, const int64_t* L, const int32_t* ks, const int32_t* dil,
                        const int32_t* causal, int64_t B, int64_t H, int64_t D, double scale,
                        const double* q, const double* k, const double* v, int64_t nrows,
                        const int64_t* rows, double* out_rows, double* lse_rows) {
    int st = check_problem(rank, L, ks, dil);
    if (st) return st;
    for (int a = 0; a < rank; ++a)
        if (ks[a] > 4096) return REF_ERR_KERNEL_SIZE;
    int64_t N = tokens_of(rank, L), ell = window_size(rank, ks);
    for (int64_t i = 0; i < nrows; ++i)
        if (rows[i] < 0 || rows[i] >= B * H * N) return REF_ERR_SHAPE;
    int fail = 0;
#pragma omp parallel
    {
        int64_t* nb = (int64_t*)malloc(sizeof(int64_t) * (size_t)ell);
        double* p = (double*)malloc(sizeof(double) * (size_t)ell);
        if (!nb || !p) {
#pragma omp atomic write
            fail = 1;
        } else {
#pragma omp for schedule(dynamic, 16)
            for (int64_t i = 0; i < nrows; ++i) {
                int64_t r = rows[i];
                int64_t slice = r / N, t = r % N;
                int64_t c = neighbours_of(rank, L, ks, dil, causal, t, nb);
                attend_row(D, scale, q + r * D, k + slice * N * D, v + slice * N * D, nb, c, p,
                           out_rows + i * D, lse_rows + i);
            }
        }
        free(nb);
        free(p);
    }
    return fail ? REF_ERR_ALLOC : REF_OK;
}

/*
 * Backward pass from the definition.  Given dO, with O and P recomputed in
 * fp64 for every query:
 *   Delta     = sum_c dO[x,c] * O[x,c]
 *   dP[x,j]   = dO[x] . v[j]                      (PN on dO and V)
 *   dA[x,j]   = P[x,j] * (dP[x,j] - Delta)
 *   dQ[x]     = scale * sum_j dA[x,j] k[j]        (NN on dA and K)
 *   dK[j]    += scale * dA[x,j] q[x]              (IN on dA and Q)
 *   dV[j]    += P[x,j] dO[x]                      (IN on P and dO)
 * One (b, h) slice per thread, so the scatter into dK/dV is race-free.
 */
int na_ref_backward(int rank, const int64_t* L, const int32_t* ks, const int32_t* dil,
                    const int32_t* causal, int64_t B, int64_t H, int64_t D, double scale,
                    const double* q, const double* k, const double* v, const double* dout,
                    double* dq, double* dk, double* dv) {
    int st = check_problem(rank, L, ks, dil);
    if (st) return st;
    for (int a = 0; a < rank; ++a)
        if (ks[a] > 4096) return REF_ERR_KERNEL_SIZE;
    int64_t N = tokens_of(rank, L), ell = window_size(rank, ks);
    int64_t slices = B * H;
    memset(dk, 0, sizeof(double) * (size_t)(slices * N * D));
    memset(dv, 0, sizeof(double) * (size_t)(slices * N * D));
    int fail = 0;
#pragma omp parallel
    {
        int64_t* nb = (int64_t*)malloc(sizeof(int64_t) * (size_t)ell);
        double* p = (double*)malloc(sizeof(double) * (size_t)ell);
        double* o = (double*)malloc(sizeof(double) * (size_t)D);
        if (!nb || !p || !o) {
#pragma omp atomic write
            fail = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t sl = 0; sl < slices; ++sl) {
                const double* qs = q + sl * N * D;
                const double* kb = k + sl * N * D;
                const double* vb = v + sl * N * D;
                const double* gs = dout + sl * N * D;
                double* dqs = dq + sl * N * D;
                double* dks = dk + sl * N * D;
                double* dvs = dv + sl * N * D;
                for (int64_t t = 0; t < N; ++t) {
                    double lse_unused;
                    int64_t cnt = neighbours_of(rank, L, ks, dil, causal, t, nb);
                    attend_row(D, scale, qs + t * D, kb, vb, nb, cnt, p, o, &lse_unused);
                    const double* g = gs + t * D;
                    double delta = 0.0;
                    for (int64_t c = 0; c < D; ++c) delta += g[c] * o[c];
                    double* dqr = dqs + t * D;
                    for (int64_t c = 0; c < D; ++c) dqr[c] = 0.0;
                    for (int64_t e = 0; e < cnt; ++e) {
                        int64_t j = nb[e];
                        const double* vr = vb + j * D;
                        double dp = 0.0;
                        for (int64_t c = 0; c < D; ++c) dp += g[c] * vr[c];
                        double da = p[e] * (dp - delta);
                        const double* kr = kb + j * D;
                        double* dkr = dks + j * D;
                        double* dvr = dvs + j * D;
                        for (int64_t c = 0; c < D; ++c) {
                            dqr[c] += scale * da * kr[c];
                            dkr[c] += scale * da * qs[t * D + c];
                            dvr[c] += p[e] * g[c];
                        }
                    }
                }
            }
        }
        free(nb);
        free(p);
        free(o);
    }
    return fail ? REF_ERR_ALLOC : REF_OK;
}

/* True when token j is among the neighbours of token t (per-axis test). */
static int is_neighbour(int rank, const int64_t* L, const int32_t* ks, const int32_t* dil,
                        const int32_t* causal, int64_t t, int64_t j, int64_t* wbuf) {
    int64_t xt[NA_REF_MAX_RANK], xj[NA_REF_MAX_RANK];
    unravel(rank, L, t, xt);
    unravel(rank, L, j, xj);
    for (int a = 0; a < rank; ++a) {
        const int32_t c = axis_window(xt[a], L[a], ks[a], dil[a], is_causal(causal, a), wbuf);
        int hit = 0;
        for (int32_t e = 0; e < c; ++e)
            if (wbuf[e] == xj[a]) hit = 1;
        if (!hit) return 0;
    }
    return 1;
}

/*
 * Backward pass for selected rows only, from the same definition:
 *   dq_rows[i] = dQ at flat query row qrows[i];
 *   dk_rows[i], dv_rows[i] = dK, dV at flat key row krows[i], summed over
 *   every query of the slice whose neighbourhood contains that key (found by
 *   scanning all queries of the slice).
 */
int na_ref_backward_rows(int rank, const int64_t* L, const int32_t* ks, const int32_t* dil,
                         const int32_t* causal, int64_t B, int64_t H, int64_t D, double scale,
                         const double* q, const double* k, const double* v, const double* dout,
                         int64_t nq, const int64_t* qrows, double* dq_rows, int64_t nk,
                         const int64_t* krows, double* dk_rows, double* dv_rows) {
    int st = check_problem(rank, L, ks, dil);
    if (st) return st;
    for (int a = 0; a < rank; ++a)
        if (ks[a] > 4096) return REF_ERR_KERNEL_SIZE;
    int64_t N = tokens_of(rank, L), ell = window_size(rank, ks);
    for (int64_t i = 0; i < nq; ++i)
        if (qrows[i] < 0 || qrows[i] >= B * H * N) return REF_ERR_SHAPE;
    for (int64_t i = 0; i < nk; ++i)
        if (krows[i] < 0 || krows[i] >= B * H * N) return REF_ERR_SHAPE;
    int fail = 0;
#pragma omp parallel
    {
        int64_t* nb = (int64_t*)malloc(sizeof(int64_t) * (size_t)ell);
        double* p = (double*)malloc(sizeof(double) * (size_t)ell);
        double* o = (double*)malloc(sizeof(double) * (size_t)D);
        int64_t* wbuf = (int64_t*)malloc(sizeof(int64_t) * 4096);
        if (!nb || !p || !o || !wbuf) {
#pragma omp atomic write
            fail = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t i = 0; i < nq; ++i) {
                int64_t r = qrows[i];
                int64_t sl = r / N, t = r % N;
                const double* kb = k + sl * N * D;
                const double* vb = v + sl * N * D;
                const double* g = dout + r * D;
                double lse_unused;
                int64_t cnt = neighbours_of(rank, L, ks, dil, causal, t, nb);
                attend_row(D, scale, q + r * D, kb, vb, nb, cnt, p, o, &lse_unused);
                double delta = 0.0;
                for (int64_t c = 0; c < D; ++c) delta += g[c] * o[c];
                double* dqr = dq_rows + i * D;
                for (int64_t c = 0; c < D; ++c) dqr[c] = 0.0;
                for (int64_t e = 0; e < cnt; ++e) {
                    const double* vr = vb + nb[e] * D;
                    double dp = 0.0;
                    for (int64_t c = 0; c < D; ++c) dp += g[c] * vr[c];
                    double da = p[e] * (dp - delta);
                    const double* kr = kb + nb[e] * D;
                    for (int64_t c = 0; c < D; ++c) dqr[c] += scale * da * kr[c];
                }
            }
#pragma omp for schedule(dynamic, 1)
            for (int64_t i = 0; i < nk; ++i) {
                int64_t r = krows[i];
                int64_t sl = r / N, j = r % N;
                const double* qs = q + sl * N * D;
                const double* kb = k + sl * N * D;
                const double* vb = v + sl * N * D;
                const double* gs = dout + sl * N * D;
                double* dkr = dk_rows + i * D;
                double* dvr = dv_rows + i * D;
                for (int64_t c = 0; c < D; ++c) {
                    dkr[c] = 0.0;
                    dvr[c] = 0.0;
                }
                for (int64_t t = 0; t < N; ++t) {
                    if (!is_neighbour(rank, L, ks, dil, causal, t, j, wbuf)) continue;
                    double lse_unused;
                    int64_t cnt = neighbours_of(rank, L, ks, dil, causal, t, nb);
                    attend_row(D, scale, qs + t * D, kb, vb, nb, cnt, p, o, &lse_unused);
                    const double* g = gs + t * D;
                    double delta = 0.0;
                    for (int64_t c = 0; c < D; ++c) delta += g[c] * o[c];
                    for (int64_t e = 0; e < cnt; ++e) {
                        if (nb[e] != j) continue;
                        const double* vr = vb + j * D;
                        double dp = 0.0;
                        for (int64_t c = 0; c < D; ++c) dp += g[c] * vr[c];
                        double da = p[e] * (dp - delta);
                        for (int64_t c = 0; c < D; ++c) {
                            dkr[c] += scale * da * qs[t * D + c];
                            dvr[c] += p[e] * g[c];
                        }
                    }
                }
            }
        }
        free(nb);
        free(p);
        free(o);
        free(wbuf);
    }
    return fail ? REF_ERR_ALLOC : REF_OK;
}

/*
 * The backward operator as the library's boundary defines it: gradients from
 * the stored forward results `out` and `lse` instead of recomputing them.
 * The probabilities come back from the logsumexp, Delta from the stored
 * output (the operators of Sec. 3.1 with P rebuilt from LSE):
 *   P[x,j]  = exp(scale * q[x].k[j] - lse[x])
 *   Delta   = sum_c dO[x,c] * out[x,c]
 *   dA[x,j] = P[x,j] * (dO[x].v[j] - Delta)
 *   dQ[x]   = scale * sum_j dA[x,j] k[j];  dK[j] += scale * dA[x,j] q[x];
 *   dV[j]  += P[x,j] dO[x].
 * When out and lse are the exact forward results this is na_ref_backward.
 *
 * dq_abs, dk_abs, dv_abs (each NULL or shaped like dq) receive the same sums
 * taken over absolute values of their terms:
 *   dq_abs[x] = scale * sum_j |dA[x,j]| |k[j]|,  dk_abs[j] = scale * sum_x |dA[x,j]| |q[x]|,
 *   dv_abs[j] = sum_x P[x,j] |dO[x]|
 * -- the magnitude a rounding of the terms (dA or P to a 16-bit type) is
 * relative to, used to bound low-precision results (standard error analysis
 * of a sum, not part of the method).
 */
int na_ref_backward_given(int rank, const int64_t* L, const int32_t* ks, const int32_t* dil,
                          const int32_t* causal, int64_t B, int64_t H, int64_t D, double scale,
                          const double* q, const double* k, const double* v, const double* out,
                          const double* lse, const double* dout, double* dq, double* dk,
                          double* dv, double* dq_abs, double* dk_abs, double* dv_abs) {
    int st = check_problem(rank, L, ks, dil);
    if (st) return st;
    for (int a = 0; a < rank; ++a)
        if (ks[a] > 4096) return REF_ERR_KERNEL_SIZE;
    int64_t N = tokens_of(rank, L), ell = window_size(rank, ks);
    int64_t slices = B * H;
    const size_t bytes = sizeof(double) * (size_t)(slices * N * D);
    memset(dk, 0, bytes);
    memset(dv, 0, bytes);
    if (dk_abs) memset(dk_abs, 0, bytes);
    if (dv_abs) memset(dv_abs, 0, bytes);
    int fail = 0;
#pragma omp parallel
    {
        int64_t* nb = (int64_t*)malloc(sizeof(int64_t) * (size_t)ell);
        if (!nb) {
#pragma omp atomic write
            fail = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t sl = 0; sl < slices; ++sl) {
                const int64_t base = sl * N * D;
                for (int64_t t = 0; t < N; ++t) {
                    const double* qr = q + base + t * D;
                    const double* g = dout + base + t * D;
                    const double* orow = out + base + t * D;
                    const double l = lse[sl * N + t];
                    int64_t cnt = neighbours_of(rank, L, ks, dil, causal, t, nb);
                    double delta = 0.0;
                    for (int64_t c = 0; c < D; ++c) delta += g[c] * orow[c];
                    double* dqr = dq + base + t * D;
                    for (int64_t c = 0; c < D; ++c) dqr[c] = 0.0;
                    if (dq_abs)
                        for (int64_t c = 0; c < D; ++c) dq_abs[base + t * D + c] = 0.0;
                    for (int64_t e = 0; e < cnt; ++e) {
                        const int64_t j = nb[e];
                        const double* kr = k + base + j * D;
                        const double* vr = v + base + j * D;
                        double s = 0.0, dp = 0.0;
                        for (int64_t c = 0; c < D; ++c) {
                            s += qr[c] * kr[c];
                            dp += g[c] * vr[c];
                        }
                        const double p = exp(scale * s - l);
                        const double da = p * (dp - delta);
                        double* dkr = dk + base + j * D;
                        double* dvr = dv + base + j * D;
                        for (int64_t c = 0; c < D; ++c) {
                            dqr[c] += scale * da * kr[c];
                            dkr[c] += scale * da * qr[c];
                            dvr[c] += p * g[c];
                        }
                        if (dq_abs)
                            for (int64_t c = 0; c < D; ++c)
                                dq_abs[base + t * D + c] += scale * fabs(da) * fabs(kr[c]);
                        if (dk_abs)
                            for (int64_t c = 0; c < D; ++c)
                                dk_abs[base + j * D + c] += scale * fabs(da) * fabs(qr[c]);
                        if (dv_abs)
                            for (int64_t c = 0; c < D; ++c)
                                dv_abs[base + j * D + c] += p * fabs(g[c]);
                    }
                }
            }
        }
        free(nb);
    }
    return fail ? REF_ERR_ALLOC : REF_OK;
}
