/* Sanitizer driver for the fp64 oracle (oracle/na_ref.c), built by
 * tests/test_sanitizers.py with -fsanitize=address,undefined: runs every entry
 * point on small problems of each rank (dilation, causal axes, even windows,
 * k = extent) and checks the outputs are finite and that the backward from
 * stored results matches the plain backward.  Exit status 0 on success. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int na_ref_neighbors(int, const int64_t*, const int32_t*, const int32_t*, const int32_t*, int64_t*);
int na_ref_axis_relation(int64_t, int32_t, int32_t, int32_t, int64_t*, int64_t*, int64_t*, int64_t*);
int na_ref_forward(int, const int64_t*, const int32_t*, const int32_t*, const int32_t*, int64_t,
                   int64_t, int64_t, double, const double*, const double*, const double*, double*,
                   double*);
int na_ref_forward_rows(int, const int64_t*, const int32_t*, const int32_t*, const int32_t*, int64_t,
                        int64_t, int64_t, double, const double*, const double*, const double*,
                        int64_t, const int64_t*, double*, double*);
int na_ref_backward(int, const int64_t*, const int32_t*, const int32_t*, const int32_t*, int64_t,
                    int64_t, int64_t, double, const double*, const double*, const double*,
                    const double*, double*, double*, double*);
int na_ref_backward_given(int, const int64_t*, const int32_t*, const int32_t*, const int32_t*,
                          int64_t, int64_t, int64_t, double, const double*, const double*,
                          const double*, const double*, const double*, const double*, double*,
                          double*, double*, double*, double*, double*);
int na_ref_backward_rows(int, const int64_t*, const int32_t*, const int32_t*, const int32_t*,
                         int64_t, int64_t, int64_t, double, const double*, const double*,
                         const double*, const double*, int64_t, const int64_t*, double*, int64_t,
                         const int64_t*, double*, double*);

static double frand(unsigned* s) {
    *s = *s * 1103515245u + 12345u;
    return ((*s >> 8) & 0xffff) / 32768.0 - 1.0;
}

static int finite_all(const double* a, int64_t n) {
    for (int64_t i = 0; i < n; ++i)
        if (!isfinite(a[i])) return 0;
    return 1;
}

struct Case { int rank; int64_t L[3]; int32_t k[3], d[3], c[3]; };

int main(void) {
    const struct Case cases[] = {
        {1, {13, 0, 0}, {4, 0, 0}, {3, 0, 0}, {0, 0, 0}},
        {1, {10, 0, 0}, {10, 0, 0}, {1, 0, 0}, {1, 0, 0}},
        {2, {9, 7, 0}, {3, 2, 0}, {2, 3, 0}, {0, 1, 0}},
        {2, {6, 6, 0}, {6, 6, 0}, {1, 1, 0}, {0, 0, 0}},
        {3, {4, 5, 6}, {3, 3, 2}, {1, 1, 3}, {1, 0, 0}},
        {3, {5, 4, 7}, {1, 4, 3}, {2, 1, 2}, {0, 0, 1}},
    };
    const int64_t B = 1, H = 2, D = 3;
    unsigned seed = 7;
    for (size_t ci = 0; ci < sizeof(cases) / sizeof(cases[0]); ++ci) {
        const struct Case* cs = &cases[ci];
        int64_t N = 1, ell = 1;
        for (int a = 0; a < cs->rank; ++a) {
            N *= cs->L[a];
            ell *= cs->k[a];
        }
        const int64_t n = B * H * N * D, nr = B * H * N;
        double *q = malloc(sizeof(double) * n), *k = malloc(sizeof(double) * n),
               *v = malloc(sizeof(double) * n), *g = malloc(sizeof(double) * n),
               *o = malloc(sizeof(double) * n), *l = malloc(sizeof(double) * nr),
               *dq = malloc(sizeof(double) * n), *dk = malloc(sizeof(double) * n),
               *dv = malloc(sizeof(double) * n), *dq2 = malloc(sizeof(double) * n),
               *dk2 = malloc(sizeof(double) * n), *dv2 = malloc(sizeof(double) * n),
               *aq = malloc(sizeof(double) * n), *ak = malloc(sizeof(double) * n),
               *av = malloc(sizeof(double) * n);
        int64_t* nb = malloc(sizeof(int64_t) * N * ell);
        for (int64_t i = 0; i < n; ++i) {
            q[i] = frand(&seed);
            k[i] = frand(&seed);
            v[i] = frand(&seed);
            g[i] = frand(&seed);
        }
        int st = na_ref_neighbors(cs->rank, cs->L, cs->k, cs->d, cs->c, nb);
        st |= na_ref_forward(cs->rank, cs->L, cs->k, cs->d, cs->c, B, H, D, 0.7, q, k, v, o, l);
        st |= na_ref_backward(cs->rank, cs->L, cs->k, cs->d, cs->c, B, H, D, 0.7, q, k, v, g, dq, dk, dv);
        st |= na_ref_backward_given(cs->rank, cs->L, cs->k, cs->d, cs->c, B, H, D, 0.7, q, k, v, o, l,
                                    g, dq2, dk2, dv2, aq, ak, av);
        int64_t rows[3] = {0, nr / 2, nr - 1};
        double ro[9], rl[3], rq[9], rk[9], rv[9];
        st |= na_ref_forward_rows(cs->rank, cs->L, cs->k, cs->d, cs->c, B, H, D, 0.7, q, k, v, 3, rows,
                                  ro, rl);
        st |= na_ref_backward_rows(cs->rank, cs->L, cs->k, cs->d, cs->c, B, H, D, 0.7, q, k, v, g, 3,
                                   rows, rq, 3, rows, rk, rv);
        for (int a = 0; a < cs->rank; ++a) {
            int64_t* r4 = malloc(sizeof(int64_t) * 4 * cs->L[a]);
            st |= na_ref_axis_relation(cs->L[a], cs->k[a], cs->d[a], cs->c[a], r4, r4 + cs->L[a],
                                       r4 + 2 * cs->L[a], r4 + 3 * cs->L[a]);
            free(r4);
        }
        if (st != 0 || !finite_all(o, n) || !finite_all(l, nr) || !finite_all(dq, n) ||
            !finite_all(dk, n) || !finite_all(dv, n)) {
            printf("FAIL case %zu status %d\n", ci, st);
            return 1;
        }
        double worst = 0.0;
        for (int64_t i = 0; i < n; ++i) {
            worst = fmax(worst, fabs(dq[i] - dq2[i]));
            worst = fmax(worst, fabs(dk[i] - dk2[i]));
            worst = fmax(worst, fabs(dv[i] - dv2[i]));
        }
        if (worst > 1e-12) {
            printf("FAIL case %zu backward_given differs by %g\n", ci, worst);
            return 1;
        }
        free(q); free(k); free(v); free(g); free(o); free(l); free(dq); free(dk); free(dv);
        free(dq2); free(dk2); free(dv2); free(aq); free(ak); free(av); free(nb);
    }
    /* invalid problems return an error before touching any buffer */
    const int64_t L1[1] = {5};
    const int32_t k1[1] = {6}, d1[1] = {1};
    if (na_ref_forward(1, L1, k1, d1, NULL, 1, 1, 2, 1.0, NULL, NULL, NULL, NULL, NULL) == 0) {
        printf("FAIL invalid window accepted\n");
        return 1;
    }
    printf("ok oracle\n");
    return 0;
}
