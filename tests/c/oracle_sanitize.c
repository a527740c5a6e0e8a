/*
 * oracle_sanitize.c -- drives every oracle entry point on small, ragged grids
 * for every op in both boundary modes, plus refused calls, so that a build
 * with AddressSanitizer and UndefinedBehaviorSanitizer (host code) checks the
 * oracle's loops for out-of-bounds accesses and undefined behaviour.  Exit
 * status 0 and "oracle-sanitize: ok" when every call returns what it should.
 */
#include <stdio.h>
#include <stdlib.h>

#include "fpde_oracle.h"

static unsigned long long rng = 88172645463325252ULL;
static double uni(void) { /* xorshift64, in [-1, 1) */
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return (double)(rng >> 11) / 4503599627370496.0 - 1.0;
}

int main(void) {
    const long shapes2[][2] = {{3, 3}, {4, 7}, {9, 5}};
    const long shapes3[][3] = {{3, 3, 3}, {4, 5, 7}, {6, 3, 5}};
    const long shapes4[][4] = {{3, 3, 3, 3}, {4, 3, 5, 6}, {5, 4, 3, 4}};
    const double coef[4] = {0.01, 2.0, 0.1, 0.3};
    int bad = 0, calls = 0;
    for (int op = 1; op <= 10; ++op) {
        int ndim, nf, nc, nr;
        if (orc_op_info(op, &ndim, &nf, &nc, &nr) != 0) {
            printf("oracle-sanitize: op_info %d failed\n", op);
            return 1;
        }
        for (int si = 0; si < 3; ++si) {
            const long* n = ndim == 2 ? shapes2[si] : ndim == 3 ? shapes3[si] : shapes4[si];
            long N = 1;
            for (int a = 0; a < ndim; ++a) N *= n[a];
            const double h[4] = {0.5, 0.25, 0.125, 0.375};
            double *f[4], *c[3], *G[4], *R[4], *g[4];
            for (int i = 0; i < nf; ++i) {
                f[i] = malloc(N * sizeof(double));
                g[i] = malloc(N * sizeof(double));
                for (long m = 0; m < N; ++m) f[i][m] = uni();
            }
            for (int i = 0; i < nc; ++i) {
                c[i] = malloc(N * sizeof(double));
                for (long m = 0; m < N; ++m) c[i][m] = uni();
            }
            for (int b = 0; b < nr; ++b) {
                G[b] = malloc(N * sizeof(double));
                R[b] = malloc(N * sizeof(double));
                for (long m = 0; m < N; ++m) G[b][m] = uni();
            }
            for (int bc = 0; bc <= 1; ++bc) {
                double L;
                const double* const* cf = (const double* const*)f;
                const double* const* cc = (const double* const*)c;
                bad |= orc_residual(op, ndim, n, h, bc, coef, cf, cc, R) != 0;
                bad |= orc_loss(op, ndim, n, h, bc, coef, cf, cc, &L) != 0;
                bad |= orc_vjp(op, ndim, n, h, bc, coef, cf, cc, (const double* const*)G, g) != 0;
                bad |= orc_grad(op, ndim, n, h, bc, coef, cf, cc, 0.5, g) != 0;
                bad |= !(L == L);
                calls += 4;
            }
            for (int i = 0; i < nf; ++i) {
                free(f[i]);
                free(g[i]);
            }
            for (int i = 0; i < nc; ++i) free(c[i]);
            for (int b = 0; b < nr; ++b) {
                free(G[b]);
                free(R[b]);
            }
        }
    }
    /* refused calls */
    const long n2[2] = {2, 5};
    const double h2[2] = {0.1, 0.1};
    double L;
    bad |= orc_loss(4, 2, n2, h2, 0, coef, NULL, NULL, &L) == 0;
    bad |= orc_op_info(0, NULL, NULL, NULL, NULL) == 0;
    if (bad) {
        printf("oracle-sanitize: a call returned an unexpected status\n");
        return 1;
    }
    printf("oracle-sanitize: ok (%d calls)\n", calls);
    return 0;
}
