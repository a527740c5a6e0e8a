/*
 * abi_c_check.c -- the C ABI of libfpde used from C alone (no Python, no
 * torch): device buffers from the HIP runtime, every entry point called on a
 * small 3-D backward-Euler Navier-Stokes grid (fpde_grid) and every four-axis
 * entry point on a small 3D+t Navier-Stokes space-time grid (fpde_grid4),
 * results compared with the CPU oracle (test infrastructure, linked by this
 * test program only).
 * Exit status 0 and a line "c-abi: ok" when every comparison holds.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "fpde.h"
#include "fpde_oracle.h"

#define CK(x)                                                                 \
    do {                                                                      \
        hipError_t e_ = (x);                                                  \
        if (e_ != hipSuccess) {                                               \
            printf("c-abi: HIP error %s at line %d\n", hipGetErrorString(e_), \
                   __LINE__);                                                 \
            exit(2);                                                          \
        }                                                                     \
    } while (0)

#define NF 4
#define NC 3
#define NR 4

static int fails = 0;

static void check(const char* what, double err, double bar) {
    printf("c-abi: %-28s rel err %.3e (bar %.0e)\n", what, err, bar);
    if (!(err <= bar)) fails++;
}

/* max |got - ref| / max |ref| over n values */
static double rel_err(const float* got, const double* ref, long n) {
    double e = 0.0, s = 0.0;
    for (long i = 0; i < n; ++i) {
        const double d = fabs((double)got[i] - ref[i]);
        if (d > e || d != d) e = d;
        if (fabs(ref[i]) > s) s = fabs(ref[i]);
    }
    return s > 0 ? e / s : e;
}

static int check_ns3d(void) {
    const long n[3] = {20, 24, 70};
    const long N = n[0] * n[1] * n[2];
    const double pi = 3.14159265358979323846;
    const double h[3] = {2 * pi / n[0], 2 * pi / n[1], 2 * pi / n[2]};
    const double coef[4] = {0.01, 0.0, 1e-2, 0.0}; /* nu, k, dt, alpha */

    /* Taylor-Green initial condition (consts) and a perturbed copy (fields) */
    float* hf[NF];
    float* hc[NC];
    float* hg[NR];
    for (int a = 0; a < NF; ++a) hf[a] = malloc(N * sizeof(float));
    for (int a = 0; a < NC; ++a) hc[a] = malloc(N * sizeof(float));
    for (int a = 0; a < NR; ++a) hg[a] = malloc(N * sizeof(float));
    for (long i = 0; i < n[0]; ++i)
        for (long j = 0; j < n[1]; ++j)
            for (long k = 0; k < n[2]; ++k) {
                const long m = (i * n[1] + j) * n[2] + k;
                const double x = i * h[0], y = j * h[1], z = k * h[2];
                const double ic[4] = {sin(x) * cos(y) * cos(z), -cos(x) * sin(y) * cos(z), 0.0,
                                      (cos(2 * x) + cos(2 * y)) * (cos(2 * z) + 2) / 16};
                for (int a = 0; a < NF; ++a)
                    hf[a][m] = (float)(ic[a] + 0.01 * sin(12.9898 * m + 78.233 * a));
                for (int a = 0; a < NC; ++a) hc[a][m] = (float)ic[a];
                for (int b = 0; b < NR; ++b) hg[b][m] = (float)cos(0.37 * m + 1.3 * b);
            }

    /* device buffers */
    float *df[NF], *dc[NC], *dR[NR], *dG[NR], *dg[NF], *dgv[NF], *dgj[NF];
    double *dloss, *ddl, *dloss_v;
    const size_t bytes = N * sizeof(float);
    for (int a = 0; a < NF; ++a) {
        CK(hipMalloc((void**)&df[a], bytes));
        CK(hipMemcpy(df[a], hf[a], bytes, hipMemcpyHostToDevice));
        CK(hipMalloc((void**)&dg[a], bytes));
        CK(hipMalloc((void**)&dgv[a], bytes));
        CK(hipMalloc((void**)&dgj[a], bytes));
    }
    for (int a = 0; a < NC; ++a) {
        CK(hipMalloc((void**)&dc[a], bytes));
        CK(hipMemcpy(dc[a], hc[a], bytes, hipMemcpyHostToDevice));
    }
    for (int b = 0; b < NR; ++b) {
        CK(hipMalloc((void**)&dR[b], bytes));
        CK(hipMalloc((void**)&dG[b], bytes));
        CK(hipMemcpy(dG[b], hg[b], bytes, hipMemcpyHostToDevice));
    }
    CK(hipMalloc((void**)&dloss, sizeof(double)));
    CK(hipMalloc((void**)&dloss_v, sizeof(double)));
    CK(hipMalloc((void**)&ddl, sizeof(double)));
    const double one = 1.0;
    CK(hipMemcpy(ddl, &one, sizeof(double), hipMemcpyHostToDevice));

    fpde_grid grid;
    memset(&grid, 0, sizeof grid);
    grid.ndim = 3;
    grid.bc_mode = 0;
    for (int a = 0; a < 3; ++a) {
        grid.n[a] = n[a];
        grid.h[a] = h[a];
    }
    const fpde_coeffs co = {coef[0], coef[1], coef[2], coef[3]};
    const float* cf[NF] = {df[0], df[1], df[2], df[3]};
    const float* cc[NC] = {dc[0], dc[1], dc[2]};
    const float* cG[NR] = {dG[0], dG[1], dG[2], dG[3]};

    int ndim, nf, nc, nr;
    if (fpde_op_info(FPDE_NS_3D_BE, &ndim, &nf, &nc, &nr) != FPDE_OK || ndim != 3 || nf != NF ||
        nc != NC || nr != NR) {
        printf("c-abi: fpde_op_info disagrees\n");
        return 1;
    }
    /* error paths: nothing is queued, a status comes back */
    if (fpde_residual_fwd(FPDE_NS_3D_BE, &grid, &co, cf, cc, NULL, NULL, NULL) != FPDE_ERR_ARG ||
        fpde_residual_bwd(FPDE_NS_3D_BE, &grid, &co, cf, cc, ddl, (float* const*)cf, NULL) !=
            FPDE_ERR_ARG ||
        fpde_residual_fwd(99, &grid, &co, cf, cc, NULL, dloss, NULL) != FPDE_ERR_ARG) {
        printf("c-abi: an invalid call was not refused\n");
        return 1;
    }
    printf("c-abi: %s; invalid calls refused (%s)\n", fpde_version(),
           fpde_status_string(FPDE_ERR_ARG));

    int st = fpde_residual_fwd(FPDE_NS_3D_BE, &grid, &co, cf, cc, dR, dloss, NULL);
    st |= fpde_residual_bwd(FPDE_NS_3D_BE, &grid, &co, cf, cc, ddl, dg, NULL);
    st |= fpde_bc_correct(FPDE_NS_3D_BE, &grid, &co, cf, cc, ddl, dg, NULL);
    st |= fpde_residual_value_and_grad(FPDE_NS_3D_BE, &grid, &co, cf, cc, ddl, dloss_v, dgv, NULL);
    st |= fpde_residual_vjp(FPDE_NS_3D_BE, &grid, &co, cf, cG, 0, dgj, NULL);
    if (st != FPDE_OK) {
        printf("c-abi: a valid call failed (%d)\n", st);
        return 1;
    }
    CK(hipDeviceSynchronize());

    /* the oracle on the same float32 inputs, widened */
    double *of[NF], *oc[NC], *oG[NR], *oR[NR], *og[NF], *oj[NF];
    for (int a = 0; a < NF; ++a) {
        of[a] = malloc(N * sizeof(double));
        og[a] = malloc(N * sizeof(double));
        oj[a] = malloc(N * sizeof(double));
        for (long m = 0; m < N; ++m) of[a][m] = hf[a][m];
    }
    for (int a = 0; a < NC; ++a) {
        oc[a] = malloc(N * sizeof(double));
        for (long m = 0; m < N; ++m) oc[a][m] = hc[a][m];
    }
    for (int b = 0; b < NR; ++b) {
        oG[b] = malloc(N * sizeof(double));
        oR[b] = malloc(N * sizeof(double));
        for (long m = 0; m < N; ++m) oG[b][m] = hg[b][m];
    }
    double L_ref;
    st = orc_loss(5, 3, n, h, 0, coef, (const double* const*)of, (const double* const*)oc, &L_ref);
    st |= orc_residual(5, 3, n, h, 0, coef, (const double* const*)of, (const double* const*)oc, oR);
    st |= orc_grad(5, 3, n, h, 0, coef, (const double* const*)of, (const double* const*)oc, 1.0, og);
    st |= orc_vjp(5, 3, n, h, 0, coef, (const double* const*)of, (const double* const*)oc,
                  (const double* const*)oG, oj);
    if (st != 0) {
        printf("c-abi: oracle failed (%d)\n", st);
        return 1;
    }

    double L, Lv;
    CK(hipMemcpy(&L, dloss, sizeof(double), hipMemcpyDeviceToHost));
    CK(hipMemcpy(&Lv, dloss_v, sizeof(double), hipMemcpyDeviceToHost));
    check("loss (fwd)", fabs(L - L_ref) / fabs(L_ref), 1e-5);
    check("loss (value_and_grad)", fabs(Lv - L_ref) / fabs(L_ref), 1e-5);
    float* buf = malloc(bytes);
    const char* names[4] = {"u", "v", "w", "p"};
    char what[64];
    for (int b = 0; b < NR; ++b) {
        CK(hipMemcpy(buf, dR[b], bytes, hipMemcpyDeviceToHost));
        snprintf(what, sizeof what, "residual %d", b);
        check(what, rel_err(buf, oR[b], N), 1e-5);
    }
    for (int a = 0; a < NF; ++a) {
        CK(hipMemcpy(buf, dg[a], bytes, hipMemcpyDeviceToHost));
        snprintf(what, sizeof what, "grad %s (bwd + bc)", names[a]);
        check(what, rel_err(buf, og[a], N), 1e-4);
        CK(hipMemcpy(buf, dgv[a], bytes, hipMemcpyDeviceToHost));
        snprintf(what, sizeof what, "grad %s (value_and_grad)", names[a]);
        check(what, rel_err(buf, og[a], N), 1e-4);
        CK(hipMemcpy(buf, dgj[a], bytes, hipMemcpyDeviceToHost));
        snprintf(what, sizeof what, "grad %s (vjp)", names[a]);
        check(what, rel_err(buf, oj[a], N), 1e-4);
    }
    return 0;
}

/* 3D+t NS on a t x x x y x z grid with several time levels, tiles and chunks
 * and a ragged last tile: the four-axis entry points against the oracle.  The
 * op has no consts (the neighbouring levels' velocities are its own fields). */
static int check_ns3dt(void) {
    enum { F4 = 4, R4 = 4 };
    const long n[4] = {6, 12, 17, 70};
    const long V = n[1] * n[2] * n[3], N = n[0] * V;
    const double pi = 3.14159265358979323846;
    const double h[4] = {1.0 / (n[0] - 1), 2 * pi / n[1], 2 * pi / n[2], 2 * pi / n[3]};
    const double coef[4] = {0.01, 0.0, 0.0, 0.0}; /* nu */
    float* hf[F4];
    float* hg[R4];
    for (int a = 0; a < F4; ++a) hf[a] = malloc(N * sizeof(float));
    for (int b = 0; b < R4; ++b) hg[b] = malloc(N * sizeof(float));
    /* a decaying Taylor-Green field, perturbed */
    for (long t = 0; t < n[0]; ++t)
        for (long i = 0; i < n[1]; ++i)
            for (long j = 0; j < n[2]; ++j)
                for (long k = 0; k < n[3]; ++k) {
                    const long m = ((t * n[1] + i) * n[2] + j) * n[3] + k;
                    const double x = i * h[1], y = j * h[2], z = k * h[3];
                    const double d = exp(-3 * coef[0] * t * h[0]);
                    const double ic[4] = {d * sin(x) * cos(y) * cos(z), -d * cos(x) * sin(y) * cos(z),
                                          0.0, d * d * (cos(2 * x) + cos(2 * y)) * (cos(2 * z) + 2) / 16};
                    for (int a = 0; a < F4; ++a)
                        hf[a][m] = (float)(ic[a] + 0.01 * sin(12.9898 * m + 78.233 * a));
                    for (int b = 0; b < R4; ++b) hg[b][m] = (float)cos(0.37 * m + 1.3 * b);
                }
    float *df[F4], *dR[R4], *dG[R4], *dg[F4], *dgv[F4], *dgj[F4];
    double *dloss, *ddl, *dloss_v;
    const size_t bytes = N * sizeof(float);
    for (int a = 0; a < F4; ++a) {
        CK(hipMalloc((void**)&df[a], bytes));
        CK(hipMemcpy(df[a], hf[a], bytes, hipMemcpyHostToDevice));
        CK(hipMalloc((void**)&dg[a], bytes));
        CK(hipMalloc((void**)&dgv[a], bytes));
        CK(hipMalloc((void**)&dgj[a], bytes));
    }
    for (int b = 0; b < R4; ++b) {
        CK(hipMalloc((void**)&dR[b], bytes));
        CK(hipMalloc((void**)&dG[b], bytes));
        CK(hipMemcpy(dG[b], hg[b], bytes, hipMemcpyHostToDevice));
    }
    CK(hipMalloc((void**)&dloss, sizeof(double)));
    CK(hipMalloc((void**)&dloss_v, sizeof(double)));
    CK(hipMalloc((void**)&ddl, sizeof(double)));
    const double dl = 0.75;
    CK(hipMemcpy(ddl, &dl, sizeof(double), hipMemcpyHostToDevice));

    fpde_grid4 grid;
    memset(&grid, 0, sizeof grid);
    grid.ndim = 4;
    grid.bc_mode = 0;
    for (int a = 0; a < 4; ++a) {
        grid.n[a] = n[a];
        grid.h[a] = h[a];
    }
    const fpde_coeffs co = {coef[0], coef[1], coef[2], coef[3]};
    const float* cf[F4] = {df[0], df[1], df[2], df[3]};
    const float* cG[R4] = {dG[0], dG[1], dG[2], dG[3]};

    int ndim, nf, nc, nr;
    if (fpde_op_info(FPDE_NS_3DT, &ndim, &nf, &nc, &nr) != FPDE_OK || ndim != 4 || nf != F4 ||
        nc != 0 || nr != R4) {
        printf("c-abi: fpde_op_info disagrees (3D+t)\n");
        return 1;
    }
    /* a four-axis op through a three-axis grid, and a three-axis grid's op
     * through fpde_grid4 with ndim 4: refused, nothing queued */
    fpde_grid g3;
    memset(&g3, 0, sizeof g3);
    g3.ndim = 3;
    for (int a = 0; a < 3; ++a) {
        g3.n[a] = n[a + 1];
        g3.h[a] = h[a + 1];
    }
    if (fpde_residual_fwd(FPDE_NS_3DT, &g3, &co, cf, NULL, NULL, dloss, NULL) != FPDE_ERR_SHAPE ||
        fpde_residual_fwd4(FPDE_NS_3D_BE, &grid, &co, cf, cf, NULL, dloss, NULL) !=
            FPDE_ERR_SHAPE) {
        printf("c-abi: a grid of the wrong rank was not refused\n");
        return 1;
    }

    int st = fpde_residual_fwd4(FPDE_NS_3DT, &grid, &co, cf, NULL, dR, dloss, NULL);
    st |= fpde_residual_bwd4(FPDE_NS_3DT, &grid, &co, cf, NULL, ddl, dg, NULL);
    st |= fpde_bc_correct4(FPDE_NS_3DT, &grid, &co, cf, NULL, ddl, dg, NULL);
    st |= fpde_residual_value_and_grad4(FPDE_NS_3DT, &grid, &co, cf, NULL, ddl, dloss_v, dgv,
                                        NULL);
    st |= fpde_residual_vjp4(FPDE_NS_3DT, &grid, &co, cf, cG, 0, dgj, NULL);
    if (st != FPDE_OK) {
        printf("c-abi: a valid four-axis call failed (%d)\n", st);
        return 1;
    }
    CK(hipDeviceSynchronize());

    double *of[F4], *oG[R4], *oR[R4], *og[F4], *oj[F4];
    for (int a = 0; a < F4; ++a) {
        of[a] = malloc(N * sizeof(double));
        og[a] = malloc(N * sizeof(double));
        oj[a] = malloc(N * sizeof(double));
        for (long m = 0; m < N; ++m) of[a][m] = hf[a][m];
    }
    for (int b = 0; b < R4; ++b) {
        oG[b] = malloc(N * sizeof(double));
        oR[b] = malloc(N * sizeof(double));
        for (long m = 0; m < N; ++m) oG[b][m] = hg[b][m];
    }
    double L_ref;
    const double* const* ocf = (const double* const*)of;
    st = orc_loss(FPDE_NS_3DT, 4, n, h, 0, coef, ocf, NULL, &L_ref);
    st |= orc_residual(FPDE_NS_3DT, 4, n, h, 0, coef, ocf, NULL, oR);
    st |= orc_grad(FPDE_NS_3DT, 4, n, h, 0, coef, ocf, NULL, dl, og);
    st |= orc_vjp(FPDE_NS_3DT, 4, n, h, 0, coef, ocf, NULL, (const double* const*)oG, oj);
    if (st != 0) {
        printf("c-abi: oracle failed on 3D+t (%d)\n", st);
        return 1;
    }
    double L, Lv;
    CK(hipMemcpy(&L, dloss, sizeof(double), hipMemcpyDeviceToHost));
    CK(hipMemcpy(&Lv, dloss_v, sizeof(double), hipMemcpyDeviceToHost));
    check("3D+t loss (fwd4)", fabs(L - L_ref) / fabs(L_ref), 1e-5);
    check("3D+t loss (value_and_grad4)", fabs(Lv - L_ref) / fabs(L_ref), 1e-5);
    float* buf = malloc(bytes);
    const char* names[4] = {"u", "v", "w", "p"};
    char what[64];
    for (int b = 0; b < R4; ++b) {
        CK(hipMemcpy(buf, dR[b], bytes, hipMemcpyDeviceToHost));
        snprintf(what, sizeof what, "3D+t residual %d", b);
        check(what, rel_err(buf, oR[b], N), 1e-5);
    }
    for (int a = 0; a < F4; ++a) {
        CK(hipMemcpy(buf, dg[a], bytes, hipMemcpyDeviceToHost));
        snprintf(what, sizeof what, "3D+t grad %s (bwd4 + bc4)", names[a]);
        check(what, rel_err(buf, og[a], N), 1e-4);
        CK(hipMemcpy(buf, dgv[a], bytes, hipMemcpyDeviceToHost));
        snprintf(what, sizeof what, "3D+t grad %s (vg4)", names[a]);
        check(what, rel_err(buf, og[a], N), 1e-4);
        CK(hipMemcpy(buf, dgj[a], bytes, hipMemcpyDeviceToHost));
        snprintf(what, sizeof what, "3D+t grad %s (vjp4)", names[a]);
        check(what, rel_err(buf, oj[a], N), 1e-4);
    }
    return 0;
}

int main(void) {
    if (check_ns3d() != 0 || check_ns3dt() != 0) return 1;
    if (fails) {
        printf("c-abi: %d comparison(s) failed\n", fails);
        return 1;
    }
    printf("c-abi: ok\n");
    return 0;
}
