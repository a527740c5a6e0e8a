/*
 * abi_host_sanitize.c -- the library's host-side argument validation under
 * AddressSanitizer and UndefinedBehaviorSanitizer (host code only; built
 * against a host-only build of the library, no GPU).  Every call below breaks
 * exactly one rule of include/fpde.h, so validation must return its status
 * before anything is queued; the "device pointers" are host addresses, which
 * validation only compares and checks for alignment.  Exit status 0 and a line
 * "abi-host-sanitize: ok" when every call returns the expected status and no
 * sanitizer reports.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "fpde.h"

static int fails = 0, calls = 0;

static void expect(const char* what, int got, int want) {
    ++calls;
    if (got != want) {
        printf("abi-host-sanitize: %s returned %d (%s), expected %d\n", what, got,
               fpde_status_string(got), want);
        ++fails;
    }
}

static float buf[64][16];  /* distinct, aligned stand-ins for device arrays */
static double dbuf[4];

static const float* const* ptrs(int first, int n, const float** store) {
    for (int i = 0; i < n; ++i) store[i] = buf[first + i];
    return store;
}

int main(void) {
    const fpde_coeffs co = {0.01, 2.0, 1e-2, 0.1};
    const float* fs[8];
    const float* cs[8];
    float* gs[8];
    for (int i = 0; i < 8; ++i) gs[i] = buf[32 + i];
    double* loss = &dbuf[0];
    const double* dl = &dbuf[1];

    /* op table, strings */
    for (int op = 0; op <= 11; ++op) {
        int nd = -1, nf = -1, nc = -1, nr = -1;
        const int st = fpde_op_info(op, &nd, &nf, &nc, &nr);
        expect("fpde_op_info", st == FPDE_OK ? (nd >= 2 && nd <= 4 && nf >= 1 && nr >= 1) : 1, 1);
        expect("fpde_op_info with null outputs", fpde_op_info(op, NULL, NULL, NULL, NULL), st);
    }
    for (int s = -10; s <= 2; ++s) expect("fpde_status_string", fpde_status_string(s) != NULL, 1);
    expect("fpde_version", fpde_version() != NULL, 1);

    /* 3-D backward-Euler NS: 4 fields, 3 consts */
    fpde_grid g;
    memset(&g, 0, sizeof g);
    g.ndim = 3;
    for (int a = 0; a < 3; ++a) {
        g.n[a] = 9;
        g.h[a] = 0.1;
    }
    const float* const* F = ptrs(0, 4, fs);
    const float* const* C = ptrs(8, 3, cs);
    const int op = FPDE_NS_3D_BE;

    expect("unknown op", fpde_residual_fwd(99, &g, &co, F, C, NULL, loss, NULL), FPDE_ERR_ARG);
    expect("null grid", fpde_residual_fwd(op, NULL, &co, F, C, NULL, loss, NULL), FPDE_ERR_ARG);
    expect("null coeffs", fpde_residual_fwd(op, &g, NULL, F, C, NULL, loss, NULL), FPDE_ERR_ARG);
    expect("null fields", fpde_residual_fwd(op, &g, &co, NULL, C, NULL, loss, NULL), FPDE_ERR_ARG);
    expect("null consts", fpde_residual_fwd(op, &g, &co, F, NULL, NULL, loss, NULL), FPDE_ERR_ARG);
    expect("null loss", fpde_residual_fwd(op, &g, &co, F, C, NULL, NULL, NULL), FPDE_ERR_ARG);
    {
        const float* bad[4] = {F[0], NULL, F[2], F[3]};
        expect("null field 1", fpde_residual_fwd(op, &g, &co, bad, C, NULL, loss, NULL), FPDE_ERR_ARG);
    }
    {
        fpde_grid b = g;
        b.bc_mode = 2;
        expect("bc_mode 2", fpde_residual_fwd(op, &b, &co, F, C, NULL, loss, NULL), FPDE_ERR_ARG);
        b = g;
        b.ndim = 2;
        expect("wrong rank", fpde_residual_fwd(op, &b, &co, F, C, NULL, loss, NULL), FPDE_ERR_SHAPE);
        b = g;
        b.n[1] = 2;
        expect("n < 3", fpde_residual_fwd(op, &b, &co, F, C, NULL, loss, NULL), FPDE_ERR_SHAPE);
        b = g;
        b.n[0] = (int64_t)1 << 31;
        expect("n = 2^31", fpde_residual_fwd(op, &b, &co, F, C, NULL, loss, NULL), FPDE_ERR_SHAPE);
        b = g;
        b.n[0] = b.n[1] = b.n[2] = ((int64_t)1 << 31) - 1;
        expect("N beyond 2^62", fpde_residual_fwd(op, &b, &co, F, C, NULL, loss, NULL), FPDE_ERR_SHAPE);
        b = g;
        b.n[1] = 1 << 15;
        b.n[2] = 1 << 14;
        expect("plane of 2^29", fpde_residual_fwd(op, &b, &co, F, C, NULL, loss, NULL), FPDE_ERR_SHAPE);
        b = g;
        b.n[0] = ((int64_t)1 << 31) - 1;  /* a long first axis: too many workgroups */
        expect("axis 0 of 2^31 - 1", fpde_residual_fwd(op, &b, &co, F, C, NULL, loss, NULL),
               FPDE_ERR_SHAPE);
        b = g;
        b.h[2] = 0.0;
        expect("h = 0", fpde_residual_fwd(op, &b, &co, F, C, NULL, loss, NULL), FPDE_ERR_SPACING);
        b = g;
        b.h[1] = NAN;
        expect("h = NaN", fpde_residual_fwd(op, &b, &co, F, C, NULL, loss, NULL), FPDE_ERR_SPACING);
        b = g;
        b.h[0] = 1e-300;  /* 1/h^2 overflows float32 */
        expect("tiny h", fpde_residual_fwd(op, &b, &co, F, C, NULL, loss, NULL), FPDE_ERR_SPACING);
    }
    {
        fpde_coeffs c = co;
        c.dt = 0.0;
        expect("dt = 0", fpde_residual_fwd(op, &g, &c, F, C, NULL, loss, NULL), FPDE_ERR_COEFF);
        c = co;
        c.nu = INFINITY;
        expect("nu = inf", fpde_residual_fwd(op, &g, &c, F, C, NULL, loss, NULL), FPDE_ERR_COEFF);
        c = co;
        c.k = 1e200;  /* k^2 overflows float32 */
        expect("huge k", fpde_residual_fwd(op, &g, &c, F, C, NULL, loss, NULL), FPDE_ERR_COEFF);
    }
    {
        const float* mis[4] = {F[0], (const float*)((const char*)F[1] + 2), F[2], F[3]};
        expect("misaligned field", fpde_residual_fwd(op, &g, &co, mis, C, NULL, loss, NULL),
               FPDE_ERR_ALIGN);
        const float* misc[3] = {C[0], C[1], (const float*)((const char*)C[2] + 1)};
        expect("misaligned const", fpde_residual_fwd(op, &g, &co, F, misc, NULL, loss, NULL),
               FPDE_ERR_ALIGN);
    }
    /* outputs: overlaps with the inputs, each other, the loss; null entries */
    {
        float* R[4] = {gs[0], gs[1], gs[2], (float*)F[3]};
        expect("residual over a field", fpde_residual_fwd(op, &g, &co, F, C, R, loss, NULL),
               FPDE_ERR_ARG);
        float* R2[4] = {gs[0], gs[1], gs[1], gs[3]};
        expect("residuals overlap", fpde_residual_fwd(op, &g, &co, F, C, R2, loss, NULL),
               FPDE_ERR_ARG);
        float* R3[4] = {gs[0], NULL, gs[2], gs[3]};
        expect("null residual", fpde_residual_fwd(op, &g, &co, F, C, R3, loss, NULL), FPDE_ERR_ARG);
        expect("loss inside a field",
               fpde_residual_fwd(op, &g, &co, F, C, NULL, (double*)(void*)buf[1], NULL),
               FPDE_ERR_ARG);
    }
    expect("bwd null dloss", fpde_residual_bwd(op, &g, &co, F, C, NULL, gs, NULL), FPDE_ERR_ARG);
    expect("bwd null grads", fpde_residual_bwd(op, &g, &co, F, C, dl, NULL, NULL), FPDE_ERR_ARG);
    {
        float* G[4] = {gs[0], gs[1], gs[2], (float*)C[1]};
        expect("bwd grad over a const", fpde_residual_bwd(op, &g, &co, F, C, dl, G, NULL),
               FPDE_ERR_ARG);
    }
    expect("bc null grads", fpde_bc_correct(op, &g, &co, F, C, dl, NULL, NULL), FPDE_ERR_ARG);
    expect("vg null loss",
           fpde_residual_value_and_grad(op, &g, &co, F, C, dl, NULL, gs, NULL), FPDE_ERR_ARG);
    expect("vg loss is dloss",
           fpde_residual_value_and_grad(op, &g, &co, F, C, dl, (double*)dl, gs, NULL),
           FPDE_ERR_ARG);
    {
        const float* S[4] = {buf[16], buf[17], buf[18], buf[19]};
        expect("vjp accumulate 2", fpde_residual_vjp(op, &g, &co, F, S, 2, gs, NULL), FPDE_ERR_ARG);
        expect("vjp null sens", fpde_residual_vjp(op, &g, &co, F, NULL, 0, gs, NULL), FPDE_ERR_ARG);
        float* G[4] = {gs[0], gs[1], (float*)S[2], gs[3]};
        expect("vjp grad over a sensitivity", fpde_residual_vjp(op, &g, &co, F, S, 0, G, NULL),
               FPDE_ERR_ARG);
    }

    /* 2-D: a long first axis; 3D+t through the four-axis entry points */
    {
        fpde_grid b;
        memset(&b, 0, sizeof b);
        b.ndim = 2;
        b.n[0] = ((int64_t)1 << 31) - 1;
        b.n[1] = 3;
        b.h[0] = b.h[1] = 0.1;
        expect("2-D axis 0 of 2^31 - 1",
               fpde_residual_fwd(FPDE_NS_2D_STEADY, &b, &co, F, NULL, NULL, loss, NULL),
               FPDE_ERR_SHAPE);
    }
    {
        fpde_grid4 b;
        memset(&b, 0, sizeof b);
        b.ndim = 4;
        for (int a = 0; a < 4; ++a) {
            b.n[a] = 5;
            b.h[a] = 0.2;
        }
        fpde_grid4 t = b;
        t.n[1] = 1 << 10;
        t.n[2] = 1 << 10;
        t.n[3] = 1 << 9;  /* a time level of 2^29 nodes */
        expect("3D+t level of 2^29", fpde_residual_fwd4(FPDE_NS_3DT, &t, &co, F, NULL, NULL, loss, NULL),
               FPDE_ERR_SHAPE);
        t = b;
        t.n[0] = ((int64_t)1 << 31) - 1;  /* many time levels: too many workgroups */
        expect("3D+t of 2^31 - 1 levels",
               fpde_residual_fwd4(FPDE_NS_3DT, &t, &co, F, NULL, NULL, loss, NULL), FPDE_ERR_SHAPE);
        t = b;
        t.h[0] = -1.0;
        expect("3D+t h_t < 0", fpde_residual_bwd4(FPDE_NS_3DT, &t, &co, F, NULL, dl, gs, NULL),
               FPDE_ERR_SPACING);
        expect("3D+t through a three-axis grid",
               fpde_residual_fwd(FPDE_NS_3DT, &g, &co, F, NULL, NULL, loss, NULL), FPDE_ERR_SHAPE);
        t = b;
        t.ndim = 3;
        expect("3D+t op through a rank-3 fpde_grid4",
               fpde_residual_fwd4(FPDE_NS_3DT, &t, &co, F, NULL, NULL, loss, NULL), FPDE_ERR_SHAPE);
    }

    if (fails) {
        printf("abi-host-sanitize: %d of %d calls failed\n", fails, calls);
        return 1;
    }
    printf("abi-host-sanitize: %d calls; ok\n", calls);
    return 0;
}
