/*
 * fpde_oracle.c -- CPU oracle for the differentiable finite-difference PDE
 * residual operator.  TEST INFRASTRUCTURE ONLY (see fpde_oracle.h): plain,
 * slow, single-threaded float64 loops, no blocking, fusion or reordering.
 *
 * What it computes, per the paper:
 *   - centred differences D1_a q = (q(m+e_a) - q(m-e_a)) / (2 h_a) and
 *     D2_a q = (q(m+e_a) - 2 q(m) + q(m-e_a)) / h_a^2            (App. A.3)
 *   - the residual of each PDE at every residual node m               (Sec. 2.1)
 *   - loss = sum over equations of the mean squared residual          (Sec. 2.2, G = dL/dres)
 *   - the gradient of the loss w.r.t. every field node, as the transpose
 *     Jacobian applied to G (Sec. 2.2, App. A.3): for each residual node m and
 *     each stencil node n of R_b(m), grad_q(n) += G_b(m) * dR_b(m)/dq(n).
 *     Each partial derivative below is the derivative of one term of the
 *     residual written beside it, so the scatter can be read against the
 *     residual term by term.
 */
#include "fpde_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define ORC_MAXD 4

typedef struct {
    int ndim;
    int periodic;           /* bc_mode 1 */
    long n[ORC_MAXD];
    long stride[ORC_MAXD];
    double h[ORC_MAXD];
    long N;                 /* all nodes */
    long M;                 /* residual nodes */
} grid_t;

typedef struct {
    double nu, k, dt, alpha;
} coef_t;

/* Field, const and residual counts per op. */
static int op_shape(int op, int* ndim, int* nf, int* nc, int* nr) {
    switch (op) {
    case 1: *ndim = 2; *nf = 1; *nc = 0; *nr = 1; return 0; /* Burgers 1D+t: u          */
    case 2: *ndim = 2; *nf = 1; *nc = 1; *nr = 1; return 0; /* Helmholtz 2D: u ; f      */
    case 3: *ndim = 3; *nf = 1; *nc = 1; *nr = 1; return 0; /* heat 3D: u ; u0          */
    case 4: *ndim = 2; *nf = 3; *nc = 0; *nr = 3; return 0; /* NS 2D: u,v,p             */
    case 5: *ndim = 3; *nf = 4; *nc = 3; *nr = 4; return 0; /* NS 3D: u,v,w,p ; prev    */
    case 6: *ndim = 3; *nf = 4; *nc = 0; *nr = 4; return 0; /* steady NS 3D: u,v,w,p    */
    case 7: *ndim = 2; *nf = 1; *nc = 1; *nr = 1; return 0; /* Poisson 2D: u ; f        */
    case 8: *ndim = 3; *nf = 1; *nc = 1; *nr = 1; return 0; /* Poisson 3D: u ; f        */
    case 9: *ndim = 3; *nf = 3; *nc = 0; *nr = 3; return 0; /* NS 2D+t: u,v,p (t,x,y)   */
    case 10: *ndim = 4; *nf = 4; *nc = 0; *nr = 4; return 0; /* NS 3D+t: u,v,w,p (t,x,y,z) */
    default: return -1;
    }
}

int orc_op_info(int op, int* ndim, int* n_fields, int* n_consts, int* n_residuals) {
    int d, f, c, r;
    if (op_shape(op, &d, &f, &c, &r)) return -1;
    if (ndim) *ndim = d;
    if (n_fields) *n_fields = f;
    if (n_consts) *n_consts = c;
    if (n_residuals) *n_residuals = r;
    return 0;
}

static int setup(int op, int ndim, const long* n, const double* h, int bc_mode,
                 const double* coef, const double* const* F, const double* const* C,
                 grid_t* g, coef_t* cf) {
    int d, nf, nc, nr, a;
    if (op_shape(op, &d, &nf, &nc, &nr)) return -1;
    if (!n || !h || !coef) return -1;
    if (ndim != d) return -2;
    if (bc_mode != 0 && bc_mode != 1) return -1;
    g->ndim = d;
    g->periodic = bc_mode;
    g->N = 1;
    g->M = 1;
    for (a = 0; a < d; a++) {
        if (n[a] < 3) return -2;
        if (!(h[a] > 0.0) || !isfinite(h[a])) return -3;
        g->n[a] = n[a];
        g->h[a] = h[a];
        g->N *= n[a];
        g->M *= bc_mode ? n[a] : (n[a] - 2);
    }
    g->stride[d - 1] = 1;
    for (a = d - 2; a >= 0; a--) g->stride[a] = g->stride[a + 1] * g->n[a + 1];
    cf->nu = coef[0];
    cf->k = coef[1];
    cf->dt = coef[2];
    cf->alpha = coef[3];
    if (!isfinite(cf->nu) || !isfinite(cf->k) || !isfinite(cf->dt) || !isfinite(cf->alpha))
        return -4;
    if ((op == 3 || op == 5) && !(cf->dt > 0.0)) return -4;
    for (a = 0; a < nf; a++)
        if (!F || !F[a]) return -1;
    for (a = 0; a < nc; a++)
        if (!C || !C[a]) return -1;
    return 0;
}

/* Index of the node m + s*e_a (s = +1 or -1); iv is the multi-index of m. */
static long nb(const grid_t* g, const long* iv, long m, int a, int s) {
    if (g->periodic) {
        long i = iv[a] + s;
        if (i < 0) i += g->n[a];
        if (i >= g->n[a]) i -= g->n[a];
        return m + (i - iv[a]) * g->stride[a];
    }
    return m + s * g->stride[a];
}

static double D1(const grid_t* g, const double* q, const long* iv, long m, int a) {
    return (q[nb(g, iv, m, a, +1)] - q[nb(g, iv, m, a, -1)]) / (2.0 * g->h[a]);
}

static double D2(const grid_t* g, const double* q, const long* iv, long m, int a) {
    return (q[nb(g, iv, m, a, +1)] - 2.0 * q[m] + q[nb(g, iv, m, a, -1)]) / (g->h[a] * g->h[a]);
}

/* Visit every residual node: call fn(m, iv) in lexicographic order. */
typedef void (*visit_fn)(const grid_t* g, long m, const long* iv, void* ctx);

static void for_each_residual_node(const grid_t* g, visit_fn fn, void* ctx) {
    long iv[ORC_MAXD], lo = g->periodic ? 0 : 1;
    int a, d = g->ndim;
    for (a = 0; a < d; a++) iv[a] = lo;
    for (;;) {
        long m = 0;
        for (a = 0; a < d; a++) m += iv[a] * g->stride[a];
        fn(g, m, iv, ctx);
        /* advance the multi-index, last axis fastest */
        for (a = d - 1; a >= 0; a--) {
            long hi = g->periodic ? g->n[a] - 1 : g->n[a] - 2;
            if (iv[a] < hi) { iv[a]++; break; }
            iv[a] = lo;
        }
        if (a < 0) return;
    }
}

/* ------------------------------------------------------------------------- */
/* Residuals R_b(m)                                                          */
/* ------------------------------------------------------------------------- */

/* Burgers on the space-time grid, axis 0 = t, axis 1 = x:
 *   R = u_t + u u_x - nu u_xx, every derivative a centred difference. */
static void res_burgers(const grid_t* g, const coef_t* c, const double* const* F,
                        const double* const* C, long m, const long* iv, double* R) {
    const double* u = F[0];
    (void)C;
    R[0] = D1(g, u, iv, m, 0) + u[m] * D1(g, u, iv, m, 1) - c->nu * D2(g, u, iv, m, 1);
}

/* Helmholtz: R = lap u + k^2 u - f. */
static void res_helmholtz(const grid_t* g, const coef_t* c, const double* const* F,
                          const double* const* C, long m, const long* iv, double* R) {
    const double* u = F[0];
    double lap = 0.0;
    int a;
    for (a = 0; a < g->ndim; a++) lap += D2(g, u, iv, m, a);
    R[0] = lap + c->k * c->k * u[m] - C[0][m];
}

/* One implicit heat step: R = (u - u0)/dt - alpha lap u. */
static void res_heat(const grid_t* g, const coef_t* c, const double* const* F,
                     const double* const* C, long m, const long* iv, double* R) {
    const double* u = F[0];
    double lap = 0.0;
    int a;
    for (a = 0; a < g->ndim; a++) lap += D2(g, u, iv, m, a);
    R[0] = (u[m] - C[0][m]) / c->dt - c->alpha * lap;
}

/* Incompressible NS, velocity component b on array axis b (u<->0, v<->1, w<->2),
 * pressure after the velocities (Sec. 2.1 for the steady 2D case):
 *   R_b = [(c_b - c_b^prev)/dt] + sum_a c_a D1_a c_b + D1_b p - nu sum_a D2_a c_b
 *   R_div = sum_a D1_a c_a
 * The bracketed time term is present for the backward-Euler step only (op 5);
 * ops 4 (2D) and 6 (3D) are steady. */
static void res_ns(const grid_t* g, const coef_t* c, const double* const* F,
                   const double* const* C, long m, const long* iv, double* R, int unsteady) {
    int d = g->ndim, a, b;
    const double* p = F[d];
    for (b = 0; b < d; b++) {
        const double* cb = F[b];
        double r = 0.0;
        if (unsteady) r += (cb[m] - C[b][m]) / c->dt;
        for (a = 0; a < d; a++) r += F[a][m] * D1(g, cb, iv, m, a);
        r += D1(g, p, iv, m, b);
        for (a = 0; a < d; a++) r -= c->nu * D2(g, cb, iv, m, a);
        R[b] = r;
    }
    R[d] = 0.0;
    for (a = 0; a < d; a++) R[d] += D1(g, F[a], iv, m, a);
}

/* Poisson: R = lap u - f. */
static void res_poisson(const grid_t* g, const coef_t* c, const double* const* F,
                        const double* const* C, long m, const long* iv, double* R) {
    const double* u = F[0];
    double lap = 0.0;
    int a;
    (void)c;
    for (a = 0; a < g->ndim; a++) lap += D2(g, u, iv, m, a);
    R[0] = lap - C[0][m];
}

/* Unsteady incompressible NS on a space-time grid: array axis 0 is t, velocity
 * component b lives on array axis b+1 (u<->1, v<->2[, w<->3]), pressure after the
 * velocities; every derivative, the time derivative included, is a centred
 * difference (the time step is the grid spacing h_0).  The 2D+t grid (op 9)
 * has ndim 3, the 3D+t grid (op 10) ndim 4; d = ndim - 1 spatial components:
 *   R_b = D1_0 c_b + sum_a c_a D1_{a+1} c_b + D1_{b+1} p - nu sum_a D2_{a+1} c_b
 *   R_div = sum_a D1_{a+1} c_a              (a, b over the spatial components) */
static void res_ns_t(const grid_t* g, const coef_t* c, const double* const* F,
                     const double* const* C, long m, const long* iv, double* R) {
    int d = g->ndim - 1, a, b;
    const double* p = F[d];
    (void)C;
    for (b = 0; b < d; b++) {
        const double* cb = F[b];
        double r = D1(g, cb, iv, m, 0);
        for (a = 0; a < d; a++) r += F[a][m] * D1(g, cb, iv, m, a + 1);
        r += D1(g, p, iv, m, b + 1);
        for (a = 0; a < d; a++) r -= c->nu * D2(g, cb, iv, m, a + 1);
        R[b] = r;
    }
    R[d] = 0.0;
    for (a = 0; a < d; a++) R[d] += D1(g, F[a], iv, m, a + 1);
}

static void residual_at(int op, const grid_t* g, const coef_t* c, const double* const* F,
                        const double* const* C, long m, const long* iv, double* R) {
    switch (op) {
    case 1: res_burgers(g, c, F, C, m, iv, R); break;
    case 2: res_helmholtz(g, c, F, C, m, iv, R); break;
    case 3: res_heat(g, c, F, C, m, iv, R); break;
    case 4: res_ns(g, c, F, C, m, iv, R, 0); break;
    case 5: res_ns(g, c, F, C, m, iv, R, 1); break;
    case 6: res_ns(g, c, F, C, m, iv, R, 0); break;
    case 7: case 8: res_poisson(g, c, F, C, m, iv, R); break;
    case 9: case 10: res_ns_t(g, c, F, C, m, iv, R); break;
    }
}

/* ------------------------------------------------------------------------- */
/* Transpose-Jacobian scatter: grad_q(n) += G_b(m) dR_b(m)/dq(n)             */
/* ------------------------------------------------------------------------- */

static void jt_burgers(const grid_t* g, const coef_t* c, const double* const* F,
                       const double* const* C, long m, const long* iv, const double* G,
                       double* const* gr) {
    const double* u = F[0];
    double* du = gr[0];
    double gm = G[0];
    double h0 = g->h[0], h1 = g->h[1];
    (void)C;
    /* u_t = (u(m+e0) - u(m-e0)) / (2 h0) */
    du[nb(g, iv, m, 0, +1)] += gm / (2.0 * h0);
    du[nb(g, iv, m, 0, -1)] -= gm / (2.0 * h0);
    /* u(m) * u_x: d/du(m) = u_x(m); d/du(m +- e1) = +- u(m) / (2 h1) */
    du[m] += gm * D1(g, u, iv, m, 1);
    du[nb(g, iv, m, 1, +1)] += gm * u[m] / (2.0 * h1);
    du[nb(g, iv, m, 1, -1)] -= gm * u[m] / (2.0 * h1);
    /* -nu u_xx: d/du(m) = 2 nu / h1^2; d/du(m +- e1) = -nu / h1^2 */
    du[m] += gm * 2.0 * c->nu / (h1 * h1);
    du[nb(g, iv, m, 1, +1)] -= gm * c->nu / (h1 * h1);
    du[nb(g, iv, m, 1, -1)] -= gm * c->nu / (h1 * h1);
}

static void jt_helmholtz(const grid_t* g, const coef_t* c, const double* const* F,
                         const double* const* C, long m, const long* iv, const double* G,
                         double* const* gr) {
    double* du = gr[0];
    double gm = G[0];
    int a;
    (void)F; (void)C;
    /* D2_a u: d/du(m) = -2/h_a^2; d/du(m +- e_a) = 1/h_a^2 */
    for (a = 0; a < g->ndim; a++) {
        double ih2 = 1.0 / (g->h[a] * g->h[a]);
        du[m] -= gm * 2.0 * ih2;
        du[nb(g, iv, m, a, +1)] += gm * ih2;
        du[nb(g, iv, m, a, -1)] += gm * ih2;
    }
    /* k^2 u: d/du(m) = k^2  (f is a constant input) */
    du[m] += gm * c->k * c->k;
}

static void jt_heat(const grid_t* g, const coef_t* c, const double* const* F,
                    const double* const* C, long m, const long* iv, const double* G,
                    double* const* gr) {
    double* du = gr[0];
    double gm = G[0];
    int a;
    (void)F; (void)C;
    /* (u - u0)/dt: d/du(m) = 1/dt */
    du[m] += gm / c->dt;
    /* -alpha D2_a u: d/du(m) = 2 alpha/h_a^2; d/du(m +- e_a) = -alpha/h_a^2 */
    for (a = 0; a < g->ndim; a++) {
        double ih2 = 1.0 / (g->h[a] * g->h[a]);
        du[m] += gm * 2.0 * c->alpha * ih2;
        du[nb(g, iv, m, a, +1)] -= gm * c->alpha * ih2;
        du[nb(g, iv, m, a, -1)] -= gm * c->alpha * ih2;
    }
}

static void jt_ns(const grid_t* g, const coef_t* c, const double* const* F,
                  const double* const* C, long m, const long* iv, const double* G,
                  double* const* gr, int unsteady) {
    int d = g->ndim, a, b;
    double* dp = gr[d];
    (void)C;
    for (b = 0; b < d; b++) {
        const double* cb = F[b];
        double gm = G[b];
        /* (c_b - c_b^prev)/dt: d/dc_b(m) = 1/dt */
        if (unsteady) gr[b][m] += gm / c->dt;
        for (a = 0; a < d; a++) {
            double i2h = 1.0 / (2.0 * g->h[a]);
            /* c_a(m) * D1_a c_b: d/dc_a(m) = D1_a c_b(m);
             *                    d/dc_b(m +- e_a) = +- c_a(m) / (2 h_a) */
            gr[a][m] += gm * D1(g, cb, iv, m, a);
            gr[b][nb(g, iv, m, a, +1)] += gm * F[a][m] * i2h;
            gr[b][nb(g, iv, m, a, -1)] -= gm * F[a][m] * i2h;
        }
        /* D1_b p: d/dp(m +- e_b) = +- 1/(2 h_b) */
        dp[nb(g, iv, m, b, +1)] += gm / (2.0 * g->h[b]);
        dp[nb(g, iv, m, b, -1)] -= gm / (2.0 * g->h[b]);
        /* -nu D2_a c_b: d/dc_b(m) = 2 nu/h_a^2; d/dc_b(m +- e_a) = -nu/h_a^2 */
        for (a = 0; a < d; a++) {
            double ih2 = 1.0 / (g->h[a] * g->h[a]);
            gr[b][m] += gm * 2.0 * c->nu * ih2;
            gr[b][nb(g, iv, m, a, +1)] -= gm * c->nu * ih2;
            gr[b][nb(g, iv, m, a, -1)] -= gm * c->nu * ih2;
        }
    }
    /* R_div = sum_a D1_a c_a: d/dc_a(m +- e_a) = +- 1/(2 h_a) */
    for (a = 0; a < d; a++) {
        gr[a][nb(g, iv, m, a, +1)] += G[d] / (2.0 * g->h[a]);
        gr[a][nb(g, iv, m, a, -1)] -= G[d] / (2.0 * g->h[a]);
    }
}

static void jt_poisson(const grid_t* g, const coef_t* c, const double* const* F,
                       const double* const* C, long m, const long* iv, const double* G,
                       double* const* gr) {
    double* du = gr[0];
    double gm = G[0];
    int a;
    (void)c; (void)F; (void)C;
    /* D2_a u: d/du(m) = -2/h_a^2; d/du(m +- e_a) = 1/h_a^2  (f is a constant input) */
    for (a = 0; a < g->ndim; a++) {
        double ih2 = 1.0 / (g->h[a] * g->h[a]);
        du[m] -= gm * 2.0 * ih2;
        du[nb(g, iv, m, a, +1)] += gm * ih2;
        du[nb(g, iv, m, a, -1)] += gm * ih2;
    }
}

static void jt_ns_t(const grid_t* g, const coef_t* c, const double* const* F,
                    const double* const* C, long m, const long* iv, const double* G,
                    double* const* gr) {
    int d = g->ndim - 1, a, b;
    double* dp = gr[d];
    (void)C;
    for (b = 0; b < d; b++) {
        const double* cb = F[b];
        double gm = G[b];
        /* D1_0 c_b: d/dc_b(m +- e_0) = +- 1/(2 h_0) */
        gr[b][nb(g, iv, m, 0, +1)] += gm / (2.0 * g->h[0]);
        gr[b][nb(g, iv, m, 0, -1)] -= gm / (2.0 * g->h[0]);
        for (a = 0; a < d; a++) {
            double i2h = 1.0 / (2.0 * g->h[a + 1]);
            /* c_a(m) * D1_{a+1} c_b: d/dc_a(m) = D1_{a+1} c_b(m);
             *                        d/dc_b(m +- e_{a+1}) = +- c_a(m) / (2 h_{a+1}) */
            gr[a][m] += gm * D1(g, cb, iv, m, a + 1);
            gr[b][nb(g, iv, m, a + 1, +1)] += gm * F[a][m] * i2h;
            gr[b][nb(g, iv, m, a + 1, -1)] -= gm * F[a][m] * i2h;
        }
        /* D1_{b+1} p: d/dp(m +- e_{b+1}) = +- 1/(2 h_{b+1}) */
        dp[nb(g, iv, m, b + 1, +1)] += gm / (2.0 * g->h[b + 1]);
        dp[nb(g, iv, m, b + 1, -1)] -= gm / (2.0 * g->h[b + 1]);
        /* -nu D2_{a+1} c_b: d/dc_b(m) = 2 nu/h^2; d/dc_b(m +- e_{a+1}) = -nu/h^2 */
        for (a = 0; a < d; a++) {
            double ih2 = 1.0 / (g->h[a + 1] * g->h[a + 1]);
            gr[b][m] += gm * 2.0 * c->nu * ih2;
            gr[b][nb(g, iv, m, a + 1, +1)] -= gm * c->nu * ih2;
            gr[b][nb(g, iv, m, a + 1, -1)] -= gm * c->nu * ih2;
        }
    }
    /* R_div = sum_a D1_{a+1} c_a: d/dc_a(m +- e_{a+1}) = +- 1/(2 h_{a+1}) */
    for (a = 0; a < d; a++) {
        gr[a][nb(g, iv, m, a + 1, +1)] += G[d] / (2.0 * g->h[a + 1]);
        gr[a][nb(g, iv, m, a + 1, -1)] -= G[d] / (2.0 * g->h[a + 1]);
    }
}

static void jt_at(int op, const grid_t* g, const coef_t* c, const double* const* F,
                  const double* const* C, long m, const long* iv, const double* G,
                  double* const* gr) {
    switch (op) {
    case 1: jt_burgers(g, c, F, C, m, iv, G, gr); break;
    case 2: jt_helmholtz(g, c, F, C, m, iv, G, gr); break;
    case 3: jt_heat(g, c, F, C, m, iv, G, gr); break;
    case 4: jt_ns(g, c, F, C, m, iv, G, gr, 0); break;
    case 5: jt_ns(g, c, F, C, m, iv, G, gr, 1); break;
    case 6: jt_ns(g, c, F, C, m, iv, G, gr, 0); break;
    case 7: case 8: jt_poisson(g, c, F, C, m, iv, G, gr); break;
    case 9: case 10: jt_ns_t(g, c, F, C, m, iv, G, gr); break;
    }
}

/* ------------------------------------------------------------------------- */
/* Entry points                                                              */
/* ------------------------------------------------------------------------- */

typedef struct {
    int op, nr;
    const coef_t* c;
    const double* const* F;
    const double* const* C;
    double* const* R;        /* residual output */
    const double* const* G;  /* vjp input */
    double* const* gr;       /* vjp output */
    double dscale;           /* orc_grad: 2 dloss / M */
    double acc;              /* orc_loss accumulator */
} ctx_t;

static void visit_residual(const grid_t* g, long m, const long* iv, void* p) {
    ctx_t* x = (ctx_t*)p;
    double r[4];
    int b;
    residual_at(x->op, g, x->c, x->F, x->C, m, iv, r);
    for (b = 0; b < x->nr; b++) x->R[b][m] = r[b];
}

static void visit_loss(const grid_t* g, long m, const long* iv, void* p) {
    ctx_t* x = (ctx_t*)p;
    double r[4];
    int b;
    residual_at(x->op, g, x->c, x->F, x->C, m, iv, r);
    for (b = 0; b < x->nr; b++) x->acc += r[b] * r[b];
}

static void visit_vjp(const grid_t* g, long m, const long* iv, void* p) {
    ctx_t* x = (ctx_t*)p;
    double gm[4];
    int b;
    for (b = 0; b < x->nr; b++) gm[b] = x->G[b][m];
    jt_at(x->op, g, x->c, x->F, x->C, m, iv, gm, x->gr);
}

static void visit_grad(const grid_t* g, long m, const long* iv, void* p) {
    ctx_t* x = (ctx_t*)p;
    double r[4];
    int b;
    residual_at(x->op, g, x->c, x->F, x->C, m, iv, r);
    for (b = 0; b < x->nr; b++) r[b] *= x->dscale; /* G_b(m) = 2 dloss R_b(m) / M */
    jt_at(x->op, g, x->c, x->F, x->C, m, iv, r, x->gr);
}

int orc_residual(int op, int ndim, const long* n, const double* h, int bc_mode,
                 const double* coef, const double* const* fields,
                 const double* const* consts, double* const* R) {
    grid_t g;
    coef_t c;
    ctx_t x;
    int d, nf, nc, nr, b, st;
    st = setup(op, ndim, n, h, bc_mode, coef, fields, consts, &g, &c);
    if (st) return st;
    op_shape(op, &d, &nf, &nc, &nr);
    if (!R) return -1;
    for (b = 0; b < nr; b++) {
        if (!R[b]) return -1;
        memset(R[b], 0, sizeof(double) * (size_t)g.N);
    }
    memset(&x, 0, sizeof x);
    x.op = op; x.nr = nr; x.c = &c; x.F = fields; x.C = consts; x.R = R;
    for_each_residual_node(&g, visit_residual, &x);
    return 0;
}

int orc_loss(int op, int ndim, const long* n, const double* h, int bc_mode,
             const double* coef, const double* const* fields,
             const double* const* consts, double* loss) {
    grid_t g;
    coef_t c;
    ctx_t x;
    int d, nf, nc, nr, st;
    st = setup(op, ndim, n, h, bc_mode, coef, fields, consts, &g, &c);
    if (st) return st;
    if (!loss) return -1;
    op_shape(op, &d, &nf, &nc, &nr);
    memset(&x, 0, sizeof x);
    x.op = op; x.nr = nr; x.c = &c; x.F = fields; x.C = consts;
    for_each_residual_node(&g, visit_loss, &x);
    *loss = x.acc / (double)g.M;
    return 0;
}

int orc_vjp(int op, int ndim, const long* n, const double* h, int bc_mode,
            const double* coef, const double* const* fields,
            const double* const* consts, const double* const* G,
            double* const* grads) {
    grid_t g;
    coef_t c;
    ctx_t x;
    int d, nf, nc, nr, b, st;
    st = setup(op, ndim, n, h, bc_mode, coef, fields, consts, &g, &c);
    if (st) return st;
    op_shape(op, &d, &nf, &nc, &nr);
    if (!G || !grads) return -1;
    for (b = 0; b < nr; b++)
        if (!G[b]) return -1;
    for (b = 0; b < nf; b++) {
        if (!grads[b]) return -1;
        memset(grads[b], 0, sizeof(double) * (size_t)g.N);
    }
    memset(&x, 0, sizeof x);
    x.op = op; x.nr = nr; x.c = &c; x.F = fields; x.C = consts; x.G = G; x.gr = grads;
    for_each_residual_node(&g, visit_vjp, &x);
    return 0;
}

int orc_grad(int op, int ndim, const long* n, const double* h, int bc_mode,
             const double* coef, const double* const* fields,
             const double* const* consts, double dloss, double* const* grads) {
    grid_t g;
    coef_t c;
    ctx_t x;
    int d, nf, nc, nr, b, st;
    st = setup(op, ndim, n, h, bc_mode, coef, fields, consts, &g, &c);
    if (st) return st;
    op_shape(op, &d, &nf, &nc, &nr);
    if (!grads) return -1;
    for (b = 0; b < nf; b++) {
        if (!grads[b]) return -1;
        memset(grads[b], 0, sizeof(double) * (size_t)g.N);
    }
    memset(&x, 0, sizeof x);
    x.op = op; x.nr = nr; x.c = &c; x.F = fields; x.C = consts; x.gr = grads;
    x.dscale = 2.0 * dloss / (double)g.M;
    for_each_residual_node(&g, visit_grad, &x);
    return 0;
}
