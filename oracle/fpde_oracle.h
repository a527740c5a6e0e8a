/*
 * fpde_oracle.h -- CPU oracle for the differentiable finite-difference PDE
 * residual operator.  TEST INFRASTRUCTURE ONLY: only the test suite, the smoke
 * check and the benchmark's CPU-baseline leg may load this library.  The GPU
 * product path never links, calls or includes it, and it shares no source with
 * the GPU path.
 *
 * Everything here is float64 on host memory, written as plain loops in the
 * order the paper states the method: centred second-order differences
 * (App. A.3), residuals on interior nodes (Sec. 2.1), mean-squared loss, and
 * the exact gradient of that loss with respect to every node of every
 * differentiated field, assembled in scatter form from the residual Jacobian
 * (the transpose-Jacobian action of Sec. 2.2, App. A.3).
 *
 * Arrays are C-contiguous with shape n[0..ndim-1] (last axis fastest).
 * Op ids: 1 Burgers 1D+t, 2 Helmholtz 2D, 3 heat 3D (one implicit step),
 *         4 steady NS 2D, 5 backward-Euler NS 3D, 6 steady NS 3D,
 *         7 Poisson 2D, 8 Poisson 3D, 9 unsteady NS 2D+t (space-time grid,
 *         ndim 3), 10 unsteady NS 3D+t (space-time grid, ndim 4: t, x, y, z).
 * coef = {nu, k, dt, alpha}; members an op does not use are ignored.
 * bc_mode 0: residuals on interior nodes only (1 <= i_a <= n_a-2 on every axis).
 * bc_mode 1: periodic wrap on every axis, residuals on all nodes.
 *
 * Return codes: 0 ok, -1 bad op / null pointer, -2 bad shape, -3 bad spacing,
 * -4 bad coefficient.
 */
#ifndef FPDE_ORACLE_H
#define FPDE_ORACLE_H

#ifdef __cplusplus
extern "C" {
#endif

int orc_op_info(int op, int* ndim, int* n_fields, int* n_consts, int* n_residuals);

/* R[b] (full-size arrays) receive residual b on the residual node set and 0 elsewhere. */
int orc_residual(int op, int ndim, const long* n, const double* h, int bc_mode,
                 const double* coef, const double* const* fields,
                 const double* const* consts, double* const* R);

/* *loss = sum over equations b of mean over the residual node set of R_b^2. */
int orc_loss(int op, int ndim, const long* n, const double* h, int bc_mode,
             const double* coef, const double* const* fields,
             const double* const* consts, double* loss);

/* grads[q] = sum_b sum_m G_b(m) dR_b(m)/dq  (full-size, overwritten).
 * G[b] are full-size arrays; only their values on the residual node set are read. */
int orc_vjp(int op, int ndim, const long* n, const double* h, int bc_mode,
            const double* coef, const double* const* fields,
            const double* const* consts, const double* const* G,
            double* const* grads);

/* Gradient of dloss * loss: orc_vjp with G_b = 2 dloss R_b / M. */
int orc_grad(int op, int ndim, const long* n, const double* h, int bc_mode,
             const double* coef, const double* const* fields,
             const double* const* consts, double dloss, double* const* grads);

#ifdef __cplusplus
}
#endif
#endif
