/*
 * fpde.h -- C ABI of libfpde: a differentiable finite-difference PDE residual
 * operator for AMD Instinct MI355X (gfx950).
 *
 * The operator follows the three-part design of FlashPDE (Sec. 2): a fused
 * forward stencil (Sec. 2.1), a discrete analytic-adjoint backward
 * (Sec. 2.2, App. A.3) and a boundary-gradient correction (Sec. 2.3, App. A.5).
 * Here the forward also reduces the mean-squared residual loss, and the
 * backward recomputes the residuals it needs instead of reading an upstream
 * sensitivity tensor, so one call sequence is
 *     fpde_residual_fwd -> fpde_residual_bwd + fpde_bc_correct.
 * fpde_residual_vjp is the general backward of Sec. 2.2: it applies the
 * transposed residual Jacobian to upstream sensitivities the caller supplies,
 * for objectives other than the mean-squared loss.
 *
 * Notation (used by every entry point):
 *   - arrays are dense C-contiguous float32, shape n[0..ndim-1], last axis
 *     fastest; h[a] is the node spacing along array axis a;
 *   - the residual set is Omega = { nodes with 1 <= i_a <= n_a - 2 on every
 *     axis }, M = prod_a (n_a - 2) (bc_mode 0); with bc_mode 1 (periodic) the
 *     grid wraps on every axis, q(m +- e_a) reading node i_a +- 1 mod n_a, and
 *     Omega is every node, M = prod_a n_a;
 *   - D1_a q(m) = (q(m+e_a) - q(m-e_a)) / (2 h_a),
 *     D2_a q(m) = (q(m+e_a) - 2 q(m) + q(m-e_a)) / h_a^2     (App. A.3);
 *   - loss L = sum over equations b of (1/M) sum_{m in Omega} R_b(m)^2;
 *   - the gradient written by bwd + bc is dloss * dL/dq for every node of
 *     every differentiated field q (boundary nodes included).
 *
 * Operators (velocity component b lives on array axis b; pressure last):
 *   FPDE_BURGERS_1DT  (ndim 2; axis 0 = t, axis 1 = x)   fields {u}        consts {}
 *       R = D1_0 u + u D1_1 u - nu D2_1 u
 *   FPDE_HELMHOLTZ_2D (ndim 2)                            fields {u}        consts {f}
 *       R = D2_0 u + D2_1 u + k^2 u - f
 *   FPDE_HEAT_3D_BE   (ndim 3; one implicit step)         fields {u}        consts {u0}
 *       R = (u - u0)/dt - alpha (D2_0 + D2_1 + D2_2) u
 *   FPDE_NS_2D_STEADY (ndim 2; the worked example of Sec. 2.1)
 *                                                         fields {u, v, p}  consts {}
 *       R_b = sum_a c_a D1_a c_b + D1_b p - nu sum_a D2_a c_b   (b = 0,1; c = (u,v))
 *       R_div = sum_a D1_a c_a
 *   FPDE_NS_3D_BE     (ndim 3; one backward-Euler step)   fields {u, v, w, p}
 *                                                         consts {u_prev, v_prev, w_prev}
 *       R_b = (c_b - c_b_prev)/dt + sum_a c_a D1_a c_b + D1_b p - nu sum_a D2_a c_b
 *       R_div = sum_a D1_a c_a
 * Adjacent operators of the paper's operator table (Sec. 4), same kernels:
 *   FPDE_NS_3D_STEADY (ndim 3)                            fields {u, v, w, p}  consts {}
 *       R_b = sum_a c_a D1_a c_b + D1_b p - nu sum_a D2_a c_b ;  R_div as above
 *   FPDE_POISSON_2D   (ndim 2)                            fields {u}        consts {f}
 *   FPDE_POISSON_3D   (ndim 3)                            fields {u}        consts {f}
 *       R = sum_a D2_a u - f
 *   FPDE_NS_2DT       (ndim 3; space-time grid: axis 0 = t, axes 1, 2 = x, y;
 *                      velocity component b on array axis b + 1)
 *                                                         fields {u, v, p}  consts {}
 *       R_b = D1_0 c_b + sum_a c_a D1_{a+1} c_b + D1_{b+1} p - nu sum_a D2_{a+1} c_b
 *       R_div = sum_a D1_{a+1} c_a            (a, b = 0, 1; the time step is h[0])
 *   FPDE_NS_3DT       (ndim 4; space-time grid: axis 0 = t, axes 1, 2, 3 = x, y, z;
 *                      velocity component b on array axis b + 1; the paper's
 *                      3d_ns_unsteady operator with a centred time difference)
 *                                                         fields {u, v, w, p}  consts {}
 *       R_b = D1_0 c_b + sum_a c_a D1_{a+1} c_b + D1_{b+1} p - nu sum_a D2_{a+1} c_b
 *       R_div = sum_a D1_{a+1} c_a            (a, b = 0, 1, 2; the time step is h[0])
 *     Four-axis grids are described by fpde_grid4 and served by the entry
 *     points ending in 4 (which take every op); fpde_grid holds three axes.
 *
 * Common argument rules:
 *   - `fields`, `consts`, `residual_out`, `sens`, `grads` are HOST arrays holding
 *     DEVICE pointers, one per array in the order listed above (`consts` may be
 *     NULL for ops without consts).  Every device array is n[0]*...*n[ndim-1]
 *     floats, 4-byte aligned, allocated on the current HIP device.
 *   - The caller owns every buffer and keeps it alive until the work queued on
 *     `stream` has completed.  The library allocates nothing and keeps no
 *     global state; calls are reentrant.
 *   - `stream` is a hipStream_t (NULL: the default stream).  All GPU work is
 *     queued asynchronously on it; the host never synchronises.
 *   - Arguments are validated on the host before anything is queued; on any
 *     error the call returns a negative fpde_status and queues nothing.
 *   - Output arrays must not overlap any input array (FPDE_ERR_ARG).
 *   - NaN/Inf in the data are not checked; they propagate.
 */
#ifndef FPDE_H
#define FPDE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum fpde_status {
    FPDE_OK = 0,
    FPDE_ERR_ARG = -1,         /* null pointer, unknown op, overlapping output */
    FPDE_ERR_SHAPE = -2,       /* ndim differs from the op's, n_a < 3, or a size too large */
    FPDE_ERR_SPACING = -3,     /* h_a <= 0 or not finite */
    FPDE_ERR_COEFF = -4,       /* non-finite coefficient, or dt <= 0 for a time-stepping op */
    FPDE_ERR_ALIGN = -5,       /* a device pointer not 4-byte aligned */
    FPDE_ERR_HIP = -6,         /* the HIP runtime reported an error while queueing */
    FPDE_ERR_UNSUPPORTED = -7  /* valid request this library version does not implement (none at present) */
} fpde_status;

typedef enum fpde_op {
    FPDE_BURGERS_1DT = 1,
    FPDE_HELMHOLTZ_2D = 2,
    FPDE_HEAT_3D_BE = 3,
    FPDE_NS_2D_STEADY = 4,
    FPDE_NS_3D_BE = 5,
    FPDE_NS_3D_STEADY = 6,
    FPDE_POISSON_2D = 7,
    FPDE_POISSON_3D = 8,
    FPDE_NS_2DT = 9,
    FPDE_NS_3DT = 10
} fpde_op;

/* Grid: rank, residual-set mode, sizes per array axis, spacings per axis.
 * bc_mode 0: the interior residual set Omega above; 1: periodic wrap on every
 * axis (the fully periodic reading of the Taylor-Green grid); other values are
 * rejected with FPDE_ERR_ARG.  Entries past ndim are ignored.
 * Limits: every n_a >= 3 and n_a < 2^31; a plane of the non-marching axes
 * (n[1]*n[2] for ndim 3, n[1] for ndim 2) holds fewer than 2^29 nodes; and every
 * launch stays below 2^31 workgroups: (n[ndim-1]/32 + 1) * (n[1] + 1) * (n[0] + 1)
 * < 2^31 for ndim 3, with 2 in place of n[1] + 1 for ndim 2 (grids up to about
 * 2^36 nodes).  Beyond any limit: FPDE_ERR_SHAPE. */
typedef struct fpde_grid {
    int32_t ndim;
    int32_t bc_mode;
    int64_t n[3];
    double h[3];
} fpde_grid;

/* The grid with up to four axes (a versioned fpde_grid: same members, one more
 * axis), taken by the entry points ending in 4.  Rules as fpde_grid; for
 * ndim 4 the limits are every n_a >= 3, n_a < 2^31, a time level of the last
 * three axes (n[1]*n[2]*n[3]) below 2^29 nodes, and
 * (n[3]/32 + 1) * (n[2] + 1) * (n[1] + 1) * n[0] < 2^31 (workgroups). */
typedef struct fpde_grid4 {
    int32_t ndim;
    int32_t bc_mode;
    int64_t n[4];
    double h[4];
} fpde_grid4;

/* PDE coefficients in float64; an op ignores the members it does not use.
 * The library derives 1/(2h), 1/h^2, nu/h^2, ... in float64 and rounds them
 * once to float32 for the kernels. */
typedef struct fpde_coeffs {
    double nu;     /* viscosity (Burgers, NS) */
    double k;      /* wave number (Helmholtz) */
    double dt;     /* time step (HEAT_3D_BE, NS_3D_BE); must be > 0 for those ops */
    double alpha;  /* diffusivity (heat) */
} fpde_coeffs;

/* Static description of an op.  Any output pointer may be NULL.
 * Returns FPDE_OK or FPDE_ERR_ARG (unknown op). */
int fpde_op_info(int op, int* ndim, int* n_fields, int* n_consts, int* n_residuals);

/* Fused forward stencil + mean-squared residual loss (Sec. 2.1).
 *   loss          device pointer to one double; OVERWRITTEN with L (not accumulated).
 *   residual_out  NULL, or a host array of n_residuals device pointers: every
 *                 node of R_b is written, R_b(m) on Omega and 0 off Omega
 *                 (periodic grids: Omega is every node).
 * Queues 2 kernels: a one-element fill that zeroes *loss, then the stencil
 * kernel (one float64 atomic add per workgroup onto *loss). */
int fpde_residual_fwd(int op, const fpde_grid* grid, const fpde_coeffs* coeffs,
                      const float* const* fields, const float* const* consts,
                      float* const* residual_out, double* loss, void* stream);

/* Interior analytic-adjoint backward, gather form (Sec. 2.2, App. A.3).
 *   dloss  device pointer to one double: the upstream derivative of the
 *          consumer's objective with respect to L (1.0 for L itself).
 *   grads  host array of n_fields device pointers; OVERWRITTEN with
 *          dloss * dL/dq on every node of the planes 1 <= i_0 <= n_0 - 2 of
 *          array axis 0 (the planes the kernel marches over), boundary columns
 *          of those planes included: there the transposed stencil is evaluated
 *          with the residuals off Omega taken as zero, which is their exact
 *          boundary term.  The end planes i_0 = 0 and i_0 = n_0 - 1 are not
 *          touched (fpde_bc_correct writes them).  Periodic grids have no
 *          boundary: every node of every plane is written.
 * The residuals are recomputed from the fields; no sensitivity tensor is read.
 * Queues 1 kernel; no atomics. */
int fpde_residual_bwd(int op, const fpde_grid* grid, const fpde_coeffs* coeffs,
                      const float* const* fields, const float* const* consts,
                      const double* dloss, float* const* grads, void* stream);

/* Boundary-gradient correction (Sec. 2.3, App. A.5): one launch over the
 * boundary nodes the backward march does not visit, the end planes i_0 = 0 and
 * i_0 = n_0 - 1.  A node whose only boundary coordinate is i_0 receives the
 * terms of its single inward neighbour's residuals; a node with a second
 * boundary coordinate (an edge or corner) touches no residual node and
 * receives 0.  Arguments as fpde_residual_bwd; OVERWRITES grads on those two
 * planes only, so bwd and bc together write every node exactly once, in
 * either order.  Queues 1 kernel.  On a periodic grid (bc_mode 1) there is no
 * boundary: the call validates its arguments and returns FPDE_OK without
 * queueing anything or writing grads. */
int fpde_bc_correct(int op, const fpde_grid* grid, const fpde_coeffs* coeffs,
                    const float* const* fields, const float* const* consts,
                    const double* dloss, float* const* grads, void* stream);

/* Value and gradient in one pass: the loss L of fpde_residual_fwd and the
 * gradient dloss * dL/dq of fpde_residual_bwd + fpde_bc_correct, from one read
 * of the fields and consts.  The gradient of the mean-squared loss needs only
 * the residuals (dL/dq = (2/M) J^T R), which the backward recomputes anyway, so
 * the forward pass of Sec. 2.1 folds into it when the upstream derivative
 * dloss is known before the call (1.0 for L itself): the backward kernel also
 * sums the squares of the residuals it evaluates.  Its march covers every plane
 * of axis 0, the end planes too: there the transposed stencil with the
 * residuals off Omega taken as zero is exactly the boundary term that
 * fpde_bc_correct writes (equal up to the float32 rounding order).
 *   dloss  device pointer to one double, as in fpde_residual_bwd.
 *   loss   device pointer to one double; OVERWRITTEN with L (not dloss * L);
 *          must not overlap any other argument array (FPDE_ERR_ARG).
 *   grads  host array of n_fields device pointers; OVERWRITTEN at every node.
 * Other arguments and errors as fpde_residual_bwd.  Queues 2 kernels: a
 * one-element fill zeroing *loss, then the backward march (one float64 atomic
 * add per workgroup onto *loss). */
int fpde_residual_value_and_grad(int op, const fpde_grid* grid, const fpde_coeffs* coeffs,
                                 const float* const* fields, const float* const* consts,
                                 const double* dloss, double* loss, float* const* grads,
                                 void* stream);

/* Explicit-sensitivity backward: the transpose-Jacobian action of the
 * residual operator on upstream residual sensitivities G_b = dObj/dR_b, the
 * form in which the backward of Sec. 2.2 receives them from autograd:
 *     grads[q](n) (+)= sum_b sum_{m in Omega} G_b(m) dR_b(m)/dq(n)
 * for every node n of every field q, boundary nodes included.
 *   sens        host array of n_residuals device pointers, full-size arrays in
 *               the residual order of the op; only the values on Omega are
 *               read (entries off Omega are ignored, whatever they hold).
 *   accumulate  0: grads are OVERWRITTEN with the action; 1: the action is
 *               ADDED to what grads hold (every node read, then written once).
 *               Any other value: FPDE_ERR_ARG.
 *   grads       host array of n_fields device pointers; every node of every
 *               array is written, so no bc call follows this one.
 * The consts enter every residual additively, so the Jacobian, and this call,
 * do not depend on them: none are passed.  grads must not overlap the fields,
 * the sensitivities or each other (FPDE_ERR_ARG).  Queues 1 kernel; no atomics. */
int fpde_residual_vjp(int op, const fpde_grid* grid, const fpde_coeffs* coeffs,
                      const float* const* fields, const float* const* sens, int accumulate,
                      float* const* grads, void* stream);

/* The same five calls for grids described by fpde_grid4: every op, four-axis
 * grids included.  Arguments, write sets and errors as the calls above, with
 * "the planes of array axis 0" read for a four-axis grid as its time levels
 * (3-D volumes).  For FPDE_NS_3DT:
 *   - fpde_residual_fwd4 queues the loss fill and one march over every interior
 *     time level; with residual_out, also a fill of zeros on the end levels
 *     (3 kernels);
 *   - fpde_residual_bwd4 writes every node of the levels 1 .. n[0] - 2 with two
 *     kernels: a march over each level (the spatial part of the transposed
 *     stencil, boundary nodes of the level included), then a march along the
 *     time axis that adds the time part (R_q(t-1) - R_q(t+1)) / (2 h_t) at every
 *     node of the spatial residual set, recomputing those residuals;
 *   - fpde_bc_correct4 writes the end levels 0 and n[0] - 1 (1 kernel);
 *   - fpde_residual_value_and_grad4 queues the fill, the level march with the
 *     loss, the time march and (bc_mode 0) the end-level kernel;
 *   - fpde_residual_vjp4 queues one march over every level; the time part comes
 *     from the sensitivities of the neighbouring levels at the node itself.
 * Queues nothing and returns an error status on invalid arguments, as above. */
int fpde_residual_fwd4(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                       const float* const* fields, const float* const* consts,
                       float* const* residual_out, double* loss, void* stream);
int fpde_residual_bwd4(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                       const float* const* fields, const float* const* consts,
                       const double* dloss, float* const* grads, void* stream);
int fpde_bc_correct4(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                     const float* const* fields, const float* const* consts,
                     const double* dloss, float* const* grads, void* stream);
int fpde_residual_value_and_grad4(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                                  const float* const* fields, const float* const* consts,
                                  const double* dloss, double* loss, float* const* grads,
                                  void* stream);
int fpde_residual_vjp4(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                       const float* const* fields, const float* const* sens, int accumulate,
                       float* const* grads, void* stream);

/* Static string naming a status code (never NULL). */
const char* fpde_status_string(int status);

/* Static version string of the library. */
const char* fpde_version(void);

#ifdef __cplusplus
}
#endif
#endif /* FPDE_H */
