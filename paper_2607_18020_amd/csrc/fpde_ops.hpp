// fpde_ops.hpp -- per-operator point arithmetic for the gfx950 kernels.
//
// Each operator is a struct with compile-time sizes and three device
// functions, all in float32:
//   residual(f, c, K, R)    R_b at one node from the 2*DIM+1-point star of every
//                           stencil field and the point values of the consts
//                           (the fused forward stencil, Sec. 2.1);
//   gather(f, r, K, g)      sum over the star of node n of R_b(m) dR_b(m)/dq(n):
//                           the transpose-Jacobian action in gather form
//                           (Sec. 2.2; the printed dL/du of the 2D NS operator is
//                           the NS case with DIM = 2), without the 2 dloss / M
//                           factor that the caller applies;
//   bc_term<AX>(f, c, K, t, g)
//                           for a boundary-face node n = m + t e_AX whose only
//                           residual neighbour is m: R_b(m) dR_b(m)/dq(n)
//                           (the boundary-gradient correction, Sec. 2.3).
// The gather splits into gather_self(f, R, K, S), its first NG partial sums,
// which need only R(n) and the star of n, and gather_rest(f, r, S, K, g), the
// neighbour terms added to them in the same order (gather = rest after self).
// The backward evaluates the self part where it evaluates R(n), from the same
// star, and carries the NG sums to the step that gathers at n.
// NFG: the gather reads the stars of the first NFG fields only (the fields the
// residual Jacobian depends on: none for a linear operator, the velocity and not
// the pressure for NS, whose pressure enters linearly).
// Star values are indexed by array axis: m[a] / p[a] hold q(n - e_a) / q(n + e_a).
//
// Evaluation order: second differences are formed as ((q+ - q) + (q- - q)) / h^2,
// differences first, and the viscous / diffusive term is kept separate from the
// advective products.  Smooth float32 fields make neighbouring values close, so
// the differences are exact and the only rounding is in the small sums; the
// algebraically equal grouped form (q+ - 2q + q-) or coefficient grouping such as
// g * (u_x + 2 nu/h^2) loses several digits on fine grids.
//
// Every multiply that feeds an add is written as fmaf, and the library is built
// with floating-point contraction off: an operator's arithmetic is then the same
// instruction sequence whichever kernel evaluates it, so two kernels that
// evaluate the same residual or gather agree bit for bit.
//
// The divergence residual sum_a D1_a c_a of a nearly divergence-free velocity is
// a near-total cancellation of terms far larger than the result, so it is summed
// in float64 (differences widened exactly, float64 1/(2h_a)) and rounded once.
#pragma once

#include <hip/hip_runtime.h>

namespace fpde {

struct Star {
    float c;
    float m[3];
    float p[3];
};

// Float32 coefficients derived on the host in float64 and rounded once.
struct KCoef {
    double i2hd[3];  // 1 / (2 h_a) in float64 (divergence residual)
    float i2h[3];    // 1 / (2 h_a)
    float ih2[3];    // 1 / h_a^2
    float nu;
    float k2;        // k^2
    float inv_dt;    // 1 / dt
    float alpha;
    float i2ht;      // 1 / (2 h_t): the time axis of a 3D+t grid (axes a above are spatial)
};

__device__ __forceinline__ float d1(const Star& s, int a, const KCoef& K) {
    return (s.p[a] - s.m[a]) * K.i2h[a];
}

template <int DIM>
__device__ __forceinline__ float lap(const Star& s, const KCoef& K) {
    float l = 0.f;
#pragma unroll
    for (int a = 0; a < DIM; ++a) l = fmaf((s.p[a] - s.c) + (s.m[a] - s.c), K.ih2[a], l);
    return l;
}

// ---------------------------------------------------------------------------
// Burgers on a space-time grid: axis 0 = t, axis 1 = x.
//   R = u_t + u u_x - nu u_xx
struct OpBurgers {
    static constexpr int DIM = 2, NF = 1, NC = 0, NR = 1, NG = 0, NFG = 1;
    static constexpr bool TIME = false;  // (see OpNS3T)

    __device__ __forceinline__ static void residual(const Star* f, const float*, const KCoef& K, float* R) {
        const Star& u = f[0];
        const float uxx = ((u.p[1] - u.c) + (u.m[1] - u.c)) * K.ih2[1];
        R[0] = fmaf(-K.nu, uxx, fmaf(u.c, d1(u, 1, K), d1(u, 0, K)));
    }

    // dL/du(n): time neighbours (R(n-e_t) - R(n+e_t))/(2dt); advective
    // R(n) u_x(n) + (R(n-e_x) u(n-e_x) - R(n+e_x) u(n+e_x))/(2dx); viscous -nu D2_x R.
    __device__ __forceinline__ static void gather(const Star* f, const Star* r, const KCoef& K, float* g) {
        const Star& u = f[0];
        const Star& R = r[0];
        float acc = (R.m[0] - R.p[0]) * K.i2h[0];
        acc = fmaf(R.c, d1(u, 1, K), acc);
        acc = fmaf(fmaf(R.m[1], u.m[1], -(R.p[1] * u.p[1])), K.i2h[1], acc);
        g[0] = fmaf(-K.nu, ((R.p[1] - R.c) + (R.m[1] - R.c)) * K.ih2[1], acc);
    }

    __device__ __forceinline__ static void gather_self(const Star*, const float*, const KCoef&, float*) {}
    __device__ __forceinline__ static void gather_rest(const Star* f, const Star* r, const float*, const KCoef& K, float* g) {
        gather(f, r, K, g);
    }

    template <int AX>
    __device__ __forceinline__ static void bc_term(const Star* f, const float* c, const KCoef& K, float t, float* g) {
        float R[1];
        residual(f, c, K, R);
        g[0] = (AX == 0) ? R[0] * t * K.i2h[0]
                         : R[0] * fmaf(t * f[0].c, K.i2h[1], -K.nu * K.ih2[1]);
    }
};

// ---------------------------------------------------------------------------
// Helmholtz: R = lap u + k^2 u - f   (self-adjoint: dL/du = k^2 R + lap R).
struct OpHelmholtz {
    static constexpr int DIM = 2, NF = 1, NC = 1, NR = 1, NG = 0, NFG = 0;
    static constexpr bool TIME = false;  // (see OpNS3T)

    __device__ __forceinline__ static void residual(const Star* f, const float* c, const KCoef& K, float* R) {
        R[0] = fmaf(K.k2, f[0].c, lap<2>(f[0], K)) - c[0];
    }

    __device__ __forceinline__ static void gather(const Star*, const Star* r, const KCoef& K, float* g) {
        g[0] = fmaf(K.k2, r[0].c, lap<2>(r[0], K));
    }
    __device__ __forceinline__ static void gather_self(const Star*, const float*, const KCoef&, float*) {}
    __device__ __forceinline__ static void gather_rest(const Star* f, const Star* r, const float*, const KCoef& K, float* g) {
        gather(f, r, K, g);
    }

    template <int AX>
    __device__ __forceinline__ static void bc_term(const Star* f, const float* c, const KCoef& K, float, float* g) {
        float R[1];
        residual(f, c, K, R);
        g[0] = R[0] * K.ih2[AX];
    }
};

// ---------------------------------------------------------------------------
// One implicit heat step: R = (u - u0)/dt - alpha lap u.
struct OpHeat {
    static constexpr int DIM = 3, NF = 1, NC = 1, NR = 1, NG = 0, NFG = 0;
    static constexpr bool TIME = false;  // (see OpNS3T)

    __device__ __forceinline__ static void residual(const Star* f, const float* c, const KCoef& K, float* R) {
        R[0] = fmaf(-K.alpha, lap<3>(f[0], K), (f[0].c - c[0]) * K.inv_dt);
    }

    __device__ __forceinline__ static void gather(const Star*, const Star* r, const KCoef& K, float* g) {
        g[0] = fmaf(-K.alpha, lap<3>(r[0], K), r[0].c * K.inv_dt);
    }
    __device__ __forceinline__ static void gather_self(const Star*, const float*, const KCoef&, float*) {}
    __device__ __forceinline__ static void gather_rest(const Star* f, const Star* r, const float*, const KCoef& K, float* g) {
        gather(f, r, K, g);
    }

    template <int AX>
    __device__ __forceinline__ static void bc_term(const Star* f, const float* c, const KCoef& K, float, float* g) {
        float R[1];
        residual(f, c, K, R);
        g[0] = -R[0] * K.alpha * K.ih2[AX];
    }
};

// ---------------------------------------------------------------------------
// Incompressible NS; velocity component b on array axis b, pressure last.
//   R_b = [(c_b - c_b_prev)/dt] + sum_a c_a D1_a c_b + D1_b p - nu lap c_b
//   R_div = sum_a D1_a c_a
// UNSTEADY selects the backward-Euler time term (consts = previous velocities).
template <int D, bool UNSTEADY>
struct OpNS {
    static constexpr int DIM = D, NF = D + 1, NC = UNSTEADY ? D : 0, NR = D + 1, NG = D, NFG = D;
    static constexpr bool TIME = false;  // (see OpNS3T)

    __device__ __forceinline__ static void residual(const Star* f, const float* c, const KCoef& K, float* R) {
        float cs[D];  // c_a / (2 h_a), shared by the D momentum equations
#pragma unroll
        for (int a = 0; a < D; ++a) cs[a] = f[a].c * K.i2h[a];
        double div = 0.0;
#pragma unroll
        for (int b = 0; b < D; ++b) {
            float r = cs[0] * (f[b].p[0] - f[b].m[0]);
#pragma unroll
            for (int a = 1; a < D; ++a) r = fmaf(cs[a], f[b].p[a] - f[b].m[a], r);
            r = fmaf(f[D].p[b] - f[D].m[b], K.i2h[b], r);
            if (UNSTEADY) r = fmaf(f[b].c - c[b], K.inv_dt, r);
            R[b] = fmaf(-K.nu, lap<D>(f[b], K), r);
            div = fma((double)f[b].p[b] - (double)f[b].m[b], K.i2hd[b], div);
        }
        R[D] = (float)div;
    }

    // dL/dc_q(n) = sum_b R_b(n) D1_q c_b(n) + [R_q(n)/dt]
    //            + sum_a (R_q(n-e_a) c_a(n-e_a) - R_q(n+e_a) c_a(n+e_a)) / (2 h_a)
    //            + (R_div(n-e_q) - R_div(n+e_q)) / (2 h_q) - nu lap R_q(n)
    // dL/dp(n)   = sum_b (R_b(n-e_b) - R_b(n+e_b)) / (2 h_b)
    // the node's own terms: S_q = sum_b R_b(n) D1_q c_b(n) [+ R_q(n)/dt]
    __device__ __forceinline__ static void gather_self(const Star* f, const float* R, const KCoef& K, float* S) {
#pragma unroll
        for (int q = 0; q < D; ++q) {
            float loc = R[0] * (f[0].p[q] - f[0].m[q]);
#pragma unroll
            for (int b = 1; b < D; ++b) loc = fmaf(R[b], f[b].p[q] - f[b].m[q], loc);
            S[q] = loc * K.i2h[q];
            if (UNSTEADY) S[q] = fmaf(R[q], K.inv_dt, S[q]);
        }
    }

    // the neighbour terms, added to S in order
    __device__ __forceinline__ static void gather_rest(const Star* f, const Star* r, const float* S, const KCoef& K, float* g) {
        float gp = 0.f;
#pragma unroll
        for (int q = 0; q < D; ++q) {
            float acc = S[q];
#pragma unroll
            for (int a = 0; a < D; ++a)
                acc = fmaf(fmaf(r[q].m[a], f[a].m[a], -(r[q].p[a] * f[a].p[a])), K.i2h[a], acc);
            acc = fmaf(r[D].m[q] - r[D].p[q], K.i2h[q], acc);
            g[q] = fmaf(-K.nu, lap<D>(r[q], K), acc);
            gp = fmaf(r[q].m[q] - r[q].p[q], K.i2h[q], gp);
        }
        g[D] = gp;
    }

    __device__ __forceinline__ static void gather(const Star* f, const Star* r, const KCoef& K, float* g) {
        float R[NR], S[D];
#pragma unroll
        for (int b = 0; b < NR; ++b) R[b] = r[b].c;
        gather_self(f, R, K, S);
        gather_rest(f, r, S, K, g);
    }

    // n = m + t e_AX: only the neighbour terms of R_b(m) reach n.
    template <int AX>
    __device__ __forceinline__ static void bc_term(const Star* f, const float* c, const KCoef& K, float t, float* g) {
        float R[NR];
        residual(f, c, K, R);
#pragma unroll
        for (int q = 0; q < D; ++q) {
            float v = R[q] * fmaf(t * f[AX].c, K.i2h[AX], -K.nu * K.ih2[AX]);
            if (q == AX) v = fmaf(R[D] * t, K.i2h[AX], v);
            g[q] = v;
        }
        g[D] = R[AX] * t * K.i2h[AX];
    }
};

using OpNS2 = OpNS<2, false>;
using OpNS3 = OpNS<3, true>;
using OpNS3S = OpNS<3, false>;  // steady 3D NS

// ---------------------------------------------------------------------------
// Poisson: R = lap u - f   (self-adjoint: dL/du = lap R).
template <int D>
struct OpPoisson {
    static constexpr int DIM = D, NF = 1, NC = 1, NR = 1, NG = 0, NFG = 0;
    static constexpr bool TIME = false;  // (see OpNS3T)

    __device__ __forceinline__ static void residual(const Star* f, const float* c, const KCoef& K, float* R) {
        R[0] = lap<D>(f[0], K) - c[0];
    }

    __device__ __forceinline__ static void gather(const Star*, const Star* r, const KCoef& K, float* g) {
        g[0] = lap<D>(r[0], K);
    }
    __device__ __forceinline__ static void gather_self(const Star*, const float*, const KCoef&, float*) {}
    __device__ __forceinline__ static void gather_rest(const Star* f, const Star* r, const float*, const KCoef& K, float* g) {
        gather(f, r, K, g);
    }

    template <int AX>
    __device__ __forceinline__ static void bc_term(const Star* f, const float* c, const KCoef& K, float, float* g) {
        float R[1];
        residual(f, c, K, R);
        g[0] = R[0] * K.ih2[AX];
    }
};

// ---------------------------------------------------------------------------
// Unsteady incompressible NS on a 2D+t space-time grid: array axis 0 is t
// (a centred difference in time, step h_0), velocity component b on array axis
// b + 1, pressure last.
//   R_b = D1_0 c_b + sum_a c_a D1_{a+1} c_b + D1_{b+1} p - nu lap_xy c_b
//   R_div = sum_a D1_{a+1} c_a                     (a, b over x and y)
struct OpNST {
    static constexpr int D = 2;  // spatial dimensions
    static constexpr int DIM = 3, NF = D + 1, NC = 0, NR = D + 1, NG = D, NFG = D;
    static constexpr bool TIME = false;  // (see OpNS3T)

    __device__ __forceinline__ static float lap_xy(const Star& s, const KCoef& K) {
        float l = 0.f;
#pragma unroll
        for (int a = 1; a <= D; ++a) l = fmaf((s.p[a] - s.c) + (s.m[a] - s.c), K.ih2[a], l);
        return l;
    }

    __device__ __forceinline__ static void residual(const Star* f, const float*, const KCoef& K, float* R) {
        float cs[D];  // c_a / (2 h_{a+1}), shared by the momentum equations
#pragma unroll
        for (int a = 0; a < D; ++a) cs[a] = f[a].c * K.i2h[a + 1];
        double div = 0.0;
#pragma unroll
        for (int b = 0; b < D; ++b) {
            float r = (f[b].p[0] - f[b].m[0]) * K.i2h[0];  // time derivative
#pragma unroll
            for (int a = 0; a < D; ++a) r = fmaf(cs[a], f[b].p[a + 1] - f[b].m[a + 1], r);
            r = fmaf(f[D].p[b + 1] - f[D].m[b + 1], K.i2h[b + 1], r);
            R[b] = fmaf(-K.nu, lap_xy(f[b], K), r);
            div = fma((double)f[b].p[b + 1] - (double)f[b].m[b + 1], K.i2hd[b + 1], div);
        }
        R[D] = (float)div;
    }

    // dL/dc_q(n) = sum_b R_b(n) D1_{q+1} c_b(n) + (R_q(n-e_0) - R_q(n+e_0)) / (2 h_0)
    //            + sum_a (R_q(n-e_{a+1}) c_a(n-e_{a+1}) - R_q(n+e_{a+1}) c_a(n+e_{a+1})) / (2 h_{a+1})
    //            + (R_div(n-e_{q+1}) - R_div(n+e_{q+1})) / (2 h_{q+1}) - nu lap_xy R_q(n)
    // dL/dp(n)   = sum_b (R_b(n-e_{b+1}) - R_b(n+e_{b+1})) / (2 h_{b+1})
    __device__ __forceinline__ static void gather_self(const Star* f, const float* R, const KCoef& K, float* S) {
#pragma unroll
        for (int q = 0; q < D; ++q) {
            float loc = R[0] * (f[0].p[q + 1] - f[0].m[q + 1]);
#pragma unroll
            for (int b = 1; b < D; ++b) loc = fmaf(R[b], f[b].p[q + 1] - f[b].m[q + 1], loc);
            S[q] = loc * K.i2h[q + 1];
        }
    }

    __device__ __forceinline__ static void gather_rest(const Star* f, const Star* r, const float* S, const KCoef& K, float* g) {
        float gp = 0.f;
#pragma unroll
        for (int q = 0; q < D; ++q) {
            float acc = fmaf(r[q].m[0] - r[q].p[0], K.i2h[0], S[q]);
#pragma unroll
            for (int a = 0; a < D; ++a)
                acc = fmaf(fmaf(r[q].m[a + 1], f[a].m[a + 1], -(r[q].p[a + 1] * f[a].p[a + 1])),
                           K.i2h[a + 1], acc);
            acc = fmaf(r[D].m[q + 1] - r[D].p[q + 1], K.i2h[q + 1], acc);
            g[q] = fmaf(-K.nu, lap_xy(r[q], K), acc);
            gp = fmaf(r[q].m[q + 1] - r[q].p[q + 1], K.i2h[q + 1], gp);
        }
        g[D] = gp;
    }

    __device__ __forceinline__ static void gather(const Star* f, const Star* r, const KCoef& K, float* g) {
        float R[NR], S[D];
#pragma unroll
        for (int b = 0; b < NR; ++b) R[b] = r[b].c;
        gather_self(f, R, K, S);
        gather_rest(f, r, S, K, g);
    }

    // n = m + t e_AX: only the neighbour terms of R_b(m) along AX reach n.
    template <int AX>
    __device__ __forceinline__ static void bc_term(const Star* f, const float* c, const KCoef& K, float t, float* g) {
        float R[NR];
        residual(f, c, K, R);
        if (AX == 0) {  // time: only the time derivative of the velocities
#pragma unroll
            for (int q = 0; q < D; ++q) g[q] = R[q] * t * K.i2h[0];
            g[D] = 0.f;
        } else {
            constexpr int S_ = AX - 1;  // the velocity component along AX
#pragma unroll
            for (int q = 0; q < D; ++q) {
                float v = R[q] * fmaf(t * f[S_].c, K.i2h[AX], -K.nu * K.ih2[AX]);
                if (q == S_) v = fmaf(R[D] * t, K.i2h[AX], v);
                g[q] = v;
            }
            g[D] = R[S_] * t * K.i2h[AX];
        }
    }
};

// ---------------------------------------------------------------------------
// Unsteady incompressible NS on a 3D+t space-time grid (t, x, y, z): array
// axis 0 is t (a centred difference in time, step h_t), velocity component b
// on array axis b + 1, pressure last.
//   R_b = D1_t c_b + sum_a c_a D1_a c_b + D1_b p - nu lap c_b      (a, b over x, y, z)
//   R_div = sum_a D1_a c_a
// The kernels run the 3-D engine on one time level t at a time (TIME): the
// stars here are spatial (index a = spatial axis a, array axis a + 1) and the
// velocities at the neighbouring time levels enter as point values, the consts
// c[0..2] = c_b(t - 1) and c[3..5] = c_b(t + 1) (TSRC / TOFF: the field and
// the time offset each const is read from).  The gather below is the spatial
// part of the transposed stencil; its time part, (R_q(t-1) - R_q(t+1)) / (2 h_t),
// needs the residuals of other time levels and is added by the time-march
// kernel (or, from given sensitivities, by the explicit-sensitivity backward).
struct OpNS3T {
    static constexpr int D = 3;  // spatial dimensions
    static constexpr int DIM = 3, NF = D + 1, NC = 2 * D, NR = D + 1, NG = D, NFG = D;
    static constexpr bool TIME = true;
    static constexpr int TSRC[2 * D] = {0, 1, 2, 0, 1, 2};
    static constexpr int TOFF[2 * D] = {-1, -1, -1, 1, 1, 1};

    __device__ __forceinline__ static void residual(const Star* f, const float* c, const KCoef& K, float* R) {
        float cs[D];  // c_a / (2 h_a), shared by the momentum equations
#pragma unroll
        for (int a = 0; a < D; ++a) cs[a] = f[a].c * K.i2h[a];
        double div = 0.0;
#pragma unroll
        for (int b = 0; b < D; ++b) {
            float r = (c[D + b] - c[b]) * K.i2ht;  // time derivative
#pragma unroll
            for (int a = 0; a < D; ++a) r = fmaf(cs[a], f[b].p[a] - f[b].m[a], r);
            r = fmaf(f[D].p[b] - f[D].m[b], K.i2h[b], r);
            R[b] = fmaf(-K.nu, lap<D>(f[b], K), r);
            div = fma((double)f[b].p[b] - (double)f[b].m[b], K.i2hd[b], div);
        }
        R[D] = (float)div;
    }

    // spatial part of dL/dc_q(n): sum_b R_b(n) D1_q c_b(n)
    //   + sum_a (R_q(n-e_a) c_a(n-e_a) - R_q(n+e_a) c_a(n+e_a)) / (2 h_a)
    //   + (R_div(n-e_q) - R_div(n+e_q)) / (2 h_q) - nu lap R_q(n);
    // dL/dp(n) = sum_b (R_b(n-e_b) - R_b(n+e_b)) / (2 h_b)
    __device__ __forceinline__ static void gather_self(const Star* f, const float* R, const KCoef& K, float* S) {
#pragma unroll
        for (int q = 0; q < D; ++q) {
            float loc = R[0] * (f[0].p[q] - f[0].m[q]);
#pragma unroll
            for (int b = 1; b < D; ++b) loc = fmaf(R[b], f[b].p[q] - f[b].m[q], loc);
            S[q] = loc * K.i2h[q];
        }
    }

    __device__ __forceinline__ static void gather_rest(const Star* f, const Star* r, const float* S, const KCoef& K, float* g) {
        float gp = 0.f;
#pragma unroll
        for (int q = 0; q < D; ++q) {
            float acc = S[q];
#pragma unroll
            for (int a = 0; a < D; ++a)
                acc = fmaf(fmaf(r[q].m[a], f[a].m[a], -(r[q].p[a] * f[a].p[a])), K.i2h[a], acc);
            acc = fmaf(r[D].m[q] - r[D].p[q], K.i2h[q], acc);
            g[q] = fmaf(-K.nu, lap<D>(r[q], K), acc);
            gp = fmaf(r[q].m[q] - r[q].p[q], K.i2h[q], gp);
        }
        g[D] = gp;
    }

    __device__ __forceinline__ static void gather(const Star* f, const Star* r, const KCoef& K, float* g) {
        float R[NR], S[D];
#pragma unroll
        for (int b = 0; b < NR; ++b) R[b] = r[b].c;
        gather_self(f, R, K, S);
        gather_rest(f, r, S, K, g);
    }

    // the time part for velocity q from the residuals (or sensitivities) of its
    // own node at t - 1 (rm) and t + 1 (rp), added after the spatial part
    __device__ __forceinline__ static void add_time(const float* rm, const float* rp, const KCoef& K, float* g) {
#pragma unroll
        for (int q = 0; q < D; ++q) g[q] = fmaf(rm[q] - rp[q], K.i2ht, g[q]);
    }

    // n = m + t e_AX on a spatial axis AX: only the neighbour terms of R_b(m) reach n
    template <int AX>
    __device__ __forceinline__ static void bc_term(const Star* f, const float* c, const KCoef& K, float t, float* g) {
        float R[NR];
        residual(f, c, K, R);
#pragma unroll
        for (int q = 0; q < D; ++q) {
            float v = R[q] * fmaf(t * f[AX].c, K.i2h[AX], -K.nu * K.ih2[AX]);
            if (q == AX) v = fmaf(R[D] * t, K.i2h[AX], v);
            g[q] = v;
        }
        g[D] = R[AX] * t * K.i2h[AX];
    }

    // n = m + t e_t (an end time level): only the time derivative of R_q(m) reaches n
    __device__ __forceinline__ static void bc_time(const Star* f, const float* c, const KCoef& K, float t, float* g) {
        float R[NR];
        residual(f, c, K, R);
#pragma unroll
        for (int q = 0; q < D; ++q) g[q] = R[q] * t * K.i2ht;
        g[D] = 0.f;
    }
};

}  // namespace fpde
