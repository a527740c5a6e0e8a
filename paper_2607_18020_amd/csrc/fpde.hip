// fpde.hip -- host side of libfpde: argument validation, launch geometry and
// the exported C entry points declared in include/fpde.h.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <type_traits>

#include "fpde.h"
#include "fpde_engine.hpp"

namespace fpde {
namespace {

// Launch geometry.  A workgroup owns a TX x TY column tile (TY = 1 for 2-D
// grids, where a "plane" is one row) and marches a chunk of planes of axis 0.
// 3-D grids: the chunk length is chosen once per call from the backward's
// tiling (at least kMinBwdBlocks workgroups) and shared by the forward and the
// backward, so that the backward, which marches each chunk top down, starts on
// the planes the forward read last (still in the memory-side infinity cache).
// 2-D grids: chunks sized for about kTargetBlocks2 workgroups per launch.
// backward tile widths: a tile's x-halo columns sit in cache lines of the
// neighbouring tiles, which L2 serves only while the two tiles march in step;
// wider tiles have fewer such lines per node
#ifndef FPDE_NS3_BWD_TX
#define FPDE_NS3_BWD_TX 128
#endif
#ifndef FPDE_HEAT_BWD_TX
#define FPDE_HEAT_BWD_TX 64
#endif
// forward tile widths (a tile's side-edge x-neighbours cost a cache line each)
#ifndef FPDE_NS3_FWD_TX
#define FPDE_NS3_FWD_TX 128
#endif
#ifndef FPDE_HEAT_FWD_TX
#define FPDE_HEAT_FWD_TX 256
#endif
#ifndef FPDE_NS3_FWD_TY
#define FPDE_NS3_FWD_TY 4
#endif
#ifndef FPDE_NS3_BWD_TY
#define FPDE_NS3_BWD_TY 8
#endif
#ifndef FPDE_NS3_MIN_BWD_BLOCKS
#define FPDE_NS3_MIN_BWD_BLOCKS 256
#endif
#ifndef FPDE_HEAT_FWD_TY
#define FPDE_HEAT_FWD_TY 4
#endif
#ifndef FPDE_HEAT_BWD_TY
#define FPDE_HEAT_BWD_TY 8
#endif
#ifndef FPDE_HEAT_MIN_BWD_BLOCKS
#define FPDE_HEAT_MIN_BWD_BLOCKS 1024
#endif
#ifndef FPDE_TX2
#define FPDE_TX2 256
#endif
// 2-D forward rows: the loss atomics of a short launch arrive together and are
// serialised on one address, so the forward uses fewer, wider workgroups
#ifndef FPDE_TX2_FWD
#define FPDE_TX2_FWD 1024
#endif
// register-queue forward: planes held per lane (the centre plane, its two
// neighbours, and Q - 3 planes in flight)
#ifndef FPDE_FWD2_Q
#define FPDE_FWD2_Q 6
#endif
// 3-D operators with one stencil field (heat, Poisson) can use the
// register-queue forward too (five loads per node and plane fit the registers);
// the LDS march is faster there (heat 256^3: 29 against 32 us), so the product
// keeps it and the checking build takes the queue, as a second algorithm
#ifndef FPDE_HEAT_FWD_QUEUE
#define FPDE_HEAT_FWD_QUEUE 0
#endif
// one stencil field and almost no arithmetic per plane: the LDS march forward
// keeps several planes in flight (an 8-slot ring), where one plane per step
// would wait for each plane's latency in turn
#ifndef FPDE_HEAT_FWD_RING
#define FPDE_HEAT_FWD_RING 8
#endif
// 2-D backward: the LDS march (bwd_kernel with one-row tiles); the checking
// build takes the register-queue march (bwdq_kernel: no LDS, no barrier; NW
// waves of 62 output columns, Q rows in registers) as a second algorithm whose
// gradients must match bit for bit.  (The queue march is no faster for the
// product: NS-2D 2048^2 37.8 against 36.7 us per step.)
#ifndef FPDE_BWD2_QUEUE
#define FPDE_BWD2_QUEUE 0
#endif
#ifndef FPDE_BWD2_NW
#define FPDE_BWD2_NW 4
#endif
#ifndef FPDE_BWD2_Q
#define FPDE_BWD2_Q 7
#endif
// 2-D one-pass value and gradient (the backward with the loss atomics)
#ifndef FPDE_TX2_VG
#define FPDE_TX2_VG 512
#endif
// explicit-sensitivity backward tiles (3-D)
#ifndef FPDE_VJP_TX3
#define FPDE_VJP_TX3 64
#endif
#ifndef FPDE_VJP_TY3
#define FPDE_VJP_TY3 4
#endif
#ifndef FPDE_VJP_HEAT_TX
#define FPDE_VJP_HEAT_TX 128
#endif
#ifndef FPDE_VJP_HEAT_TY
#define FPDE_VJP_HEAT_TY 8
#endif
#ifndef FPDE_VJP_TARGET3
#define FPDE_VJP_TARGET3 512
#endif
#ifndef FPDE_BLOCKS2
#define FPDE_BLOCKS2 1024
#endif
// The backward marches each chunk top-down (see above).
#ifndef FPDE_BWD_REVERSE
#define FPDE_BWD_REVERSE 1
#endif
constexpr int kTX2 = FPDE_TX2, kTX2F = FPDE_TX2_FWD, kTX2V = FPDE_TX2_VG,
              kTargetBlocks2 = FPDE_BLOCKS2;
constexpr bool kBwdReverse = FPDE_BWD_REVERSE != 0;

// 3-D grids: forward tile TXF x TYf, backward tile TXB x TYb, explicit-sensitivity
// backward tile TXV x TYV
template <int TXF_, int TYF, int TXB_, int TYB, int MINB, int TXV_, int TYV_, bool QF = false,
          int RF = 4>
struct Geo3 {
    static constexpr bool D3 = true;
    static constexpr bool FWD_QUEUE = QF;  // forward: fwdq_kernel (else the LDS march)
    static constexpr int FWD_RING = RF;    // LDS march forward: slots of its plane ring
    static constexpr int TXF = TXF_, TYf = TYF, TXB = TXB_, TYb = TYB, MIN_BWD_BLOCKS = MINB;
    static constexpr int TXV = TXV_, TYV = TYV_;
};
// 2-D grids: one-row tiles of kTX2 nodes for every kernel
struct Geo2 {
    static constexpr bool D3 = false;
    static constexpr bool FWD_QUEUE = true;  // (the 2-D forward is always fwdq_kernel)
};
// several fields with nonlinear coupling (NS)
using GeoNS3 = Geo3<FPDE_NS3_FWD_TX, FPDE_NS3_FWD_TY, FPDE_NS3_BWD_TX, FPDE_NS3_BWD_TY,
                    FPDE_NS3_MIN_BWD_BLOCKS, FPDE_VJP_TX3, FPDE_VJP_TY3>;
// 3D+t NS: the level march reads six time-neighbour velocities per node besides
// the four fields, which do not fit the 128 registers of a 1024-thread backward
// tile: 768-thread backward tiles (at 20 x 128^3, 5% faster than 512 threads)
#ifndef FPDE_NS4_BWD_TX
#define FPDE_NS4_BWD_TX 128
#endif
#ifndef FPDE_NS4_BWD_TY
#define FPDE_NS4_BWD_TY 6
#endif
// workgroups per launch: a time level is a 3-D volume of its own, so whole-level
// chunks leave few workgroups (and a last round of them mostly idle) on the
// smaller volumes of space-time grids; chunks are cut for many rounds instead
#ifndef FPDE_NS4_MIN_BLOCKS
#define FPDE_NS4_MIN_BLOCKS 2048
#endif
using GeoNS4 = Geo3<FPDE_NS3_FWD_TX, FPDE_NS3_FWD_TY, FPDE_NS4_BWD_TX, FPDE_NS4_BWD_TY,
                    FPDE_NS4_MIN_BLOCKS, FPDE_VJP_TX3, FPDE_VJP_TY3>;
// one field, a Laplacian (heat, Poisson)
using GeoHeat = Geo3<FPDE_HEAT_FWD_TX, FPDE_HEAT_FWD_TY, FPDE_HEAT_BWD_TX, FPDE_HEAT_BWD_TY,
                     FPDE_HEAT_MIN_BWD_BLOCKS, FPDE_VJP_HEAT_TX, FPDE_VJP_HEAT_TY,
                     FPDE_HEAT_FWD_QUEUE != 0, FPDE_HEAT_FWD_RING>;

template <class OP_, class GEO_>
struct OpTag {
    using OP = OP_;    // point functions (fpde_ops.hpp)
    using GEO = GEO_;  // launch shapes
};

// f(OpTag<...>{}) for the op, FPDE_ERR_ARG for an unknown op: the one table
// that maps an op id to its point functions and launch shapes.
template <class F>
int with_op(int op, F&& f) {
    switch (op) {
    case FPDE_BURGERS_1DT: return f(OpTag<OpBurgers, Geo2>{});
    case FPDE_HELMHOLTZ_2D: return f(OpTag<OpHelmholtz, Geo2>{});
    case FPDE_HEAT_3D_BE: return f(OpTag<OpHeat, GeoHeat>{});
    case FPDE_NS_2D_STEADY: return f(OpTag<OpNS2, Geo2>{});
    case FPDE_NS_3D_BE: return f(OpTag<OpNS3, GeoNS3>{});
    case FPDE_NS_3D_STEADY: return f(OpTag<OpNS3S, GeoNS3>{});
    case FPDE_POISSON_2D: return f(OpTag<OpPoisson<2>, Geo2>{});
    case FPDE_POISSON_3D: return f(OpTag<OpPoisson<3>, GeoHeat>{});
    case FPDE_NS_2DT: return f(OpTag<OpNST, GeoNS3>{});
    // 3D+t: the 3-D marches run on one time level per workgroup
    case FPDE_NS_3DT: return f(OpTag<OpNS3T, GeoNS4>{});
    }
    return FPDE_ERR_ARG;
}

struct OpDesc {
    int ndim, nf, nc, nr;
    bool time;  // 3D+t: the grid has a time axis 0 before the DIM axes the kernels march
};

bool op_desc(int op, OpDesc* d) {
    return with_op(op, [&](auto tag) {
        using OP = typename decltype(tag)::OP;
        // (a 3D+t operator's consts are its own fields at the neighbouring time
        // levels, which the kernels address themselves: the caller passes none)
        *d = {OP::DIM + (OP::TIME ? 1 : 0), OP::NF, OP::TIME ? 0 : OP::NC, OP::NR, OP::TIME};
        return FPDE_OK;
    }) == FPDE_OK;
}

// ops with a time step dt among their coefficients
bool uses_dt(int op) { return op == FPDE_HEAT_3D_BE || op == FPDE_NS_3D_BE; }

struct Req {
    int op;
    OpDesc d;
    Dims dims;
    KCoef K;
    double inv_M, two_over_M;
    long long N, M;
    Ptrs P;
    hipStream_t stream;
};

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

bool finite_pos(double v) { return isfinite(v) && v > 0.0; }

// Validates everything except the outputs; fills req.  need_consts: the call
// reads the const arrays (the explicit-sensitivity backward does not).
int validate_common(int op, const fpde_grid4* g, const fpde_coeffs* c, const float* const* fields,
                    const float* const* consts, Req* r, bool need_consts = true) {
    if (!op_desc(op, &r->d)) return FPDE_ERR_ARG;
    if (!g || !c || !fields) return FPDE_ERR_ARG;
    if (!need_consts) consts = nullptr;
    const int nc = need_consts ? r->d.nc : 0;
    if (nc > 0 && !consts) return FPDE_ERR_ARG;
    for (int f = 0; f < r->d.nf; ++f)
        if (!fields[f]) return FPDE_ERR_ARG;
    for (int j = 0; j < nc; ++j)
        if (!consts[j]) return FPDE_ERR_ARG;
    if (g->bc_mode != 0 && g->bc_mode != 1) return FPDE_ERR_ARG;
    if (g->ndim != r->d.ndim) return FPDE_ERR_SHAPE;
    const int D = r->d.ndim;
    const bool per = g->bc_mode == 1;
    long long N = 1, M = 1;
    for (int a = 0; a < D; ++a) {
        if (g->n[a] < 3 || g->n[a] >= (1LL << 31)) return FPDE_ERR_SHAPE;
        if (N > (1LL << 62) / g->n[a]) return FPDE_ERR_SHAPE;
        N *= g->n[a];
        M *= per ? g->n[a] : g->n[a] - 2;  // periodic: a residual at every node
    }
    // plane of the last two axes (one row for 2-D grids) addressed with 32-bit byte
    // offsets; a 3D+t grid's time level (the last three axes) as well
    if ((D >= 3 ? g->n[D - 2] * g->n[D - 1] : g->n[1]) >= (1LL << 29)) return FPDE_ERR_SHAPE;
    if (D == 4 && g->n[1] * g->n[2] * g->n[3] >= (1LL << 29)) return FPDE_ERR_SHAPE;
    for (int a = 0; a < D; ++a)
        if (!finite_pos(g->h[a])) return FPDE_ERR_SPACING;
    if (!isfinite(c->nu) || !isfinite(c->k) || !isfinite(c->dt) || !isfinite(c->alpha))
        return FPDE_ERR_COEFF;
    if (uses_dt(op) && !(c->dt > 0.0)) return FPDE_ERR_COEFF;

    // float32 kernel coefficients, derived in float64; a 3D+t grid's kernel axes
    // are its spatial axes 1..3, and its time axis 0 has a coefficient of its own
    const int A0 = r->d.time ? 1 : 0;  // first array axis the kernels march
    KCoef K;
    memset(&K, 0, sizeof K);
    for (int a = 0; a < D - A0; ++a) {
        const double h = g->h[a + A0];
        K.i2hd[a] = 1.0 / (2.0 * h);
        K.i2h[a] = (float)(1.0 / (2.0 * h));
        K.ih2[a] = (float)(1.0 / (h * h));
        if (!isfinite(K.i2h[a]) || !isfinite(K.ih2[a]) || K.ih2[a] == 0.f) return FPDE_ERR_SPACING;
    }
    if (r->d.time) {
        K.i2ht = (float)(1.0 / (2.0 * g->h[0]));
        if (!isfinite(K.i2ht)) return FPDE_ERR_SPACING;
    }
    K.nu = (float)c->nu;
    K.k2 = (float)(c->k * c->k);
    K.inv_dt = uses_dt(op) ? (float)(1.0 / c->dt) : 0.f;
    K.alpha = (float)c->alpha;
    if (!isfinite(K.nu) || !isfinite(K.k2) || !isfinite(K.inv_dt) || !isfinite(K.alpha))
        return FPDE_ERR_COEFF;

    for (int f = 0; f < r->d.nf; ++f)
        if ((uintptr_t)fields[f] & 3u) return FPDE_ERR_ALIGN;
    for (int j = 0; j < nc; ++j)
        if ((uintptr_t)consts[j] & 3u) return FPDE_ERR_ALIGN;

    r->op = op;
    r->K = K;
    r->N = N;
    r->M = M;
    r->inv_M = 1.0 / (double)M;
    r->two_over_M = 2.0 / (double)M;
    memset(&r->P, 0, sizeof r->P);
    for (int f = 0; f < r->d.nf; ++f) r->P.f[f] = fields[f];
    for (int j = 0; j < nc; ++j) r->P.c[j] = consts[j];

    Dims& dm = r->dims;  // sizes only; tiles and chunks are set per launch
    dm.nz = (int)g->n[A0];
    dm.ny = (D - A0 == 3) ? (int)g->n[A0 + 1] : 1;
    dm.nx = (int)g->n[D - 1];
    dm.tiles_x = dm.tiles_y = dm.zc = dm.nblocks = 0;
    dm.per = per ? 1 : 0;
    dm.zlo = per ? 0 : 1;  // the marched planes: 1 .. n0-2, or all of them
    dm.nt = r->d.time ? (int)g->n[0] : 1;
    dm.nlev = 1;  // (set per launch for 3D+t grids)
    dm.lev0 = 0;
    dm.vol = r->d.time ? (long long)dm.nz * dm.ny * dm.nx : 0;
    // every launch shape used below must have fewer than 2^31 workgroups
    // (in 64 bits: an extent of axis 0 may be up to 2^31 - 1)
    if (((long long)dm.nx / 32 + 1) * ((long long)dm.ny + 1) * ((long long)dm.nz + 1) * dm.nt >=
        (1LL << 31))
        return FPDE_ERR_SHAPE;
    return FPDE_OK;
}

// The time levels a 3D+t launch covers: those with residuals (1 .. nt-2), or
// every level (periodic grids; the explicit-sensitivity backward, which writes
// every node).  No-op for other grids.
Dims levels(const Dims& n, bool all) {
    Dims dm = n;
    if (dm.nt > 1) {
        const bool every = all || dm.per;
        dm.lev0 = every ? 0 : 1;
        dm.nlev = every ? dm.nt : dm.nt - 2;
    }
    return dm;
}

// Tiles of TX x TY columns; chunks of zc planes along axis 0.
Dims tile_dims(const Dims& n, int TX, int TY, int zc) {
    Dims dm = n;
    dm.tiles_x = (dm.nx + TX - 1) / TX;
    dm.tiles_y = (dm.ny + TY - 1) / TY;
    const int nplanes = dm.nz - 2 * dm.zlo;
    dm.zc = zc;
    const long long nch = (nplanes + zc - 1) / zc;
    dm.nblocks = (int)((long long)dm.tiles_x * dm.tiles_y * nch * dm.nlev);
    return dm;
}

// Chunk length giving a launch with TX x TY tiles about `target` workgroups
// (each chunk at least one plane; 3D+t grids: over all launched levels, and at
// least kMinChunkT planes, as a chunk of a few planes re-reads its halo planes
// and its march prologue for little work).
constexpr int kMinChunkT = 8;
int chunk_planes(const Dims& n, int TX, int TY, int target) {
    const long long tiles =
        (long long)((n.nx + TX - 1) / TX) * ((n.ny + TY - 1) / TY) * n.nlev;
    const int nplanes = n.nz - 2 * n.zlo;
    long long nch = (target + tiles - 1) / tiles;
    if (n.nt > 1 && nch > (nplanes + kMinChunkT - 1) / kMinChunkT)
        nch = (nplanes + kMinChunkT - 1) / kMinChunkT;
    if (nch < 1) nch = 1;
    if (nch > nplanes) nch = nplanes;
    return (int)((nplanes + nch - 1) / nch);
}

int check_outputs(const Req& r, const fpde_grid4*, const float* const* fields,
                  const float* const* consts, float* const* outs, int nout, const void* extra,
                  size_t extra_bytes) {
    const size_t bytes = (size_t)r.N * sizeof(float);
    for (int o = 0; o < nout; ++o) {
        if (!outs[o]) return FPDE_ERR_ARG;
        if ((uintptr_t)outs[o] & 3u) return FPDE_ERR_ALIGN;
        for (int f = 0; f < r.d.nf; ++f)
            if (overlaps(outs[o], bytes, fields[f], bytes)) return FPDE_ERR_ARG;
        for (int j = 0; j < r.d.nc; ++j)
            if (overlaps(outs[o], bytes, consts[j], bytes)) return FPDE_ERR_ARG;
        for (int p = 0; p < o; ++p)
            if (overlaps(outs[o], bytes, outs[p], bytes)) return FPDE_ERR_ARG;
        if (extra && overlaps(outs[o], bytes, extra, extra_bytes)) return FPDE_ERR_ARG;
    }
    return FPDE_OK;
}

template <class T>
struct ident {
    using type = T;
};

// Queues kernel k on stream s and returns the status of that launch alone:
// hipLaunchKernel's own return value.  The thread's last-error state, which the
// caller may have left set by an earlier call, is neither read nor cleared.
// (The arguments take the kernel's parameter types, so each is passed in the
// layout the kernel expects.)
template <class... P>
int launch(void (*k)(P...), dim3 grid, dim3 block, hipStream_t s,
           typename ident<P>::type... args) {
    void* a[] = {(void*)&args...};
    return hipLaunchKernel(reinterpret_cast<const void*>(k), grid, block, a, 0, s) == hipSuccess
               ? FPDE_OK
               : FPDE_ERR_HIP;
}

int zero_loss(const Req& r, double* loss) {
    return launch(fill_f64_kernel, dim3(1), dim3(1), r.stream, loss, 0.0);
}

// ---- launches, per op type

// f(std::bool_constant<v>{}) for a runtime flag v: kernels take flags that
// decide their per-step control flow (periodic wrap, ...) as template arguments
template <class F>
void with_flag(bool v, F&& f) {
    if (v) f(std::true_type{});
    else f(std::false_type{});
}

template <class OP, int TX, int TY, int RD>
int launch_fwd(const Req& r, bool store, double* loss, int zc) {
    const Dims dm = tile_dims(r.dims, TX, TY, zc);
    int st = zero_loss(r, loss);
    if (st != FPDE_OK) return st;
    if (OP::TIME && store && !dm.per) {  // the end time levels hold no residual node
        st = launch(zero_levels_kernel<OP::NR>, dim3((unsigned)((2 * dm.vol + 255) / 256)),
                    dim3(256), r.stream, r.P, dm);
        if (st != FPDE_OK) return st;
    }
    with_flag(store, [&](auto sr) {
        with_flag(dm.per, [&](auto per) {
            st = launch(fwd_kernel<OP, TX, TY, decltype(sr)::value, decltype(per)::value, RD>,
                        dim3(dm.nblocks), dim3(TX * TY), r.stream, r.P, dm, r.K, r.inv_M, loss);
        });
    });
    return st;
}

// the register-queue forward (no LDS, no barrier)
template <class OP, int TX, int TY>
int launch_fwdq(const Req& r, bool store, double* loss, int zc) {
    const Dims dm = tile_dims(r.dims, TX, TY, zc);
    int st = zero_loss(r, loss);
    if (st != FPDE_OK) return st;
    with_flag(store, [&](auto sr) {
        with_flag(dm.per, [&](auto per) {
            st = launch(fwdq_kernel<OP, TX, TY, FPDE_FWD2_Q, decltype(sr)::value,
                                    decltype(per)::value>,
                        dim3(dm.nblocks), dim3(TX * TY), r.stream, r.P, dm, r.K, r.inv_M, loss);
        });
    });
    return st;
}

template <class OP, int TX, int TY>
int launch_bwd(const Req& r, const double* dloss, int zc, double* loss) {
    const Dims dm = tile_dims(r.dims, TX, TY, zc);
    // value and gradient in one pass when loss is given
    int st = loss ? zero_loss(r, loss) : FPDE_OK;
    if (st != FPDE_OK) return st;
    with_flag(loss != nullptr, [&](auto lo) {
        with_flag(dm.per, [&](auto per) {
            st = launch(bwd_kernel<OP, TX, TY, kBwdReverse, decltype(lo)::value,
                                   decltype(per)::value>,
                        dim3(dm.nblocks), dim3(TX * TY), r.stream, r.P, dm, r.K, dloss,
                        r.two_over_M, r.inv_M, loss);
        });
    });
    return st;
}

// 2-D register-queue backward (the gradient alone)
template <class OP>
int launch_bwdq(const Req& r, const double* dloss, int zc) {
    constexpr int NW = FPDE_BWD2_NW;
    const Dims dm = tile_dims(r.dims, 62 * NW, 1, zc);
    int st = FPDE_OK;
    with_flag(dm.per, [&](auto per) {
        st = launch(bwdq_kernel<OP, NW, FPDE_BWD2_Q, decltype(per)::value>, dim3(dm.nblocks),
                    dim3(64 * NW), r.stream, r.P, dm, r.K, dloss, r.two_over_M);
    });
    return st;
}

// 3-D: the chunk length shared by the forward and the backward
template <class GEO>
int zc3(const Req& r) {
    return chunk_planes(r.dims, GEO::TXB, GEO::TYb, GEO::MIN_BWD_BLOCKS);
}
int zc2(const Req& r) { return chunk_planes(r.dims, kTX2, 1, kTargetBlocks2); }

template <class OP>
int launch_bc(const Req& r, const double* dloss) {
    if constexpr (OP::TIME) {
        // 3D+t: the two end time levels, 256 consecutive nodes of a level per
        // workgroup (fewer than 2^31: a level holds fewer than 2^29 nodes)
        const long long nb = 2 * ((r.dims.vol + 255) / 256);
        return launch(bc4_kernel<OP>, dim3((unsigned)nb), dim3(256), r.stream, r.P, r.dims, r.K,
                      dloss, r.two_over_M);
    } else {
        // the two end planes of axis 0: one workgroup per 256-node segment of each row
        // (fewer than 2^31 of them: the node count of a plane is below 2^29)
        const long long nb = 2LL * r.dims.ny * ((r.dims.nx + 255) / 256);
        return launch(bc_kernel<OP>, dim3((unsigned)nb), dim3(256), r.stream, r.P, r.dims, r.K,
                      dloss, r.two_over_M);
    }
}

// 3D+t: the time part of the backward, one lane per spatial node marching the
// time levels (after the level march, which wrote the spatial part)
template <class OP>
int launch_tm(const Req& r, const double* dloss) {
    int st = FPDE_OK;
    with_flag(r.dims.per, [&](auto per) {
        st = launch(tm_kernel<OP, decltype(per)::value>,
                    dim3((unsigned)((r.dims.vol + 255) / 256)), dim3(256), r.stream, r.P, r.dims,
                    r.K, dloss, r.two_over_M);
    });
    return st;
}

// Explicit-sensitivity backward: every plane of axis 0 is marched (zlo = 0),
// on a 3D+t grid in every time level.
template <class OP, int TX, int TY>
int launch_vjp(const Req& r, bool acc, int target) {
    Dims base = levels(r.dims, true);
    base.zlo = 0;
    const Dims dm = tile_dims(base, TX, TY, chunk_planes(base, TX, TY, target));
    int st = FPDE_OK;
    with_flag(acc, [&](auto ac) {
        with_flag(dm.per, [&](auto per) {
            st = launch(vjp_kernel<OP, TX, TY, decltype(ac)::value, decltype(per)::value>,
                        dim3(dm.nblocks), dim3(TX * TY), r.stream, r.P, dm, r.K);
        });
    });
    return st;
}

int run_vjp(const Req& r, bool acc) {
    return with_op(r.op, [&](auto tag) {
        using OP = typename decltype(tag)::OP;
        using GEO = typename decltype(tag)::GEO;
        if constexpr (GEO::D3)
            return launch_vjp<OP, GEO::TXV, GEO::TYV>(
                r, acc, OP::TIME ? GEO::MIN_BWD_BLOCKS : FPDE_VJP_TARGET3);
        else
            return launch_vjp<OP, kTX2, 1>(r, acc, kTargetBlocks2);
    });
}

int run_fwd(const Req& r0, bool store, double* loss) {
    Req r = r0;
    r.dims = levels(r0.dims, false);
    return with_op(r.op, [&](auto tag) {
        using OP = typename decltype(tag)::OP;
        using GEO = typename decltype(tag)::GEO;
        if constexpr (GEO::D3 && GEO::FWD_QUEUE)
            return launch_fwdq<OP, GEO::TXF, GEO::TYf>(r, store, loss, zc3<GEO>(r));
        else if constexpr (GEO::D3)
            return launch_fwd<OP, GEO::TXF, GEO::TYf, GEO::FWD_RING>(r, store, loss, zc3<GEO>(r));
        else
            return launch_fwdq<OP, kTX2F, 1>(r, store, loss, zc2(r));
    });
}

// loss: nullptr for the gradient alone (planes 1 .. n0-2; the boundary kernel
// writes the end planes), else also the loss (fused value and grad), marching
// every plane: at the end planes the gather with the residuals off the residual
// set taken as zero is their exact boundary term, so no boundary kernel follows
//
// 3D+t grids: the level march covers every plane of each level with residuals
// (the boundary planes of the level included, as above), the time march then
// adds the time part, and with the loss the end time levels follow (bc_mode 0).
int run_bwd(const Req& r0, const double* dloss, double* loss = nullptr) {
    Req r = r0;
    r.dims = levels(r0.dims, false);
    if (loss || r.d.time) r.dims.zlo = 0;
    return with_op(r.op, [&](auto tag) {
        using OP = typename decltype(tag)::OP;
        using GEO = typename decltype(tag)::GEO;
        if constexpr (OP::TIME) {
            int st = launch_bwd<OP, GEO::TXB, GEO::TYb>(r, dloss, zc3<GEO>(r), loss);
            if (st == FPDE_OK) st = launch_tm<OP>(r, dloss);
            if (st == FPDE_OK && loss && !r.dims.per) st = launch_bc<OP>(r, dloss);
            return st;
        } else if constexpr (GEO::D3)
            return launch_bwd<OP, GEO::TXB, GEO::TYb>(r, dloss, zc3<GEO>(r), loss);
        else if (loss)
            return launch_bwd<OP, kTX2V, 1>(r, dloss, zc2(r), loss);
        else if (FPDE_BWD2_QUEUE)
            return launch_bwdq<OP>(r, dloss, zc2(r));
        else
            return launch_bwd<OP, kTX2, 1>(r, dloss, zc2(r), loss);
    });
}

int run_bc(const Req& r, const double* dloss) {
    if (r.dims.per) return FPDE_OK;  // a periodic grid has no boundary: the march wrote every node
    return with_op(r.op, [&](auto tag) {
        return launch_bc<typename decltype(tag)::OP>(r, dloss);
    });
}

int prepare_grad_call(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                      const float* const* fields, const float* const* consts, const double* dloss,
                      float* const* grads, void* stream, Req* r) {
    int st = validate_common(op, grid, coeffs, fields, consts, r);
    if (st != FPDE_OK) return st;
    if (!dloss || !grads) return FPDE_ERR_ARG;
    if ((uintptr_t)dloss & 7u) return FPDE_ERR_ALIGN;
    st = check_outputs(*r, grid, fields, consts, grads, r->d.nf, dloss, sizeof(double));
    if (st != FPDE_OK) return st;
    for (int f = 0; f < r->d.nf; ++f) r->P.out[f] = grads[f];
    r->stream = (hipStream_t)stream;
    return FPDE_OK;
}

}  // namespace
}  // namespace fpde

using namespace fpde;

extern "C" int fpde_op_info(int op, int* ndim, int* n_fields, int* n_consts, int* n_residuals) {
    OpDesc d;
    if (!op_desc(op, &d)) return FPDE_ERR_ARG;
    if (ndim) *ndim = d.ndim;
    if (n_fields) *n_fields = d.nf;
    if (n_consts) *n_consts = d.nc;
    if (n_residuals) *n_residuals = d.nr;
    return FPDE_OK;
}

static int fwd_impl(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                                 const float* const* fields, const float* const* consts,
                                 float* const* residual_out, double* loss, void* stream) {
    Req r;
    int st = validate_common(op, grid, coeffs, fields, consts, &r);
    if (st != FPDE_OK) return st;
    if (!loss) return FPDE_ERR_ARG;
    if ((uintptr_t)loss & 7u) return FPDE_ERR_ALIGN;
    const size_t bytes = (size_t)r.N * sizeof(float);
    for (int f = 0; f < r.d.nf; ++f)
        if (overlaps(loss, sizeof(double), fields[f], bytes)) return FPDE_ERR_ARG;
    for (int j = 0; j < r.d.nc; ++j)
        if (overlaps(loss, sizeof(double), consts[j], bytes)) return FPDE_ERR_ARG;
    if (residual_out) {
        st = check_outputs(r, grid, fields, consts, residual_out, r.d.nr, loss, sizeof(double));
        if (st != FPDE_OK) return st;
        for (int b = 0; b < r.d.nr; ++b) r.P.out[b] = residual_out[b];
    }
    r.stream = (hipStream_t)stream;
    return run_fwd(r, residual_out != nullptr, loss);
}

static int bwd_impl(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                                 const float* const* fields, const float* const* consts,
                                 const double* dloss, float* const* grads, void* stream) {
    Req r;
    const int st = prepare_grad_call(op, grid, coeffs, fields, consts, dloss, grads, stream, &r);
    if (st != FPDE_OK) return st;
    return run_bwd(r, dloss);
}

static int bc_impl(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                               const float* const* fields, const float* const* consts,
                               const double* dloss, float* const* grads, void* stream) {
    Req r;
    const int st = prepare_grad_call(op, grid, coeffs, fields, consts, dloss, grads, stream, &r);
    if (st != FPDE_OK) return st;
    return run_bc(r, dloss);
}

static int value_and_grad_impl(int op, const fpde_grid4* grid,
                                            const fpde_coeffs* coeffs, const float* const* fields,
                                            const float* const* consts, const double* dloss,
                                            double* loss, float* const* grads, void* stream) {
    Req r;
    int st = prepare_grad_call(op, grid, coeffs, fields, consts, dloss, grads, stream, &r);
    if (st != FPDE_OK) return st;
    if (!loss) return FPDE_ERR_ARG;
    if ((uintptr_t)loss & 7u) return FPDE_ERR_ALIGN;
    const size_t bytes = (size_t)r.N * sizeof(float);
    if (overlaps(loss, sizeof(double), dloss, sizeof(double))) return FPDE_ERR_ARG;
    for (int f = 0; f < r.d.nf; ++f)
        if (overlaps(loss, sizeof(double), fields[f], bytes) ||
            overlaps(loss, sizeof(double), grads[f], bytes))
            return FPDE_ERR_ARG;
    for (int j = 0; j < r.d.nc; ++j)
        if (overlaps(loss, sizeof(double), consts[j], bytes)) return FPDE_ERR_ARG;
    return run_bwd(r, dloss, loss);
}

static int vjp_impl(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                                 const float* const* fields, const float* const* sens,
                                 int accumulate, float* const* grads, void* stream) {
    Req r;
    int st = validate_common(op, grid, coeffs, fields, nullptr, &r, false);
    if (st != FPDE_OK) return st;
    if (!sens || !grads) return FPDE_ERR_ARG;
    if (accumulate != 0 && accumulate != 1) return FPDE_ERR_ARG;
    const size_t bytes = (size_t)r.N * sizeof(float);
    for (int b = 0; b < r.d.nr; ++b) {
        if (!sens[b]) return FPDE_ERR_ARG;
        if ((uintptr_t)sens[b] & 3u) return FPDE_ERR_ALIGN;
    }
    for (int f = 0; f < r.d.nf; ++f) {
        if (!grads[f]) return FPDE_ERR_ARG;
        if ((uintptr_t)grads[f] & 3u) return FPDE_ERR_ALIGN;
        for (int q = 0; q < r.d.nf; ++q)
            if (overlaps(grads[f], bytes, fields[q], bytes)) return FPDE_ERR_ARG;
        for (int b = 0; b < r.d.nr; ++b)
            if (overlaps(grads[f], bytes, sens[b], bytes)) return FPDE_ERR_ARG;
        for (int q = 0; q < f; ++q)
            if (overlaps(grads[f], bytes, grads[q], bytes)) return FPDE_ERR_ARG;
    }
    for (int b = 0; b < r.d.nr; ++b) r.P.s[b] = sens[b];
    for (int f = 0; f < r.d.nf; ++f) r.P.out[f] = grads[f];
    r.stream = (hipStream_t)stream;
    return run_vjp(r, accumulate == 1);
}

// fpde_grid (three axes) as fpde_grid4; ndim is checked against the op's later
static const fpde_grid4* widen(const fpde_grid* g, fpde_grid4* w) {
    if (!g) return nullptr;
    memset(w, 0, sizeof *w);
    w->ndim = g->ndim > 3 ? -1 : g->ndim;  // (four axes do not fit an fpde_grid)
    w->bc_mode = g->bc_mode;
    for (int a = 0; a < 3; ++a) {
        w->n[a] = g->n[a];
        w->h[a] = g->h[a];
    }
    return w;
}

extern "C" int fpde_residual_fwd(int op, const fpde_grid* grid, const fpde_coeffs* coeffs,
                                 const float* const* fields, const float* const* consts,
                                 float* const* residual_out, double* loss, void* stream) {
    fpde_grid4 w;
    return fwd_impl(op, widen(grid, &w), coeffs, fields, consts, residual_out, loss, stream);
}

extern "C" int fpde_residual_bwd(int op, const fpde_grid* grid, const fpde_coeffs* coeffs,
                                 const float* const* fields, const float* const* consts,
                                 const double* dloss, float* const* grads, void* stream) {
    fpde_grid4 w;
    return bwd_impl(op, widen(grid, &w), coeffs, fields, consts, dloss, grads, stream);
}

extern "C" int fpde_bc_correct(int op, const fpde_grid* grid, const fpde_coeffs* coeffs,
                               const float* const* fields, const float* const* consts,
                               const double* dloss, float* const* grads, void* stream) {
    fpde_grid4 w;
    return bc_impl(op, widen(grid, &w), coeffs, fields, consts, dloss, grads, stream);
}

extern "C" int fpde_residual_value_and_grad(int op, const fpde_grid* grid,
                                            const fpde_coeffs* coeffs, const float* const* fields,
                                            const float* const* consts, const double* dloss,
                                            double* loss, float* const* grads, void* stream) {
    fpde_grid4 w;
    return value_and_grad_impl(op, widen(grid, &w), coeffs, fields, consts, dloss, loss, grads,
                               stream);
}

extern "C" int fpde_residual_vjp(int op, const fpde_grid* grid, const fpde_coeffs* coeffs,
                                 const float* const* fields, const float* const* sens,
                                 int accumulate, float* const* grads, void* stream) {
    fpde_grid4 w;
    return vjp_impl(op, widen(grid, &w), coeffs, fields, sens, accumulate, grads, stream);
}

extern "C" int fpde_residual_fwd4(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                                  const float* const* fields, const float* const* consts,
                                  float* const* residual_out, double* loss, void* stream) {
    return fwd_impl(op, grid, coeffs, fields, consts, residual_out, loss, stream);
}

extern "C" int fpde_residual_bwd4(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                                  const float* const* fields, const float* const* consts,
                                  const double* dloss, float* const* grads, void* stream) {
    return bwd_impl(op, grid, coeffs, fields, consts, dloss, grads, stream);
}

extern "C" int fpde_bc_correct4(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                                const float* const* fields, const float* const* consts,
                                const double* dloss, float* const* grads, void* stream) {
    return bc_impl(op, grid, coeffs, fields, consts, dloss, grads, stream);
}

extern "C" int fpde_residual_value_and_grad4(int op, const fpde_grid4* grid,
                                             const fpde_coeffs* coeffs, const float* const* fields,
                                             const float* const* consts, const double* dloss,
                                             double* loss, float* const* grads, void* stream) {
    return value_and_grad_impl(op, grid, coeffs, fields, consts, dloss, loss, grads, stream);
}

extern "C" int fpde_residual_vjp4(int op, const fpde_grid4* grid, const fpde_coeffs* coeffs,
                                  const float* const* fields, const float* const* sens,
                                  int accumulate, float* const* grads, void* stream) {
    return vjp_impl(op, grid, coeffs, fields, sens, accumulate, grads, stream);
}

extern "C" const char* fpde_status_string(int status) {
    switch (status) {
    case FPDE_OK: return "FPDE_OK";
    case FPDE_ERR_ARG: return "FPDE_ERR_ARG: null pointer, unknown op or overlapping output";
    case FPDE_ERR_SHAPE: return "FPDE_ERR_SHAPE: wrong rank, n_a < 3 or size too large";
    case FPDE_ERR_SPACING: return "FPDE_ERR_SPACING: grid spacing not positive and finite";
    case FPDE_ERR_COEFF: return "FPDE_ERR_COEFF: non-finite coefficient or dt <= 0";
    case FPDE_ERR_ALIGN: return "FPDE_ERR_ALIGN: misaligned device pointer";
    case FPDE_ERR_HIP: return "FPDE_ERR_HIP: HIP runtime error while queueing work";
    case FPDE_ERR_UNSUPPORTED: return "FPDE_ERR_UNSUPPORTED: request not implemented by this library version";
    default: return "unknown fpde status";
    }
}

extern "C" const char* fpde_version(void) { return "fpde 0.2 gfx950"; }
