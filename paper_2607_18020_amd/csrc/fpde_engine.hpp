// fpde_engine.hpp -- gfx950 kernels of the FD residual operator.
//
// Grid geometry: array axis 0 is the march axis ("z"); the last axis is x
// (fastest, coalesced); for 3-D grids axis 1 is y.  A workgroup owns a TX x TY
// column tile of the (y, x) plane (TY = 1 for 2-D grids, where the "plane" is a
// row segment) and marches a chunk of ZC planes along axis 0:
//   * the in-plane neighbours come from a halo tile of the current plane in LDS;
//   * the axis-0 neighbours come from a per-thread register queue (planes
//     z-1, z, z+1 of the thread's own column);
// so every input element is read from HBM once per chunk plus the halo.
//
// Forward: one residual per interior node, sum of squares accumulated in a
// per-thread float64 register, reduced with DPP across the wavefront and through
// LDS across waves, then ONE float64 atomic add per workgroup (Sec. 2.1 fused
// stencil, with the loss fused as well).
//
// Backward: gather form of the transposed stencil (Sec. 2.2).  The residuals
// that the gather needs are recomputed, never read: at step z the workgroup
// evaluates R(z+1) on the tile plus a one-node ring into an LDS tile, so the
// gather for plane z reads R(z) (in-plane star, LDS), R(z+1) (LDS) and R(z-1)
// (register queue).  Field planes live in a 4-slot LDS ring (tile plus a
// two-node halo); the next plane is prefetched into registers one step ahead.
// Every node of the visited planes 1..nz-2 is written exactly once (boundary
// columns included: there the residuals off the residual set are zero, which
// the LDS tiles already hold); no atomics.
//
// Boundary correction: a 1-D launch over the two end planes of axis 0, the
// boundary nodes the march does not visit (Sec. 2.3).
//
// Workgroup-to-tile order is XCD-aware: consecutive workgroup ids are spread
// round-robin over the 8 XCDs, so the id is remapped such that each XCD gets a
// contiguous run of tiles (neighbouring tiles, which share halos, then share
// that XCD's L2).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "fpde_ops.hpp"

namespace fpde {

struct Ptrs {
    const float* f[4];
    const float* c[3];
    float* out[4];
};

struct Dims {
    int nz, ny, nx;         // ny = 1 for 2-D grids
    int tiles_x, tiles_y;   // tiles_y = 1 for 2-D grids
    int zc, nblocks;        // planes per chunk, workgroups launched
};

__device__ __forceinline__ int remap_xcd(int b, int nb) {
    const int nb8 = nb & ~7;
    if (b >= nb8) return b;
    return (b & 7) * (nb8 >> 3) + (b >> 3);
}

// ---------------------------------------------------------------------------
// Wavefront and workgroup sums.

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_f64(double v) {
    const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), CTRL, ROW_MASK, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), CTRL, ROW_MASK, 0xF, false);
    return __hiloint2double(hi, lo);
}

// Sum over the 64 lanes; the total is valid in lane 63.
__device__ __forceinline__ double wave_sum_f64(double v) {
    v += dpp_f64<0xB1, 0xF>(v);   // quad_perm [1,0,3,2]
    v += dpp_f64<0x4E, 0xF>(v);   // quad_perm [2,3,0,1]
    v += dpp_f64<0x141, 0xF>(v);  // row_half_mirror: 8-lane sums
    v += dpp_f64<0x140, 0xF>(v);  // row_mirror: 16-lane row sums
    v += dpp_f64<0x142, 0xA>(v);  // row_bcast:15 -> rows 1, 3
    v += dpp_f64<0x143, 0xC>(v);  // row_bcast:31 -> rows 2, 3
    return v;
}

template <int NT>
__device__ __forceinline__ void block_atomic_sum(double v, double* dst) {
    __shared__ double part[NT / 64];
    v = wave_sum_f64(v);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (lane == 63) part[w] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        double s = 0.0;
#pragma unroll
        for (int i = 0; i < NT / 64; ++i) s += part[i];
        atomicAdd(dst, s);
    }
}

__global__ void fill_f64_kernel(double* p, double v) { *p = v; }

// Tile-ring enumeration: ring index r -> (ly, lx) on a (TY + 2*HYR) x (TX + 2)
// tile with a one-node ring (HYR = 1 for 3-D, 0 for 2-D).
template <int TX, int TY, int DIM>
struct Ring {
    static constexpr int COUNT = (DIM == 3) ? 2 * (TX + 2) + 2 * TY : 2;
    __device__ static void pos(int r, int& ly, int& lx) {
        if (DIM == 2) {
            ly = 0;
            lx = r ? TX + 1 : 0;
            return;
        }
        if (r < TX + 2) { ly = 0; lx = r; return; }
        r -= TX + 2;
        if (r < TX + 2) { ly = TY + 1; lx = r; return; }
        r -= TX + 2;
        if (r < TY) { ly = 1 + r; lx = 0; return; }
        r -= TY;
        ly = 1 + r;
        lx = TX + 1;
    }
};

struct TileCoord {
    int gx0, gy0, z0, z1;
};

template <int TX, int TY>
__device__ __forceinline__ TileCoord tile_coord(const Dims& D) {
    int lb = remap_xcd(blockIdx.x, D.nblocks);
    const int bx = lb % D.tiles_x;
    lb /= D.tiles_x;
    const int by = lb % D.tiles_y;
    const int ch = lb / D.tiles_y;
    TileCoord tc;
    tc.gx0 = bx * TX;
    tc.gy0 = by * TY;
    tc.z0 = 1 + ch * D.zc;
    tc.z1 = min(tc.z0 + D.zc, D.nz - 1);
    return tc;
}

// ---------------------------------------------------------------------------
// Global-memory access in the marching kernels: one raw buffer resource per
// plane (base = the plane's first byte, built in SGPRs) and a 32-bit per-thread
// byte offset, so a load is a single buffer_load_dword with no per-lane
// address arithmetic.  num_records is the plane size: an offset past it reads 0.
// Positions outside the array use offset 0 and a select to zero.

template <int V>
using IC = std::integral_constant<int, V>;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t plane_rsrc(const float* p, int z,
                                                             uint32_t pbytes) {
    return __builtin_amdgcn_make_buffer_rsrc(
        (void*)(reinterpret_cast<const char*>(p) + (uint64_t)z * pbytes), (short)0, (int)pbytes,
        0x00020000);
}

__device__ __forceinline__ float bld(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
}

__device__ __forceinline__ void bst(__amdgpu_buffer_rsrc_t r, uint32_t off, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)off, 0, 0);
}

// ---------------------------------------------------------------------------
// Forward: residuals of one chunk of planes + fused sum of squares.

#ifndef FPDE_FWD_MINW
#define FPDE_FWD_MINW 1
#endif
#ifndef FPDE_BWD_MINW
#define FPDE_BWD_MINW 1
#endif

template <class OP, int TX, int TY, bool STORE_R>
__global__ __launch_bounds__(TX* TY, FPDE_FWD_MINW) void fwd_kernel(Ptrs P, Dims D, KCoef K, double inv_M,
                                                     double* loss) {
    constexpr int DIM = OP::DIM, NF = OP::NF, NC = OP::NC, NR = OP::NR, NT = TX * TY;
    constexpr int NC1 = NC > 0 ? NC : 1;
    constexpr int HY = (DIM == 3) ? 1 : 0;
    constexpr int LY = TY + 2 * HY, LX = TX + 2;
    static_assert(DIM == 3 || TY == 1, "2-D grids use one-row tiles");
    static_assert(Ring<TX, TY, DIM>::COUNT <= NT, "ring larger than the workgroup");
    __shared__ float sF[2][NF][LY][LX];

    const int t = threadIdx.x, tx = t % TX, ty = t / TX;
    const TileCoord tc = tile_coord<TX, TY>(D);
    const int z0 = tc.z0, z1 = tc.z1;
    const int gx = tc.gx0 + tx, gy = (DIM == 3) ? tc.gy0 + ty : 0;
    const uint32_t pbytes = (uint32_t)D.ny * (uint32_t)D.nx * 4u;
    const bool inarr = gx < D.nx && gy < D.ny;
    const bool interior = gx >= 1 && gx <= D.nx - 2 && (DIM == 2 || (gy >= 1 && gy <= D.ny - 2));
    const uint32_t cb = inarr ? (uint32_t)(gy * D.nx + gx) * 4u : 0u;

    // fixed halo-ring slot of this thread (if any)
    const bool has_ring = t < Ring<TX, TY, DIM>::COUNT;
    int rly = 0, rlx = 0;
    if (has_ring) Ring<TX, TY, DIM>::pos(t, rly, rlx);
    const int rgy = (DIM == 3) ? tc.gy0 - 1 + rly : 0, rgx = tc.gx0 - 1 + rlx;
    const bool ring_in = has_ring && rgx >= 0 && rgx < D.nx && rgy >= 0 && rgy < D.ny;
    const uint32_t rb = ring_in ? (uint32_t)(rgy * D.nx + rgx) * 4u : 0u;

    // Register queue of the own column: planes z-1, z, z+1 and the prefetched
    // z+2 live in q[(j)&3], q[(j+1)&3], q[(j+2)&3], q[(j+3)&3] at step j = z - z0;
    // the ring values and consts of plane z (and prefetched z+1) alternate.
    float q[4][NF], rv[2][NF], cv[2][NC1];
#pragma unroll
    for (int f = 0; f < NF; ++f) {
        const float a = bld(plane_rsrc(P.f[f], z0 - 1, pbytes), cb);
        const float b = bld(plane_rsrc(P.f[f], z0, pbytes), cb);
        const float c = bld(plane_rsrc(P.f[f], z0 + 1, pbytes), cb);
        const float r = bld(plane_rsrc(P.f[f], z0, pbytes), rb);
        q[0][f] = inarr ? a : 0.f;
        q[1][f] = inarr ? b : 0.f;
        q[2][f] = inarr ? c : 0.f;
        q[3][f] = 0.f;
        rv[0][f] = ring_in ? r : 0.f;
        rv[1][f] = 0.f;
    }
#pragma unroll
    for (int j = 0; j < NC1; ++j) {
        cv[0][j] = NC ? bld(plane_rsrc(P.c[j], z0, pbytes), cb) : 0.f;
        cv[1][j] = 0.f;
    }

    double acc = 0.0;
    auto step = [&](auto jc, int z) __attribute__((always_inline)) {
        constexpr int J = decltype(jc)::value;
        constexpr int QM = J & 3, QZ = (J + 1) & 3, QP = (J + 2) & 3, QN = (J + 3) & 3;
        constexpr int CUR = J & 1, NXT = (J + 1) & 1, BUF = J & 1;
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            sF[BUF][f][ty + HY][tx + 1] = q[QZ][f];
            if (has_ring) sF[BUF][f][rly][rlx] = rv[CUR][f];
        }
        if (z + 1 < z1) {  // prefetch plane z+2 of the own column, ring and consts of z+1
#pragma unroll
            for (int f = 0; f < NF; ++f) {
                // branch-free: threads without a ring node load a valid address too
                const float v = bld(plane_rsrc(P.f[f], z + 2, pbytes), cb);
                const float w = bld(plane_rsrc(P.f[f], z + 1, pbytes), rb);
                q[QN][f] = inarr ? v : 0.f;
                rv[NXT][f] = ring_in ? w : 0.f;
            }
#pragma unroll
            for (int j = 0; j < NC; ++j) cv[NXT][j] = bld(plane_rsrc(P.c[j], z + 1, pbytes), cb);
        }
        __syncthreads();
        Star s[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            s[f].c = q[QZ][f];
            s[f].m[0] = q[QM][f];
            s[f].p[0] = q[QP][f];
            s[f].m[DIM - 1] = sF[BUF][f][ty + HY][tx];
            s[f].p[DIM - 1] = sF[BUF][f][ty + HY][tx + 2];
            if (DIM == 3) {
                s[f].m[1] = sF[BUF][f][ty][tx + 1];
                s[f].p[1] = sF[BUF][f][ty + 2][tx + 1];
            }
        }
        float R[NR];
        OP::residual(s, cv[CUR], K, R);
        float ss = 0.f;
#pragma unroll
        for (int b = 0; b < NR; ++b) ss = fmaf(R[b], R[b], ss);
        acc += (double)(interior ? ss : 0.f);
        if (STORE_R && interior) {
#pragma unroll
            for (int b = 0; b < NR; ++b) bst(plane_rsrc(P.out[b], z, pbytes), cb, R[b]);
        }
    };

    int z = z0;
    for (; z + 4 <= z1; z += 4) {  // four steps bring the queue and the buffers back
        step(IC<0>{}, z);
        step(IC<1>{}, z + 1);
        step(IC<2>{}, z + 2);
        step(IC<3>{}, z + 3);
    }
    if (z < z1) step(IC<0>{}, z);
    if (z + 1 < z1) step(IC<1>{}, z + 1);
    if (z + 2 < z1) step(IC<2>{}, z + 2);
    block_atomic_sum<NT>(acc * inv_M, loss);
}

// ---------------------------------------------------------------------------
// Backward: gather-form transposed stencil with residual recompute.
//
// Per step z: plane z+3 is queued from memory straight into the LDS slot of
// plane z-1; R(z+1) is evaluated on the tile and its one-node ring into an LDS
// tile; the gather at plane z reads the in-plane neighbours of R(z) from LDS and
// R(z-1), R(z), R(z+1) of its own column from a register queue; one barrier.

template <class OP, int TX, int TY>
struct BwdGeo {
    static constexpr int DIM = OP::DIM, NT = TX * TY;
    static constexpr int HY = (DIM == 3) ? 2 : 0;   // field-slot halo (y)
    static constexpr int FLY = TY + 2 * HY, FLX = TX + 4;
    static constexpr int RHY = (DIM == 3) ? 1 : 0;  // R-tile halo (y)
    static constexpr int RLY = TY + 2 * RHY, RLX = TX + 2;
    static constexpr int FSZ = FLY * FLX;
    static constexpr int KP = (FSZ + NT - 1) / NT;  // prefetch elements per thread
};

template <class OP, int TX, int TY>
__global__ __launch_bounds__(TX* TY, FPDE_BWD_MINW) void bwd_kernel(Ptrs P, Dims D, KCoef K,
                                                     const double* dloss, double two_over_M) {
    using G = BwdGeo<OP, TX, TY>;
    constexpr int DIM = OP::DIM, NF = OP::NF, NC = OP::NC, NR = OP::NR, NT = G::NT;
    constexpr int NC1 = NC > 0 ? NC : 1;
    constexpr int HY = G::HY, FLY = G::FLY, FLX = G::FLX, RHY = G::RHY, RLY = G::RLY,
                  RLX = G::RLX, FSZ = G::FSZ, KP = G::KP;
    static_assert(DIM == 3 || TY == 1, "2-D grids use one-row tiles");
    static_assert(Ring<TX, TY, DIM>::COUNT <= NT, "ring larger than the workgroup");
    // field planes in a 4-slot ring: plane pz lives in slot (pz - z0 + 1) & 3
    __shared__ float sF[4][NF][FLY][FLX];
    // residual tiles: R(zr) lives in buffer (zr - z0) & 1
    __shared__ float sR[2][NR][RLY][RLX];

    const int t = threadIdx.x, tx = t % TX, ty = t / TX;
    const TileCoord tc = tile_coord<TX, TY>(D);
    const int z0 = tc.z0, z1 = tc.z1;
    const int gx = tc.gx0 + tx, gy = (DIM == 3) ? tc.gy0 + ty : 0;
    const uint32_t pbytes = (uint32_t)D.ny * (uint32_t)D.nx * 4u;
    const bool inarr = gx < D.nx && gy < D.ny;
    const uint32_t cb = inarr ? (uint32_t)(gy * D.nx + gx) * 4u : 0u;
    const float scale = (float)(two_over_M * (*dloss));

    // This thread's share of a field plane (tile + 2-node halo): element
    // i = t + k*NT of the slot, in slot order, so that the 64 lanes of a wave
    // fill 64 consecutive LDS words.  Planes go straight from memory into LDS
    // (buffer_load_dword ... lds); a position outside the array gets an offset
    // past the descriptor's range, which the buffer unit reads as 0.
    constexpr uint32_t kOff = 0x80000000u;
    uint32_t poff[KP];
#pragma unroll
    for (int k = 0; k < KP; ++k) {
        const int i = t + k * NT;
        const int ly = i / FLX, lx = i % FLX;
        const int py = (DIM == 3) ? tc.gy0 - HY + ly : 0, px = tc.gx0 - 2 + lx;
        const bool ok = i < FSZ && px >= 0 && px < D.nx && py >= 0 && py < D.ny;
        poff[k] = ok ? (uint32_t)(py * D.nx + px) * 4u : kOff;
    }
    const int wbase = t & ~63;  // first element of this wave in each round
    // queue plane pz (uniform) into LDS slot `slot`; planes outside the grid read as 0
    auto load_plane = [&](int pz, int slot) __attribute__((always_inline)) {
        const bool zok = pz >= 0 && pz < D.nz;
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
                (void*)(reinterpret_cast<const char*>(P.f[f]) +
                        (uint64_t)(zok ? pz : 0) * pbytes),
                (short)0, zok ? (int)pbytes : 0, 0x00020000);
#pragma unroll
            for (int k = 0; k < KP; ++k) {
                if (KP * NT == FSZ || t + k * NT < FSZ) {
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(
                        r, (__attribute__((address_space(3))) void*)(&sF[slot][f][0][0] + wbase + k * NT),
                        4, (int)poff[k], 0, 0, 0);
                }
            }
        }
    };

    // residual positions of this thread on the R tile: its own column and, for
    // the first threads, one node of the ring; their in-plane part of the
    // residual-set test and their const offsets are fixed for the whole march
    const int oly = ty + RHY, olx = tx + 1;
    const bool own_om = gx >= 1 && gx <= D.nx - 2 && (DIM == 2 || (gy >= 1 && gy <= D.ny - 2));
    const bool has_ring = t < Ring<TX, TY, DIM>::COUNT;
    int rly = 0, rlx = 0;
    if (has_ring) Ring<TX, TY, DIM>::pos(t, rly, rlx);
    const int rgy = (DIM == 3) ? tc.gy0 - RHY + rly : 0, rgx = tc.gx0 - 1 + rlx;
    const bool ring_om = has_ring && rgx >= 1 && rgx <= D.nx - 2 &&
                         (DIM == 2 || (rgy >= 1 && rgy <= D.ny - 2));
    const uint32_t rcb = ring_om ? (uint32_t)(rgy * D.nx + rgx) * 4u : 0u;

    // R(zr) at R-tile position (ly, lx) from field slots sm (zr-1), sc (zr), sp (zr+1);
    // written to sR[dst] and returned in R (zero off the residual set)
    auto r_at = [&](int zr, int sm, int sc, int sp, int dst, int ly, int lx, bool om_xy,
                    const float* cc, float* R) __attribute__((always_inline)) {
        const int fy = ly + (HY - RHY), fx = lx + 1;
        Star s[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            s[f].c = sF[sc][f][fy][fx];
            s[f].m[0] = sF[sm][f][fy][fx];
            s[f].p[0] = sF[sp][f][fy][fx];
            s[f].m[DIM - 1] = sF[sc][f][fy][fx - 1];
            s[f].p[DIM - 1] = sF[sc][f][fy][fx + 1];
            if (DIM == 3) {
                s[f].m[1] = sF[sc][f][fy - 1][fx];
                s[f].p[1] = sF[sc][f][fy + 1][fx];
            }
        }
        OP::residual(s, cc, K, R);
        const bool om = om_xy && zr >= 1 && zr <= D.nz - 2;
#pragma unroll
        for (int b = 0; b < NR; ++b) {
            R[b] = om ? R[b] : 0.f;
            sR[dst][b][ly][lx] = R[b];
        }
    };
    // consts of the R-tile positions, for the plane whose residuals come next
    // (loaded one step ahead so that their latency hides behind a step)
    float cown[NC1], cring[NC1];
    auto load_consts = [&](int zr) __attribute__((always_inline)) {  // zr uniform, in range
#pragma unroll
        for (int j = 0; j < NC; ++j) {
            const __amdgpu_buffer_rsrc_t r = plane_rsrc(P.c[j], zr, pbytes);
            cown[j] = bld(r, cb);
            cring[j] = bld(r, rcb);
        }
    };
    // R(zr) on the whole R tile; the own column's values are returned in Rown
    auto r_tile = [&](int zr, int sm, int sc, int sp, int dst, float* Rown)
                      __attribute__((always_inline)) {
        r_at(zr, sm, sc, sp, dst, oly, olx, own_om, cown, Rown);
        if (has_ring) {
            float Rr[NR];
            r_at(zr, sm, sc, sp, dst, rly, rlx, ring_om, cring, Rr);
        }
    };

    // ---- prologue: planes z0-1 .. z0+2 in slots 0..3; R(z0) tile; the own
    // column's R(z0-1), R(z0) and fields of plane z0-1 in registers
    for (int j = 0; j < 4; ++j) load_plane(z0 - 1 + j, j);
    float fzm2[NF];
#pragma unroll
    for (int f = 0; f < NF; ++f) {
        const float v = bld(plane_rsrc(P.f[f], z0 >= 2 ? z0 - 2 : 0, pbytes), cb);
        fzm2[f] = (inarr && z0 >= 2) ? v : 0.f;
    }
    load_consts(z0);
    __syncthreads();
    float fzm[NF], rzm[NR], rzc[NR], rzp[NR];
    r_tile(z0, 0, 1, 2, 0, rzc);
    {
        const int fy = ty + HY, fx = tx + 2;
        Star s[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            s[f].c = sF[0][f][fy][fx];
            s[f].m[0] = fzm2[f];
            s[f].p[0] = sF[1][f][fy][fx];
            s[f].m[DIM - 1] = sF[0][f][fy][fx - 1];
            s[f].p[DIM - 1] = sF[0][f][fy][fx + 1];
            if (DIM == 3) {
                s[f].m[1] = sF[0][f][fy - 1][fx];
                s[f].p[1] = sF[0][f][fy + 1][fx];
            }
            fzm[f] = s[f].c;
        }
        float cc[NC1];
#pragma unroll
        for (int j = 0; j < NC; ++j) cc[j] = bld(plane_rsrc(P.c[j], z0 - 1, pbytes), cb);
        OP::residual(s, cc, K, rzm);
        const bool om = own_om && z0 - 1 >= 1;
#pragma unroll
        for (int b = 0; b < NR; ++b) rzm[b] = om ? rzm[b] : 0.f;
    }
    load_consts(z0 + 1);
    __syncthreads();

    // ---- march.  Step z: issue the loads of plane z+3; R(z+1) on the R tile; the
    // gather at plane z; plane z+3 into the slot of plane z-1; one barrier.  Every
    // LDS buffer a step writes was last read before the previous step's barrier.
    auto step = [&](auto jc, int z) __attribute__((always_inline)) {
        constexpr int J = decltype(jc)::value;  // (z - z0) & 3
        // field slots of planes z-1 (reused for z+3), z, z+1, z+2; R tiles of R(z), R(z+1)
        constexpr int SM = J & 3, SC = (J + 1) & 3, SP = (J + 2) & 3, SQ = (J + 3) & 3;
        constexpr int RC = J & 1, RP = (J + 1) & 1;
        const bool more = z + 1 < z1;
        if (more) load_plane(z + 3, SM);  // the slot of plane z-1, unread in this step
        r_tile(z + 1, SC, SP, SQ, RP, rzp);
        if (more) load_consts(z + 2);
        const int fy = ty + HY, fx = tx + 2, ry = ty + RHY, rx = tx + 1;
        Star fs[NF], rs[NR];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            fs[f].c = sF[SC][f][fy][fx];
            fs[f].m[0] = fzm[f];
            fs[f].p[0] = sF[SP][f][fy][fx];
            fs[f].m[DIM - 1] = sF[SC][f][fy][fx - 1];
            fs[f].p[DIM - 1] = sF[SC][f][fy][fx + 1];
            if (DIM == 3) {
                fs[f].m[1] = sF[SC][f][fy - 1][fx];
                fs[f].p[1] = sF[SC][f][fy + 1][fx];
            }
        }
#pragma unroll
        for (int b = 0; b < NR; ++b) {
            rs[b].c = rzc[b];
            rs[b].m[0] = rzm[b];
            rs[b].p[0] = rzp[b];
            rs[b].m[DIM - 1] = sR[RC][b][ry][rx - 1];
            rs[b].p[DIM - 1] = sR[RC][b][ry][rx + 1];
            if (DIM == 3) {
                rs[b].m[1] = sR[RC][b][ry - 1][rx];
                rs[b].p[1] = sR[RC][b][ry + 1][rx];
            }
        }
        float g[NF];
        OP::gather(fs, rs, K, g);
        if (inarr) {
#pragma unroll
            for (int f = 0; f < NF; ++f) bst(plane_rsrc(P.out[f], z, pbytes), cb, scale * g[f]);
        }
#pragma unroll
        for (int f = 0; f < NF; ++f) fzm[f] = fs[f].c;
#pragma unroll
        for (int b = 0; b < NR; ++b) {
            rzm[b] = rzc[b];
            rzc[b] = rzp[b];
        }
        __syncthreads();  // (waits for the plane loads into LDS as well)
    };

    int z = z0;
    for (; z + 4 <= z1; z += 4) {  // slot and buffer indices are constants in each copy
        step(IC<0>{}, z);
        step(IC<1>{}, z + 1);
        step(IC<2>{}, z + 2);
        step(IC<3>{}, z + 3);
    }
    if (z < z1) step(IC<0>{}, z);
    if (z + 1 < z1) step(IC<1>{}, z + 1);
    if (z + 2 < z1) step(IC<2>{}, z + 2);
}

// ---------------------------------------------------------------------------
// Boundary-gradient correction: the two end planes of axis 0 (i0 = 0 and
// i0 = nz - 1), which the march never visits.  A node whose only boundary
// coordinate is i0 receives the terms of its inward neighbour's residuals; a
// node with another boundary coordinate as well (an edge or corner) touches no
// residual node and gets 0.  (Boundary nodes of the other axes lie on visited
// planes: the march evaluates the same transposed stencil there with the
// residuals taken as zero off the residual set, which is exactly their
// correction term.)

template <class OP>
__device__ __forceinline__ void bc_node0(const Ptrs& P, const KCoef& K, const long long* str,
                                         long long node, bool low, float* g) {
    constexpr int DIM = OP::DIM, NF = OP::NF, NC = OP::NC;
    const float t = low ? -1.f : 1.f;  // node = m + t e_0
    const long long m = low ? node + str[0] : node - str[0];
    Star s[NF];
#pragma unroll
    for (int f = 0; f < NF; ++f) {
        const float* q = P.f[f];
        s[f].c = q[m];
#pragma unroll
        for (int a = 0; a < DIM; ++a) {
            s[f].m[a] = q[m - str[a]];
            s[f].p[a] = q[m + str[a]];
        }
    }
    float cc[NC > 0 ? NC : 1];
#pragma unroll
    for (int j = 0; j < NC; ++j) cc[j] = P.c[j][m];
    OP::template bc_term<0>(s, cc, K, t, g);
}

template <class OP>
__global__ __launch_bounds__(256) void bc_kernel(Ptrs P, Dims D, KCoef K, const double* dloss,
                                                 double two_over_M) {
    constexpr int DIM = OP::DIM, NF = OP::NF;
    const float scale = (float)(two_over_M * (*dloss));
    const long long nz = D.nz, ny = D.ny, nx = D.nx;
    const long long plane = ny * nx;
    const long long total = 2 * plane;
    const long long str[3] = {plane, (DIM == 3) ? nx : 1, 1};
    for (long long idx = blockIdx.x * 256LL + threadIdx.x; idx < total;
         idx += (long long)gridDim.x * 256LL) {
        const bool low = idx < plane;
        const long long r = low ? idx : idx - plane;
        const long long node = (low ? 0 : (nz - 1) * plane) + r;
        const long long i1 = (DIM == 3) ? r / nx : r;
        const long long i2 = r % nx;
        const bool edge = (DIM == 3) ? (i1 == 0 || i1 == ny - 1 || i2 == 0 || i2 == nx - 1)
                                     : (i1 == 0 || i1 == nx - 1);
        float g[NF];
        if (!edge) {
            bc_node0<OP>(P, K, str, node, low, g);
#pragma unroll
            for (int f = 0; f < NF; ++f) g[f] *= scale;
        } else {
#pragma unroll
            for (int f = 0; f < NF; ++f) g[f] = 0.f;
        }
#pragma unroll
        for (int f = 0; f < NF; ++f) P.out[f][node] = g[f];
    }
}

}  // namespace fpde
