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
// Forward: residuals of one chunk of planes + fused sum of squares.

template <class OP, int TX, int TY, bool STORE_R>
__global__ __launch_bounds__(TX* TY) void fwd_kernel(Ptrs P, Dims D, KCoef K, double inv_M,
                                                     double* loss) {
    constexpr int DIM = OP::DIM, NF = OP::NF, NC = OP::NC, NR = OP::NR, NT = TX * TY;
    constexpr int HY = (DIM == 3) ? 1 : 0;
    constexpr int LY = TY + 2 * HY, LX = TX + 2;
    static_assert(DIM == 3 || TY == 1, "2-D grids use one-row tiles");
    static_assert(Ring<TX, TY, DIM>::COUNT <= NT, "ring larger than the workgroup");
    __shared__ float sF[2][NF][LY][LX];

    const int t = threadIdx.x, tx = t % TX, ty = t / TX;
    const TileCoord tc = tile_coord<TX, TY>(D);
    const int gx = tc.gx0 + tx, gy = (DIM == 3) ? tc.gy0 + ty : 0;
    const long long plane = (long long)D.ny * D.nx;
    const bool inarr = gx < D.nx && gy < D.ny;
    const bool interior = gx >= 1 && gx <= D.nx - 2 && (DIM == 2 || (gy >= 1 && gy <= D.ny - 2));
    const int col = gy * D.nx + gx;

    // fixed halo-ring slot of this thread (if any)
    const bool has_ring = t < Ring<TX, TY, DIM>::COUNT;
    int rly = 0, rlx = 0;
    if (has_ring) Ring<TX, TY, DIM>::pos(t, rly, rlx);
    const int rgy = (DIM == 3) ? tc.gy0 - 1 + rly : 0, rgx = tc.gx0 - 1 + rlx;
    const bool ring_in = has_ring && rgx >= 0 && rgx < D.nx && rgy >= 0 && rgy < D.ny;
    const int rcol = ring_in ? rgy * D.nx + rgx : 0;

    // register queue of the own column (planes z-1, z, z+1), the ring value of the
    // current plane, the consts of the current plane, and their prefetched successors
    float q[NF][3], qn[NF], rc[NF], rn[NF];
    float cc[NC > 0 ? NC : 1], cn[NC > 0 ? NC : 1];
#pragma unroll
    for (int f = 0; f < NF; ++f) {
        q[f][0] = inarr ? P.f[f][(long long)(tc.z0 - 1) * plane + col] : 0.f;
        q[f][1] = inarr ? P.f[f][(long long)tc.z0 * plane + col] : 0.f;
        q[f][2] = inarr ? P.f[f][(long long)(tc.z0 + 1) * plane + col] : 0.f;
        rc[f] = ring_in ? P.f[f][(long long)tc.z0 * plane + rcol] : 0.f;
        qn[f] = 0.f;
        rn[f] = 0.f;
    }
#pragma unroll
    for (int j = 0; j < NC; ++j) {
        cc[j] = interior ? P.c[j][(long long)tc.z0 * plane + col] : 0.f;
        cn[j] = 0.f;
    }

    double acc = 0.0;
    int buf = 0;
    for (int z = tc.z0; z < tc.z1; ++z) {
        const long long zo = (long long)z * plane;
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            sF[buf][f][ty + HY][tx + 1] = q[f][1];
            if (has_ring) sF[buf][f][rly][rlx] = rc[f];
        }
        if (z + 1 < tc.z1) {  // prefetch plane z+1's ring and consts, plane z+2's column
#pragma unroll
            for (int f = 0; f < NF; ++f) {
                qn[f] = inarr ? P.f[f][zo + 2 * plane + col] : 0.f;
                rn[f] = ring_in ? P.f[f][zo + plane + rcol] : 0.f;
            }
#pragma unroll
            for (int j = 0; j < NC; ++j) cn[j] = interior ? P.c[j][zo + plane + col] : 0.f;
        }
        __syncthreads();
        if (interior) {
            Star s[NF];
#pragma unroll
            for (int f = 0; f < NF; ++f) {
                s[f].c = q[f][1];
                s[f].m[0] = q[f][0];
                s[f].p[0] = q[f][2];
                s[f].m[DIM - 1] = sF[buf][f][ty + HY][tx];
                s[f].p[DIM - 1] = sF[buf][f][ty + HY][tx + 2];
                if (DIM == 3) {
                    s[f].m[1] = sF[buf][f][ty][tx + 1];
                    s[f].p[1] = sF[buf][f][ty + 2][tx + 1];
                }
            }
            float R[NR];
            OP::residual(s, cc, K, R);
            float ss = 0.f;
#pragma unroll
            for (int b = 0; b < NR; ++b) {
                ss += R[b] * R[b];
                if (STORE_R) P.out[b][zo + col] = R[b];
            }
            acc += (double)ss;
        }
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            q[f][0] = q[f][1];
            q[f][1] = q[f][2];
            q[f][2] = qn[f];
            rc[f] = rn[f];
        }
#pragma unroll
        for (int j = 0; j < NC; ++j) cc[j] = cn[j];
        buf ^= 1;
    }
    block_atomic_sum<NT>(acc * inv_M, loss);
}

// ---------------------------------------------------------------------------
// Backward: gather-form transposed stencil with residual recompute.

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
__global__ __launch_bounds__(TX* TY) void bwd_kernel(Ptrs P, Dims D, KCoef K,
                                                     const double* dloss, double two_over_M) {
    using G = BwdGeo<OP, TX, TY>;
    constexpr int DIM = OP::DIM, NF = OP::NF, NC = OP::NC, NR = OP::NR, NT = G::NT;
    constexpr int HY = G::HY, FLY = G::FLY, FLX = G::FLX, RHY = G::RHY, RLY = G::RLY,
                  RLX = G::RLX, FSZ = G::FSZ, KP = G::KP;
    static_assert(DIM == 3 || TY == 1, "2-D grids use one-row tiles");
    static_assert(Ring<TX, TY, DIM>::COUNT <= NT, "ring larger than the workgroup");
    __shared__ float sF[4][NF][FLY][FLX];
    __shared__ float sR[2][NR][RLY][RLX];

    const int t = threadIdx.x, tx = t % TX, ty = t / TX;
    const TileCoord tc = tile_coord<TX, TY>(D);
    const int gx = tc.gx0 + tx, gy = (DIM == 3) ? tc.gy0 + ty : 0;
    const long long plane = (long long)D.ny * D.nx;
    const bool inarr = gx < D.nx && gy < D.ny;
    const bool interior = gx >= 1 && gx <= D.nx - 2 && (DIM == 2 || (gy >= 1 && gy <= D.ny - 2));
    const int col = gy * D.nx + gx;
    const float scale = (float)(two_over_M * (*dloss));

    // Per-thread prefetch slots of a field plane (tile + 2-node halo).
    int pofs[KP];
    bool pok[KP];
#pragma unroll
    for (int k = 0; k < KP; ++k) {
        const int i = t + k * NT;
        const int ly = i / FLX, lx = i % FLX;
        const int py = (DIM == 3) ? tc.gy0 - HY + ly : 0, px = tc.gx0 - 2 + lx;
        pok[k] = i < FSZ && px >= 0 && px < D.nx && py >= 0 && py < D.ny;
        pofs[k] = pok[k] ? py * D.nx + px : 0;
    }
    float pre[NF][KP];
    auto load_plane = [&](int z) {
        const bool zok = z >= 0 && z < D.nz;
        const long long zo = (long long)(zok ? z : 0) * plane;
#pragma unroll
        for (int f = 0; f < NF; ++f)
#pragma unroll
            for (int k = 0; k < KP; ++k) pre[f][k] = (zok && pok[k]) ? P.f[f][zo + pofs[k]] : 0.f;
    };
    auto store_plane = [&](int slot) {
#pragma unroll
        for (int k = 0; k < KP; ++k) {
            const int i = t + k * NT;
            if (i < FSZ) {
#pragma unroll
                for (int f = 0; f < NF; ++f) (&sF[slot][f][0][0])[i] = pre[f][k];
            }
        }
    };

    // Residuals at plane zr on R-tile position (ly, lx) -> sR[dst].
    auto r_at = [&](int zr, int sm, int sc, int sp, int dst, int ly, int lx) {
        const int ry = (DIM == 3) ? tc.gy0 - RHY + ly : 0, rx = tc.gx0 - 1 + lx;
        const bool om = zr >= 1 && zr <= D.nz - 2 && rx >= 1 && rx <= D.nx - 2 &&
                        (DIM == 2 || (ry >= 1 && ry <= D.ny - 2));
        float R[NR];
        if (om) {
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
            float cc[NC > 0 ? NC : 1];
            const long long o = (long long)zr * plane + ry * D.nx + rx;
#pragma unroll
            for (int j = 0; j < NC; ++j) cc[j] = P.c[j][o];
            OP::residual(s, cc, K, R);
        } else {
#pragma unroll
            for (int b = 0; b < NR; ++b) R[b] = 0.f;
        }
#pragma unroll
        for (int b = 0; b < NR; ++b) sR[dst][b][ly][lx] = R[b];
    };
    const bool has_ring = t < Ring<TX, TY, DIM>::COUNT;
    int rly = 0, rlx = 0;
    if (has_ring) Ring<TX, TY, DIM>::pos(t, rly, rlx);
    auto r_tile = [&](int zr, int sm, int sc, int sp, int dst) {
        r_at(zr, sm, sc, sp, dst, ty + RHY, tx + 1);
        if (has_ring) r_at(zr, sm, sc, sp, dst, rly, rlx);
    };

    // ---- prologue: planes z0-1, z0, z0+1 in LDS; R(z0) tile; R(z0-1) own column
    const int z0 = tc.z0, z1 = tc.z1;
    for (int pz = z0 - 1; pz <= z0 + 1; ++pz) {
        load_plane(pz);
        store_plane(pz & 3);
    }
    float fzm[NF], rzm[NR];
    float fzm2[NF];
#pragma unroll
    for (int f = 0; f < NF; ++f)
        fzm2[f] = (inarr && z0 >= 2) ? P.f[f][(long long)(z0 - 2) * plane + col] : 0.f;
    __syncthreads();
    r_tile(z0, (z0 - 1) & 3, z0 & 3, (z0 + 1) & 3, z0 & 1);
    {
        const int s1 = (z0 - 1) & 3, s0 = z0 & 3;
        const int fy = ty + HY, fx = tx + 2;
#pragma unroll
        for (int f = 0; f < NF; ++f) fzm[f] = sF[s1][f][fy][fx];
        if (interior && z0 - 1 >= 1) {
            Star s[NF];
#pragma unroll
            for (int f = 0; f < NF; ++f) {
                s[f].c = sF[s1][f][fy][fx];
                s[f].m[0] = fzm2[f];
                s[f].p[0] = sF[s0][f][fy][fx];
                s[f].m[DIM - 1] = sF[s1][f][fy][fx - 1];
                s[f].p[DIM - 1] = sF[s1][f][fy][fx + 1];
                if (DIM == 3) {
                    s[f].m[1] = sF[s1][f][fy - 1][fx];
                    s[f].p[1] = sF[s1][f][fy + 1][fx];
                }
            }
            float cc[NC > 0 ? NC : 1];
#pragma unroll
            for (int j = 0; j < NC; ++j) cc[j] = P.c[j][(long long)(z0 - 1) * plane + col];
            OP::residual(s, cc, K, rzm);
        } else {
#pragma unroll
            for (int b = 0; b < NR; ++b) rzm[b] = 0.f;
        }
    }
    load_plane(z0 + 2);

    // ---- march
    for (int z = z0; z < z1; ++z) {
        store_plane((z + 2) & 3);
        if (z + 1 < z1) load_plane(z + 3);
        __syncthreads();
        r_tile(z + 1, z & 3, (z + 1) & 3, (z + 2) & 3, (z + 1) & 1);
        __syncthreads();
        if (inarr) {
            const int sc = z & 3, sp = (z + 1) & 3, rc = z & 1, rp = (z + 1) & 1;
            const int fy = ty + HY, fx = tx + 2, ry = ty + RHY, rx = tx + 1;
            Star fs[NF], rs[NR];
#pragma unroll
            for (int f = 0; f < NF; ++f) {
                fs[f].c = sF[sc][f][fy][fx];
                fs[f].m[0] = fzm[f];
                fs[f].p[0] = sF[sp][f][fy][fx];
                fs[f].m[DIM - 1] = sF[sc][f][fy][fx - 1];
                fs[f].p[DIM - 1] = sF[sc][f][fy][fx + 1];
                if (DIM == 3) {
                    fs[f].m[1] = sF[sc][f][fy - 1][fx];
                    fs[f].p[1] = sF[sc][f][fy + 1][fx];
                }
            }
#pragma unroll
            for (int b = 0; b < NR; ++b) {
                rs[b].c = sR[rc][b][ry][rx];
                rs[b].m[0] = rzm[b];
                rs[b].p[0] = sR[rp][b][ry][rx];
                rs[b].m[DIM - 1] = sR[rc][b][ry][rx - 1];
                rs[b].p[DIM - 1] = sR[rc][b][ry][rx + 1];
                if (DIM == 3) {
                    rs[b].m[1] = sR[rc][b][ry - 1][rx];
                    rs[b].p[1] = sR[rc][b][ry + 1][rx];
                }
            }
            float g[NF];
            OP::gather(fs, rs, K, g);
            const long long o = (long long)z * plane + col;
#pragma unroll
            for (int f = 0; f < NF; ++f) P.out[f][o] = scale * g[f];
#pragma unroll
            for (int f = 0; f < NF; ++f) fzm[f] = fs[f].c;
#pragma unroll
            for (int b = 0; b < NR; ++b) rzm[b] = rs[b].c;
        }
    }
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
