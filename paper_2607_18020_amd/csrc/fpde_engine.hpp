// fpde_engine.hpp -- gfx950 kernels of the FD residual operator.
//
// Grid geometry: array axis 0 is the march axis ("z"); the last axis is x
// (fastest, coalesced); for 3-D grids axis 1 is y.  A workgroup owns a TX x TY
// column tile of the (y, x) plane (TY = 1 for 2-D grids, where the "plane" is a
// row segment) and marches a chunk of planes along axis 0.  Each plane region
// streams from memory straight into a ring of LDS slots, so every input element
// is read from HBM once per chunk plus the halo; the 7-point star of a node is
// read from the slots of planes z-1, z, z+1.  (The register-queue forward,
// fwdq_kernel, keeps its planes in per-lane registers instead.)
//
// Forward: one residual per interior node, sum of squares accumulated in a
// per-thread float64 register, reduced with DPP across the wavefront and through
// LDS across waves, then ONE float64 atomic add per workgroup (Sec. 2.1 fused
// stencil, with the loss fused as well).
//
// Backward: gather form of the transposed stencil (Sec. 2.2).  The residuals
// that the gather needs are recomputed, never read: at step z the workgroup
// evaluates R(z+1) on the tile plus a one-node ring into an LDS tile, so the
// gather for plane z reads R(z) (in-plane star, LDS), R(z+1) and R(z-1) of its
// own column (registers).  Every node of the visited planes is written exactly
// once (boundary columns included: there the residuals off the residual set are
// zero, which the LDS tiles already hold); no atomics.  The planes visited are
// 1..nz-2, or all of them on a periodic grid and in the one-pass value and
// gradient (the end planes' terms then come from the same gather).
//
// Boundary correction: one workgroup per row segment of the two end planes of
// axis 0, the boundary nodes the three-call backward does not visit (Sec. 2.3).
//
// Workgroup-to-tile order is XCD-aware: consecutive workgroup ids are spread
// round-robin over the 8 XCDs, so the id is remapped such that each XCD gets a
// contiguous run of tiles (neighbouring tiles, which share halos, then share
// that XCD's L2).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "fpde_ops.hpp"

// Minimum waves per SIMD requested from the compiler for the marching kernels
// (the second launch bound, which caps their VGPRs; 1 leaves the compiler free).
// The forward asks for 4, so that two 8-wave workgroups share a CU with at most
// 128 VGPRs each.
#ifndef FPDE_FWD_MINW
#define FPDE_FWD_MINW 4
#endif
#ifndef FPDE_BWD_MINW
#define FPDE_BWD_MINW 1
#endif
#ifndef FPDE_VJP_MINW
#define FPDE_VJP_MINW 1
#endif

namespace fpde {

struct Ptrs {
    const float* f[4];
    const float* c[6];
    float* out[4];
    const float* s[4];  // caller-given residual sensitivities (explicit-sensitivity backward)
};

struct Dims {
    int nz, ny, nx;         // ny = 1 for 2-D grids
    int tiles_x, tiles_y;   // tiles_y = 1 for 2-D grids
    int zc, nblocks;        // planes per chunk, workgroups launched
    int per;                // periodic wrap on every axis (residual at every node); the
                            // marching kernels take it as their template argument PER
    int zlo;                // first marched plane: 1, or 0 when periodic or when the
                            // backward march also covers the end planes (value and grad)
    // 3D+t grids (operators with TIME): the 3-D volume (nz, ny, nx) of one time
    // level is what the kernels march; a launch covers the levels lev0 ..
    // lev0 + nlev - 1 of the nt levels, vol nodes apart.  Other grids: nlev = nt
    // = 1, lev0 = 0, vol = 0.
    int nt, nlev, lev0;
    long long vol;
};

// i in [-n, 2n) wrapped into [0, n) (periodic grids; a ragged tile reaches past n)
__device__ __forceinline__ int wrap_idx(int i, int n) {
    return i < 0 ? i + n : (i >= n ? (i >= 2 * n ? i % n : i - n) : i);
}

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
    int lev;  // time level (3D+t grids; 0 otherwise)
};

// Workgroup -> (time level, x tile, y tile, chunk), the time level fastest: the
// workgroups of neighbouring levels of one tile and chunk then run together on
// one XCD, and the point values one reads from the other's level are in L2.
template <int TX, int TY>
__device__ __forceinline__ TileCoord tile_coord(const Dims& D) {
    int lb = remap_xcd(blockIdx.x, D.nblocks);
    const int lev = D.lev0 + lb % D.nlev;
    lb /= D.nlev;
    const int bx = lb % D.tiles_x;
    lb /= D.tiles_x;
    const int by = lb % D.tiles_y;
    const int ch = lb / D.tiles_y;
    TileCoord tc;
    tc.gx0 = bx * TX;
    tc.gy0 = by * TY;
    tc.z0 = D.zlo + ch * D.zc;
    tc.z1 = min(tc.z0 + D.zc, D.nz - D.zlo);
    tc.lev = lev;
    return tc;
}

// A 3D+t operator's arrays at time level lev: the fields, outputs and
// sensitivities move to the level, and each const becomes the field TSRC[j] at
// level lev + TOFF[j] (wrapped on a periodic grid).  No-op for other operators.
template <class OP>
__device__ __forceinline__ void time_level(Ptrs& P, const Dims& D, int lev) {
    if constexpr (OP::TIME) {
        const long long off = (long long)lev * D.vol;
        const float* base[OP::NF];
#pragma unroll
        for (int f = 0; f < OP::NF; ++f) {
            base[f] = P.f[f];
            P.f[f] += off;
            P.out[f] += off;
        }
#pragma unroll
        for (int j = 0; j < OP::NC; ++j) {
            int l = lev + OP::TOFF[j];
            l = l < 0 ? l + D.nt : (l >= D.nt ? l - D.nt : l);
            P.c[j] = base[OP::TSRC[j]] + (long long)l * D.vol;
        }
#pragma unroll
        for (int b = 0; b < OP::NR; ++b) P.s[b] += off;
    }
}

// ---------------------------------------------------------------------------
// Global-memory access in the marching kernels: one raw buffer resource per
// plane (base = the plane's first byte, built in SGPRs) and a 32-bit per-thread
// byte offset, so a load is a single buffer_load_dword with no per-lane
// address arithmetic.  num_records is the plane size: an offset past it reads 0.
// Positions outside the array use offset 0 and a select to zero.

template <int V>
using IC = std::integral_constant<int, V>;

// The LDS ring slots are N (4 or 8) distinct __shared__ arrays, picked by a
// compile-time index modulo N.  Distinct objects let the compiler see that a
// slot being filled by buffer_load ... lds is not one being read, so the reads
// of a step do not wait for the plane that the same step queues.  (Slots 4..7
// of a 4-slot ring are one-element placeholders that nothing references.)
#define FPDE_SLOT_RING_N(T, NAME, N, D1, D2)                                              \
    static_assert((N) == 4 || (N) == 8, "rings of 4 or 8 slots");                         \
    __shared__ T NAME##0[D1][D2], NAME##1[D1][D2], NAME##2[D1][D2], NAME##3[D1][D2];      \
    __shared__ T NAME##4[(N) > 4 ? (D1) : 1][(N) > 4 ? (D2) : 1],                         \
        NAME##5[(N) > 4 ? (D1) : 1][(N) > 4 ? (D2) : 1],                                  \
        NAME##6[(N) > 4 ? (D1) : 1][(N) > 4 ? (D2) : 1],                                  \
        NAME##7[(N) > 4 ? (D1) : 1][(N) > 4 ? (D2) : 1];                                  \
    auto NAME = [&](auto sc) __attribute__((always_inline)) -> T(*)[D2] {                 \
        constexpr int S_ = decltype(sc)::value % (N);                                     \
        if constexpr (S_ == 0) return NAME##0;                                            \
        else if constexpr (S_ == 1) return NAME##1;                                       \
        else if constexpr (S_ == 2) return NAME##2;                                       \
        else if constexpr (S_ == 3) return NAME##3;                                       \
        else if constexpr (S_ == 4) return reinterpret_cast<T(*)[D2]>(&NAME##4[0][0]);    \
        else if constexpr (S_ == 5) return reinterpret_cast<T(*)[D2]>(&NAME##5[0][0]);    \
        else if constexpr (S_ == 6) return reinterpret_cast<T(*)[D2]>(&NAME##6[0][0]);    \
        else return reinterpret_cast<T(*)[D2]>(&NAME##7[0][0]);                           \
    }
#define FPDE_SLOT_RING(T, NAME, D1, D2) FPDE_SLOT_RING_N(T, NAME, 4, D1, D2)

// Checking build (FPDE_LDS_POISON): every LDS array of a marching kernel is
// filled with NaN before the march, so that a read of a location no load or
// residual evaluation has written shows up as NaN in the outputs.
#ifndef FPDE_LDS_POISON
#define FPDE_LDS_POISON 0
#endif
__device__ __forceinline__ void poison_lds(float* p, int n) {
    if (FPDE_LDS_POISON)
        for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = __int_as_float(0x7fc00000);
}
#define FPDE_POISON_RING(NAME)                                              \
    do {                                                                    \
        if (FPDE_LDS_POISON) {                                              \
            poison_lds(&NAME##0[0][0], (int)(sizeof(NAME##0) / 4));         \
            poison_lds(&NAME##1[0][0], (int)(sizeof(NAME##1) / 4));         \
            poison_lds(&NAME##2[0][0], (int)(sizeof(NAME##2) / 4));         \
            poison_lds(&NAME##3[0][0], (int)(sizeof(NAME##3) / 4));         \
            poison_lds(&NAME##4[0][0], (int)(sizeof(NAME##4) / 4));         \
            poison_lds(&NAME##5[0][0], (int)(sizeof(NAME##5) / 4));         \
            poison_lds(&NAME##6[0][0], (int)(sizeof(NAME##6) / 4));         \
            poison_lds(&NAME##7[0][0], (int)(sizeof(NAME##7) / 4));         \
        }                                                                   \
    } while (0)

// Descriptor words must sit in SGPRs.  Their inputs are wave-uniform by
// construction (kernel arguments and march counters), but after control flow
// joins the compiler can lose track of that and wrap each load in a
// readfirstlane loop; rebuilding the base and the size from lane 0 keeps the
// descriptor scalar.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t uniform_rsrc(const void* base, int nbytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    // (readfirstlane returns int: widen through uint32_t, not by sign extension)
    const uint64_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint64_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(hi << 32 | lo), (short)0,
                                             __builtin_amdgcn_readfirstlane(nbytes), 0x00020000);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t plane_rsrc(const float* p, int z,
                                                             uint32_t pbytes) {
    return uniform_rsrc(reinterpret_cast<const char*>(p) + (uint64_t)z * pbytes, (int)pbytes);
}

// Plane z if ok, else an empty range: every access through it reads 0 and
// fetches nothing.  Keeps a step's memory operations unconditional, so that
// the number of them in flight does not depend on the path taken.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t plane_rsrc_if(const float* p, int z,
                                                                uint32_t pbytes, bool ok) {
    return uniform_rsrc(reinterpret_cast<const char*>(p) + (ok ? (uint64_t)z * pbytes : 0),
                        ok ? (int)pbytes : 0);
}

// A store offset past every plane's range (planes hold fewer than 2^29 nodes):
// the hardware drops such a store.
constexpr uint32_t kDropOff = 0x80000000u;

// AUX: the cache-policy bits of the access (0: default; 2: non-temporal).
// Outputs (gradients, residuals) are written once and not read again by the
// operator: they are stored non-temporally, so that they neither evict the
// halo rows that neighbouring tiles share in L2 nor leave dirty lines in the
// caches for the next kernel to write back.
constexpr int kStream = 2;

template <int AUX = 0>
__device__ __forceinline__ float bld(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, AUX));
}

template <int AUX = 0>
__device__ __forceinline__ void bst(__amdgpu_buffer_rsrc_t r, uint32_t off, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)off, 0, AUX);
}



// An opaque copy of v, made once per march step.  LDS addresses derived from it
// are recomputed in the step (one add each) instead of being hoisted out of the
// march: with buffers beyond the 64 KB reach of a ds_read offset, the hoisted
// addresses would hold many VGPRs for the whole loop.  Only when LDS_BYTES, the
// kernel's LDS footprint, exceeds that reach (else v itself).
template <int LDS_BYTES>
__device__ __forceinline__ int fresh(int v) {
    if constexpr (LDS_BYTES > 65536) asm volatile("" : "+v"(v));
    return v;
}

// ---------------------------------------------------------------------------
// Streaming a plane region straight into LDS.  A workgroup's slot holds the
// region's FSZ elements (tile plus halo, row-major) padded to a multiple of 64,
// and element i is loaded by thread i mod NT in round i / NT: the 64 lanes of a
// wave fill 64 consecutive LDS words (buffer_load_dword ... lds, M0 = the
// wave's base).  Every wave issues the same KP loads per array and plane, so
// that the number of loads in flight does not depend on the wave (the
// compiler's wait counts are exact only then): a wave whose part of a round
// lies past the slot sends it to the 64-word spill line after the slot (slot
// arrays hold FSZS words).  Elements outside the array, and the padding, carry
// an offset past the descriptor's range and read as 0 without a memory access;
// so does a whole plane outside the grid.

template <int FSZ, int NT>
struct PlaneStream {
    static constexpr int FSZP = (FSZ + 63) / 64 * 64;  // padded slot size (elements)
    static constexpr int FSZS = FSZP + 64;              // with the spill line
    static constexpr int KP = (FSZP + NT - 1) / NT;     // load rounds
    static constexpr uint32_t kOff = 0x80000000u;
    uint32_t off[KP];  // byte offset of this thread's element in each round
    uint32_t wl;       // first element of this wave (uniform)

    // node_of(i, lin): in-plane linear node index of element i; false if outside the array
    template <class F>
    __device__ __forceinline__ void init(int t, F node_of) {
        wl = __builtin_amdgcn_readfirstlane((uint32_t)(t & ~63));
#pragma unroll
        for (int k = 0; k < KP; ++k) {
            const int i = t + k * NT;
            int lin = 0;
            const bool ok = i < FSZ && node_of(i, lin);
            off[k] = ok ? (uint32_t)lin * 4u : kOff;
        }
    }
    // queue plane pz (uniform) of the NF arrays src[0..NF) into slot base pointers
    template <int NF>
    __device__ __forceinline__ void load(const float* const* src, int pz, int nz, uint32_t pbytes,
                                         float* const* dst) const {
        const bool zok = pz >= 0 && pz < nz;
        const uint64_t zoff = zok ? (uint64_t)pz * pbytes : 0;
        const int nrec = zok ? (int)pbytes : 0;
        __amdgpu_buffer_rsrc_t r[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f)
            r[f] = uniform_rsrc(reinterpret_cast<const char*>(src[f]) + zoff, nrec);
#pragma unroll
        for (int k = 0; k < KP; ++k) {
            // rounds that the slot fills completely hold a part of every wave
            const bool in = (k + 1) * NT <= FSZP || wl + k * NT < (uint32_t)FSZP;
            const uint32_t at = in ? wl + k * NT : (uint32_t)FSZP;  // uniform
#pragma unroll
            for (int f = 0; f < NF; ++f)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    r[f], (__attribute__((address_space(3))) void*)(dst[f] + at), 4, (int)off[k], 0,
                    0, 0);
        }
    }
};

// ---------------------------------------------------------------------------
// Forward: residuals of one chunk of planes + fused sum of squares.  Each plane
// (tile rows plus one row above and below, and the side-edge x-neighbours)
// streams from memory straight into an LDS ring of RD slots; the 7-point star
// of every field is read from the slots of planes z-1, z, z+1.  One barrier per
// step: plane z + RD - 2 streams into the slot of plane z-2 while plane z is
// evaluated, and the consts come CD - 1 planes ahead into registers.  The sum
// of squares is accumulated per thread in float64, reduced with DPP across the
// wavefront and through LDS across waves, then added with ONE float64 atomic
// per workgroup.
//
// RD = 4: the plane queued in a step is read in the next one, and the barrier
// waits for it (the operators with several fields, whose arithmetic per step
// covers a plane's latency; their LDS holds no more slots anyway).  RD = 8: the
// plane queued in a step is read five steps later, so that an operator with
// one field and almost no arithmetic per step keeps several planes in flight;
// the barrier waits, by an explicit count, only for the plane queued four
// steps earlier, which the next step reads first.

template <class F, int... I>
__device__ __forceinline__ void unroll_seq(F&& f, std::integer_sequence<int, I...>) {
    (f(IC<I>{}), ...);
}

// Waits until at most N vector-memory operations of this wave are in flight
// and its LDS operations are done, then the workgroup barrier.
template <int N>
__device__ __forceinline__ void barrier_after() {
    static_assert(N >= 0 && N <= 63, "vmcnt counts 0 .. 63");
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

template <class OP, int TX, int TY, bool STORE_R, bool PER, int RD = 4>
__global__ __launch_bounds__(TX* TY, FPDE_FWD_MINW) void fwd_kernel(Ptrs P, Dims D, KCoef K,
                                                                    double inv_M, double* loss) {
    constexpr int DIM = OP::DIM, NF = OP::NF, NC = OP::NC, NR = OP::NR, NT = TX * TY;
    constexpr int NC1 = NC > 0 ? NC : 1;
    constexpr int CD = RD / 2;  // const queue: planes z .. z + CD - 1 in registers
    constexpr int HY = (DIM == 3) ? 1 : 0;
    // A slot holds the tile's own TX columns for TY + 2 HY rows, so that every
    // wavefront's plane load is one aligned 64-node row segment (a halo column in
    // each row would misalign them all), followed by one 64-element group with
    // the x-neighbours across the tile's side edges: element LY*TX + r is the
    // left neighbour of own row r, element LY*TX + TY + r the right one.  Each of
    // those is a cache line of its own, so tiles are made wide.
    constexpr int LY = TY + 2 * HY, LX = TX, XG = LY * LX;
    static_assert(TX % 64 == 0, "a wavefront loads whole aligned row segments");
    static_assert(2 * TY <= 64, "the side-edge neighbours fill one 64-element group");
    using PS = PlaneStream<XG + 64, NT>;
    static_assert(DIM == 3 || TY == 1, "2-D grids use one-row tiles");
    FPDE_SLOT_RING_N(float, sF, RD, NF, PS::FSZS);
    // vector-memory operations a wave issues per step, in this order: the plane
    // loads (every wave the same number), the const loads, the residual stores
    constexpr int kPlaneOps = PS::KP * NF, kStepOps = kPlaneOps + NC + (STORE_R ? NR : 0);
    // At the end of step w, step w + 1 needs plane z + 2, queued in step
    // w - (RD - 4), or for w < RD - 4 in the prologue (RD - 1 plane groups, then
    // CD - 1 const groups); the operations issued after it may stay in flight:
    //   w >= RD - 4:  (kStepOps - kPlaneOps) + (RD - 4) kStepOps
    //   w <  RD - 4:  (RD - 5 - w) kPlaneOps + (CD - 1) NC + (w + 1) kStepOps
    constexpr int kInFlight = (kStepOps - kPlaneOps) + (RD - 4) * kStepOps;
    constexpr auto in_flight_early = [](int w) {
        const int k = (RD - 5 - w) * kPlaneOps + (CD - 1) * NC + (w + 1) * kStepOps;
        return k < kInFlight ? k : kInFlight;
    };
    static_assert(RD == 4 || kInFlight <= 63, "a vmcnt wait counts at most 63 operations");
    static_assert(RD == 4 || RD == 8, "rings of 4 or 8 slots");

    const int t = threadIdx.x, tx = t % TX, ty = t / TX;
    FPDE_POISON_RING(sF);
    if (FPDE_LDS_POISON) __syncthreads();
    const TileCoord tc = tile_coord<TX, TY>(D);
    time_level<OP>(P, D, tc.lev);
    const int z0 = tc.z0, z1 = tc.z1, L = z1 - z0;
    const int gx = tc.gx0 + tx, gy = (DIM == 3) ? tc.gy0 + ty : 0;
    const uint32_t pbytes = (uint32_t)D.ny * (uint32_t)D.nx * 4u;
    const bool inarr = gx < D.nx && gy < D.ny;
    const bool interior =
        PER ? inarr : gx >= 1 && gx <= D.nx - 2 && (DIM == 2 || (gy >= 1 && gy <= D.ny - 2));
    const uint32_t cb = inarr ? (uint32_t)(gy * D.nx + gx) * 4u : 0u;
    auto zw = [&](int z) { return PER ? wrap_idx(z, D.nz) : z; };  // plane index

    PS ps;
    ps.init(t, [&](int i, int& lin) {
        int py, px;
        if (i < XG) {
            py = (DIM == 3) ? tc.gy0 - HY + i / LX : 0;
            px = tc.gx0 + i % LX;
        } else {
            const int j = i - XG, side = j / TY;
            py = (DIM == 3) ? tc.gy0 + j % TY : 0;
            px = side == 0 ? tc.gx0 - 1 : tc.gx0 + TX;
            if (side > 1) return false;
        }
        if (PER) {  // every position is a node of the wrapped grid
            px = wrap_idx(px, D.nx);
            py = wrap_idx(py, D.ny);
        }
        lin = py * D.nx + px;
        return px >= 0 && px < D.nx && py >= 0 && py < D.ny;
    });
    auto load_plane = [&](int pz, auto slot) __attribute__((always_inline)) {
        float* dst[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f) dst[f] = &sF(slot)[f][0];
        ps.template load<NF>(P.f, pz, D.nz, pbytes, dst);
    };
    float cv[CD][NC1];
    auto load_consts = [&](int pz, bool ok, float* c) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < NC; ++j)
            c[j] = bld(plane_rsrc_if(P.c[j], pz, pbytes, ok), cb);
    };

    // The end planes of axis 0, which the march does not visit, hold no residual
    // node: the first and the last chunk write their zeros.  (Whole rows are
    // written, boundary columns included, so that no cache line of R is stored
    // in part.)
    if (STORE_R && !PER) {
        const uint32_t so = inarr ? cb : kDropOff;
#pragma unroll
        for (int b = 0; b < NR; ++b) {
            if (z0 == 1) bst<kStream>(plane_rsrc(P.out[b], 0, pbytes), so, 0.f);
            if (z1 == D.nz - 1) bst<kStream>(plane_rsrc(P.out[b], D.nz - 1, pbytes), so, 0.f);
        }
    }

    // plane z0 + j lives in slot (j + 1) % RD; prologue: planes z0 - 1 .. z0 + RD - 3
    // (planes past the chunk's stencil, or past the grid, are harmless: unread, or
    // read as 0), consts of planes z0 .. z0 + CD - 2
    unroll_seq([&](auto jc) __attribute__((always_inline)) {
        constexpr int J = decltype(jc)::value;  // slot J holds plane z0 + J - 1
        load_plane(J == 1 ? z0 : zw(z0 + J - 1), IC<J>{});
    }, std::make_integer_sequence<int, RD - 1>{});
    // (the plane loads first, as in the steps: the wait counts assume that order)
    __builtin_amdgcn_sched_barrier(0);
    unroll_seq([&](auto jc) __attribute__((always_inline)) {
        constexpr int J = decltype(jc)::value;
        load_consts(z0 + J, J == 0 || J < L, cv[J]);  // (a chunk holds a plane at least)
    }, std::make_integer_sequence<int, CD - 1>{});
    __syncthreads();

    const int own = (ty + HY) * LX + tx;  // own node in a slot
    // its x-neighbours: in the row, or in the side-edge group
    const int xm = tx == 0 ? XG + ty : own - 1, xp = tx == TX - 1 ? XG + TY + ty : own + 1;
    double acc = 0.0;
    auto step = [&](auto jc, int w) __attribute__((always_inline)) {
        constexpr int J = decltype(jc)::value;  // w % RD
        constexpr int SM = J % RD, SC = (J + 1) % RD, SP = (J + 2) % RD, SQ = (J + RD - 1) % RD;
        constexpr int CUR = J % CD, NXT = (J + CD - 1) % CD;
        const int z = z0 + w;
        // plane z + RD - 2 goes to the slot of plane z - 2, last read before the
        // previous barrier; it is in the chunk's stencil if z + RD - 2 <= z1
        load_plane(w + RD - 3 < L ? zw(z + RD - 2) : -1, IC<SQ>{});
        // the plane loads go first: the barrier then waits for them alone, not
        // for the const loads queued after them for later steps
        __builtin_amdgcn_sched_barrier(0);
        load_consts(z + CD - 1, w + CD - 1 < L, cv[NXT]);
        Star s[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const float* c = &sF(IC<SC>{})[f][own];
            s[f].c = c[0];
            s[f].m[0] = sF(IC<SM>{})[f][own];
            s[f].p[0] = sF(IC<SP>{})[f][own];
            s[f].m[DIM - 1] = sF(IC<SC>{})[f][xm];
            s[f].p[DIM - 1] = sF(IC<SC>{})[f][xp];
            if (DIM == 3) {
                s[f].m[1] = c[-LX];
                s[f].p[1] = c[LX];
            }
        }
        float R[NR];
        OP::residual(s, cv[CUR], K, R);
        float ss = 0.f;
#pragma unroll
        for (int b = 0; b < NR; ++b) ss = fmaf(R[b], R[b], ss);
        acc += (double)(interior ? ss : 0.f);
        // the step's arithmetic feeds nothing but acc: pin acc here, or the compiler
        // may sink that arithmetic past the barriers and keep several steps' loads live
        asm volatile("" : "+v"(acc));
        if (STORE_R) {  // every node of the plane: R on the residual set, 0 off it
            const uint32_t so = inarr ? cb : kDropOff;
#pragma unroll
            for (int b = 0; b < NR; ++b)
                bst<kStream>(plane_rsrc(P.out[b], z, pbytes), so, interior ? R[b] : 0.f);
        }
        if constexpr (RD == 4) {
            __syncthreads();  // (waits for the plane loads into LDS as well)
        } else {
            // the plane step w + 1 reads first, and every earlier operation, has
            // landed (operations retire in order); the LDS reads of this step are
            // done; then the workgroup's barrier (w is uniform)
            if (w >= RD - 4) barrier_after<kInFlight>();
            else if (w == 0) barrier_after<in_flight_early(0)>();
            else if (w == 1) barrier_after<in_flight_early(1)>();
            else if (w == 2) barrier_after<in_flight_early(2)>();
            else barrier_after<in_flight_early(3)>();
        }
    };

    int w = 0;
    for (; w + RD <= L; w += RD)  // slot indices are constants in each copy
        unroll_seq([&](auto jc) __attribute__((always_inline)) {
            step(jc, w + decltype(jc)::value);
        }, std::make_integer_sequence<int, RD>{});
    unroll_seq([&](auto jc) __attribute__((always_inline)) {
        if (w + decltype(jc)::value < L) step(jc, w + decltype(jc)::value);
    }, std::make_integer_sequence<int, RD - 1>{});
    // nothing still streams into LDS when the workgroup's LDS is reused below
    // or handed to the next workgroup
    if constexpr (RD != 4) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    block_atomic_sum<NT>(acc * inv_M, loss);
}

// ---------------------------------------------------------------------------
// Register-queue forward (2-D grids, and 3-D operators with one stencil field):
// residuals of one chunk of planes + fused sum of squares, with no LDS and no
// barrier.  A workgroup owns a TX x TY tile of columns (TY = 1 on 2-D grids,
// where a plane is a row); each lane marches its column down the chunk and
// keeps, for every field, the centre and in-plane neighbours of its column
// (x -+ 1, and y -+ 1 on 3-D grids) for Q planes in a register queue: the plane
// evaluated, its two neighbours and Q - 3 planes in flight, each loaded Q - 3
// steps before it becomes the centre plane.  Where a plane region is a few
// kilobytes, a march with one barrier per plane waits for each plane's latency
// in turn; here each wave keeps several planes of loads in flight on its own.
// The neighbour loads fall in the cache lines of neighbouring lanes' (x) or
// waves' (y) centre loads, so HBM sees each field once.  Planes outside the
// chunk's stencil and outside the grid are read through empty descriptors (0,
// no access).


template <class OP, int TX, int TY, int Q, bool STORE_R, bool PER>
__global__ __launch_bounds__(TX* TY) void fwdq_kernel(Ptrs P, Dims D, KCoef K, double inv_M,
                                                      double* loss) {
    constexpr int DIM = OP::DIM, NF = OP::NF, NC = OP::NC, NR = OP::NR, NT = TX * TY;
    constexpr int NC1 = NC > 0 ? NC : 1;
    constexpr int NV = 2 * DIM - 1;  // centre, x -+ 1 [, y -+ 1]
    static_assert(DIM == 3 || TY == 1, "2-D grids use one-row tiles");
    static_assert(Q >= 4, "planes z - 1, z, z + 1 and at least one plane in flight");
    constexpr uint32_t kOff = 0x80000000u;  // past every plane's range: reads 0
    const int t = threadIdx.x, tx = t % TX, ty = t / TX;
    const TileCoord tc = tile_coord<TX, TY>(D);
    time_level<OP>(P, D, tc.lev);
    const int z0 = tc.z0, z1 = tc.z1, L = z1 - z0;
    const int gx = tc.gx0 + tx, gy = (DIM == 3) ? tc.gy0 + ty : 0;
    const uint32_t pbytes = (uint32_t)D.ny * (uint32_t)D.nx * 4u;
    const bool inarr = gx < D.nx && gy < D.ny;
    const bool interior =
        PER ? inarr : gx >= 1 && gx <= D.nx - 2 && (DIM == 2 || (gy >= 1 && gy <= D.ny - 2));
    // byte offsets of the centre and in-plane neighbours within a plane
    auto at = [&](int y, int x) -> uint32_t {
        if (!inarr) return kOff;
        if (PER) {
            x = wrap_idx(x, D.nx);
            y = wrap_idx(y, D.ny);
        } else if (x < 0 || x >= D.nx || y < 0 || y >= D.ny) {
            return kOff;
        }
        return (uint32_t)(y * D.nx + x) * 4u;
    };
    uint32_t off[NV];
    off[0] = at(gy, gx);
    off[1] = at(gy, gx - 1);
    off[2] = at(gy, gx + 1);
    if constexpr (DIM == 3) {
        off[3] = at(gy - 1, gx);
        off[4] = at(gy + 1, gx);
    }

    // the queue: plane z0 - 1 + k lives in slot k % Q
    float qv[Q][NF][NV], qk[Q][NC1];
    auto load_plane = [&](int z, auto slot) __attribute__((always_inline)) {  // z uniform
        constexpr int S_ = decltype(slot)::value;
        // the planes the chunk's residuals read: z0 - 1 .. z1
        const bool ok = z >= z0 - 1 && z <= z1 && (PER || (z >= 0 && z < D.nz));
        const int zr = PER ? wrap_idx(z, D.nz) : z;
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const __amdgpu_buffer_rsrc_t r = plane_rsrc_if(P.f[f], zr, pbytes, ok);
#pragma unroll
            for (int v = 0; v < NV; ++v) qv[S_][f][v] = bld(r, off[v]);
        }
#pragma unroll
        for (int j = 0; j < NC; ++j)
            qk[S_][j] = bld(plane_rsrc_if(P.c[j], zr, pbytes, ok), off[0]);
    };

    // the end planes of axis 0 hold no residual node: the first and the last chunk
    // write their zeros (every column, so that no cache line of R is stored in part)
    if (STORE_R && !PER) {
        const uint32_t so = inarr ? off[0] : kDropOff;
#pragma unroll
        for (int b = 0; b < NR; ++b) {
            if (z0 == 1) bst<kStream>(plane_rsrc(P.out[b], 0, pbytes), so, 0.f);
            if (z1 == D.nz - 1) bst<kStream>(plane_rsrc(P.out[b], D.nz - 1, pbytes), so, 0.f);
        }
    }

    unroll_seq([&](auto k) __attribute__((always_inline)) {
        load_plane(z0 - 1 + decltype(k)::value, k);
    }, std::make_integer_sequence<int, Q - 1>{});

    double acc = 0.0;
    auto step = [&](auto jc, int w) __attribute__((always_inline)) {
        constexpr int J = decltype(jc)::value;  // w % Q
        constexpr int SM = J % Q, SC = (J + 1) % Q, SP = (J + 2) % Q, SN = (J + Q - 1) % Q;
        // plane z + Q - 2 goes to the slot of plane z - 2, read last in the previous step
        load_plane(z0 + w + Q - 2, IC<SN>{});
        Star st[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            st[f].c = qv[SC][f][0];
            st[f].m[0] = qv[SM][f][0];
            st[f].p[0] = qv[SP][f][0];
            st[f].m[DIM - 1] = qv[SC][f][1];
            st[f].p[DIM - 1] = qv[SC][f][2];
            if constexpr (DIM == 3) {
                st[f].m[1] = qv[SC][f][3];
                st[f].p[1] = qv[SC][f][4];
            }
        }
        float R[NR];
        OP::residual(st, qk[SC], K, R);
        float ss = 0.f;
#pragma unroll
        for (int b = 0; b < NR; ++b) ss = fmaf(R[b], R[b], ss);
        acc += (double)(interior ? ss : 0.f);
        if (STORE_R) {  // every node of the plane: R on the residual set, 0 off it
            const uint32_t so = inarr ? off[0] : kDropOff;
            const int z = PER ? wrap_idx(z0 + w, D.nz) : z0 + w;
#pragma unroll
            for (int b = 0; b < NR; ++b)
                bst<kStream>(plane_rsrc(P.out[b], z, pbytes), so, interior ? R[b] : 0.f);
        }
    };

    int w = 0;
    for (; w + Q <= L; w += Q)  // slot indices are constants in each copy
        unroll_seq([&](auto j) __attribute__((always_inline)) {
            step(j, w + decltype(j)::value);
        }, std::make_integer_sequence<int, Q>{});
    unroll_seq([&](auto j) __attribute__((always_inline)) {
        if (w + decltype(j)::value < L) step(j, w + decltype(j)::value);
    }, std::make_integer_sequence<int, Q - 1>{});
    block_atomic_sum<NT>(acc * inv_M, loss);
}

// ---------------------------------------------------------------------------
// Backward: gather-form transposed stencil with residual recompute.
//
// Per step z: plane z+3 is queued from memory straight into the LDS slot of
// plane z-1; R(z+1) is evaluated on the tile and its one-node ring into an LDS
// tile; the gather at plane z reads the in-plane neighbours of R(z) from LDS and
// R(z-1), R(z), R(z+1) of its own column from a register queue; one barrier.
//
// LOSS: the value and the gradient in one pass.  Every residual of the chunk's
// planes is evaluated here anyway (own column, once per step), so the kernel
// also adds their squares to the loss as the forward does (float32 sum over
// the equations, float64 accumulation, one float64 atomic per workgroup onto
// *loss, which the host zeroes first): the fields are read once for both.

template <class OP, int TX, int TY, bool REV, bool LOSS, bool PER>
__global__ __launch_bounds__(TX* TY, FPDE_BWD_MINW) void bwd_kernel(Ptrs P, Dims D, KCoef K,
                                                                    const double* dloss,
                                                                    double two_over_M,
                                                                    double inv_M, double* loss) {
    constexpr int DIM = OP::DIM, NF = OP::NF, NC = OP::NC, NR = OP::NR, NT = TX * TY;
    constexpr int NC1 = NC > 0 ? NC : 1, NG = OP::NG, NG1 = NG > 0 ? NG : 1;
    constexpr int HY = (DIM == 3) ? 2 : 0;   // field-slot halo (y)
    constexpr int FLY = TY + 2 * HY, FLX = TX + 4;
    constexpr int RHY = (DIM == 3) ? 1 : 0;  // R-tile halo (y)
    constexpr int RLY = TY + 2 * RHY, RLX = TX + 2;
    using PS = PlaneStream<FLY * FLX, NT>;
    static_assert(DIM == 3 || TY == 1, "2-D grids use one-row tiles");
    static_assert(Ring<TX, TY, DIM>::COUNT <= NT, "ring larger than the workgroup");
    // The chunk [z0, z1) of axis 0 is marched in steps w = 0 .. L-1 over the
    // physical planes ph(w) = z0 + w, or z1 - 1 - w when REV (top down).
    // Field planes of march steps live in a 4-slot ring: step w in slot (w + 1) & 3;
    // residual tiles: R of step w in buffer w & 1.
    FPDE_SLOT_RING(float, sF, NF, PS::FSZS);
    __shared__ float sR[2][NR][RLY * RLX];
    constexpr int kLds = (4 * NF * PS::FSZS + 2 * NR * RLY * RLX) * 4;

    const int t = threadIdx.x, tx = t % TX, ty = t / TX;
    FPDE_POISON_RING(sF);
    poison_lds(&sR[0][0][0], (int)(sizeof(sR) / 4));
    if (FPDE_LDS_POISON) __syncthreads();
    const TileCoord tc = tile_coord<TX, TY>(D);
    time_level<OP>(P, D, tc.lev);
    const int z0 = tc.z0, z1 = tc.z1, L = z1 - z0;
    auto ph = [&](int w) {  // (wrapped into the grid when periodic)
        const int p = REV ? z1 - 1 - w : z0 + w;
        return PER ? wrap_idx(p, D.nz) : p;
    };
    const int gx = tc.gx0 + tx, gy = (DIM == 3) ? tc.gy0 + ty : 0;
    const uint32_t pbytes = (uint32_t)D.ny * (uint32_t)D.nx * 4u;
    const bool inarr = gx < D.nx && gy < D.ny;
    const uint32_t cb = inarr ? (uint32_t)(gy * D.nx + gx) * 4u : 0u;
    // offset of the node whose residual this lane evaluates: its own, or on a
    // periodic grid the wrapped one (a ragged tile's first lane past the last
    // column holds the residual that column's gather needs as its x+1 term)
    const uint32_t cbr =
        PER ? (uint32_t)(wrap_idx(gy, D.ny) * D.nx + wrap_idx(gx, D.nx)) * 4u : cb;
    const float scale = (float)(two_over_M * (*dloss));

    PS ps;
    ps.init(t, [&](int i, int& lin) {
        int py = (DIM == 3) ? tc.gy0 - HY + i / FLX : 0, px = tc.gx0 - 2 + i % FLX;
        if (PER) {  // every position is a node of the wrapped grid
            px = wrap_idx(px, D.nx);
            py = wrap_idx(py, D.ny);
        }
        lin = py * D.nx + px;
        return px >= 0 && px < D.nx && py >= 0 && py < D.ny;
    });
    auto load_plane = [&](int pz, auto slot) __attribute__((always_inline)) {
        float* dst[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f) dst[f] = &sF(slot)[f][0];
        ps.template load<NF>(P.f, pz, D.nz, pbytes, dst);
    };

    // residual positions of this thread on the R tile: its own column and, for
    // the first threads, one node of the ring; their in-plane part of the
    // residual-set test and their const offsets are fixed for the whole march
    const bool own_om =
        PER || (gx >= 1 && gx <= D.nx - 2 && (DIM == 2 || (gy >= 1 && gy <= D.ny - 2)));
    const bool has_ring = t < Ring<TX, TY, DIM>::COUNT;
    int rly = 0, rlx = 0;
    if (has_ring) Ring<TX, TY, DIM>::pos(t, rly, rlx);
    const int rgy = (DIM == 3) ? tc.gy0 - RHY + rly : 0, rgx = tc.gx0 - 1 + rlx;
    const bool ring_om = has_ring && (PER || (rgx >= 1 && rgx <= D.nx - 2 &&
                                                (DIM == 2 || (rgy >= 1 && rgy <= D.ny - 2))));
    const uint32_t rcb =
        !ring_om ? 0u
        : PER  ? (uint32_t)(wrap_idx(rgy, D.ny) * D.nx + wrap_idx(rgx, D.nx)) * 4u
                 : (uint32_t)(rgy * D.nx + rgx) * 4u;

    // R at physical plane zr, at node fi of a field slot and ri of an R tile, from
    // the field slots of the previous (sb), same (sc) and next (sn) march steps;
    // written to sR[dst] and returned in R (zero off the residual set); with S,
    // also the gather's self terms at that node
    auto r_at = [&](int zr, auto sb, auto sc, auto sn, int dst, int fi, int ri, bool om_xy,
                    const float* cc, float* R, float* S) __attribute__((always_inline)) {
        Star s[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const float* c = &sF(sc)[f][fi];
            const float vb = sF(sb)[f][fi], vn = sF(sn)[f][fi];
            s[f].c = c[0];
            s[f].m[0] = REV ? vn : vb;  // physical z-1, z+1
            s[f].p[0] = REV ? vb : vn;
            s[f].m[DIM - 1] = c[-1];
            s[f].p[DIM - 1] = c[1];
            if (DIM == 3) {
                s[f].m[1] = c[-FLX];
                s[f].p[1] = c[FLX];
            }
        }
        OP::residual(s, cc, K, R);
        const bool om = om_xy && (PER || (zr >= 1 && zr <= D.nz - 2));
#pragma unroll
        for (int b = 0; b < NR; ++b) {
            R[b] = om ? R[b] : 0.f;
            sR[dst][b][ri] = R[b];
        }
        if (S) OP::gather_self(s, R, K, S);
    };
    // consts of the R-tile positions, for the plane whose residuals come next
    // (loaded one step ahead so that their latency hides behind a step)
    float cown[NC1], cring[NC1];
    // (a march over every plane, end planes included, reaches past the grid: such
    // planes read as 0, and their residuals are masked to 0 anyway)
    auto load_consts = [&](int zr, bool ok) __attribute__((always_inline)) {  // zr uniform
        ok = ok && zr >= 0 && zr < D.nz;
#pragma unroll
        for (int j = 0; j < NC; ++j) {
            const __amdgpu_buffer_rsrc_t r = plane_rsrc_if(P.c[j], zr, pbytes, ok);
            cown[j] = bld(r, cbr);
            cring[j] = bld(r, rcb);
        }
    };
    // positions in a field slot and in an R tile: the own node, and the ring node
    const int fown = (ty + HY) * FLX + tx + 2;   // own node in a field slot
    const int rown = (ty + RHY) * RLX + tx + 1;  // own node in an R tile
    const int fring = (rly + HY - RHY) * FLX + rlx + 1, rring = rly * RLX + rlx;  // ring node

    // R on the whole R tile; the own column's R and gather self terms are returned
    // in Rown, Sown.  fo, ro, fr, rr: a step's copies of fown, rown, fring, rring
    auto r_tile = [&](int zr, auto sb, auto sc, auto sn, int dst, float* Rown, float* Sown, int fo,
                      int ro, int fr, int rr) __attribute__((always_inline)) {
        r_at(zr, sb, sc, sn, dst, fo, ro, own_om, cown, Rown, Sown);
        if (has_ring) {
            float Rr[NR];
            r_at(zr, sb, sc, sn, dst, fr, rr, ring_om, cring, Rr, nullptr);
        }
    };

    // ---- prologue: march steps -1 .. 2 in slots 0..3; R of step 0 on the tile;
    // the own column's R of steps -1, 0 and fields of step -1 in registers
    load_plane(ph(-1), IC<0>{});
    load_plane(ph(0), IC<1>{});
    load_plane(ph(1), IC<2>{});
    load_plane(ph(2), IC<3>{});
    float fzm2[NF];
    {
        const int pz = ph(-2);
        const bool zok = pz >= 0 && pz < D.nz;
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const float v = bld(plane_rsrc(P.f[f], zok ? pz : 0, pbytes), cbr);
            fzm2[f] = ((inarr || PER) && zok) ? v : 0.f;
        }
    }
    load_consts(ph(0), true);
    __syncthreads();
    // own column: fields of the previous step; R of the previous, current and next
    // steps; gather self terms of the current and next steps
    float fzm[NF], rzm[NR], rzc[NR], rzp[NR], sgc[NG1], sgp[NG1];
    r_tile(ph(0), IC<0>{}, IC<1>{}, IC<2>{}, 0, rzc, sgc, fown, rown, fring, rring);
    {
        Star s[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const float* c = &sF(IC<0>{})[f][fown];
            const float nxt = sF(IC<1>{})[f][fown];
            s[f].c = c[0];
            s[f].m[0] = REV ? nxt : fzm2[f];
            s[f].p[0] = REV ? fzm2[f] : nxt;
            s[f].m[DIM - 1] = c[-1];
            s[f].p[DIM - 1] = c[1];
            if (DIM == 3) {
                s[f].m[1] = c[-FLX];
                s[f].p[1] = c[FLX];
            }
            fzm[f] = s[f].c;
        }
        const int pz = ph(-1);  // past the grid when the march covers the end planes
        const bool pok = pz >= 0 && pz < D.nz;
        float cc[NC1];
#pragma unroll
        for (int j = 0; j < NC; ++j) cc[j] = bld(plane_rsrc_if(P.c[j], pz, pbytes, pok), cbr);
        OP::residual(s, cc, K, rzm);
        const bool om = own_om && (PER || (pz >= 1 && pz <= D.nz - 2));
#pragma unroll
        for (int b = 0; b < NR; ++b) rzm[b] = om ? rzm[b] : 0.f;
    }
    load_consts(ph(1), true);  // step 0 evaluates R of step 1 (in range for L >= 1)
    __syncthreads();

    // ---- march.  Step w: issue the loads of step w+3; R of step w+1 on the R tile;
    // the gather at step w; step w+3's plane goes to the slot of step w-1; one
    // barrier.  Every LDS buffer a step writes was last read before the previous
    // step's barrier.
    double acc = 0.0;  // LOSS: sum of squares of the own column's residuals
    auto step = [&](auto jc, int w) __attribute__((always_inline)) {
        constexpr int J = decltype(jc)::value;  // w & 3
        // field slots of steps w-1 (reused for w+3), w, w+1, w+2; R tiles of w, w+1
        constexpr int SB = J & 3, SC = (J + 1) & 3, SN = (J + 2) & 3, SQ = (J + 3) & 3;
        constexpr int RC = J & 1, RN = (J + 1) & 1;
        const bool more = w + 1 < L;
        // step w+3's plane goes to the slot of step w-1, unread in this step; an
        // empty plane after the chunk's last step
        load_plane(more ? ph(w + 3) : -1, IC<SB>{});
        __builtin_amdgcn_sched_barrier(0);  // (the plane loads first, as in the forward)
        const int fos = fown, ros = rown;
        // (the ring's addresses, used by a few waves only, are not held across the march)
        r_tile(ph(w + 1), IC<SC>{}, IC<SN>{}, IC<SQ>{}, RN, rzp, sgp, fos, ros, fresh<kLds>(fring),
               fresh<kLds>(rring));
        load_consts(ph(w + 2), more);  // step w+1 evaluates R of step w+2 (<= L: in range)
        Star fs[NF], rs[NR];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const float* c = &sF(IC<SC>{})[f][fos];
            const float fnext = sF(IC<SN>{})[f][fos];
            fs[f].c = c[0];
            fs[f].m[0] = REV ? fnext : fzm[f];
            fs[f].p[0] = REV ? fzm[f] : fnext;
            fs[f].m[DIM - 1] = c[-1];
            fs[f].p[DIM - 1] = c[1];
            if (DIM == 3) {
                fs[f].m[1] = c[-FLX];
                fs[f].p[1] = c[FLX];
            }
        }
#pragma unroll
        for (int b = 0; b < NR; ++b) {
            const float* c = &sR[RC][b][ros];
            rs[b].c = rzc[b];
            rs[b].m[0] = REV ? rzp[b] : rzm[b];
            rs[b].p[0] = REV ? rzm[b] : rzp[b];
            rs[b].m[DIM - 1] = c[-1];
            rs[b].p[DIM - 1] = c[1];
            if (DIM == 3) {
                rs[b].m[1] = c[-RLX];
                rs[b].p[1] = c[RLX];
            }
        }
        if (LOSS) {  // R of step w (zero off the residual set); a lane past the
                     // grid's edge holds a wrapped duplicate on a periodic grid
            float ss = 0.f;
#pragma unroll
            for (int b = 0; b < NR; ++b) ss = fmaf(rzc[b], rzc[b], ss);
            acc += (double)(inarr ? ss : 0.f);
            asm volatile("" : "+v"(acc));
        }
        float g[NF];
        OP::gather_rest(fs, rs, sgc, K, g);
        {
            const int pz = ph(w);
            const uint32_t so = inarr ? cb : kDropOff;
#pragma unroll
            for (int f = 0; f < NF; ++f)
                bst<kStream>(plane_rsrc(P.out[f], pz, pbytes), so, scale * g[f]);
        }
#pragma unroll
        for (int f = 0; f < NF; ++f) fzm[f] = fs[f].c;
#pragma unroll
        for (int b = 0; b < NR; ++b) {
            rzm[b] = rzc[b];
            rzc[b] = rzp[b];
        }
#pragma unroll
        for (int q = 0; q < NG; ++q) sgc[q] = sgp[q];
        __syncthreads();  // (waits for the plane loads into LDS as well)
    };

    int w = 0;
    for (; w + 4 <= L; w += 4) {  // slot and buffer indices are constants in each copy
        step(IC<0>{}, w);
        step(IC<1>{}, w + 1);
        step(IC<2>{}, w + 2);
        step(IC<3>{}, w + 3);
    }
    if (w < L) step(IC<0>{}, w);
    if (w + 1 < L) step(IC<1>{}, w + 1);
    if (w + 2 < L) step(IC<2>{}, w + 2);
    if (LOSS) block_atomic_sum<NT>(acc * inv_M, loss);
}

// ---------------------------------------------------------------------------
// 2-D backward with a register queue: no LDS and no barrier.  A row of a 2-D
// grid is a few kilobytes, so the LDS march above waits once per row for a
// barrier and that row's loads.  Here each lane marches one column down its
// chunk of rows, keeping for every field the values at x - 1, x, x + 1 of Q
// rows in registers (each row loaded Q - 5 steps before its first use), and
// its own residuals R of the rows z - 1, z, z + 1.  The gather at (z, x) needs
// R at x -+ 1 as well: the neighbouring lanes hold them, and a DPP wavefront
// shift by one lane brings them over.  So that every lane has both neighbours,
// the two edge lanes of each wave evaluate residuals only (at the columns
// before and after the wave's 62 output columns), and a workgroup of NW waves
// writes 62 NW columns.  Every node of the marched rows is written once, the
// boundary columns included (R is zero off the residual set); no atomics.

// v of lane i - 1 (wave_shr:1) or of lane i + 1 (wave_shl:1); the lanes at the
// wave's ends receive 0
__device__ __forceinline__ float lane_prev(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x138, 0xF, 0xF, false));
}
__device__ __forceinline__ float lane_next(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x130, 0xF, 0xF, false));
}

template <class OP, int NW, int Q, bool PER>
__global__ __launch_bounds__(NW * 64) void bwdq_kernel(Ptrs P, Dims D, KCoef K, const double* dloss,
                                                     double two_over_M) {
    constexpr int NF = OP::NF, NC = OP::NC, NR = OP::NR, NG = OP::NG;
    constexpr int NC1 = NC > 0 ? NC : 1, NG1 = NG > 0 ? NG : 1;
    constexpr int TXO = 62 * NW;  // output columns per workgroup
    static_assert(OP::DIM == 2, "rows of a 2-D grid");
    static_assert(Q >= 6, "rows z - 1 .. z + 2 in use and at least one row in flight");
    constexpr uint32_t kOff = 0x80000000u;  // past every row's range: reads 0
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    const TileCoord tc = tile_coord<TXO, 1>(D);
    const int z0 = tc.z0, z1 = tc.z1, L = z1 - z0;
    const int c = tc.gx0 + wv * 62 + lane - 1;  // this lane's column (-1 .. past the grid)
    const bool out_lane = lane >= 1 && lane <= 62 && c < D.nx;  // writes a gradient
    // the lane's residual is that of its column, or of the wrapped column on a
    // periodic grid (the edge lanes hold the x -+ 1 residuals of the output lanes)
    const bool own_om = PER ? (c >= -D.nx && c < 2 * D.nx) : (c >= 1 && c <= D.nx - 2);
    const uint32_t pbytes = (uint32_t)D.nx * 4u;
    auto at = [&](int x) -> uint32_t {
        if (PER) return (uint32_t)wrap_idx(x, D.nx) * 4u;
        return (x >= 0 && x < D.nx) ? (uint32_t)x * 4u : kOff;
    };
    const uint32_t off[3] = {at(c - 1), at(c), at(c + 1)};
    const uint32_t so = out_lane ? (uint32_t)c * 4u : kDropOff;
    const float scale = (float)(two_over_M * (*dloss));

    // the queue: row z0 - 2 + k lives in slot k % Q; rows z0 - 2 .. z1 + 1 are read
    float qv[Q][NF][3], qk[Q][NC1];
    auto load_row = [&](int k, auto slot) __attribute__((always_inline)) {
        constexpr int S_ = decltype(slot)::value;
        const int z = z0 - 2 + k;
        const bool ok = z <= z1 + 1 && (PER || (z >= 0 && z < D.nz));
        const int zr = PER ? wrap_idx(z, D.nz) : z;
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const __amdgpu_buffer_rsrc_t r = plane_rsrc_if(P.f[f], zr, pbytes, ok);
#pragma unroll
            for (int v = 0; v < 3; ++v) qv[S_][f][v] = bld(r, off[v]);
        }
#pragma unroll
        for (int j = 0; j < NC; ++j) qk[S_][j] = bld(plane_rsrc_if(P.c[j], zr, pbytes, ok), off[1]);
    };
    // R at the row of slot K1 from the rows of slots K0, K1, K2 (zero off the
    // residual set), and the gather's self terms there
    auto r_row = [&](auto k0, auto k1, auto k2, int z, float* R, float* S) __attribute__((always_inline)) {
        constexpr int A = decltype(k0)::value, B = decltype(k1)::value, C = decltype(k2)::value;
        Star s[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            s[f].c = qv[B][f][1];
            s[f].m[0] = qv[A][f][1];
            s[f].p[0] = qv[C][f][1];
            s[f].m[1] = qv[B][f][0];
            s[f].p[1] = qv[B][f][2];
        }
        OP::residual(s, qk[B], K, R);
        const bool om = own_om && (PER || (z >= 1 && z <= D.nz - 2));
#pragma unroll
        for (int b = 0; b < NR; ++b) R[b] = om ? R[b] : 0.f;
        OP::gather_self(s, R, K, S);
    };

    unroll_seq([&](auto k) __attribute__((always_inline)) {
        load_row(decltype(k)::value, k);
    }, std::make_integer_sequence<int, Q - 1>{});
    float Rm[NR], Rc[NR], Sm[NG1], Sc[NG1];
    r_row(IC<0>{}, IC<1>{}, IC<2>{}, z0 - 1, Rm, Sm);
    r_row(IC<1>{}, IC<2>{}, IC<3>{}, z0, Rc, Sc);

    auto step = [&](auto jc, int w) __attribute__((always_inline)) {
        constexpr int J = decltype(jc)::value;  // w % Q
        // slots of the rows z - 1, z, z + 1, z + 2 (k = w + 1 .. w + 4), and of the row
        // loaded now (k = w + Q - 1, in the slot of row z - 3, last read a step ago)
        constexpr int K1 = (J + 1) % Q, K2 = (J + 2) % Q, K3 = (J + 3) % Q, K4 = (J + 4) % Q;
        constexpr int KN = (J + Q - 1) % Q;
        const int z = z0 + w;
        load_row(w + Q - 1, IC<KN>{});
        float Rp[NR], Sp[NG1];
        r_row(IC<K2>{}, IC<K3>{}, IC<K4>{}, z + 1, Rp, Sp);
        Star fs[NF], rs[NR];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            fs[f].c = qv[K2][f][1];
            fs[f].m[0] = qv[K1][f][1];
            fs[f].p[0] = qv[K3][f][1];
            fs[f].m[1] = qv[K2][f][0];
            fs[f].p[1] = qv[K2][f][2];
        }
#pragma unroll
        for (int b = 0; b < NR; ++b) {
            rs[b].c = Rc[b];
            rs[b].m[0] = Rm[b];
            rs[b].p[0] = Rp[b];
            rs[b].m[1] = lane_prev(Rc[b]);
            rs[b].p[1] = lane_next(Rc[b]);
        }
        float g[NF];
        OP::gather_rest(fs, rs, Sc, K, g);
        const int zr = PER ? wrap_idx(z, D.nz) : z;
#pragma unroll
        for (int f = 0; f < NF; ++f) bst<kStream>(plane_rsrc(P.out[f], zr, pbytes), so, scale * g[f]);
#pragma unroll
        for (int b = 0; b < NR; ++b) {
            Rm[b] = Rc[b];
            Rc[b] = Rp[b];
        }
#pragma unroll
        for (int q = 0; q < NG; ++q) Sc[q] = Sp[q];
        (void)Sm;
    };

    int w = 0;
    for (; w + Q <= L; w += Q)  // slot indices are constants in each copy
        unroll_seq([&](auto j) __attribute__((always_inline)) {
            step(j, w + decltype(j)::value);
        }, std::make_integer_sequence<int, Q>{});
    unroll_seq([&](auto j) __attribute__((always_inline)) {
        if (w + decltype(j)::value < L) step(j, w + decltype(j)::value);
    }, std::make_integer_sequence<int, Q - 1>{});
}

// ---------------------------------------------------------------------------
// Explicit-sensitivity backward: grads (=, or += when ACC) J^T G for caller-given
// residual sensitivities G_b = dL/dR_b (Sec. 2.2).  The gather is the one above
// with G in place of the recomputed residuals, so no residual, const or ring is
// needed: the fields the Jacobian depends on (OP::NFG of them: none for a linear
// operator, no pressure for NS) and the sensitivities, each with a radius-1
// halo, stream through one LDS ring with the forward's slot layout, and the
// march covers every plane 0..nz-1, writing
// every node once (boundary shell included: G is zero off the residual set,
// which the loads enforce with out-of-range offsets, whatever the arrays hold
// there).

template <class OP, int TX, int TY, bool ACC, bool PER>
__global__ __launch_bounds__(TX* TY, FPDE_VJP_MINW) void vjp_kernel(Ptrs P, Dims D, KCoef K) {
    constexpr int DIM = OP::DIM, NF = OP::NF, NR = OP::NR, NT = TX * TY;
    constexpr int NFG = OP::NFG;  // fields the Jacobian depends on (the others are not read)
    static_assert(NT <= 1024, "a workgroup holds at most 1024 threads");
    constexpr int NA = NFG + NR;  // arrays per slot: those fields, then the sensitivities
    constexpr int HY = (DIM == 3) ? 1 : 0;
    constexpr int LY = TY + 2 * HY, LX = TX, XG = LY * LX;
    static_assert(TX % 64 == 0, "a wavefront loads whole aligned row segments");
    static_assert(2 * TY <= 64, "the side-edge neighbours fill one 64-element group");
    using PS = PlaneStream<XG + 64, NT>;
    static_assert(DIM == 3 || TY == 1, "2-D grids use one-row tiles");
    FPDE_SLOT_RING(float, sF, NA, PS::FSZS);

    const int t = threadIdx.x, tx = t % TX, ty = t / TX;
    FPDE_POISON_RING(sF);
    if (FPDE_LDS_POISON) __syncthreads();
    const TileCoord tc = tile_coord<TX, TY>(D);  // (D.zlo = 0: every plane)
    // 3D+t grids: the sensitivities of the velocity residuals at the own node of
    // the neighbouring time levels (the time part of the transposed stencil),
    // read as 0 off the residual set
    const float* st[2][3] = {};
    bool lok[2] = {false, false};
    if constexpr (OP::TIME) {
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            int l = tc.lev + (k ? 1 : -1);
            lok[k] = PER || (l >= 1 && l <= D.nt - 2);
            l = l < 0 ? l + D.nt : (l >= D.nt ? l - D.nt : l);
#pragma unroll
            for (int q = 0; q < 3; ++q) st[k][q] = P.s[q] + (long long)l * D.vol;
        }
    }
    time_level<OP>(P, D, tc.lev);
    const int z0 = tc.z0, z1 = tc.z1, L = z1 - z0;
    const int gx = tc.gx0 + tx, gy = (DIM == 3) ? tc.gy0 + ty : 0;
    const uint32_t pbytes = (uint32_t)D.ny * (uint32_t)D.nx * 4u;
    const bool inarr = gx < D.nx && gy < D.ny;
    const uint32_t cb = inarr ? (uint32_t)(gy * D.nx + gx) * 4u : 0u;
    auto zw = [&](int z) { return PER ? wrap_idx(z, D.nz) : z; };  // plane index
    // own node on the residual set in the plane (the time-neighbour loads)
    const uint32_t cbo =
        (inarr && (PER || (gx >= 1 && gx <= D.nx - 2 && (DIM == 2 || (gy >= 1 && gy <= D.ny - 2)))))
            ? cb
            : 0x80000000u;

    // slot element -> grid position (the forward's layout); for the
    // sensitivities, positions off the residual set read as 0
    auto node_at = [&](int i, int& lin, bool omega) {
        int py, px;
        if (i < XG) {
            py = (DIM == 3) ? tc.gy0 - HY + i / LX : 0;
            px = tc.gx0 + i % LX;
        } else {
            const int j = i - XG, side = j / TY;
            py = (DIM == 3) ? tc.gy0 + j % TY : 0;
            px = side == 0 ? tc.gx0 - 1 : tc.gx0 + TX;
            if (side > 1) return false;
        }
        if (PER) {
            px = wrap_idx(px, D.nx);
            py = wrap_idx(py, D.ny);
        }
        lin = py * D.nx + px;
        if (omega && !PER)
            return px >= 1 && px <= D.nx - 2 && (DIM == 2 || (py >= 1 && py <= D.ny - 2));
        return px >= 0 && px < D.nx && py >= 0 && py < D.ny;
    };
    PS psf, psg;
    if constexpr (NFG > 0) psf.init(t, [&](int i, int& lin) { return node_at(i, lin, false); });
    psg.init(t, [&](int i, int& lin) { return node_at(i, lin, true); });
    // plane pz (wrapped or -1) of the fields and the sensitivities into a slot;
    // the sensitivities of a plane off the residual set read as 0
    // (3D+t: the end time levels hold no residual node, so none of their
    // sensitivities is read either)
    const bool lev_om = !OP::TIME || PER || (tc.lev >= 1 && tc.lev <= D.nt - 2);
    auto load_plane = [&](int pz, auto slot) __attribute__((always_inline)) {
        float* dst[NA];
#pragma unroll
        for (int a = 0; a < NA; ++a) dst[a] = &sF(slot)[a][0];
        if constexpr (NFG > 0) psf.template load<NFG>(P.f, pz, D.nz, pbytes, dst);
        const bool gok = lev_om && (PER || (pz >= 1 && pz <= D.nz - 2));
        psg.template load<NR>(P.s, gok ? pz : -1, D.nz, pbytes, dst + NFG);
    };
    float gq[2][NF];  // accumulate mode: the stored gradients of the next plane
    auto load_old = [&](int pz, bool ok, float* o) __attribute__((always_inline)) {
        if (ACC) {
#pragma unroll
            for (int f = 0; f < NF; ++f) o[f] = bld(plane_rsrc_if(P.out[f], pz, pbytes, ok), cb);
        }
    };
    float gt[2][2][3];  // 3D+t: [plane slot][t - 1, t + 1][velocity] of the next plane
    auto load_gt = [&](int pz, bool ok, float (*o)[3]) __attribute__((always_inline)) {
        if constexpr (OP::TIME) {
            ok = ok && (PER || (pz >= 1 && pz <= D.nz - 2));
#pragma unroll
            for (int k = 0; k < 2; ++k)
#pragma unroll
                for (int q = 0; q < 3; ++q)
                    o[k][q] = bld(plane_rsrc_if(st[k][q], pz, pbytes, ok && lok[k]), cbo);
        }
    };

    // plane z0 + j lives in slot (j + 1) & 3; prologue: planes z0-1, z0, z0+1
    load_plane(zw(z0 - 1), IC<0>{});
    load_plane(z0, IC<1>{});
    load_plane(zw(z0 + 1), IC<2>{});
    load_old(z0, true, gq[0]);
    load_gt(z0, true, gt[0]);
    __syncthreads();

    const int own = (ty + HY) * LX + tx;  // own node in a slot
    const int xm = tx == 0 ? XG + ty : own - 1, xp = tx == TX - 1 ? XG + TY + ty : own + 1;
    auto star = [&](auto sm, auto sc, auto sp, int a, Star& sv) __attribute__((always_inline)) {
        const float* c = &sF(sc)[a][0];
        sv.c = c[own];
        sv.m[0] = sF(sm)[a][own];
        sv.p[0] = sF(sp)[a][own];
        sv.m[DIM - 1] = c[xm];
        sv.p[DIM - 1] = c[xp];
        if (DIM == 3) {
            sv.m[1] = c[own - LX];
            sv.p[1] = c[own + LX];
        }
    };
    auto step = [&](auto jc, int w) __attribute__((always_inline)) {
        constexpr int J = decltype(jc)::value;  // w & 3
        constexpr int SM = J & 3, SC = (J + 1) & 3, SP = (J + 2) & 3, SQ = (J + 3) & 3;
        constexpr int CUR = J & 1, NXT = (J + 1) & 1;
        const int z = z0 + w;
        const bool more = w + 1 < L;
        // plane z+2 goes to the slot of plane z-2, last read before the previous barrier
        load_plane(more ? zw(z + 2) : -1, IC<SQ>{});
        __builtin_amdgcn_sched_barrier(0);  // (the plane loads first, as in the forward)
        load_old(z + 1, more, gq[NXT]);
        load_gt(zw(z + 1), more, gt[NXT]);
        Star fs[NF] = {}, gs[NR];
#pragma unroll
        for (int f = 0; f < NFG; ++f) star(IC<SM>{}, IC<SC>{}, IC<SP>{}, f, fs[f]);
#pragma unroll
        for (int b = 0; b < NR; ++b) star(IC<SM>{}, IC<SC>{}, IC<SP>{}, NFG + b, gs[b]);
        float g[NF];
        OP::gather(fs, gs, K, g);
        if constexpr (OP::TIME) OP::add_time(gt[CUR][0], gt[CUR][1], K, g);
        const uint32_t so = inarr ? cb : kDropOff;
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            float v = g[f];
            if (ACC) {
                // the stored value plus the action, each rounded on its own: the
                // add is kept apart from the product that formed the action
                asm volatile("" : "+v"(v));
                v = gq[CUR][f] + v;
            }
            bst<kStream>(plane_rsrc(P.out[f], z, pbytes), so, v);
        }
        __syncthreads();  // (waits for the plane loads into LDS as well)
    };

    int w = 0;
    for (; w + 4 <= L; w += 4) {  // slot indices are constants in each copy
        step(IC<0>{}, w);
        step(IC<1>{}, w + 1);
        step(IC<2>{}, w + 2);
        step(IC<3>{}, w + 3);
    }
    if (w < L) step(IC<0>{}, w);
    if (w + 1 < L) step(IC<1>{}, w + 1);
    if (w + 2 < L) step(IC<2>{}, w + 2);
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

// One workgroup per 256-node segment of one row (axis 1 for 3-D grids; the
// single row of a 2-D grid's plane) of one end plane, so that a workgroup's rows
// are uniform: an edge row holds only zeros and loads nothing.  Every load goes
// through a plane's buffer descriptor with a 32-bit byte offset.
template <class OP>
__global__ __launch_bounds__(256) void bc_kernel(Ptrs P, Dims D, KCoef K, const double* dloss,
                                                 double two_over_M) {
    constexpr int DIM = OP::DIM, NF = OP::NF, NC = OP::NC;
    const int segs = (D.nx + 255) / 256;
    int blk = blockIdx.x;
    const int seg = blk % segs;
    blk /= segs;
    const int i1 = blk % D.ny;           // row of the plane (0 for 2-D grids)
    const bool low = blk / D.ny == 0;    // plane 0, else plane nz - 1
    const int i2 = seg * 256 + (int)threadIdx.x;
    if (i2 >= D.nx) return;
    const int zn = low ? 0 : D.nz - 1;   // the node's plane
    const int zm = low ? 1 : D.nz - 2;   // its inward neighbour's (the residual's) plane
    const uint32_t pbytes = (uint32_t)D.ny * (uint32_t)D.nx * 4u;
    const uint32_t off = (uint32_t)(i1 * D.nx + i2) * 4u;
    const bool edge_row = DIM == 3 && (i1 == 0 || i1 == D.ny - 1);
    float g[NF];
#pragma unroll
    for (int f = 0; f < NF; ++f) g[f] = 0.f;
    if (!edge_row && i2 >= 1 && i2 <= D.nx - 2) {
        const uint32_t dy = (uint32_t)D.nx * 4u;
        Star st[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const __amdgpu_buffer_rsrc_t rc = plane_rsrc(P.f[f], zm, pbytes);
            st[f].c = bld(rc, off);
            st[f].m[0] = bld(plane_rsrc(P.f[f], zm - 1, pbytes), off);
            st[f].p[0] = bld(plane_rsrc(P.f[f], zm + 1, pbytes), off);
            st[f].m[DIM - 1] = bld(rc, off - 4u);
            st[f].p[DIM - 1] = bld(rc, off + 4u);
            if (DIM == 3) {
                st[f].m[1] = bld(rc, off - dy);
                st[f].p[1] = bld(rc, off + dy);
            }
        }
        float cc[NC > 0 ? NC : 1];
#pragma unroll
        for (int j = 0; j < NC; ++j) cc[j] = bld(plane_rsrc(P.c[j], zm, pbytes), off);
        OP::template bc_term<0>(st, cc, K, low ? -1.f : 1.f, g);  // node = m + t e_0
        const float scale = (float)(two_over_M * (*dloss));
#pragma unroll
        for (int f = 0; f < NF; ++f) g[f] *= scale;
    }
#pragma unroll
    for (int f = 0; f < NF; ++f) bst<kStream>(plane_rsrc(P.out[f], zn, pbytes), off, g[f]);
}

// ---------------------------------------------------------------------------
// 3D+t grids (operators with TIME).  The marching kernels above run on one time
// level per workgroup: their residuals read the velocities of the neighbouring
// levels as point values, and their gather is the spatial part of the
// transposed stencil.  The time part of the gather,
//     dL/dc_q(n) += (R_q(n - e_t) - R_q(n + e_t)) / (2 h_t),
// needs residuals of other time levels, which another workgroup evaluates.  So
// tm_kernel recomputes them: one lane per spatial node marches the time levels
// and keeps R_q of the levels t - 1, t, t + 1 in registers, so every residual is
// evaluated once; each node's gradient is read, the time part added, and
// written once (the march's spatial part is already there).  Only nodes on the
// spatial residual set have a time part (R is zero off it).
//
// The residual of level L reads the stars at L and the node's velocities at
// L -+ 1, which are the centres of the stars at L -+ 1.  The lane loads the stars
// of each level once, one level ahead of the residual it evaluates, and keeps
// the stars of L + 1 and the centre velocities of L - 1 in registers: a point
// value fetched once for a residual and again, a level later, for a star would
// come from HBM twice, since a whole level of every field passes through L2 in
// between.

// The stars of every field at one spatial node of level lev (lev in range),
// loaded through the level's buffer descriptors (o: the node's byte offset in a
// level, n[6]: its neighbours' at -+ one node along the three spatial axes).
template <class OP>
__device__ __forceinline__ void stars_at_level(const Ptrs& P, int lev, uint32_t vbytes, uint32_t o,
                                               const uint32_t* n, Star* st) {
    constexpr int NF = OP::NF, D3 = OP::D;
#pragma unroll
    for (int f = 0; f < NF; ++f) {
        const __amdgpu_buffer_rsrc_t r = plane_rsrc(P.f[f], lev, vbytes);
        st[f].c = f < D3 ? bld(r, o) : 0.f;  // (the pressure's own value enters no residual)
#pragma unroll
        for (int a = 0; a < D3; ++a) {
            st[f].m[a] = bld(r, n[2 * a]);
            st[f].p[a] = bld(r, n[2 * a + 1]);
        }
    }
}

// Lanes: one per spatial node of a level, 256 consecutive nodes per workgroup,
// in launch order or (FPDE_TM_REMAP) XCD-contiguous.  Each lane marches the
// time levels on its own, so the rows that neighbouring workgroups share meet
// in L2 only while those workgroups run at the same time.  At 20 x 128^3 this
// order was the fastest of the lane blocks tried (2 x 2 x 64 up to 4 x 4 x 64
// nodes, and 128-wide blocks of 1 to 8 rows: 1-8% slower), and the
// XCD-contiguous order 3-4% slower; unlike a block, it leaves no lane idle
// whatever the extent of the last axis.
#ifndef FPDE_TM_REMAP
#define FPDE_TM_REMAP 0
#endif

template <class OP, bool PER>
__global__ __launch_bounds__(256) void tm_kernel(Ptrs P, Dims D, KCoef K, const double* dloss,
                                                 double two_over_M) {
    constexpr int NF = OP::NF, D3 = OP::D;
    static_assert(OP::NC == 2 * D3, "consts: the velocities at t - 1, then at t + 1");
    const int blk = FPDE_TM_REMAP ? remap_xcd((int)blockIdx.x, (int)gridDim.x) : (int)blockIdx.x;
    const int idx = blk * 256 + (int)threadIdx.x;  // (vol < 2^29)
    if (idx >= (int)D.vol) return;
    const int i3 = idx % D.nx, r = idx / D.nx, i2 = r % D.ny, i1 = r / D.ny;
    if (!PER && !(i1 >= 1 && i1 <= D.nz - 2 && i2 >= 1 && i2 <= D.ny - 2 && i3 >= 1 &&
                  i3 <= D.nx - 2))
        return;  // off the spatial residual set: no time part
    const uint32_t vbytes = (uint32_t)D.vol * 4u;
    const uint32_t o = (uint32_t)idx * 4u;
    // neighbours along x (array axis 1), y, z: -+1, wrapped on a periodic grid
    uint32_t n[6];
    {
        const int sx = D.ny * D.nx, sy = D.nx;
        auto at = [&](int a1, int a2, int a3) -> uint32_t {
            if (PER) {
                a1 = wrap_idx(a1, D.nz);
                a2 = wrap_idx(a2, D.ny);
                a3 = wrap_idx(a3, D.nx);
            }
            return (uint32_t)(a1 * sx + a2 * sy + a3) * 4u;
        };
        n[0] = at(i1 - 1, i2, i3);
        n[1] = at(i1 + 1, i2, i3);
        n[2] = at(i1, i2 - 1, i3);
        n[3] = at(i1, i2 + 1, i3);
        n[4] = at(i1, i2, i3 - 1);
        n[5] = at(i1, i2, i3 + 1);
    }
    const float scale = (float)(two_over_M * (*dloss));
    // levels whose gradient gets the time part: those the march wrote (all of
    // them on a periodic grid, else 1 .. nt - 2, whose residual neighbours are
    // the levels 0 .. nt - 1 with R zero at the end levels); nt >= 3
    const int t0 = PER ? 0 : 1, t1 = PER ? D.nt - 1 : D.nt - 2;
    // the march state: the next residual is that of level L, from the stars of
    // L (sc) and the centre velocities of L - 1 (vm) and L + 1 (loaded with the
    // stars of L + 1, which become sc for the next level)
    int L;
    Star sc[NF];
    float vm[D3];
    auto next_R = [&](float* R) __attribute__((always_inline)) {
        if (!PER && L > D.nt - 2) {  // level nt - 1: R = 0 and no level beyond it
#pragma unroll
            for (int q = 0; q < D3; ++q) R[q] = 0.f;
            ++L;
            return;
        }
        Star sn[NF];
        stars_at_level<OP>(P, PER ? wrap_idx(L + 1, D.nt) : L + 1, vbytes, o, n, sn);
        float c[2 * D3], Rf[OP::NR];
#pragma unroll
        for (int b = 0; b < D3; ++b) {
            c[b] = vm[b];
            c[D3 + b] = sn[b].c;
        }
        OP::residual(sc, c, K, Rf);
#pragma unroll
        for (int q = 0; q < D3; ++q) {
            R[q] = Rf[q];
            vm[q] = sc[q].c;
        }
#pragma unroll
        for (int f = 0; f < NF; ++f) sc[f] = sn[f];
        ++L;
    };
    float Rm[D3], Rc[D3], Rp[D3];
    if (PER) {  // from level -1 (= nt - 1): the residual of t0 - 1 is evaluated too
        L = -1;
        stars_at_level<OP>(P, D.nt - 1, vbytes, o, n, sc);
        const int l2 = D.nt - 2;
#pragma unroll
        for (int b = 0; b < D3; ++b) vm[b] = bld(plane_rsrc(P.f[b], l2, vbytes), o);
        next_R(Rm);
    } else {  // R(0) = 0; the march starts at level 1 with the velocities of level 0
        L = 1;
        stars_at_level<OP>(P, 1, vbytes, o, n, sc);
#pragma unroll
        for (int b = 0; b < D3; ++b) {
            vm[b] = bld(plane_rsrc(P.f[b], 0, vbytes), o);
            Rm[b] = 0.f;
        }
    }
    next_R(Rc);
    for (int t = t0; t <= t1; ++t) {
        next_R(Rp);  // R of level t + 1
        float tp[D3] = {};
        OP::add_time(Rm, Rp, K, tp);
#pragma unroll
        for (int q = 0; q < D3; ++q) {
            const __amdgpu_buffer_rsrc_t rg = plane_rsrc(P.out[q], t, vbytes);
            const float g = bld(rg, o);
            bst<kStream>(rg, o, fmaf(scale, tp[q], g));
            Rm[q] = Rc[q];
            Rc[q] = Rp[q];
        }
    }
}

// Boundary-gradient correction on a 3D+t grid: the end time levels t = 0 and
// t = nt - 1 (the end planes of array axis 0), which the level marches do not
// visit.  A node whose only boundary coordinate is t receives the time term of
// its inward neighbour's residuals (level 1 or nt - 2); a node on the spatial
// boundary as well touches no residual node and gets 0.  One workgroup per 256
// consecutive nodes of a level (the first half of the workgroups covers level 0).
template <class OP>
__global__ __launch_bounds__(256) void bc4_kernel(Ptrs P, Dims D, KCoef K, const double* dloss,
                                                  double two_over_M) {
    constexpr int NF = OP::NF, NC = OP::NC, D3 = OP::D;
    const int per_level = (int)((D.vol + 255) / 256);
    const int blk = remap_xcd((int)blockIdx.x, 2 * per_level);  // (neighbours through one L2)
    const bool low = blk < per_level;
    const int idx = (blk - (low ? 0 : per_level)) * 256 + (int)threadIdx.x;
    if (idx >= (int)D.vol) return;
    const int i3 = idx % D.nx, rr = idx / D.nx, i2 = rr % D.ny, i1 = rr / D.ny;
    const int tn = low ? 0 : D.nt - 1;  // the node's level
    const int tm = low ? 1 : D.nt - 2;  // its inward neighbour's (the residual's)
    const uint32_t vbytes = (uint32_t)D.vol * 4u;
    const int sx = D.ny * D.nx, sy = D.nx;
    const uint32_t off = (uint32_t)(i1 * sx + i2 * sy + i3) * 4u;
    float g[NF];
#pragma unroll
    for (int f = 0; f < NF; ++f) g[f] = 0.f;
    if (i1 >= 1 && i1 <= D.nz - 2 && i2 >= 1 && i2 <= D.ny - 2 && i3 >= 1 && i3 <= D.nx - 2 &&
        D.nt >= 3) {
        const uint32_t d[3] = {(uint32_t)sx * 4u, (uint32_t)sy * 4u, 4u};
        Star st[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const __amdgpu_buffer_rsrc_t r = plane_rsrc(P.f[f], tm, vbytes);
            st[f].c = bld(r, off);
#pragma unroll
            for (int a = 0; a < D3; ++a) {
                st[f].m[a] = bld(r, off - d[a]);
                st[f].p[a] = bld(r, off + d[a]);
            }
        }
        float c[NC];
#pragma unroll
        for (int j = 0; j < NC; ++j)
            c[j] = bld(plane_rsrc(P.f[OP::TSRC[j]], tm + OP::TOFF[j], vbytes), off);
        OP::bc_time(st, c, K, low ? -1.f : 1.f, g);
        const float scale = (float)(two_over_M * (*dloss));
#pragma unroll
        for (int f = 0; f < NF; ++f) g[f] *= scale;
    }
#pragma unroll
    for (int f = 0; f < NF; ++f) bst<kStream>(plane_rsrc(P.out[f], tn, vbytes), off, g[f]);
}

// Zeros of the residual arrays on the end time levels of a 3D+t grid (no
// residual node there), for the forward that stores the residuals: the level
// marches write every other node.
template <int NR>
__global__ __launch_bounds__(256) void zero_levels_kernel(Ptrs P, Dims D) {
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= 2 * D.vol) return;
    const long long at = i < D.vol ? i : i - D.vol + (long long)(D.nt - 1) * D.vol;
#pragma unroll
    for (int b = 0; b < NR; ++b) P.out[b][at] = 0.f;
}

}  // namespace fpde
