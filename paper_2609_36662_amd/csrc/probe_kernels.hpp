// Streaming-pattern probes (measurement only; no operation of the paper).
//
// A probe moves the bytes of a set of streams with no arithmetic, so its time
// is what the device sustains for that access pattern: the practical ceiling
// of a kernel that makes the same loads and stores.  Streams come in five
// classes, in this order in the argument list:
//   A  4-byte streams read and written back in place (unchanged contents),
//   B  4-byte streams read,
//   C  2-byte streams read,
//   D  2-byte streams written: the upper halves of stream 0's words,
//   E  4-byte streams written: stream 0's words,
// and the counts of the classes are template parameters, so every load and
// store is straight-line code (with runtime per-stream branches the compiler
// waits for each store before the next).  When no stream is read, written
// streams receive the index of each run of 4.  Words of read-only streams are
// folded into one value per lane that decides an improbable store, so no load
// can be dropped.
//
// Shapes:
//   run      the round kernel's window loop: a lane owns R runs of 4 elements
//            per window (R = 1: one run, the fp32 round's; R = 2: two runs 256
//            apart, the bf16 round's and the per-GPU kernels'; R = 8: eight
//            runs 256 apart, the standalone reset's with three or more fp32
//            replicas), at a 32-bit offset from a wave-uniform window base;
//   serial   a workgroup stages a tile of every read stream in LDS with direct
//            global-to-LDS loads, stream after stream, waiting for stream s
//            before it issues stream s + 2 (two streams' loads in flight per
//            workgroup at most), then stores the tile stream by stream;
//   tile     the same tiles with every stream's loads issued at once, waited
//            for together, then stored: read and write phases of up to 160 KB
//            per workgroup;
//   phased   read and write phases of the whole grid: every workgroup loads
//            its tile of every stream (3 runs of 4 per lane into LDS with
//            direct loads, 4 more into registers: 280 KB per workgroup over ten
//            streams), waits for them, meets every other workgroup at a grid
//            barrier, stores the tile, waits, and meets them again, so the
//            device reads and writes in alternating phases of about 70 MB
//            (cooperative launch, one workgroup per compute unit).
// Run shapes skip the last n mod 4 elements, tile shapes the elements past the
// last whole tile (4 runs of 4 per lane: 4,096 elements).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "round_kernels.hpp"

namespace autoloco {

constexpr int kProbeMaxStreams = 18;          // theta, v and 16 replicas
constexpr int kProbeTileStreams = 10;         // the tile shapes' LDS holds this many
constexpr int kProbeTileQuads = 4;            // runs of 4 per lane per stream per tile
constexpr int kProbePieces = 40;              // LDS pieces of 4 KB (one run per lane of a workgroup)

enum ProbeShape { PROBE_RUN = 0, PROBE_SERIAL = 1, PROBE_TILE = 2, PROBE_PHASED = 3 };

struct ProbeArgs {
    void* ptr[kProbeMaxStreams];
    int64_t n;                          // elements per stream
    uint32_t sentinel;                  // the improbable value that triggers the sink store
    uint32_t mask;                      // 0: XORed into words written back in place, so the
                                        // compiler cannot drop a store of the word it loaded
    uint32_t* sink;                     // [gridDim.x]
};

// Upper halves of two 32-bit words packed into one (2-byte copy of a 4-byte stream).
__device__ __forceinline__ uint32_t hi_pair(uint32_t lo, uint32_t hi) { return (lo >> 16) | (hi & 0xffff0000u); }

// Window loop, R runs of 4 elements per lane per window.
template <int R, int A, int B, int C, int D, int E>
__global__ void __launch_bounds__(kBlock) probe_run_kernel(ProbeArgs a) {
    constexpr int N4 = A + B;                  // 4-byte streams read (classes A, B)
    constexpr bool SRC = N4 > 0;               // stream 0 feeds the written streams
    const int64_t nq = a.n / 4;
    const int64_t qstride = (int64_t)gridDim.x * kBlock * R;
    uint32_t fold = 0;
    for (int64_t qb = (int64_t)blockIdx.x * kBlock * R; qb < nq; qb += qstride) {
        if (qb + threadIdx.x >= nq) continue;
        const bool full = qb + (int64_t)kBlock * R <= nq;     // wave-uniform: every run in range
        u32x4 w4[N4 > 0 ? N4 : 1][R];
        u32x2r w2[C > 0 ? C : 1][R];
#pragma unroll
        for (int h = 0; h < R; ++h) {
            if (h > 0 && !full && qb + h * kBlock + threadIdx.x >= nq) continue;
            const uint32_t run = h * kBlock + threadIdx.x;
#pragma unroll
            for (int s = 0; s < N4; ++s) w4[s][h] = ld_u4_at(static_cast<const uint32_t*>(a.ptr[s]) + qb * 4, run * 16u);
#pragma unroll
            for (int s = 0; s < C; ++s)
                w2[s][h] = ld_u2_at(static_cast<const uint16_t*>(a.ptr[N4 + s]) + qb * 4, run * 8u);
        }
#pragma unroll
        for (int h = 0; h < R; ++h) {
            if (h > 0 && !full && qb + h * kBlock + threadIdx.x >= nq) continue;
            const uint32_t run = h * kBlock + threadIdx.x;
            const uint32_t x = (uint32_t)qb + run;
#pragma unroll
            for (int s = 0; s < A; ++s)
                st_u4_at(static_cast<uint32_t*>(a.ptr[s]) + qb * 4, run * 16u, w4[s][h] ^ a.mask);
#pragma unroll
            for (int s = A; s < N4; ++s) fold ^= w4[s][h][0] ^ w4[s][h][1] ^ w4[s][h][2] ^ w4[s][h][3];
#pragma unroll
            for (int s = 0; s < C; ++s) fold ^= w2[s][h][0] ^ w2[s][h][1];
#pragma unroll
            for (int s = 0; s < D; ++s) {
                u32x2r v = {x, x};
                if constexpr (SRC) v = u32x2r{hi_pair(w4[0][h][0], w4[0][h][1]), hi_pair(w4[0][h][2], w4[0][h][3])};
                st_u2_at(static_cast<uint16_t*>(a.ptr[N4 + C + s]) + qb * 4, run * 8u, v);
            }
#pragma unroll
            for (int s = 0; s < E; ++s) {
                u32x4 v = {x, x, x, x};
                if constexpr (SRC) v = w4[0][h];
                st_u4_at(static_cast<uint32_t*>(a.ptr[N4 + C + D + s]) + qb * 4, run * 16u, v);
            }
        }
    }
    if (fold == a.sentinel) a.sink[blockIdx.x] = fold;
}

// vmcnt wait with the other counters left alone (gfx9 encoding: vmcnt in bits
// 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
#define AUTOLOCO_WAIT_VMCNT(c) __builtin_amdgcn_s_waitcnt(((c) & 0xF) | (((c) >> 4) << 14) | 0x70 | 0xF00)

// Tile shapes, 4-byte streams of classes A (in place), B (read) and E
// (written).  Run u of wave w covers quads [u * 256 + w * 64, +64) of the tile
// and lands in LDS piece (stream * 4 + u), at the wave's 1 KB slice of it.  A
// wave reads back only what it loaded itself, so no barrier is needed between
// the direct loads and the LDS reads once the wave's own counter shows them
// complete.
template <bool SERIAL, int A, int B, int E>
__global__ void __launch_bounds__(kBlock) probe_tile_kernel(ProbeArgs a) {
    constexpr int U = kProbeTileQuads;
    constexpr int NR = A + B;                  // streams loaded into LDS
    static_assert(NR * U <= kProbePieces && NR + E <= kProbeTileStreams, "LDS holds the tile");
    __shared__ u32x4 lds[(NR > 0 ? NR : 1) * U * kBlock];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    constexpr int64_t tq = (int64_t)U * kBlock;    // quads per stream per tile
    const int64_t ntiles = a.n / 4 / tq;
    uint32_t fold = 0;
    for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const int64_t w0 = t * tq * 4;             // first element of the tile
#pragma unroll
        for (int s = 0; s < NR; ++s) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t* src = static_cast<const uint32_t*>(a.ptr[s]) + w0 + (int64_t)(u * kBlock + threadIdx.x) * 4;
                __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)src,
                                                 (void __attribute__((address_space(3)))*)(lds + (s * U + u) * kBlock + wave * 64),
                                                 16, 0, 0);
            }
            // SERIAL: before the next stream is issued, the one before this has
            // landed (at most U loads, this stream's, still out; anything issued
            // earlier, the last tile's stores included, has completed, by
            // in-order completion), so two streams at most are in flight.
            if constexpr (SERIAL) {
                if (s >= 1) AUTOLOCO_WAIT_VMCNT(U);
            }
        }
        AUTOLOCO_WAIT_VMCNT(0);                    // every piece of this tile is in LDS
        __asm__ volatile("" ::: "memory");         // no LDS read moves above the wait
#pragma unroll
        for (int s = 0; s < NR + E; ++s) {
            const int from = s < NR ? s : 0;
            u32x4 x[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (NR > 0) {
                    x[u] = lds[(from * U + u) * kBlock + wave * 64 + lane];
                } else {
                    const uint32_t i = (uint32_t)(t * tq) + u * kBlock + threadIdx.x;
                    x[u] = u32x4{i, i, i, i};
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (s >= A && s < NR)
                    fold ^= x[u][0] ^ x[u][1] ^ x[u][2] ^ x[u][3];
                else
                    st_u4_at(static_cast<uint32_t*>(a.ptr[s]) + w0, (uint32_t)(u * kBlock + threadIdx.x) * 16u,
                             x[u] ^ a.mask);
            }
        }
        // the LDS reads above have returned before the next tile's direct
        // loads overwrite the pieces
        __builtin_amdgcn_s_waitcnt(0xC07F);        // lgkmcnt(0)
        __asm__ volatile("" ::: "memory");
    }
    AUTOLOCO_WAIT_VMCNT(0);
    if (fold == a.sentinel) a.sink[blockIdx.x] = fold;
}

// Phased shape: runs of 4 per lane per stream per tile held in LDS and in
// registers, and the polls after which a grid barrier gives up.
constexpr int kPhaseLdsRuns = 3;
constexpr int kPhaseRegRuns = 4;
constexpr int kPhaseStreams = 10;
constexpr uint32_t kPhaseSpin = 1u << 22;

// Grid barrier of a cooperative launch (every workgroup resident at once).
// sync[0] counts arrivals over the whole launch (target: the barrier's number
// times the grid), sync[1] is set by a workgroup that gave up.  Thread 0 adds
// its arrival and polls, sleeping between polls; after kPhaseSpin polls, or as
// soon as another workgroup has given up, it sets sync[1] and reports failure,
// and every workgroup then leaves its loop, so the grid always drains.  The
// decision reaches the workgroup's other threads through LDS, so they all take
// the same branch.  Vector memory atomics only.
__device__ __forceinline__ bool phase_barrier(uint32_t* sync, uint32_t target, uint32_t* ok) {
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t good = 1;
        __hip_atomic_fetch_add(sync, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        for (uint32_t i = 0; __hip_atomic_load(sync, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target; ++i) {
            if (i >= kPhaseSpin || __hip_atomic_load(sync + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
                __hip_atomic_store(sync + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                good = 0;
                break;
            }
            __builtin_amdgcn_s_sleep(2);
        }
        *ok = good;
    }
    __syncthreads();
    return *ok != 0;
}

// Phased shape, A 4-byte streams read and written back in place.  Tile t
// (workgroup b's in round r: t = r * grid + b) covers 7 * 256 quads of every
// stream; run u of lane i is quad u * 256 + i.  Only whole rounds of tiles over
// the grid are moved (every workgroup meets every barrier).
template <int A>
__global__ void __launch_bounds__(kBlock, 1) probe_phase_kernel(ProbeArgs a, uint32_t* sync) {
    constexpr int UL = kPhaseLdsRuns, UR = kPhaseRegRuns, U = UL + UR;
    __shared__ u32x4 lds[A * UL * kBlock];
    __shared__ uint32_t ok;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    constexpr int64_t tq = (int64_t)U * kBlock;
    const int64_t rounds = a.n / 4 / tq / gridDim.x;
    uint32_t target = 0;
    for (int64_t r = 0; r < rounds; ++r) {
        const int64_t w0 = (r * gridDim.x + blockIdx.x) * tq * 4;
        u32x4 x[A][UR];
#pragma unroll
        for (int s = 0; s < A; ++s) {
#pragma unroll
            for (int u = 0; u < UL; ++u) {
                const uint32_t* src = static_cast<const uint32_t*>(a.ptr[s]) + w0 + (int64_t)(u * kBlock + threadIdx.x) * 4;
                __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)src,
                                                 (void __attribute__((address_space(3)))*)(lds + (s * UL + u) * kBlock + wave * 64),
                                                 16, 0, 0);
            }
#pragma unroll
            for (int u = 0; u < UR; ++u)
                x[s][u] = ld_u4_at(static_cast<const uint32_t*>(a.ptr[s]) + w0, (uint32_t)((UL + u) * kBlock + threadIdx.x) * 16u);
        }
        // the read phase ends when this workgroup's loads have all landed
        __asm__ volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0);
        __asm__ volatile("" ::: "memory");
        target += gridDim.x;
        if (!phase_barrier(sync, target, &ok)) break;
#pragma unroll
        for (int s = 0; s < A; ++s) {
#pragma unroll
            for (int u = 0; u < UL; ++u)
                st_u4_at(static_cast<uint32_t*>(a.ptr[s]) + w0, (uint32_t)(u * kBlock + threadIdx.x) * 16u,
                         lds[(s * UL + u) * kBlock + wave * 64 + lane] ^ a.mask);
#pragma unroll
            for (int u = 0; u < UR; ++u)
                st_u4_at(static_cast<uint32_t*>(a.ptr[s]) + w0, (uint32_t)((UL + u) * kBlock + threadIdx.x) * 16u,
                         x[s][u] ^ a.mask);
        }
        // the write phase ends when the stores are done (and the LDS reads have
        // returned, before the next round's direct loads reuse the pieces)
        __asm__ volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0);
        __asm__ volatile("" ::: "memory");
        target += gridDim.x;
        if (!phase_barrier(sync, target, &ok)) break;
    }
}

// Launches the phased probe over kPhaseStreams streams in place as a
// cooperative launch; sync: two zeroed words (see phase_barrier).
hipError_t launch_probe_phased(int blocks, hipStream_t stream, const ProbeArgs& a, uint32_t* sync);
// Workgroups of the phased probe that fit on one compute unit.
int probe_phased_occupancy();

// One instantiated pattern: shape, runs per lane (run shape), class counts.
struct ProbePattern {
    int shape, r, a, b, c, d, e;
};

// Whether an instance matches p exactly.
bool probe_available(const ProbePattern& p);
// Launches the instance that matches p exactly; hipErrorInvalidValue if none.
hipError_t launch_probe(const ProbePattern& p, int blocks, hipStream_t stream, const ProbeArgs& a);

}  // namespace autoloco
