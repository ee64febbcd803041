// Deterministic reductions of per-thread fp64 sums, shared by the streaming
// kernels.  Every stage adds in a fixed order (wavefront butterfly, the waves
// of a workgroup in index order through LDS, the workgroups in index order in
// the last workgroup to finish), so with a fixed grid the result is the same
// bit for bit on every run.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace autoloco {

constexpr int kMaxK = 16;
constexpr int kMaxSums = 2 * kMaxK + 1;
constexpr int kMaxWaves = 16;  // up to 1024 threads per workgroup

// Sums acc[0..NS) over a workgroup of NT threads; thread j < NS returns sum j.
template <int NS, int NT>
__device__ __forceinline__ double block_reduce(double (&acc)[NS], double* lds) {
    constexpr int NW = NT / 64;
#pragma unroll
    for (int j = 0; j < NS; ++j) {
        double v = acc[j];
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
        acc[j] = v;
    }
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    if (lane == 0) {
#pragma unroll
        for (int j = 0; j < NS; ++j) lds[wave * NS + j] = acc[j];
    }
    __syncthreads();
    double t = 0.0;
    if (threadIdx.x < NS) {
        t = lds[threadIdx.x];
#pragma unroll
        for (int w = 1; w < NW; ++w) t += lds[w * NS + threadIdx.x];
    }
    __syncthreads();
    return t;
}

// Stage 1 writes this workgroup's partial sums; the last workgroup to arrive
// (agent-scope ticket) adds all partials in workgroup order into sums[] and
// resets the ticket for the next launch.
template <int NS, int NT>
__device__ __forceinline__ void grid_reduce(double (&acc)[NS], double* partials, unsigned int* ticket,
                                            double* sums) {
    __shared__ double lds[kMaxWaves * kMaxSums];
    __shared__ int is_last;
    const double part = block_reduce<NS, NT>(acc, lds);
    if (threadIdx.x < NS)
        __hip_atomic_store(&partials[(int64_t)blockIdx.x * NS + threadIdx.x], part, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        const unsigned int prev = __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        is_last = (prev == gridDim.x - 1);
    }
    __syncthreads();
    if (!is_last) return;
    __threadfence();
    double tot[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) tot[j] = 0.0;
    for (unsigned int b = threadIdx.x; b < gridDim.x; b += NT) {
#pragma unroll
        for (int j = 0; j < NS; ++j)
            tot[j] += __hip_atomic_load(&partials[(int64_t)b * NS + j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const double fin = block_reduce<NS, NT>(tot, lds);
    if (threadIdx.x < NS) sums[threadIdx.x] = fin;
    if (threadIdx.x == 0) __hip_atomic_store(ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace autoloco
