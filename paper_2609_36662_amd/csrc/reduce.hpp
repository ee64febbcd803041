// Deterministic reductions of per-thread fp64 sums, shared by the streaming
// kernels.  Every stage adds in a fixed order (wavefront butterfly, the waves
// of a workgroup in index order through LDS, then the workgroups' partials in
// index order in a one-workgroup finishing kernel), so with a fixed grid the
// result is the same bit for bit on every run.
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

// Stage 1: this workgroup's sums into partials[blockIdx.x][NS] with plain
// stores.  Stage 2 is finish_sums_kernel, launched after the producing kernel
// on the same stream (the stream order makes the partials visible to it), so
// no workgroup takes a device-scope fence or a ticket at its end.
template <int NS, int NT>
__device__ __forceinline__ void store_partials(double (&acc)[NS], double* partials) {
    __shared__ double lds[kMaxWaves * kMaxSums];
    const double part = block_reduce<NS, NT>(acc, lds);
    if (threadIdx.x < NS) partials[(int64_t)blockIdx.x * NS + threadIdx.x] = part;
}

// Stage 2, one workgroup of NT threads (NT = the producer's workgroup size):
// thread t adds the partials of workgroups t, t + NT, ... in that order, then
// the workgroup reduces those as in stage 1; sums[0..NS) receives the totals.
template <int NS, int NT>
__global__ void __launch_bounds__(NT) finish_sums_kernel(const double* partials, int nblocks, double* sums,
                                                         double* host_copy) {
    __shared__ double lds[kMaxWaves * kMaxSums];
    double tot[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) tot[j] = 0.0;
    for (int b = threadIdx.x; b < nblocks; b += NT) {
#pragma unroll
        for (int j = 0; j < NS; ++j) tot[j] += partials[(int64_t)b * NS + j];
    }
    const double fin = block_reduce<NS, NT>(tot, lds);
    if (threadIdx.x < NS) {
        sums[threadIdx.x] = fin;
        if (host_copy != nullptr) host_copy[threadIdx.x] = fin;
    }
}

// Launches finish_sums_kernel for ns in 1..kMaxSums and nt in {256, 512};
// host_copy (may be null): a device view of coherent host memory that receives
// the sums as well, so no copy is needed to bring them to the host.
hipError_t launch_finish_sums(int ns, int nt, int nblocks, const double* partials, double* sums,
                              hipStream_t stream, double* host_copy = nullptr);

}  // namespace autoloco
