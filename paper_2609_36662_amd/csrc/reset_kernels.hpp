// Standalone replica reset (Alg. "AutoLoCo outer interval": every worker
// starts the next interval from the synchronised parameters) on gfx950: theta
// read once, every replica written once (bf16 replicas rounded to nearest
// even).  Bound by HBM bandwidth; no arithmetic beyond the bf16 narrowing.
#pragma once

#include "round_kernels.hpp"

namespace autoloco {

// Quad q of the span at element wb written into every replica.
template <int K, int RT>
__device__ __forceinline__ void store_quad(const RoundArgs& a, int64_t wb, uint32_t q, f32x4 t) {
    if constexpr (RT == RT_F32) {
#pragma unroll
        for (int k = 0; k < K; ++k) st_f4_at(static_cast<float*>(a.replicas[k]) + wb, q * 16u, t);
    } else {
        const u32x2r w = {bf16_pack(t[0], t[1]), bf16_pack(t[2], t[3])};
#pragma unroll
        for (int k = 0; k < K; ++k) st_u2_at(static_cast<uint16_t*>(a.replicas[k]) + wb, q * 8u, w);   // bf16: 8 B a quad
    }
}

// theta_k <- theta for every replica.  A workgroup takes U consecutive windows
// of 256 quads of theta per iteration (U * 4 KB), loads them all, then writes
// them into every replica, so that each replica receives one contiguous run of
// U * 4 KB (fp32) or U * 2 KB (bf16) per workgroup and iteration.  A lane owns
// quad u * 256 + lane of the span, at a 32-bit offset from the wave-uniform
// span base, so every load and store instruction of a wavefront covers one
// contiguous run (1 KB of theta, 1 KB of an fp32 replica, 512 B of a bf16 one).
// The launcher picks U per replica type and K (longer runs pay off for
// three or more fp32 replicas, whose writes dominate the traffic).
template <int K, int RT, int U>
__global__ void __launch_bounds__(kBlock) reset_kernel(RoundArgs a) {
    const int64_t nq = a.n / 4;
    constexpr int64_t span = (int64_t)kBlock * U;      // quads per workgroup and iteration
    const int64_t qstride = (int64_t)gridDim.x * span;
    const int64_t gtid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    for (int64_t qb = (int64_t)blockIdx.x * span; qb < nq; qb += qstride) {
        const int64_t wb = qb * 4;                     // element index of the span's first quad
        if (qb + span <= nq) {                         // a whole span (wave-uniform): no per-lane test
            f32x4 t[U];
#pragma unroll
            for (int u = 0; u < U; ++u) t[u] = ld_f4_at(a.theta + wb, (u * kBlock + threadIdx.x) * 16u);
#pragma unroll
            for (int u = 0; u < U; ++u) store_quad<K, RT>(a, wb, u * kBlock + threadIdx.x, t[u]);
        } else {                                       // the last, shorter span: quad by quad
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t q = u * kBlock + threadIdx.x;
                if (qb + q < nq) store_quad<K, RT>(a, wb, q, ld_f4_at(a.theta + wb, q * 16u));
            }
        }
    }
    const int64_t tail0 = nq * 4;
    if (gtid < a.n - tail0) {
        const int64_t j = tail0 + gtid;
        const float t = a.theta[j];
#pragma unroll
        for (int k = 0; k < K; ++k) {
            if constexpr (RT == RT_F32)
                static_cast<float*>(a.replicas[k])[j] = t;
            else
                static_cast<uint16_t*>(a.replicas[k])[j] = (uint16_t)bf16_rne(t);
        }
    }
}

hipError_t launch_reset(int rt, int k, int blocks, hipStream_t stream, const RoundArgs& a);

}  // namespace autoloco
