// Standalone replica reset (Alg. "AutoLoCo outer interval": every worker
// starts the next interval from the synchronised parameters) on gfx950: theta
// read once, every replica written once (bf16 replicas rounded to nearest
// even).  Bound by HBM bandwidth; no arithmetic beyond the bf16 narrowing.
#pragma once

#include "round_kernels.hpp"

namespace autoloco {

// theta_k <- theta for every replica.  The round kernel's window loop: a lane
// owns one quad per window of 256 (fp32 replicas) or two, 256 quads apart
// (bf16), at a 32-bit offset from a wave-uniform window base, so every load
// and store instruction of a wavefront covers one contiguous run (1 KB of
// theta, 1 KB of an fp32 replica, 512 B of a bf16 one).
template <int K, int RT>
__global__ void __launch_bounds__(kBlock) reset_kernel(RoundArgs a) {
    constexpr int R = RT == RT_F32 ? 1 : 2;   // quads per lane per window
    const int64_t nq = a.n / 4;
    const int64_t qstride = (int64_t)gridDim.x * kBlock * R;
    const int64_t gtid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    for (int64_t qb = (int64_t)blockIdx.x * kBlock * R; qb < nq; qb += qstride) {
        if (qb + threadIdx.x >= nq) continue;
        const bool ok1 = R == 2 && qb + kBlock + threadIdx.x < nq;
        const int64_t wb = qb * 4;
        if constexpr (RT == RT_F32) {
            const uint32_t fo = threadIdx.x * 16u;
            const f32x4 t = ld_f4_at(a.theta + wb, fo);
#pragma unroll
            for (int k = 0; k < K; ++k) st_f4_at(static_cast<float*>(a.replicas[k]) + wb, fo, t);
        } else {
            f32x4 t[2] = {};
            t[0] = ld_f4_at(a.theta + wb, threadIdx.x * 16u);
            if (ok1) t[1] = ld_f4_at(a.theta + wb, (kBlock + threadIdx.x) * 16u);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                if (h == 1 && !ok1) continue;
                const uint32_t fo = (h * kBlock + threadIdx.x) * 8u;   // byte offset in bf16 buffers
                const u32x2r w = {bf16_pack(t[h][0], t[h][1]), bf16_pack(t[h][2], t[h][3])};
#pragma unroll
                for (int k = 0; k < K; ++k) st_u2_at(static_cast<uint16_t*>(a.replicas[k]) + wb, fo, w);
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
