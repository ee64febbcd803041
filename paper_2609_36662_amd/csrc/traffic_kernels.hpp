// Measurement reference for the fused round kernel (no operation of the
// paper): its loads and stores without its arithmetic.
#pragma once

#include "round_kernels.hpp"

namespace autoloco {

// The fused round's memory traffic with none of its arithmetic: the same
// window loop, launch shape, loads and stores (theta, v and every replica read
// once and written once, in the same order), each 32-bit word written back
// XOR `mask`.  Called with mask = 0 it leaves every buffer as it was (the mask
// only keeps the compiler from dropping the stores); the last n mod 4
// parameters are not touched.  Its time is what the device sustains for the
// round's access pattern: the practical ceiling of the fused round.
template <int K, int RT>
__global__ void __launch_bounds__(kBlock) traffic_kernel(RoundArgs a, uint32_t mask) {
    constexpr int R = RT == RT_F32 ? 1 : 2;   // quads per lane per window, as in round_kernel
    const int64_t nq = a.n / 4;
    const int64_t qstride = (int64_t)gridDim.x * kBlock * R;
    for (int64_t qb = (int64_t)blockIdx.x * kBlock * R; qb < nq; qb += qstride) {
        if (qb + threadIdx.x >= nq) continue;
        const bool ok1 = R == 2 && qb + kBlock + threadIdx.x < nq;
        const int64_t wb = qb * 4;
        float* const th_w = a.theta + wb;
        float* const mo_w = a.momentum + wb;
        if constexpr (RT == RT_F32) {
            const uint32_t fo = threadIdx.x * 16u;
            const u32x4 t = ld_u4_at(th_w, fo), m = ld_u4_at(mo_w, fo);
            u32x4 r[K];
#pragma unroll
            for (int k = 0; k < K; ++k) r[k] = ld_u4_at(static_cast<const float*>(a.replicas[k]) + wb, fo);
            st_u4_at(th_w, fo, t ^ mask);
            st_u4_at(mo_w, fo, m ^ mask);
#pragma unroll
            for (int k = 0; k < K; ++k) st_u4_at(static_cast<float*>(a.replicas[k]) + wb, fo, r[k] ^ mask);
        } else {
            u32x4 t[2] = {}, m[2] = {};
            u32x2r r[K][2] = {};
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                if (h == 1 && !ok1) continue;
                const uint32_t fo = (h * kBlock + threadIdx.x) * 16u;
                t[h] = ld_u4_at(th_w, fo);
                m[h] = ld_u4_at(mo_w, fo);
#pragma unroll
                for (int k = 0; k < K; ++k) r[k][h] = ld_u2_at(static_cast<const uint16_t*>(a.replicas[k]) + wb, fo / 2);
            }
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                if (h == 1 && !ok1) continue;
                const uint32_t fo = (h * kBlock + threadIdx.x) * 16u;
                st_u4_at(th_w, fo, t[h] ^ mask);
                st_u4_at(mo_w, fo, m[h] ^ mask);
#pragma unroll
                for (int k = 0; k < K; ++k)
                    st_u2_at(static_cast<uint16_t*>(a.replicas[k]) + wb, fo / 2, r[k][h] ^ mask);
            }
        }
    }
}

hipError_t launch_traffic(int rt, int k, int blocks, hipStream_t stream, const RoundArgs& a, uint32_t mask);

}  // namespace autoloco
