// One GPU's share of a round in the paper's topology (one worker replica per
// GPU), with BF16 pseudo-gradient payloads, on gfx950.  Between the two
// kernels a collective moves payload shards (all-to-all: GPU s receives shard
// s of every worker's payload); after the second an all-gather of theta'
// shards rebuilds theta on every GPU, and the reset copies it into the
// worker's replica.  The arithmetic is that of the fused BF16-payload round,
// so the decomposition gives the same bits.
//
//   rank_payload_kernel  (worker r, all n parameters)
//       Delta = theta - theta_r (FP32); payload = bf16(Delta); S_r = sum Delta^2
//   shard_step_kernel    (shard s, its n_s parameters, K payload shards)
//       mean = bf16(fp32(sum_k payload_k (float64, worker order) * 1/K))
//       M_s = sum mean^2; v' = mu v + mean*scale; theta' = theta - eta (mean*scale + mu v')
//
// Both stream 16-byte vectors (8 parameters per lane) and reduce their one sum
// with the deterministic two-stage reduction.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "reduce.hpp"
#include "round_kernels.hpp"

namespace autoloco {

struct RankPayloadArgs {
    const float* theta;
    const void* replica;
    uint16_t* payload;
    int64_t n;
    double* partials;
    unsigned int* ticket;
    double* sums;
};

struct ShardArgs {
    float* theta;
    float* momentum;
    const uint16_t* payloads[kMaxK];
    uint16_t* mean_out;   // or null
    int64_t n;
    float mu, eta, scale;
    double inv_k64;
    double* partials;
    unsigned int* ticket;
    double* sums;
};

template <int RT>
__global__ void __launch_bounds__(kBlock) rank_payload_kernel(RankPayloadArgs a) {
    double acc[1] = {0.0};
    const int64_t nvec = a.n / 8;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < nvec; i += stride) {
        const int64_t o = 8 * i;
        const f32x4 t0 = ld_f4(a.theta + o), t1 = ld_f4(a.theta + o + 4);
        float r[8];
        if constexpr (RT == RT_F32) {
            const f32x4 r0 = ld_f4(static_cast<const float*>(a.replica) + o);
            const f32x4 r1 = ld_f4(static_cast<const float*>(a.replica) + o + 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                r[e] = r0[e];
                r[4 + e] = r1[e];
            }
        } else {
            const u32x4 w = ld_u4(static_cast<const uint16_t*>(a.replica) + o);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                r[2 * e] = bf16_lo(w[e]);
                r[2 * e + 1] = bf16_hi(w[e]);
            }
        }
        float d[8], s = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            d[e] = t0[e] - r[e];
            d[4 + e] = t1[e] - r[4 + e];
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) s = __builtin_fmaf(d[e], d[e], s);
        acc[0] += (double)s;
        st_u4(a.payload + o, u32x4{bf16_pack(d[0], d[1]), bf16_pack(d[2], d[3]), bf16_pack(d[4], d[5]),
                                   bf16_pack(d[6], d[7])});
    }
    if (blockIdx.x == 0 && threadIdx.x < (a.n & 7)) {
        const int64_t j = nvec * 8 + threadIdx.x;
        float r;
        if constexpr (RT == RT_F32)
            r = static_cast<const float*>(a.replica)[j];
        else
            r = __uint_as_float((uint32_t) static_cast<const uint16_t*>(a.replica)[j] << 16);
        const float d = a.theta[j] - r;
        acc[0] += (double)(d * d);
        a.payload[j] = (uint16_t)bf16_rne(d);
    }
    grid_reduce<1, kBlock>(acc, a.partials, a.ticket, a.sums);
}

// The received mean of one parameter from its K payloads, and the step.
template <int K>
__device__ __forceinline__ float shard_one(const ShardArgs& a, const float (&b)[K], float th, float v, float& th_new,
                                           float& v_new, uint32_t& pb) {
    double sum = 0.0;
#pragma unroll
    for (int k = 0; k < K; ++k) sum += (double)b[k];
    pb = bf16_rne((float)(sum * a.inv_k64));
    const float mean = __uint_as_float(pb << 16);
    const float dt = mean * a.scale;
    v_new = __builtin_fmaf(a.mu, v, dt);
    const float dir = __builtin_fmaf(a.mu, v_new, dt);
    th_new = __builtin_fmaf(-a.eta, dir, th);
    return mean;
}

template <int K>
__global__ void __launch_bounds__(kBlock) shard_step_kernel(ShardArgs a) {
    double acc[1] = {0.0};
    const int64_t nvec = a.n / 8;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < nvec; i += stride) {
        const int64_t o = 8 * i;
        const f32x4 t0 = ld_f4(a.theta + o), t1 = ld_f4(a.theta + o + 4);
        const f32x4 v0 = ld_f4(a.momentum + o), v1 = ld_f4(a.momentum + o + 4);
        float b[K][8];
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const u32x4 w = ld_u4(a.payloads[k] + o);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                b[k][2 * e] = bf16_lo(w[e]);
                b[k][2 * e + 1] = bf16_hi(w[e]);
            }
        }
        float th[8], v[8], th_new[8], v_new[8], m = 0.f;
        uint32_t pb[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            th[e] = t0[e];
            th[4 + e] = t1[e];
            v[e] = v0[e];
            v[4 + e] = v1[e];
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            float be[K];
#pragma unroll
            for (int k = 0; k < K; ++k) be[k] = b[k][e];
            const float mean = shard_one<K>(a, be, th[e], v[e], th_new[e], v_new[e], pb[e]);
            m = __builtin_fmaf(mean, mean, m);
        }
        acc[0] += (double)m;
        st_f4(a.theta + o, f32x4{th_new[0], th_new[1], th_new[2], th_new[3]});
        st_f4(a.theta + o + 4, f32x4{th_new[4], th_new[5], th_new[6], th_new[7]});
        st_f4(a.momentum + o, f32x4{v_new[0], v_new[1], v_new[2], v_new[3]});
        st_f4(a.momentum + o + 4, f32x4{v_new[4], v_new[5], v_new[6], v_new[7]});
        if (a.mean_out != nullptr)
            st_u4(a.mean_out + o, u32x4{pb[0] | pb[1] << 16, pb[2] | pb[3] << 16, pb[4] | pb[5] << 16,
                                        pb[6] | pb[7] << 16});
    }
    if (blockIdx.x == 0 && threadIdx.x < (a.n & 7)) {
        const int64_t j = nvec * 8 + threadIdx.x;
        float be[K];
#pragma unroll
        for (int k = 0; k < K; ++k) be[k] = __uint_as_float((uint32_t)a.payloads[k][j] << 16);
        float th_new, v_new;
        uint32_t pb;
        const float mean = shard_one<K>(a, be, a.theta[j], a.momentum[j], th_new, v_new, pb);
        acc[0] += (double)(mean * mean);
        a.theta[j] = th_new;
        a.momentum[j] = v_new;
        if (a.mean_out != nullptr) a.mean_out[j] = (uint16_t)pb;
    }
    grid_reduce<1, kBlock>(acc, a.partials, a.ticket, a.sums);
}

hipError_t launch_rank_payload(int rt, int blocks, hipStream_t s, const RankPayloadArgs& a);
hipError_t launch_shard_step(int k, int blocks, hipStream_t s, const ShardArgs& a);

}  // namespace autoloco
