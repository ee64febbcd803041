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
// Both reduce their one sum with the deterministic two-stage reduction.
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
    double* partials;     // [gridDim.x] per-workgroup sums
};

struct ShardArgs {
    float* theta;
    float* momentum;
    const uint16_t* payloads[kMaxK];
    uint16_t* mean_out;   // or null
    int64_t n;
    float mu, eta, scale;
    double inv_k64;
    double* partials;     // [gridDim.x] per-workgroup sums
};

// Both kernels walk runs of 4 parameters ("quads"); a lane owns two quads per
// window of 512, 256 quads apart, at a 32-bit offset from a wave-uniform window
// base, so every wavefront instruction covers one contiguous run (1 KB of fp32,
// 512 B of bf16) and no cache line is written in parts.  The last n mod 4
// parameters go to threads of workgroup 0.
// One window of rank_payload_kernel for one lane: its two quads (FULL: both in
// range, a wave-uniform fact; else only those below `left` quads from the
// window's start), both loaded before any store (the payload store could alias
// the inputs as far as the compiler knows, so it would not move a later load
// above it).  Returns the lane's fp32 sum of squares over the window.
template <int RT, bool FULL>
__device__ __forceinline__ float payload_window(const RankPayloadArgs& a, int64_t wb, int64_t left) {
    f32x4 t[2], r4[2];
    u32x2r rw[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint32_t run = h * kBlock + threadIdx.x;
        if (!FULL && run >= left) continue;
        t[h] = ld_f4_at(a.theta + wb, run * 16u);
        if constexpr (RT == RT_F32)
            r4[h] = ld_f4_at(static_cast<const float*>(a.replica) + wb, run * 16u);
        else
            rw[h] = ld_u2_at(static_cast<const uint16_t*>(a.replica) + wb, run * 8u);
    }
    float s = 0.f;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint32_t run = h * kBlock + threadIdx.x;
        if (!FULL && run >= left) continue;
        float r[4];
        if constexpr (RT == RT_F32) {
#pragma unroll
            for (int e = 0; e < 4; ++e) r[e] = r4[h][e];
        } else {
            r[0] = bf16_lo(rw[h][0]);
            r[1] = bf16_hi(rw[h][0]);
            r[2] = bf16_lo(rw[h][1]);
            r[3] = bf16_hi(rw[h][1]);
        }
        float d[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            d[e] = t[h][e] - r[e];
            s = __builtin_fmaf(d[e], d[e], s);
        }
        st_u2_at(a.payload + wb, run * 8u, u32x2r{bf16_pack(d[0], d[1]), bf16_pack(d[2], d[3])});
    }
    return s;
}

template <int RT>
__global__ void __launch_bounds__(kBlock) rank_payload_kernel(RankPayloadArgs a) {
    double acc[1] = {0.0};
    const int64_t nq = a.n / 4;
    const int64_t stride = (int64_t)gridDim.x * kBlock * 2;
    for (int64_t qb = (int64_t)blockIdx.x * kBlock * 2; qb < nq; qb += stride) {
        const int64_t wb = qb * 4;                       // first parameter of the window
        if (qb + 2 * kBlock <= nq)                       // a whole window: no per-lane test
            acc[0] += (double)payload_window<RT, true>(a, wb, 0);
        else if (qb + threadIdx.x < nq)                  // the last, shorter window
            acc[0] += (double)payload_window<RT, false>(a, wb, nq - qb);
    }
    if (blockIdx.x == 0 && threadIdx.x < (a.n & 3)) {
        const int64_t j = nq * 4 + threadIdx.x;
        float r;
        if constexpr (RT == RT_F32)
            r = static_cast<const float*>(a.replica)[j];
        else
            r = __uint_as_float((uint32_t) static_cast<const uint16_t*>(a.replica)[j] << 16);
        const float d = a.theta[j] - r;
        acc[0] += (double)(d * d);
        a.payload[j] = (uint16_t)bf16_rne(d);
    }
    store_partials<1, kBlock>(acc, a.partials);
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

// One window of shard_step_kernel for one lane (FULL and left as in
// payload_window); returns the lane's fp32 sum of the squared means.
template <int K, bool FULL>
__device__ __forceinline__ float shard_window(const ShardArgs& a, int64_t wb, int64_t left) {
    f32x4 t4[2], v4[2];
    u32x2r w[K][2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint32_t run = h * kBlock + threadIdx.x;
        if (!FULL && run >= left) continue;
        t4[h] = ld_f4_at(a.theta + wb, run * 16u);
        v4[h] = ld_f4_at(a.momentum + wb, run * 16u);
#pragma unroll
        for (int k = 0; k < K; ++k) w[k][h] = ld_u2_at(a.payloads[k] + wb, run * 8u);
    }
    float m = 0.f;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint32_t run = h * kBlock + threadIdx.x;
        if (!FULL && run >= left) continue;
        float th_new[4], v_new[4];
        uint32_t pb[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float be[K];
#pragma unroll
            for (int k = 0; k < K; ++k) be[k] = (e & 1) ? bf16_hi(w[k][h][e >> 1]) : bf16_lo(w[k][h][e >> 1]);
            const float mean = shard_one<K>(a, be, t4[h][e], v4[h][e], th_new[e], v_new[e], pb[e]);
            m = __builtin_fmaf(mean, mean, m);
        }
        st_f4_at(a.theta + wb, run * 16u, f32x4{th_new[0], th_new[1], th_new[2], th_new[3]});
        st_f4_at(a.momentum + wb, run * 16u, f32x4{v_new[0], v_new[1], v_new[2], v_new[3]});
        if (a.mean_out != nullptr)
            st_u2_at(a.mean_out + wb, run * 8u, u32x2r{pb[0] | pb[1] << 16, pb[2] | pb[3] << 16});
    }
    return m;
}

template <int K>
__global__ void __launch_bounds__(kBlock) shard_step_kernel(ShardArgs a) {
    double acc[1] = {0.0};
    const int64_t nq = a.n / 4;
    const int64_t stride = (int64_t)gridDim.x * kBlock * 2;
    for (int64_t qb = (int64_t)blockIdx.x * kBlock * 2; qb < nq; qb += stride) {
        const int64_t wb = qb * 4;                       // first parameter of the window
        if (qb + 2 * kBlock <= nq)                       // a whole window: no per-lane test
            acc[0] += (double)shard_window<K, true>(a, wb, 0);
        else if (qb + threadIdx.x < nq)                  // the last, shorter window
            acc[0] += (double)shard_window<K, false>(a, wb, nq - qb);
    }
    if (blockIdx.x == 0 && threadIdx.x < (a.n & 3)) {
        const int64_t j = nq * 4 + threadIdx.x;
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
    store_partials<1, kBlock>(acc, a.partials);
}

hipError_t launch_rank_payload(int rt, int blocks, hipStream_t s, const RankPayloadArgs& a);
hipError_t launch_shard_step(int k, int blocks, hipStream_t s, const ShardArgs& a);

}  // namespace autoloco
