// Inner AdamW step of K workers on gfx950 (the local inner loops between two
// synchronisations; settings of Table "Training settings": AdamW with
// coefficients (beta1, beta2), weight decay, gradient-norm clipping; App. G.1:
// FP32 master parameters and AdamW states, BF16 compute copy).
//
// Two streaming passes, both bound by HBM bandwidth:
//   grad_norm_kernel  reads every worker's gradient once and sums g^2 per
//                     worker (fp32 per vector, fp64 per lane, then the same
//                     deterministic two-stage reduction as the round), so the
//                     clipping coefficient sees the worker's whole gradient;
//   adamw_kernel      one grid row per worker: reads theta, m, v and g once,
//                     writes theta, m, v once (and the BF16 copy of theta):
//                       c      = min(1, max_norm / (||g|| + 1e-6))   (from pass 1)
//                       g      = c g
//                       theta  = theta (1 - lr wd)
//                       m      = beta1 m + (1 - beta1) g
//                       v      = beta2 v + (1 - beta2) g^2
//                       theta -= (lr / (1 - beta1^t)) m / (sqrt(v) / sqrt(1 - beta2^t) + eps)
// The clipping coefficient is computed in fp64 by every workgroup from the
// sums pass 1 left in device memory, so the step needs no host round trip.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "reduce.hpp"
#include "round_kernels.hpp"

namespace autoloco {

struct GradNormArgs {
    const float* grads[kMaxK];
    int64_t n;
    double* partials;      // [gridDim.x][K] per-workgroup squared norms
};

struct AdamWArgs {
    float* params[kMaxK];
    float* exp_avg[kMaxK];
    float* exp_avg_sq[kMaxK];
    const float* grads[kMaxK];
    uint16_t* copy[kMaxK];   // BF16 copies of the new parameters, or all null
    int64_t n;
    const double* norm_sq;   // [K] squared gradient norms, or null (no clipping)
    double max_norm;
    float decay;             // 1 - lr * weight_decay
    float beta1, beta2;
    float omb1, omb2;        // 1 - beta1, 1 - beta2
    float step_size;         // lr / (1 - beta1^t)
    float inv_sqrt_bc2;      // 1 / sqrt(1 - beta2^t)
    float eps;
    uint32_t mask;           // traffic reference only: 0 (a value the compiler cannot see)
};

template <int K>
__global__ void __launch_bounds__(kBlock) grad_norm_kernel(GradNormArgs a) {
    double acc[K];
#pragma unroll
    for (int k = 0; k < K; ++k) acc[k] = 0.0;
    const int64_t nvec = a.n / 4;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < nvec; i += stride) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const f32x4 g = ld_f4(a.grads[k] + 4 * i);
            float s = g[0] * g[0];
            s = __builtin_fmaf(g[1], g[1], s);
            s = __builtin_fmaf(g[2], g[2], s);
            s = __builtin_fmaf(g[3], g[3], s);
            acc[k] += (double)s;
        }
    }
    if (blockIdx.x == 0 && threadIdx.x < (a.n & 3)) {
        const int64_t j = nvec * 4 + threadIdx.x;
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const float g = a.grads[k][j];
            acc[k] += (double)(g * g);
        }
    }
    store_partials<K, kBlock>(acc, a.partials);
}

// Clipping coefficient from a squared norm; NaN stays NaN.
__device__ __forceinline__ float clip_coef(double norm_sq, double max_norm) {
    const double c = max_norm / (sqrt(norm_sq) + 1e-6);
    return (float)(c > 1.0 ? 1.0 : c);
}

__device__ __forceinline__ void adamw_one(const AdamWArgs& a, float coef, float& p, float& m, float& v, float g) {
    g *= coef;
    const float pd = p * a.decay;
    m = __builtin_fmaf(a.beta1, m, a.omb1 * g);
    v = __builtin_fmaf(a.beta2, v, (a.omb2 * g) * g);
    const float denom = __builtin_fmaf(__builtin_sqrtf(v), a.inv_sqrt_bc2, a.eps);
    p = pd - a.step_size * (m / denom);
}

typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));

// One element of the traffic reference: the loaded words go back unchanged
// (a.mask is 0), and the gradient word is folded into the parameter's through
// the same mask so that its load stays.
__device__ __forceinline__ void adamw_keep(const AdamWArgs& a, float& p, float& m, float& v, float g) {
    p = __uint_as_float(__float_as_uint(p) ^ (__float_as_uint(g) & a.mask));
    m = __uint_as_float(__float_as_uint(m) ^ a.mask);
    v = __uint_as_float(__float_as_uint(v) ^ a.mask);
}

// TRAFFIC: the traffic reference of this kernel -- the same grid, loop, loads and
// stores, none of the arithmetic; θ, m and v keep their bits and the BF16 copy
// receives the rounding of the unchanged θ (what the last step wrote there).
template <bool COPY, bool TRAFFIC>
__global__ void __launch_bounds__(kBlock) adamw_kernel(AdamWArgs a) {
    const int k = blockIdx.y;
    const float coef = !TRAFFIC && a.norm_sq != nullptr ? clip_coef(a.norm_sq[k], a.max_norm) : 1.0f;
    float* __restrict__ p = a.params[k];
    float* __restrict__ m = a.exp_avg[k];
    float* __restrict__ v = a.exp_avg_sq[k];
    const float* __restrict__ g = a.grads[k];
    uint16_t* __restrict__ c = a.copy[k];
    const int64_t nvec = a.n / 4;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < nvec; i += stride) {
        f32x4 pv = ld_f4(p + 4 * i), mv = ld_f4(m + 4 * i), vv = ld_f4(v + 4 * i);
        const f32x4 gv = ld_f4(g + 4 * i);
        float pe[4], me[4], ve[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            pe[e] = pv[e];
            me[e] = mv[e];
            ve[e] = vv[e];
            if constexpr (TRAFFIC)
                adamw_keep(a, pe[e], me[e], ve[e], gv[e]);
            else
                adamw_one(a, coef, pe[e], me[e], ve[e], gv[e]);
        }
        st_f4(p + 4 * i, f32x4{pe[0], pe[1], pe[2], pe[3]});
        st_f4(m + 4 * i, f32x4{me[0], me[1], me[2], me[3]});
        st_f4(v + 4 * i, f32x4{ve[0], ve[1], ve[2], ve[3]});
        if constexpr (COPY)
            __builtin_nontemporal_store(u32x2v{bf16_pack(pe[0], pe[1]), bf16_pack(pe[2], pe[3])},
                                        reinterpret_cast<u32x2v*>(c + 4 * i));
    }
    if (blockIdx.x == 0 && threadIdx.x < (a.n & 3)) {
        const int64_t j = nvec * 4 + threadIdx.x;
        float pe = p[j], me = m[j], ve = v[j];
        if constexpr (TRAFFIC)
            adamw_keep(a, pe, me, ve, g[j]);
        else
            adamw_one(a, coef, pe, me, ve, g[j]);
        p[j] = pe;
        m[j] = me;
        v[j] = ve;
        if constexpr (COPY) c[j] = (uint16_t)bf16_rne(pe);
    }
}

hipError_t launch_grad_norm(int k, int blocks, hipStream_t s, const GradNormArgs& a);
hipError_t launch_adamw(bool copy, bool traffic, int k, int blocks_per_worker, hipStream_t s, const AdamWArgs& a);

}  // namespace autoloco
