// A synchronisation round whose pseudo-gradient average travels through the
// INT8 blockwise codec (App. G.1), on gfx950.
//
// One workgroup of 512 threads owns one codec block of 4,096 parameters at a
// time (8 parameters per thread), so every buffer is still read once and
// written once.  Per block:
//   Delta_k = theta - theta_k                                (fp32)
//   S_k += Delta_k^2                 D is measured before quantisation
//   s_k = max|Delta_k| / 127 (1 for a zero block, at least 2^-126)
//   q = clip(rne(Delta_k / s_k), -127, 127);  Delta^_k = q s_k    (fp32)
//   mean = fp32(sum_k Delta^_k (fp64, worker order) * fp64(1/K))
//   the mean is encoded and decoded once more (same rule)  -> Delta_agg
//   Q_k += (Delta_k - Delta_agg)^2, M += Delta_agg^2          C uses the aggregate
//   corrected Nesterov step with Delta_agg, reset of the replicas
// The two block maxima (the K worker maxima, then the mean's) are exact and
// order-independent: a wavefront butterfly of fmaxf and the waves through LDS.
// Every codec step runs in fp32 with IEEE division and round-to-nearest-even,
// so the codes are the same integers the FP32 definition gives.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "reduce.hpp"
#include "round_kernels.hpp"

namespace autoloco {

constexpr int kCodecBlock = 4096;

struct Int8Args {
    float* theta;
    float* momentum;
    void* replicas[kMaxK];
    int64_t n;
    float mu, eta, scale;
    double inv_k;
    int8_t* mean_codes;   // [n] or null
    float* mean_scales;   // [ceil(n / 4096)] or null
    double* partials;
    unsigned int* ticket;
    double* sums;
};

__device__ __forceinline__ float codec_scale(float amax) {
    if (amax == 0.0f) return 1.0f;
    const float s = amax / 127.0f;
    return s < 0x1p-126f ? 0x1p-126f : s;
}

__device__ __forceinline__ float codec_q(float x, float s) {
    float q = __builtin_rintf(x / s);
    q = q < -127.0f ? -127.0f : q;
    return q > 127.0f ? 127.0f : q;
}

// Maximum of NV values over the workgroup (every thread gets the result).
template <int NV, int NT>
__device__ __forceinline__ void block_max(float (&v)[NV], float* lds) {
    constexpr int NW = NT / 64;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        float x = v[j];
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
        v[j] = x;
    }
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    if (lane == 0) {
#pragma unroll
        for (int j = 0; j < NV; ++j) lds[wave * NV + j] = v[j];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        float x = lds[j];
#pragma unroll
        for (int w = 1; w < NW; ++w) x = fmaxf(x, lds[w * NV + j]);
        v[j] = x;
    }
    __syncthreads();
}

constexpr int kInt8Threads = 512;  // one codec block of 4,096 parameters per workgroup

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Thread t of a workgroup owns parameters blk*4096 + g*2048 + 4t + e for
// g in {0,1}, e in 0..3: every load and store instruction of a wavefront
// covers one contiguous 1 KB (fp32) or 512 B (bf16) run.
template <int K, int RT, bool STATS, bool RESET>
__global__ void __launch_bounds__(kInt8Threads) int8_round_kernel(Int8Args a) {
    constexpr int NT = kInt8Threads;
    constexpr int V = 8;
    constexpr int NS = STATS ? 2 * K + 1 : 1;
    __shared__ float lds_max[kMaxWaves * kMaxK];

    double acc[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) acc[j] = 0.0;

    const int64_t nblocks = (a.n + kCodecBlock - 1) / kCodecBlock;
    for (int64_t blk = blockIdx.x; blk < nblocks; blk += gridDim.x) {
        int64_t off[2];
        int valid[2];
#pragma unroll
        for (int g = 0; g < 2; ++g) {
            off[g] = blk * kCodecBlock + g * (kCodecBlock / 2) + (int64_t)threadIdx.x * 4;
            const int64_t left = a.n - off[g];
            valid[g] = left >= 4 ? 4 : (left > 0 ? (int)left : 0);
        }

        float th[V], v[V], d[K][V];
#pragma unroll
        for (int g = 0; g < 2; ++g) {
            const int64_t o = off[g];
            if (valid[g] == 4) {
                const f32x4 t4 = ld_f4(a.theta + o), v4 = ld_f4(a.momentum + o);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    th[4 * g + e] = t4[e];
                    v[4 * g + e] = v4[e];
                }
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    if constexpr (RT == RT_F32) {
                        const f32x4 r4 = ld_f4(static_cast<const float*>(a.replicas[k]) + o);
#pragma unroll
                        for (int e = 0; e < 4; ++e) d[k][4 * g + e] = th[4 * g + e] - r4[e];
                    } else {
                        const u32x2 w = __builtin_nontemporal_load(
                            reinterpret_cast<const u32x2*>(static_cast<const uint16_t*>(a.replicas[k]) + o));
                        d[k][4 * g + 0] = th[4 * g + 0] - bf16_lo(w[0]);
                        d[k][4 * g + 1] = th[4 * g + 1] - bf16_hi(w[0]);
                        d[k][4 * g + 2] = th[4 * g + 2] - bf16_lo(w[1]);
                        d[k][4 * g + 3] = th[4 * g + 3] - bf16_hi(w[1]);
                    }
                }
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const bool in = e < valid[g];
                    th[4 * g + e] = in ? a.theta[o + e] : 0.0f;
                    v[4 * g + e] = in ? a.momentum[o + e] : 0.0f;
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        float r = 0.0f;
                        if (in) {
                            if constexpr (RT == RT_F32)
                                r = static_cast<const float*>(a.replicas[k])[o + e];
                            else
                                r = __uint_as_float((uint32_t) static_cast<const uint16_t*>(a.replicas[k])[o + e] << 16);
                        }
                        d[k][4 * g + e] = in ? th[4 * g + e] - r : 0.0f;
                    }
                }
            }
        }

        // local-drift energy before quantisation
        if constexpr (STATS) {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                float s = 0.f;
#pragma unroll
                for (int e = 0; e < V; ++e) s = __builtin_fmaf(d[k][e], d[k][e], s);
                acc[k] += (double)s;
            }
        }

        // worker block scales
        float amax[K];
#pragma unroll
        for (int k = 0; k < K; ++k) {
            float m = 0.f;
#pragma unroll
            for (int e = 0; e < V; ++e) m = fmaxf(m, fabsf(d[k][e]));
            amax[k] = m;
        }
        block_max<K, NT>(amax, lds_max);

        // decode every worker and average: fp64 sum in worker order, times fp64(1/K)
        double sum[V];
#pragma unroll
        for (int e = 0; e < V; ++e) sum[e] = 0.0;
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const float s = codec_scale(amax[k]);
#pragma unroll
            for (int e = 0; e < V; ++e) sum[e] += (double)(codec_q(d[k][e], s) * s);
        }
        float mean[V];
        float mmax[1] = {0.f};
#pragma unroll
        for (int e = 0; e < V; ++e) {
            mean[e] = (float)(sum[e] * a.inv_k);
            mmax[0] = fmaxf(mmax[0], fabsf(mean[e]));
        }
        block_max<1, NT>(mmax, lds_max);
        const float sm = codec_scale(mmax[0]);

        float agg[V], qm[V];
#pragma unroll
        for (int e = 0; e < V; ++e) {
            qm[e] = codec_q(mean[e], sm);
            agg[e] = e % 4 < valid[e / 4] ? qm[e] * sm : 0.0f;
        }
        if (a.mean_codes != nullptr) {
#pragma unroll
            for (int g = 0; g < 2; ++g) {
                if (valid[g] == 4) {
                    uint32_t w = 0;
#pragma unroll
                    for (int e = 0; e < 4; ++e) w |= (uint32_t)(uint8_t)(int8_t)qm[4 * g + e] << (8 * e);
                    __builtin_nontemporal_store(w, reinterpret_cast<uint32_t*>(a.mean_codes + off[g]));
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (e < valid[g]) a.mean_codes[off[g] + e] = (int8_t)qm[4 * g + e];
                }
            }
            if (threadIdx.x == 0) a.mean_scales[blk] = sm;
        }

        if constexpr (STATS) {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                float q = 0.f;
#pragma unroll
                for (int e = 0; e < V; ++e) {
                    const float t = d[k][e] - agg[e];
                    q = __builtin_fmaf(t, t, q);
                }
                acc[K + k] += (double)q;
            }
            float m = 0.f;
#pragma unroll
            for (int e = 0; e < V; ++e) m = __builtin_fmaf(agg[e], agg[e], m);
            acc[2 * K] += (double)m;
        }

        // corrected Nesterov step with the decoded aggregate, and the reset
        float th_new[V], v_new[V];
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const float dt = agg[e] * a.scale;
            v_new[e] = __builtin_fmaf(a.mu, v[e], dt);
            const float dir = __builtin_fmaf(a.mu, v_new[e], dt);
            th_new[e] = __builtin_fmaf(-a.eta, dir, th[e]);
        }
#pragma unroll
        for (int g = 0; g < 2; ++g) {
            const int64_t o = off[g];
            const float* tn = th_new + 4 * g;
            const float* vn = v_new + 4 * g;
            if (valid[g] == 4) {
                st_f4(a.theta + o, f32x4{tn[0], tn[1], tn[2], tn[3]});
                st_f4(a.momentum + o, f32x4{vn[0], vn[1], vn[2], vn[3]});
                if constexpr (RESET) {
                    if constexpr (RT == RT_F32) {
                        const f32x4 t4 = {tn[0], tn[1], tn[2], tn[3]};
#pragma unroll
                        for (int k = 0; k < K; ++k) st_f4(static_cast<float*>(a.replicas[k]) + o, t4);
                    } else {
                        const u32x2 w = {bf16_pack(tn[0], tn[1]), bf16_pack(tn[2], tn[3])};
#pragma unroll
                        for (int k = 0; k < K; ++k)
                            __builtin_nontemporal_store(w, reinterpret_cast<u32x2*>(static_cast<uint16_t*>(a.replicas[k]) + o));
                    }
                }
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if (e < valid[g]) {
                        a.theta[o + e] = tn[e];
                        a.momentum[o + e] = vn[e];
                        if constexpr (RESET) {
#pragma unroll
                            for (int k = 0; k < K; ++k) {
                                if constexpr (RT == RT_F32)
                                    static_cast<float*>(a.replicas[k])[o + e] = tn[e];
                                else
                                    static_cast<uint16_t*>(a.replicas[k])[o + e] = (uint16_t)bf16_rne(tn[e]);
                            }
                        }
                    }
                }
            }
        }
    }

    if constexpr (STATS) grid_reduce<NS, NT>(acc, a.partials, a.ticket, a.sums);
}

typedef hipError_t (*Int8Launcher)(int k, int blocks, hipStream_t stream, const Int8Args& a);
// one per (replica type, stats, reset): launch_int8_<rt>_s<stats>r<reset>
hipError_t launch_int8_f32_s0r0(int, int, hipStream_t, const Int8Args&);
hipError_t launch_int8_f32_s0r1(int, int, hipStream_t, const Int8Args&);
hipError_t launch_int8_f32_s1r0(int, int, hipStream_t, const Int8Args&);
hipError_t launch_int8_f32_s1r1(int, int, hipStream_t, const Int8Args&);
hipError_t launch_int8_bf16_s0r0(int, int, hipStream_t, const Int8Args&);
hipError_t launch_int8_bf16_s0r1(int, int, hipStream_t, const Int8Args&);
hipError_t launch_int8_bf16_s1r0(int, int, hipStream_t, const Int8Args&);
hipError_t launch_int8_bf16_s1r1(int, int, hipStream_t, const Int8Args&);
int occupancy_int8_f32_s1r1(int k);
int occupancy_int8_bf16_s1r1(int k);

}  // namespace autoloco
