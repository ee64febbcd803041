// Streaming kernels of one AutoLoCo synchronisation round on gfx950.
//
// One pass over the parameters reads theta_t, v_{t-1} and the K worker
// replicas once, and (depending on the mode) writes theta_{t+1}, v_t and the
// K reset replicas once.  Per parameter j:
//   Delta_k   = theta[j] - theta_k[j]                  (Alg. "AutoLoCo outer interval")
//   Delta_bar = (sum_k Delta_k) * (1/K)                pairwise tree over k in index order
//   S_k += Delta_k^2, Q_k += (Delta_k - Delta_bar)^2, M += Delta_bar^2
//                                                      (eq. adaptive-h-core-diagnostics; App. C.1)
//   Dt = Delta_bar * scale   (scale = 1/rho when normalising, else 1; eq. normalized-pseudo-gradient)
//   v' = mu v + Dt; d = Dt + mu v'; theta' = theta - eta d   (eq. autoloco-corrected-nesterov)
//   theta_k[j] = theta'  (fp32, or bf16 rounded to nearest even)
//
// Nothing here is a contraction, so no matrix cores are used: the work is
// bound by HBM bandwidth.  Each lane moves 16-byte vectors (4 fp32 or 8 bf16
// parameters) with non-temporal loads and stores so the streams do not
// displace one another in the caches, in a grid-stride loop over a fixed
// grid.  Elementwise arithmetic is fp32; the squared sums of one vector are
// added in fp32 and then into per-lane fp64 running sums.  The 2K+1 sums are
// reduced deterministically: a wavefront butterfly, then the waves of the
// workgroup in order through LDS into one partial per workgroup (a plain
// store), then a one-workgroup kernel launched after this one on the same
// stream adds the partials in workgroup order.  With the grid fixed, every
// run adds the same numbers in the same order, so the statistics are
// bit-identical between runs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "reduce.hpp"

namespace autoloco {

constexpr int kBlock = 256;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2r __attribute__((ext_vector_type(2)));

enum ReplicaType { RT_F32 = 0, RT_BF16 = 1 };
// Modes 5..8 are modes 1..4 with the worker average taken through BF16
// pseudo-gradient payloads.
enum Mode { MODE_STATS = 0, MODE_UPDATE = 1, MODE_UPDATE_STATS = 2, MODE_UPDATE_RESET = 3,
            MODE_UPDATE_STATS_RESET = 4, MODE_P_UPDATE = 5, MODE_P_UPDATE_STATS = 6, MODE_P_UPDATE_RESET = 7,
            MODE_P_UPDATE_STATS_RESET = 8, MODE_COUNT = 9 };

struct RoundArgs {
    float* theta;
    float* momentum;
    void* replicas[kMaxK];
    int64_t n;
    float mu, eta, scale, inv_k;
    double* partials;      // [gridDim.x][2K+1] per-workgroup sums
    uint16_t* payload;     // BF16 payload modes: [n] bits of the received mean, or null
    double inv_k64;        // 1/K in float64 (BF16 payload modes)
};

// ------------------------------------------------------------------ memory --
__device__ __forceinline__ f32x4 ld_f4(const float* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
}
__device__ __forceinline__ void st_f4(float* p, f32x4 v) {
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(p));
}
__device__ __forceinline__ u32x4 ld_u4(const void* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ void st_u4(void* p, u32x4 v) {
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

// Same, at a wave-uniform base plus a 32-bit per-lane byte offset (lets the
// compiler keep the base in scalar registers).
__device__ __forceinline__ f32x4 ld_f4_at(const void* base, uint32_t off) {
    return __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(static_cast<const char*>(base) + off));
}
__device__ __forceinline__ void st_f4_at(void* base, uint32_t off, f32x4 v) {
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(static_cast<char*>(base) + off));
}
__device__ __forceinline__ u32x4 ld_u4_at(const void* base, uint32_t off) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(static_cast<const char*>(base) + off));
}
__device__ __forceinline__ void st_u4_at(void* base, uint32_t off, u32x4 v) {
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(static_cast<char*>(base) + off));
}
__device__ __forceinline__ u32x2r ld_u2_at(const void* base, uint32_t off) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x2r*>(static_cast<const char*>(base) + off));
}
__device__ __forceinline__ void st_u2_at(void* base, uint32_t off, u32x2r v) {
    __builtin_nontemporal_store(v, reinterpret_cast<u32x2r*>(static_cast<char*>(base) + off));
}

// bf16 <-> fp32.  Widening is exact.  Narrowing is gfx950's conversion
// instruction (one for a pair): round to nearest, ties to even, subnormals and
// infinities kept, overflow to infinity; a NaN stays a quiet NaN with the top
// of its payload.  (Over all 2^32 inputs other than NaN it gives the bits of
// the integer formulation (u + 0x7FFF + lsb) >> 16, checked on MI355X.)
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ uint32_t bf16_pack(float lo, float hi) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}
__device__ __forceinline__ uint32_t bf16_rne(float x) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(x));
}

// ------------------------------------------------------------- arithmetic --
template <int LO, int CNT, int K>
__device__ __forceinline__ float tree_sum(const float (&d)[K]) {
    if constexpr (CNT == 1) {
        return d[LO];
    } else {
        constexpr int H = CNT / 2;
        return tree_sum<LO, H, K>(d) + tree_sum<LO + H, CNT - H, K>(d);
    }
}

// One parameter: pseudo-gradients, their mean, the squared-sum terms and the
// corrected Nesterov step.  With BF16P the mean is the one every worker
// receives when the pseudo-gradients travel as BF16: each Delta_k rounded to
// BF16 (nearest even), their float64 sum in worker order times float64(1/K)
// rounded to FP32, then to BF16 (its bits go to pb); the squared sums use the
// unrounded Delta_k and that received mean.
// Only the fused multiply-adds written out are fused: without the pragma the
// compiler may fold the mean's product into Delta_k - mean in some kernel
// variants and not in others, and the standalone and fused statistics would
// then differ in their last bits.
template <int K, bool STATS, bool UPDATE, bool BF16P>
__device__ __forceinline__ void one_param(float th, float v, const float (&r)[K], const RoundArgs& a,
                                          float (&s)[K], float (&q)[K], float& m, float& th_new,
                                          float& v_new, uint32_t& pb) {
#pragma clang fp contract(off)
    float d[K];
#pragma unroll
    for (int k = 0; k < K; ++k) d[k] = th - r[k];
    float mean;
    if constexpr (BF16P) {
        double sum = 0.0;
#pragma unroll
        for (int k = 0; k < K; ++k) sum += (double)__uint_as_float(bf16_rne(d[k]) << 16);
        pb = bf16_rne((float)(sum * a.inv_k64));
        mean = __uint_as_float(pb << 16);
    } else {
        mean = tree_sum<0, K, K>(d) * a.inv_k;
    }
    if constexpr (STATS) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            s[k] = __builtin_fmaf(d[k], d[k], s[k]);
            const float e = d[k] - mean;
            q[k] = __builtin_fmaf(e, e, q[k]);
        }
        m = __builtin_fmaf(mean, mean, m);
    }
    if constexpr (UPDATE) {
        const float dt = mean * a.scale;
        v_new = __builtin_fmaf(a.mu, v, dt);
        const float dir = __builtin_fmaf(a.mu, v_new, dt);
        th_new = __builtin_fmaf(-a.eta, dir, th);
    }
}

// Windows the statistics-only mode loads ahead: enough for about 512 bytes of
// loads per lane (from K = 5 with fp32 replicas and from K = 6 with bf16 the
// default grid holds one wave per SIMD), at most 8, within 200 registers for the
// loaded words (below those K, whose grid keeps three workgroups per compute
// unit, 100 with fp32 replicas and 64 with bf16, so that three waves per SIMD
// still fit).  Per window a lane loads (K + 1) quads of fp32, or with bf16
// replicas two of theta and 2K words.
template <int K, int RT>
constexpr int stats_unroll() {
    const int words = RT == RT_F32 ? 4 * (K + 1) : 4 * K + 8;
    const int bytes = RT == RT_F32 ? 16 * (K + 1) : 32 + 16 * K;
    const int cap = K >= (RT == RT_F32 ? 5 : 6) ? 200 : (RT == RT_F32 ? 100 : 64);
    int u = (512 + bytes - 1) / bytes;
    if (u > 8) u = 8;
    while (u > 1 && u * words > cap) --u;
    return u;
}

// ------------------------------------------------------------ round kernel --
template <int K, int RT, bool STATS, bool UPDATE, bool RESET, bool BF16P = false>
__global__ void __launch_bounds__(kBlock) round_kernel(RoundArgs a) {
    constexpr int NS = STATS ? 2 * K + 1 : 1;
    double acc[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) acc[j] = 0.0;

    // Parameters in runs of 4 ("quads": 16 bytes of fp32, 8 of bf16).  The
    // loop walks wave-uniform windows: each stream's window base stays in
    // scalar registers and a lane adds only its 32-bit offset.  fp32 replicas:
    // a lane owns one quad per window of 256; bf16 replicas: two, 256 quads
    // apart (a window of 512), so every load and store instruction of a
    // wavefront covers one contiguous run (1 KB of fp32, 512 B of bf16) and no
    // cache line is written in parts.
    constexpr int R = RT == RT_F32 ? 1 : 2;   // quads per lane per window
    constexpr int V = 4 * R;                  // parameters per lane per window
    const int64_t nq = a.n / 4;
    const int64_t qstride = (int64_t)gridDim.x * kBlock * R;
    const int64_t gtid = (int64_t)blockIdx.x * kBlock + threadIdx.x;

    if constexpr (!UPDATE) {
        // Statistics only, so no stores to overlap the loads with: U windows of
        // the thread's grid-stride sequence are loaded before any of them is
        // added up, in that same order, which keeps every per-thread sum what one
        // window per iteration gives, bit for bit, with U times the loads in
        // flight.
        constexpr int U = stats_unroll<K, RT>();
        for (int64_t qb0 = (int64_t)blockIdx.x * kBlock * R; qb0 < nq; qb0 += U * qstride) {
            f32x4 tq[U][R];
            f32x4 rf[RT == RT_F32 ? U : 1][RT == RT_F32 ? K : 1];
            u32x2r rw[RT == RT_BF16 ? U : 1][RT == RT_BF16 ? K : 1][R];
            bool live[U], ok1[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t qb = qb0 + u * qstride;
                live[u] = qb + threadIdx.x < nq;
                ok1[u] = R == 2 && qb + kBlock + threadIdx.x < nq;
                if (!live[u]) continue;
                const int64_t wb = qb * 4;
#pragma unroll
                for (int h = 0; h < R; ++h) {
                    if (h == 1 && !ok1[u]) continue;
                    const uint32_t fo = (h * kBlock + threadIdx.x) * 16u;
                    tq[u][h] = ld_f4_at(a.theta + wb, fo);
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        if constexpr (RT == RT_F32)
                            rf[u][k] = ld_f4_at(static_cast<const float*>(a.replicas[k]) + wb, fo);
                        else
                            rw[u][k][h] = ld_u2_at(static_cast<const uint16_t*>(a.replicas[k]) + wb, fo / 2);
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (!live[u]) break;   // the later windows lie past the end as well
                float th[V], r[K][V];
#pragma unroll
                for (int h = 0; h < R; ++h) {
                    const bool z = h == 1 && !ok1[u];
#pragma unroll
                    for (int e = 0; e < 4; ++e) th[4 * h + e] = z ? 0.f : tq[u][h][e];
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        if constexpr (RT == RT_F32) {
#pragma unroll
                            for (int e = 0; e < 4; ++e) r[k][e] = rf[u][k][e];
                        } else {
                            const u32x2r w = z ? u32x2r{0u, 0u} : rw[u][k][h];
                            r[k][4 * h] = bf16_lo(w[0]);
                            r[k][4 * h + 1] = bf16_hi(w[0]);
                            r[k][4 * h + 2] = bf16_lo(w[1]);
                            r[k][4 * h + 3] = bf16_hi(w[1]);
                        }
                    }
                }
                float s[K], q[K], m = 0.f;
#pragma unroll
                for (int k = 0; k < K; ++k) s[k] = q[k] = 0.f;
#pragma unroll
                for (int e = 0; e < V; ++e) {
                    float re[K];
#pragma unroll
                    for (int k = 0; k < K; ++k) re[k] = r[k][e];
                    float tn, vn;
                    uint32_t pbe;
                    one_param<K, STATS, UPDATE, BF16P>(th[e], 0.f, re, a, s, q, m, tn, vn, pbe);
                }
                if constexpr (STATS) {
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        acc[k] += (double)s[k];
                        acc[K + k] += (double)q[k];
                    }
                    acc[2 * K] += (double)m;
                }
            }
        }
    } else {
        for (int64_t qb = (int64_t)blockIdx.x * kBlock * R; qb < nq; qb += qstride) {
            if (qb + threadIdx.x >= nq) continue;
            // run 1 (bf16) exists unless this is the last, shorter window
            const bool ok1 = R == 2 && qb + kBlock + threadIdx.x < nq;
            const int64_t wb = qb * 4;                        // first parameter of the window
            float* const th_w = a.theta + wb;
            float* const mo_w = UPDATE ? a.momentum + wb : nullptr;
            float th[V], v[V], r[K][V];
#pragma unroll
            for (int h = 0; h < R; ++h) {
                const uint32_t fo = (h * kBlock + threadIdx.x) * 16u;   // byte offset in fp32 buffers
                if (h == 1 && !ok1) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        th[4 * h + e] = v[4 * h + e] = 0.f;
#pragma unroll
                        for (int k = 0; k < K; ++k) r[k][4 * h + e] = 0.f;
                    }
                    continue;
                }
                const f32x4 t4 = ld_f4_at(th_w, fo);
#pragma unroll
                for (int e = 0; e < 4; ++e) th[4 * h + e] = t4[e];
                if constexpr (UPDATE) {
                    const f32x4 v4 = ld_f4_at(mo_w, fo);
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[4 * h + e] = v4[e];
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[4 * h + e] = 0.f;
                }
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    if constexpr (RT == RT_F32) {
                        const f32x4 r4 = ld_f4_at(static_cast<const float*>(a.replicas[k]) + wb, fo);
#pragma unroll
                        for (int e = 0; e < 4; ++e) r[k][e] = r4[e];
                    } else {
                        const u32x2r w = ld_u2_at(static_cast<const uint16_t*>(a.replicas[k]) + wb, fo / 2);
                        r[k][4 * h] = bf16_lo(w[0]);
                        r[k][4 * h + 1] = bf16_hi(w[0]);
                        r[k][4 * h + 2] = bf16_lo(w[1]);
                        r[k][4 * h + 3] = bf16_hi(w[1]);
                    }
                }
            }

            float s[K], q[K], m = 0.f;
#pragma unroll
            for (int k = 0; k < K; ++k) s[k] = q[k] = 0.f;
            float th_new[V], v_new[V];
            uint32_t pb[V];
#pragma unroll
            for (int e = 0; e < V; ++e) {
                float re[K];
#pragma unroll
                for (int k = 0; k < K; ++k) re[k] = r[k][e];
                one_param<K, STATS, UPDATE, BF16P>(th[e], v[e], re, a, s, q, m, th_new[e], v_new[e], pb[e]);
            }
            if constexpr (STATS) {
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    acc[k] += (double)s[k];
                    acc[K + k] += (double)q[k];
                }
                acc[2 * K] += (double)m;
            }
#pragma unroll
            for (int h = 0; h < R; ++h) {
                if (h == 1 && !ok1) continue;
                const uint32_t fo = (h * kBlock + threadIdx.x) * 16u;
                if constexpr (BF16P) {
                    // 2 bytes per parameter: 8 per quad
                    if (a.payload != nullptr)
                        st_u2_at(a.payload + wb, fo / 2, u32x2r{pb[4 * h] | pb[4 * h + 1] << 16,
                                                                pb[4 * h + 2] | pb[4 * h + 3] << 16});
                }
                if constexpr (UPDATE) {
                    const f32x4 o = {th_new[4 * h], th_new[4 * h + 1], th_new[4 * h + 2], th_new[4 * h + 3]};
                    st_f4_at(th_w, fo, o);
                    st_f4_at(mo_w, fo, f32x4{v_new[4 * h], v_new[4 * h + 1], v_new[4 * h + 2], v_new[4 * h + 3]});
                    if constexpr (RESET) {
                        if constexpr (RT == RT_F32) {
#pragma unroll
                            for (int k = 0; k < K; ++k) st_f4_at(static_cast<float*>(a.replicas[k]) + wb, fo, o);
                        } else {
                            const u32x2r w = {bf16_pack(o[0], o[1]), bf16_pack(o[2], o[3])};
#pragma unroll
                            for (int k = 0; k < K; ++k) st_u2_at(static_cast<uint16_t*>(a.replicas[k]) + wb, fo / 2, w);
                        }
                    }
                }
            }
        }
    }

    // Ragged tail: the last n mod 4 parameters, one per thread of workgroup 0.
    const int64_t tail0 = nq * 4;
    if (gtid < a.n - tail0) {
        const int64_t j = tail0 + gtid;
        const float th = a.theta[j];
        const float v = UPDATE ? a.momentum[j] : 0.f;
        float r[K];
#pragma unroll
        for (int k = 0; k < K; ++k) {
            if constexpr (RT == RT_F32)
                r[k] = static_cast<const float*>(a.replicas[k])[j];
            else
                r[k] = __uint_as_float((uint32_t) static_cast<const uint16_t*>(a.replicas[k])[j] << 16);
        }
        float s[K], q[K], m = 0.f, th_new = 0.f, v_new = 0.f;
        uint32_t pb = 0;
#pragma unroll
        for (int k = 0; k < K; ++k) s[k] = q[k] = 0.f;
        one_param<K, STATS, UPDATE, BF16P>(th, v, r, a, s, q, m, th_new, v_new, pb);
        if constexpr (BF16P) {
            if (a.payload != nullptr) a.payload[j] = (uint16_t)pb;
        }
        if constexpr (STATS) {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                acc[k] += (double)s[k];
                acc[K + k] += (double)q[k];
            }
            acc[2 * K] += (double)m;
        }
        if constexpr (UPDATE) {
            a.theta[j] = th_new;
            a.momentum[j] = v_new;
            if constexpr (RESET) {
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    if constexpr (RT == RT_F32)
                        static_cast<float*>(a.replicas[k])[j] = th_new;
                    else
                        static_cast<uint16_t*>(a.replicas[k])[j] = (uint16_t)bf16_rne(th_new);
                }
            }
        }
    }

    if constexpr (STATS) store_partials<NS, kBlock>(acc, a.partials);
}

// Launchers, one per (replica type, mode) translation unit.
typedef hipError_t (*RoundLauncher)(int k, int blocks, hipStream_t stream, const RoundArgs& a);
hipError_t launch_round_f32_m0(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_f32_m1(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_f32_m2(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_f32_m3(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_f32_m4(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_bf16_m0(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_bf16_m1(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_bf16_m2(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_bf16_m3(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_bf16_m4(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_f32_m5(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_f32_m6(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_f32_m7(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_f32_m8(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_bf16_m5(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_bf16_m6(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_bf16_m7(int, int, hipStream_t, const RoundArgs&);
hipError_t launch_round_bf16_m8(int, int, hipStream_t, const RoundArgs&);
// Resident workgroups per compute unit of the fused (update + stats + reset) kernel.
int occupancy_round_f32_m4(int k);
int occupancy_round_bf16_m4(int k);
int occupancy_round_f32_m8(int k);
int occupancy_round_bf16_m8(int k);

}  // namespace autoloco
