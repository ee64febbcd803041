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
// order-independent: lane exchanges (DPP) inside each wavefront, then the
// waves through LDS, with one barrier each.
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
    double* partials;     // [gridDim.x][2K+1] per-workgroup sums
};

__device__ __forceinline__ float codec_scale(float amax) {
    if (amax == 0.0f) return 1.0f;
    const float s = amax / 127.0f;
    return s < 0x1p-126f ? 0x1p-126f : s;
}

// Codes of x[0..NV) at scale s (r = fp32(1/s)): the integers nearest
// fp32(x / s), ties to even, clipped to +-127.  t = x * r differs from
// fp32(x / s) by at most (3u + u^2) |x / s| <= 2.28e-5 here (u = 2^-24,
// |x / s| <= 127.00003), so rint(t) is the same integer unless t lies within
// 3e-5 of a half-integer; only then (about 6e-5 of the elements) is the IEEE
// quotient formed.  t - rint(t) is exact (Sterbenz); where the compiler fuses
// the product into it, the test value is x r - rint(t) rounded once, within
// u |x / s| of the exact one, which the margin covers as well.  The common path
// has no per-element test: each lane keeps the largest |t - rint(t)| of its
// elements, and one wavefront-uniform branch leads to the quotients when some
// lane's exceeds the bound.  A NaN t drops out of that maximum, which is
// harmless: t is NaN only when x is NaN, or infinite in a block whose scale is
// infinite (r = 0), and the quotient is NaN then too.
// The clip is implied by the scale and costs no instruction: s is the block's
// largest magnitude over 127 rounded once (or the larger 2^-126), so |t| and
// |fp32(x / s)| are at most 127 (1 + 3 * 2^-24) < 127.5 for every x of the
// block, and their nearest integers lie in [-127, 127].  (A non-finite block
// has an infinite scale and decodes to non-finite values either way.)
// x(e) gives element e (evaluated again on the rare path).
template <int NV, typename X>
__device__ __forceinline__ void codec_q(X x, float s, float r, float (&q)[NV]) {
    constexpr float kNear = 0.5f - 3.0e-5f;
    float dev = 0.0f;
#pragma unroll
    for (int e = 0; e < NV; ++e) {
        const float t = x(e) * r;
        q[e] = __builtin_rintf(t);
        dev = fmaxf(dev, fabsf(t - q[e]));
    }
    if (__builtin_amdgcn_ballot_w64(dev >= kNear) != 0) {
#pragma unroll
        for (int e = 0; e < NV; ++e)
            if (!(fabsf(x(e) * r - q[e]) < kNear)) q[e] = __builtin_rintf(x(e) / s);
    }
}

// Maximum over the 64 lanes of a wavefront of a non-negative float (or NaN),
// compared as its bit pattern, which orders non-negative floats as numbers:
// DPP exchanges within each row of 16 lanes, then the four row results are read
// out as wave-uniform values.
__device__ __forceinline__ uint32_t wave_max_bits(uint32_t x) {
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x141, 0xF, 0xF, false));  // row_half_mirror
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x140, 0xF, 0xF, false));  // row_mirror
    const uint32_t a = max((uint32_t)__builtin_amdgcn_readlane((int)x, 0), (uint32_t)__builtin_amdgcn_readlane((int)x, 16));
    const uint32_t b = max((uint32_t)__builtin_amdgcn_readlane((int)x, 32), (uint32_t)__builtin_amdgcn_readlane((int)x, 48));
    return max(a, b);
}

// Maximum of NV non-negative values over the workgroup (every thread gets the
// result).  One barrier: the caller gives each use within a loop iteration its
// own LDS region, so a wave that runs ahead into the next iteration writes a
// region every other wave has finished reading (they all passed a later
// barrier of this iteration after reading it).  Every thread of the workgroup
// must be active.
template <int NV, int NT>
__device__ __forceinline__ void block_max(float (&v)[NV], uint32_t* lds) {
    constexpr int NW = NT / 64;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const uint32_t m = wave_max_bits(__float_as_uint(v[j]));
        if (lane == 0) lds[j * NW + wave] = m;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        uint32_t x = lds[j * NW];
#pragma unroll
        for (int w = 1; w < NW; ++w) x = max(x, lds[j * NW + w]);
        v[j] = __uint_as_float(x);
    }
}

// Block maxima of up to 8 workers' non-negative values (compared as their bit
// patterns) over a workgroup of NW waves; returns worker (lane mod 8)'s in
// every lane.  Instead of one wavefront reduction per worker, a halving
// exchange inside each group of 8 lanes (partners 7 - i, i ^ 1, i ^ 2; every
// lane sends the half of its values its partner keeps) leaves lane i with the
// group's maximum of worker w(i) = 4 b2 + 2 b0 + b1 (b_j the bits of i), a
// rotation by 8 lanes joins the two groups of each row of 16, and every wave
// stores its 4 row values per worker.  After the one barrier each lane reads
// the 4 NW values of its worker (rows 16-byte aligned, 4 words apart in bank
// order, so the 8 workers' reads fall in distinct banks).  The same reuse rule
// as block_max holds for the LDS region.
constexpr int kWorkerMaxStride(int nw) { return 4 * nw + 4; }
template <int K, int NW>
__device__ __forceinline__ float worker_block_max(const float (&v)[K], uint32_t* lds) {
    static_assert(K <= 8, "at most 8 workers");
    constexpr int S = kWorkerMaxStride(NW);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t m[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) m[j] = j < K ? __float_as_uint(v[j]) : 0u;
    const bool lo = (lane & 4) == 0, even = (lane & 1) == 0, b1 = (lane & 2) != 0;
    uint32_t a4[4], a2[2];
#pragma unroll
    for (int j = 0; j < 4; ++j) {   // partner 7 - i (row_half_mirror): the low lane keeps workers 0..3
        const uint32_t send = lo ? m[j + 4] : m[j], keep = lo ? m[j] : m[j + 4];
        a4[j] = max(keep, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)send, 0x141, 0xF, 0xF, false));
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {   // partner i ^ 1 (quad_perm 1,0,3,2)
        const uint32_t send = even ? a4[j + 2] : a4[j], keep = even ? a4[j] : a4[j + 2];
        a2[j] = max(keep, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)send, 0xB1, 0xF, 0xF, false));
    }
    uint32_t c;
    {                               // partner i ^ 2 (quad_perm 2,3,0,1)
        const uint32_t send = b1 ? a2[0] : a2[1], keep = b1 ? a2[1] : a2[0];
        c = max(keep, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)send, 0x4E, 0xF, 0xF, false));
    }
    c = max(c, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)c, 0x128, 0xF, 0xF, false));   // row_ror:8
    const int w = (lane & 4) + ((lane & 1) << 1) + ((lane & 2) >> 1);
    if ((lane & 8) == 0) lds[w * S + wave * 4 + (lane >> 4)] = c;
    __syncthreads();
    const uint32_t* p = lds + (lane & 7) * S;
    uint32_t r = 0;
#pragma unroll
    for (int i = 0; i < 4 * NW; ++i) r = max(r, p[i]);
    return __uint_as_float(r);
}

constexpr int kInt8Threads = 512;  // one codec block of 4,096 parameters per workgroup

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <bool B>
struct BoolC {
    static constexpr bool value = B;
};

// Each thread of a workgroup owns 8 parameters of a codec block: two runs of
// 4, 2,048 apart, so every wavefront instruction covers one contiguous run
// (1 KB of fp32, 512 B of bf16) and no cache line is written in parts.  The loop runs over the full blocks, in which
// every load and store is a whole vector; the one shorter last block, if any,
// goes through a second instance of the same body with per-element accesses.
// The next block of a workgroup is loaded while the current one is encoded:
// up to 8 bf16 workers its raw replica words, theta and momentum go to
// registers (the block barriers wait for LDS traffic only), pseudo-gradients
// are formed from the raw words where they are used, and each thread's fp64
// sums live in LDS slots of its own, which leaves the registers for it;
// up to 8 fp32 workers its theta and replica vectors go straight to LDS
// (global_load_lds_dwordx4, no registers), each wave into pieces only it reads
// back, behind an explicit count of the vector memory instructions issued
// after them (the compiler does not order these loads against later LDS
// reads by itself).
template <int K, int RT, bool STATS, bool RESET>
__global__ void __launch_bounds__(kInt8Threads) int8_round_kernel(Int8Args a) {
    constexpr int NT = kInt8Threads;
    constexpr int V = 8;
    constexpr int NS = STATS ? 2 * K + 1 : 1;
    constexpr int G = 2;   // runs of W parameters per thread
    constexpr int W = V / G;
    constexpr bool PF = RT == RT_BF16 && K <= 8;
    // fp32 replicas up to 8 workers: the next block's theta and replica vectors
    // stream into LDS (direct global-to-LDS loads, no registers) while the
    // current block is encoded; (K + 1) * 16 KB of LDS
    constexpr bool LP = RT == RT_F32 && K <= 8;
    constexpr int NW = NT / 64;
    constexpr int KW = RT == RT_BF16 ? K : 1;   // raw bf16 replica words held per thread
    // worker block maxima
    __shared__ uint32_t lds_max[K <= 8 ? 8 * kWorkerMaxStride(NT / 64) : NT / 64 * K];
    __shared__ uint32_t lds_mmax[NT / 64];      // the mean's block maximum
    // prefetched vectors, [stream (theta, replica 0..K-1)][run][wave][lane];
    // every wave reads back only the 1 KB pieces it loaded itself
    __shared__ f32x4 lds_pf[LP ? (K + 1) * G * NT : 1];

    // per-thread fp64 sums: in registers, or with the bf16 prefetch (which holds
    // many registers) in this thread's own LDS slots, [sum][thread]
    constexpr bool AL = PF;
    double acc[AL ? 1 : NS];
    __shared__ double lds_acc[AL ? NS * NT : 1];
    auto acc_add = [&](int j, double x) {
        if constexpr (AL)
            lds_acc[j * NT + threadIdx.x] += x;
        else
            acc[j] += x;
    };
#pragma unroll
    for (int j = 0; j < NS; ++j) {
        if constexpr (AL)
            lds_acc[j * NT + threadIdx.x] = 0.0;
        else
            acc[j] = 0.0;
    }

    const int64_t nfull = a.n / kCodecBlock;
    const int64_t nblocks = (a.n + kCodecBlock - 1) / kCodecBlock;

    // LDS prefetch: this wave's piece of stream s, run g
    const int wave = threadIdx.x >> 6;
    auto pf_piece = [&](int s, int g) { return lds_pf + ((s * G + g) * NW + wave) * 64; };
    // Issues the (K + 1) * G direct loads of full block b: lane l's 16 bytes
    // land at its wave's piece + 16 l.
    auto pf_issue = [&](int64_t b) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int64_t o = b * kCodecBlock + g * (kCodecBlock / 2) + (int64_t)threadIdx.x * W;
#pragma unroll
            for (int s = 0; s <= K; ++s) {
                const float* src = s == 0 ? a.theta + o : static_cast<const float*>(a.replicas[s - 1]) + o;
                __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)src,
                                                 (void __attribute__((address_space(3)))*)pf_piece(s, g), 16, 0, 0);
            }
        }
    };

    // bf16: raw words (two per run), theta and (full blocks) momentum of one
    // block (full: vector loads; else per element, zero beyond n)
    // two register sets for the bf16 prefetch: the loop takes blocks in pairs and
    // the sets swap roles (current / next) instead of being copied
    u32x2 wA[KW][G], wB[PF ? KW : 1][G];
    float tA[V], tB[PF ? V : 1];
    float mA[PF ? V : 1], mB[PF ? V : 1];
    auto load_bf16 = [&](int64_t b, auto& w, float (&t)[V], auto& m, auto full_c) {
        constexpr bool FULL = decltype(full_c)::value;
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int64_t o = b * kCodecBlock + g * (kCodecBlock / 2) + (int64_t)threadIdx.x * W;
            if constexpr (FULL) {
                const f32x4 t4 = ld_f4(a.theta + o);
#pragma unroll
                for (int e = 0; e < W; ++e) t[g * W + e] = t4[e];
                if constexpr (PF) {
                    const f32x4 m4 = ld_f4(a.momentum + o);
#pragma unroll
                    for (int e = 0; e < W; ++e) m[g * W + e] = m4[e];
                }
#pragma unroll
                for (int k = 0; k < KW; ++k)
                    w[k][g] = __builtin_nontemporal_load(
                        reinterpret_cast<const u32x2*>(static_cast<const uint16_t*>(a.replicas[k]) + o));
            } else {
                const int64_t left = a.n - o;
#pragma unroll
                for (int e = 0; e < W; ++e) t[g * W + e] = e < left ? a.theta[o + e] : 0.0f;
#pragma unroll
                for (int k = 0; k < KW; ++k) {
                    const uint16_t* r = static_cast<const uint16_t*>(a.replicas[k]) + o;
                    uint32_t h[W];
#pragma unroll
                    for (int e = 0; e < W; ++e) h[e] = e < left ? r[e] : 0u;
                    w[k][g] = u32x2{h[0] | h[1] << 16, h[2] | h[3] << 16};
                }
            }
        }
    };

    auto body = [&](int64_t blk, auto full_c, auto& cw, auto& cth, auto& cm, auto& nw, auto& nth, auto& nm) {
        constexpr bool FULL = decltype(full_c)::value;
        int64_t off[G];
        int valid[G];
        bool ok[V];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            off[g] = blk * kCodecBlock + g * (kCodecBlock / 2) + (int64_t)threadIdx.x * W;
            if constexpr (FULL) {
                valid[g] = W;
            } else {
                const int64_t left = a.n - off[g];
                valid[g] = left >= W ? W : (left > 0 ? (int)left : 0);
            }
#pragma unroll
            for (int e = 0; e < W; ++e) ok[g * W + e] = e < valid[g];
        }

        float th[V], v[V], d[RT == RT_F32 ? K : 1][V];
        if constexpr (RT == RT_BF16) {
            // momentum: from the prefetch, or loaded first (the update waits for
            // it, and in-order completion then leaves the loads below in flight)
            if constexpr (PF && FULL) {
#pragma unroll
                for (int e = 0; e < V; ++e) v[e] = cm[e];
            } else
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const int64_t o = off[g];
                if constexpr (FULL) {
                    const f32x4 v4 = ld_f4(a.momentum + o);
#pragma unroll
                    for (int e = 0; e < W; ++e) v[g * W + e] = v4[e];
                } else {
#pragma unroll
                    for (int e = 0; e < W; ++e) v[g * W + e] = e < valid[g] ? a.momentum[o + e] : 0.0f;
                }
            }
            if constexpr (PF && FULL) {
                // next full block of this workgroup; on its last one, this block again
                // (every iteration issues the same loads)
                const int64_t nb = blk + gridDim.x < nfull ? blk + gridDim.x : blk;
                load_bf16(nb, nw, nth, nm, BoolC<true>{});
            } else {
                load_bf16(blk, cw, cth, cm, full_c);
            }
#pragma unroll
            for (int e = 0; e < V; ++e) th[e] = cth[e];
        } else {
            if constexpr (FULL && LP) {
                // This block's direct loads were issued in the previous iteration
                // (or before the loop), and every vector memory instruction issued
                // after them is one of that iteration's stores: G of theta, G of
                // v and, with the reset, G of each replica (more with the encoded
                // mean).  In-order completion makes "at most that many
                // outstanding" imply the loads have landed in LDS.
                constexpr int after = G * (2 + (RESET ? K : 0));
                __builtin_amdgcn_s_waitcnt((after & 0xF) | ((after >> 4) << 14) | 0x70 | 0xF00);
            }
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const int64_t o = off[g];
                if constexpr (FULL && LP) {
                    // theta and the replicas from the LDS prefetch (complete: see the
                    // wait above), momentum from memory
                    const int lane = threadIdx.x & 63;
                    const f32x4 t4 = pf_piece(0, g)[lane], v4 = ld_f4(a.momentum + o);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        th[g * W + e] = t4[e];
                        v[g * W + e] = v4[e];
                    }
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        const f32x4 r4 = pf_piece(k + 1, g)[lane];
#pragma unroll
                        for (int e = 0; e < 4; ++e) d[k][g * W + e] = th[g * W + e] - r4[e];
                    }
                } else if constexpr (FULL) {
                    const f32x4 t4 = ld_f4(a.theta + o), v4 = ld_f4(a.momentum + o);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        th[g * W + e] = t4[e];
                        v[g * W + e] = v4[e];
                    }
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        const f32x4 r4 = ld_f4(static_cast<const float*>(a.replicas[k]) + o);
#pragma unroll
                        for (int e = 0; e < 4; ++e) d[k][g * W + e] = th[g * W + e] - r4[e];
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < W; ++e) {
                        const bool in = e < valid[g];
                        const int x = g * W + e;
                        th[x] = in ? a.theta[o + e] : 0.0f;
                        v[x] = in ? a.momentum[o + e] : 0.0f;
#pragma unroll
                        for (int k = 0; k < K; ++k)
                            d[k][x] = in ? th[x] - static_cast<const float*>(a.replicas[k])[o + e] : 0.0f;
                    }
                }
            }
        }
        if constexpr (RT == RT_F32 && LP && FULL) {
            // every LDS read of this block has returned before the next block's
            // direct loads overwrite the pieces; then issue them (on the last
            // block of this workgroup, this block again, so every iteration
            // issues the same instructions; those values are not used)
            __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
            pf_issue(blk + gridDim.x < nfull ? blk + gridDim.x : blk);
        }
        // pseudo-gradient k of parameter e (bf16: from the raw replica word)
        auto D = [&](int k, int e) -> float {
            if constexpr (RT == RT_F32)
                return d[k][e];
            else
                return th[e] - ((e & 1) ? bf16_hi(cw[k][e / W][(e % W) >> 1]) : bf16_lo(cw[k][e / W][(e % W) >> 1]));
        };

        // local-drift energy before quantisation
        if constexpr (STATS) {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                float s = 0.f;
#pragma unroll
                for (int e = 0; e < V; ++e) s = __builtin_fmaf(D(k, e), D(k, e), s);
                acc_add(k, (double)s);
            }
        }

        // worker block scales
        float amax[K];
#pragma unroll
        for (int k = 0; k < K; ++k) {
            float m = 0.f;
#pragma unroll
            for (int e = 0; e < V; ++e) m = fmaxf(m, fabsf(D(k, e)));
            amax[k] = m;
        }
        float am_lane = 0.0f;   // up to 8 workers: worker (lane mod 8)'s block maximum
        if constexpr (K <= 8)
            am_lane = worker_block_max<K, NT / 64>(amax, lds_max);
        else
            block_max<K, NT>(amax, lds_max);

        // The K scales and their reciprocals are the same in every lane: lane k
        // computes worker k's (one IEEE division of each kind for all workers
        // instead of K), and every lane reads them back.
        float scale_k[K], recip_k[K];
        {
            const int lane = threadIdx.x & 63;
            float am = am_lane;
            if constexpr (K > 8) {
                am = amax[0];
#pragma unroll
                for (int k = 1; k < K; ++k) am = lane == k ? amax[k] : am;
            }
            const float sv = codec_scale(am);
            const float rv = 1.0f / sv;
#pragma unroll
            for (int k = 0; k < K; ++k) {
                scale_k[k] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sv), k));
                recip_k[k] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(rv), k));
            }
        }

        // decode every worker and average: fp64 sum in worker order, times fp64(1/K)
        double sum[V];
#pragma unroll
        for (int e = 0; e < V; ++e) sum[e] = 0.0;
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const float s = scale_k[k];
            const float r = recip_k[k];
            float q[V];
            codec_q<V>([&](int e) { return D(k, e); }, s, r, q);
#pragma unroll
            for (int e = 0; e < V; ++e) sum[e] += (double)(q[e] * s);
        }
        float mean[V];
        float mmax[1] = {0.f};
#pragma unroll
        for (int e = 0; e < V; ++e) {
            mean[e] = (float)(sum[e] * a.inv_k);
            mmax[0] = fmaxf(mmax[0], fabsf(mean[e]));
        }
        block_max<1, NT>(mmax, lds_mmax);
        const float sm = codec_scale(mmax[0]);
        const float rm = 1.0f / sm;

        float agg[V], qm[V];
        codec_q<V>([&](int e) { return mean[e]; }, sm, rm, qm);
#pragma unroll
        for (int e = 0; e < V; ++e) agg[e] = ok[e] ? qm[e] * sm : 0.0f;
        if (a.mean_codes != nullptr) {
#pragma unroll
            for (int g = 0; g < G; ++g) {
                if (FULL || valid[g] == W) {
                    uint32_t w[W / 4];
#pragma unroll
                    for (int h = 0; h < W / 4; ++h) {
                        w[h] = 0;
#pragma unroll
                        for (int e = 0; e < 4; ++e) w[h] |= (uint32_t)(uint8_t)(int8_t)qm[g * W + 4 * h + e] << (8 * e);
                    }
                    if constexpr (W == 4)
                        __builtin_nontemporal_store(w[0], reinterpret_cast<uint32_t*>(a.mean_codes + off[g]));
                    else
                        __builtin_nontemporal_store(u32x2{w[0], w[1]}, reinterpret_cast<u32x2*>(a.mean_codes + off[g]));
                } else {
#pragma unroll
                    for (int e = 0; e < W; ++e)
                        if (e < valid[g]) a.mean_codes[off[g] + e] = (int8_t)qm[g * W + e];
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
                    const float t = D(k, e) - agg[e];
                    q = __builtin_fmaf(t, t, q);
                }
                acc_add(K + k, (double)q);
            }
            float m = 0.f;
#pragma unroll
            for (int e = 0; e < V; ++e) m = __builtin_fmaf(agg[e], agg[e], m);
            acc_add(2 * K, (double)m);
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
        for (int g = 0; g < G; ++g) {
            const int64_t o = off[g];
            const float* tn = th_new + g * W;
            const float* vn = v_new + g * W;
            if (FULL || valid[g] == W) {
#pragma unroll
                for (int h = 0; h < W / 4; ++h) {
                    st_f4(a.theta + o + 4 * h, f32x4{tn[4 * h], tn[4 * h + 1], tn[4 * h + 2], tn[4 * h + 3]});
                    st_f4(a.momentum + o + 4 * h, f32x4{vn[4 * h], vn[4 * h + 1], vn[4 * h + 2], vn[4 * h + 3]});
                }
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
                for (int e = 0; e < W; ++e) {
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
    };

    if constexpr (PF) {
        if (blockIdx.x < nfull) load_bf16(blockIdx.x, wA, tA, mA, BoolC<true>{});
        // the first block's words are complete before the loop
        __builtin_amdgcn_s_waitcnt(0);
        // blocks in pairs: the first of a pair prefetches into B, the second into A
        for (int64_t blk = blockIdx.x; blk < nfull; blk += 2 * (int64_t)gridDim.x) {
            body(blk, BoolC<true>{}, wA, tA, mA, wB, tB, mB);
            if (blk + gridDim.x >= nfull) break;
            body(blk + gridDim.x, BoolC<true>{}, wB, tB, mB, wA, tA, mA);
        }
    } else {
        if constexpr (LP) {
            if (blockIdx.x < nfull) pf_issue(blockIdx.x);
            __builtin_amdgcn_s_waitcnt(0);   // the first block's pieces are in LDS
        }
        for (int64_t blk = blockIdx.x; blk < nfull; blk += gridDim.x) body(blk, BoolC<true>{}, wA, tA, mA, wB, tB, mB);
        // the last iteration's direct loads (a re-read, unused) land before anything
        // else uses this workgroup's LDS or the workgroup ends
        if constexpr (LP) __builtin_amdgcn_s_waitcnt(0);
    }
    // the shorter last block belongs to the workgroup the grid stride gives it
    if (nfull < nblocks && nfull % gridDim.x == blockIdx.x) body(nfull, BoolC<false>{}, wA, tA, mA, wB, tB, mB);

    if constexpr (STATS) {
        if constexpr (AL) {
            double r[NS];
#pragma unroll
            for (int j = 0; j < NS; ++j) r[j] = lds_acc[j * NT + threadIdx.x];
            store_partials<NS, NT>(r, a.partials);
        } else {
            store_partials<NS, NT>(acc, a.partials);
        }
    }
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
