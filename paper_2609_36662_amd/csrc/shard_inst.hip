// Launchers of the per-GPU kernels of the one-replica-per-GPU round.
#include "shard_kernels.hpp"

namespace autoloco {

namespace {

template <int K>
hipError_t shard_k(int blocks, hipStream_t s, const ShardArgs& a) {
    hipLaunchKernelGGL(shard_step_kernel<K>, dim3(blocks), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

using ShardFn = hipError_t (*)(int, hipStream_t, const ShardArgs&);

}  // namespace

hipError_t launch_rank_payload(int rt, int blocks, hipStream_t s, const RankPayloadArgs& a) {
    if (rt == RT_BF16)
        hipLaunchKernelGGL(rank_payload_kernel<RT_BF16>, dim3(blocks), dim3(kBlock), 0, s, a);
    else
        hipLaunchKernelGGL(rank_payload_kernel<RT_F32>, dim3(blocks), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_shard_step(int k, int blocks, hipStream_t s, const ShardArgs& a) {
    static const ShardFn table[kMaxK + 1] = {
        nullptr,    shard_k<1>,  shard_k<2>,  shard_k<3>,  shard_k<4>,  shard_k<5>,  shard_k<6>,  shard_k<7>,  shard_k<8>,
        shard_k<9>, shard_k<10>, shard_k<11>, shard_k<12>, shard_k<13>, shard_k<14>, shard_k<15>, shard_k<16>};
    if (k < 1 || k > kMaxK) return hipErrorInvalidValue;
    return table[k](blocks, s, a);
}

}  // namespace autoloco
