// Launchers of the inner AdamW kernels.
#include "adamw_kernels.hpp"

namespace autoloco {

namespace {

template <int K>
hipError_t grad_norm_k(int blocks, hipStream_t s, const GradNormArgs& a) {
    hipLaunchKernelGGL(grad_norm_kernel<K>, dim3(blocks), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

using GradNormFn = hipError_t (*)(int, hipStream_t, const GradNormArgs&);

}  // namespace

hipError_t launch_grad_norm(int k, int blocks, hipStream_t s, const GradNormArgs& a) {
    static const GradNormFn table[kMaxK + 1] = {
        nullptr,         grad_norm_k<1>,  grad_norm_k<2>,  grad_norm_k<3>,  grad_norm_k<4>,  grad_norm_k<5>,
        grad_norm_k<6>,  grad_norm_k<7>,  grad_norm_k<8>,  grad_norm_k<9>,  grad_norm_k<10>, grad_norm_k<11>,
        grad_norm_k<12>, grad_norm_k<13>, grad_norm_k<14>, grad_norm_k<15>, grad_norm_k<16>};
    if (k < 1 || k > kMaxK) return hipErrorInvalidValue;
    return table[k](blocks, s, a);
}

hipError_t launch_adamw(bool copy, bool traffic, int k, int blocks_per_worker, hipStream_t s, const AdamWArgs& a) {
    if (k < 1 || k > kMaxK) return hipErrorInvalidValue;
    const dim3 grid(blocks_per_worker, k);
    if (traffic) {
        if (copy)
            hipLaunchKernelGGL((adamw_kernel<true, true>), grid, dim3(kBlock), 0, s, a);
        else
            hipLaunchKernelGGL((adamw_kernel<false, true>), grid, dim3(kBlock), 0, s, a);
    } else if (copy) {
        hipLaunchKernelGGL((adamw_kernel<true, false>), grid, dim3(kBlock), 0, s, a);
    } else {
        hipLaunchKernelGGL((adamw_kernel<false, false>), grid, dim3(kBlock), 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace autoloco
