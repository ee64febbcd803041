// Instances of the second reduction stage: one per number of sums (1..33:
// one norm, K norms, or the round's 2K+1 sums) and producer workgroup size.
#include <utility>

#include "reduce.hpp"

namespace autoloco {
namespace {

template <int NS>
hipError_t finish_ns(int nt, int nblocks, const double* partials, double* sums, hipStream_t s, double* h) {
    if (nt == 512)
        hipLaunchKernelGGL((finish_sums_kernel<NS, 512>), dim3(1), dim3(512), 0, s, partials, nblocks, sums, h);
    else if (nt == 256)
        hipLaunchKernelGGL((finish_sums_kernel<NS, 256>), dim3(1), dim3(256), 0, s, partials, nblocks, sums, h);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

template <int... I>
struct Table {
    static hipError_t go(int ns, int nt, int nblocks, const double* p, double* s, hipStream_t st, double* h) {
        hipError_t e = hipErrorInvalidValue;
        ((ns == I + 1 ? (e = finish_ns<I + 1>(nt, nblocks, p, s, st, h), true) : false) || ...);
        return e;
    }
};

template <int... I>
Table<I...> make_table(std::integer_sequence<int, I...>);

}  // namespace

hipError_t launch_finish_sums(int ns, int nt, int nblocks, const double* partials, double* sums,
                              hipStream_t stream, double* host_copy) {
    if (ns < 1 || ns > kMaxSums || nblocks < 1) return hipErrorInvalidValue;
    using T = decltype(make_table(std::make_integer_sequence<int, kMaxSums>{}));
    return T::go(ns, nt, nblocks, partials, sums, stream, host_copy);
}

}  // namespace autoloco
