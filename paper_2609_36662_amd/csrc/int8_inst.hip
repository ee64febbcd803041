// One (replica type, stats, reset) slice of the INT8-codec round kernels, for
// every K.  Compiled once per slice with -DAL_RT=<0|1> -DAL_RTNAME=<f32|bf16>
// -DAL_STATS=<0|1> -DAL_RESET=<0|1>.
#include "int8_kernels.hpp"

#if !defined(AL_RT) || !defined(AL_RTNAME) || !defined(AL_STATS) || !defined(AL_RESET)
#error "AL_RT, AL_RTNAME, AL_STATS and AL_RESET must be defined"
#endif

#define AL_CAT4(a, b, c, d) a##b##_s##c##r##d
#define AL_LNAME(rt, s, r) AL_CAT4(launch_int8_, rt, s, r)
#define AL_ONAME(rt, s, r) AL_CAT4(occupancy_int8_, rt, s, r)

namespace autoloco {
namespace {

template <int K>
hipError_t launch_k(int blocks, hipStream_t stream, const Int8Args& a) {
    hipLaunchKernelGGL((int8_round_kernel<K, AL_RT, AL_STATS != 0, AL_RESET != 0>), dim3(blocks), dim3(kInt8Threads),
                       0, stream, a);
    return hipGetLastError();
}

template <int K>
int occ_k() {
    int b = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, int8_round_kernel<K, AL_RT, AL_STATS != 0, AL_RESET != 0>,
                                                     kInt8Threads, 0) != hipSuccess)
        return 0;
    return b;
}

}  // namespace

hipError_t AL_LNAME(AL_RTNAME, AL_STATS, AL_RESET)(int k, int blocks, hipStream_t stream, const Int8Args& a) {
    switch (k) {
        case 1: return launch_k<1>(blocks, stream, a);
        case 2: return launch_k<2>(blocks, stream, a);
        case 3: return launch_k<3>(blocks, stream, a);
        case 4: return launch_k<4>(blocks, stream, a);
        case 5: return launch_k<5>(blocks, stream, a);
        case 6: return launch_k<6>(blocks, stream, a);
        case 7: return launch_k<7>(blocks, stream, a);
        case 8: return launch_k<8>(blocks, stream, a);
        case 9: return launch_k<9>(blocks, stream, a);
        case 10: return launch_k<10>(blocks, stream, a);
        case 11: return launch_k<11>(blocks, stream, a);
        case 12: return launch_k<12>(blocks, stream, a);
        case 13: return launch_k<13>(blocks, stream, a);
        case 14: return launch_k<14>(blocks, stream, a);
        case 15: return launch_k<15>(blocks, stream, a);
        case 16: return launch_k<16>(blocks, stream, a);
        default: return hipErrorInvalidValue;
    }
}

#if AL_STATS && AL_RESET
int AL_ONAME(AL_RTNAME, AL_STATS, AL_RESET)(int k) {
    switch (k) {
        case 1: return occ_k<1>();
        case 2: return occ_k<2>();
        case 3: return occ_k<3>();
        case 4: return occ_k<4>();
        case 5: return occ_k<5>();
        case 6: return occ_k<6>();
        case 7: return occ_k<7>();
        case 8: return occ_k<8>();
        case 9: return occ_k<9>();
        case 10: return occ_k<10>();
        case 11: return occ_k<11>();
        case 12: return occ_k<12>();
        case 13: return occ_k<13>();
        case 14: return occ_k<14>();
        case 15: return occ_k<15>();
        case 16: return occ_k<16>();
        default: return 0;
    }
}
#endif

}  // namespace autoloco
