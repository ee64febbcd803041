// One (replica type, mode) slice of the round kernels, for every K.
// Compiled once per slice with -DAL_RT=<0|1> -DAL_RTNAME=<f32|bf16> -DAL_MODE=<0..8>,
// so the template instances build in parallel.
#include "round_kernels.hpp"

#if !defined(AL_RT) || !defined(AL_MODE) || !defined(AL_RTNAME)
#error "AL_RT, AL_RTNAME and AL_MODE must be defined"
#endif

#define AL_CAT(a, b, c) a##b##_m##c
#define AL_NAME(rt, m) AL_CAT(launch_round_, rt, m)
#define AL_OCC_NAME(rt, m) AL_CAT(occupancy_round_, rt, m)

namespace autoloco {
namespace {

constexpr bool kBf16p = AL_MODE >= MODE_P_UPDATE;
constexpr int kBase = kBf16p ? AL_MODE - 4 : AL_MODE;   // the plain mode with the same outputs
constexpr bool kStats = kBase == MODE_STATS || kBase == MODE_UPDATE_STATS || kBase == MODE_UPDATE_STATS_RESET;
constexpr bool kUpdate = kBase != MODE_STATS;
constexpr bool kReset = kBase == MODE_UPDATE_RESET || kBase == MODE_UPDATE_STATS_RESET;

template <int K>
hipError_t launch_k(int blocks, hipStream_t stream, const RoundArgs& a) {
    hipLaunchKernelGGL((round_kernel<K, AL_RT, kStats, kUpdate, kReset, kBf16p>), dim3(blocks), dim3(kBlock), 0, stream,
                       a);
    return hipGetLastError();
}

template <int K>
int occ_k() {
    int blocks = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, round_kernel<K, AL_RT, kStats, kUpdate, kReset, kBf16p>, kBlock,
                                                     0) != hipSuccess)
        return 0;
    return blocks;
}

}  // namespace

int AL_OCC_NAME(AL_RTNAME, AL_MODE)(int k) {
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

hipError_t AL_NAME(AL_RTNAME, AL_MODE)(int k, int blocks, hipStream_t stream, const RoundArgs& a) {
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

}  // namespace autoloco
