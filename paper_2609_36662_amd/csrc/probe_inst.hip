// Instances and launcher of the streaming-pattern probes.  Each entry is
// (runs per lane, class counts A, B, C, D, E); see probe_kernels.hpp.
#include "probe_kernels.hpp"

namespace autoloco {

namespace {

typedef void (*ProbeFn)(ProbeArgs);

struct ProbeEntry {
    ProbePattern p;
    ProbeFn fn;
};

// the run shape: the ceiling table's patterns, then the traffic of the reset
// (theta read, K replicas written: fp32 with one run per lane below three
// replicas and eight from three on, or bf16 with two runs per lane), of
// the worker payload (theta and the replica read, the payload written) and of
// the shard step (theta and v in place, K payload shards read, the mean
// written or not)
#define AUTOLOCO_PROBE_RUNS(X)                                                                         \
    X(1, 10, 0, 0, 0, 0) X(1, 6, 0, 0, 0, 0) X(1, 4, 0, 0, 0, 0) X(1, 2, 0, 0, 0, 0) X(1, 1, 0, 0, 0, 0) \
    X(1, 0, 10, 0, 0, 0) X(1, 0, 8, 0, 0, 0) X(1, 0, 4, 0, 0, 0) X(1, 0, 2, 0, 0, 0) X(1, 0, 1, 0, 0, 0) \
    X(1, 0, 0, 0, 0, 10) X(1, 0, 0, 0, 0, 1) X(1, 0, 5, 0, 0, 5)                                         \
    X(1, 0, 1, 0, 0, 1) X(1, 0, 1, 0, 0, 2) X(1, 0, 1, 0, 0, 4) X(1, 0, 1, 0, 0, 8) X(1, 0, 1, 0, 0, 16) \
    X(2, 10, 0, 0, 0, 0) X(2, 0, 10, 0, 0, 0)                                                          \
    X(2, 0, 1, 0, 1, 0) X(2, 0, 1, 0, 4, 0) X(2, 0, 1, 0, 8, 0) X(2, 0, 1, 0, 16, 0)                     \
    X(2, 0, 2, 0, 1, 0) X(2, 0, 1, 1, 1, 0)                                                            \
    X(2, 2, 0, 1, 1, 0) X(2, 2, 0, 2, 1, 0) X(2, 2, 0, 4, 1, 0) X(2, 2, 0, 8, 1, 0) X(2, 2, 0, 16, 1, 0) \
    X(2, 2, 0, 4, 0, 0) X(2, 2, 0, 8, 0, 0)                                                            \
    X(8, 10, 0, 0, 0, 0) X(8, 0, 10, 0, 0, 0) X(8, 0, 0, 0, 0, 10)                                     \
    X(8, 0, 1, 0, 0, 4) X(8, 0, 1, 0, 0, 8) X(8, 0, 1, 0, 0, 16)

// the tile shapes: 10 streams in place, read, or written
#define AUTOLOCO_PROBE_TILES(X) X(10, 0, 0) X(0, 10, 0) X(0, 0, 10)

#define AUTOLOCO_RUN_ENTRY(R, A, B, C, D, E) {{PROBE_RUN, R, A, B, C, D, E}, probe_run_kernel<R, A, B, C, D, E>},
#define AUTOLOCO_SERIAL_ENTRY(A, B, E) {{PROBE_SERIAL, 0, A, B, 0, 0, E}, probe_tile_kernel<true, A, B, E>},
#define AUTOLOCO_TILE_ENTRY(A, B, E) {{PROBE_TILE, 0, A, B, 0, 0, E}, probe_tile_kernel<false, A, B, E>},

const ProbeEntry kProbes[] = {
    AUTOLOCO_PROBE_RUNS(AUTOLOCO_RUN_ENTRY) AUTOLOCO_PROBE_TILES(AUTOLOCO_SERIAL_ENTRY)
        AUTOLOCO_PROBE_TILES(AUTOLOCO_TILE_ENTRY)};

bool same(const ProbePattern& x, const ProbePattern& y) {
    return x.shape == y.shape && (x.shape != PROBE_RUN || x.r == y.r) && x.a == y.a && x.b == y.b && x.c == y.c &&
           x.d == y.d && x.e == y.e;
}

}  // namespace

bool probe_available(const ProbePattern& p) {
    for (const ProbeEntry& e : kProbes)
        if (same(e.p, p)) return true;
    return false;
}

hipError_t launch_probe_phased(int blocks, hipStream_t stream, const ProbeArgs& a, uint32_t* sync) {
    ProbeArgs args = a;
    uint32_t* sy = sync;
    void* params[] = {&args, &sy};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(probe_phase_kernel<kPhaseStreams>), dim3(blocks),
                                      dim3(kBlock), params, 0, stream);
}

int probe_phased_occupancy() {
    int b = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, probe_phase_kernel<kPhaseStreams>, kBlock, 0) != hipSuccess)
        return 0;
    return b;
}

hipError_t launch_probe(const ProbePattern& p, int blocks, hipStream_t s, const ProbeArgs& a) {
    for (const ProbeEntry& e : kProbes) {
        if (!same(e.p, p)) continue;
        hipLaunchKernelGGL(e.fn, dim3(blocks), dim3(kBlock), 0, s, a);
        return hipGetLastError();
    }
    return hipErrorInvalidValue;
}

}  // namespace autoloco
