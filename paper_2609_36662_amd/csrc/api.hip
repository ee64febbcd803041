// Device entry points of the C ABI: context, argument validation, launch
// shape and dispatch to the round kernels.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "autoloco.h"
#include "adamw_kernels.hpp"
#include "shard_kernels.hpp"
#include "int8_kernels.hpp"
#include "probe_kernels.hpp"
#include "reset_kernels.hpp"
#include "round_kernels.hpp"
#include "traffic_kernels.hpp"

// Hash of the sources the library was built from (set by the build).
#ifndef AUTOLOCO_BUILD_ID
#define AUTOLOCO_BUILD_ID "unknown"
#endif

using namespace autoloco;

namespace {

constexpr int kMaxBlocks = 16384;   // scratch sized for this many workgroups

// Workgroups whose partial sums the static scratch below holds: the default
// grid is one workgroup per compute unit from K = 5 (fp32 replicas) or 6 (bf16)
// and three below (768 on MI355X).
constexpr int kStaticBlocks = 1024;

}  // namespace

// Reduction scratch of autoloco_outer_step_static on every device: per-workgroup
// partial sums [kStaticBlocks][33], then the 33 final sums (270 KB).  In host
// code the name stands for the variable, not for its device address: host code
// uses only the address hipGetSymbolAddress returns with the device current.
static __device__ __align__(256) double scratch[kStaticBlocks * kMaxSums + kMaxSums];

struct autoloco_ctx {
    int device = 0;
    hipStream_t stream = nullptr;
    int num_cus = 0;
    int grid_limit = 0;
    int occupancy[2][AUTOLOCO_MAX_K + 1] = {};  // resident workgroups per CU, by replica type and k
    int occupancy_int8[2][AUTOLOCO_MAX_K + 1] = {};
    int occupancy_bf16p[2][AUTOLOCO_MAX_K + 1] = {};  // the BF16-payload round
    double* partials = nullptr;
    double* sums = nullptr;
    double* host_sums = nullptr;
    double* host_sums_dev = nullptr;  // device view of host_sums (coherent host memory), or null
    bool timing = false;
    bool timed_valid = false;
    hipEvent_t ev_start = nullptr, ev_stop = nullptr, ev_mid = nullptr;
    bool adamw_timed = false;     // the last timed call was an AdamW step
    bool adamw_norm_ran = false;  // ... and it ran the norm pass (ev_start..ev_mid)
    std::string err;
};

namespace {

// Makes the context's device current for the duration of a call.
struct DeviceGuard {
    int prev = -1;
    bool ok = true;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        if (prev != dev) ok = hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

int fail(autoloco_ctx* ctx, int code, const std::string& msg) {
    if (ctx) ctx->err = msg;
    return code;
}

int hip_fail(autoloco_ctx* ctx, hipError_t e, const char* what) {
    return fail(ctx, AUTOLOCO_E_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

size_t replica_size(int32_t dtype) { return dtype == AUTOLOCO_BF16 ? 2 : 4; }

// The kernels dereference every buffer on the context's device: host memory
// and memory of another device are rejected before anything is launched.
int check_device_ptr(autoloco_ctx* ctx, uintptr_t p, const char* name) {
    hipPointerAttribute_t at;
    std::memset(&at, 0, sizeof(at));
    if (hipPointerGetAttributes(&at, reinterpret_cast<const void*>(p)) != hipSuccess) {
        (void)hipGetLastError();
        return fail(ctx, AUTOLOCO_E_INVALID, std::string(name) + " is not device memory");
    }
    if (at.type == hipMemoryTypeManaged || at.isManaged) return AUTOLOCO_OK;
    if (at.type != hipMemoryTypeDevice) return fail(ctx, AUTOLOCO_E_INVALID, std::string(name) + " is not device memory");
    if (at.device != ctx->device)
        return fail(ctx, AUTOLOCO_E_INVALID, std::string(name) + " is on device " + std::to_string(at.device) +
                                                 ", the context's is " + std::to_string(ctx->device));
    return AUTOLOCO_OK;
}

// Default grid: from K = 5 with fp32 replicas and from K = 6 with bf16 one
// workgroup per compute unit (4 waves), below that three, or fewer if fewer fit
// (the fused kernel's occupancy).  Measured on MI355X (256 CUs) with the
// round's buffers spread in HBM, 1.1B K = 8 fp32: fused round 14.14-14.27 ms at
// 256 workgroups against 14.37-14.57 at 768 (the traffic reference alike), and
// no mode slower (statistics only 6.28 against 6.37 ms, with its windows loaded
// ahead); 3B K = 8 bf16, GPT-2 small K = 8 and K = 12-16 gain 1-3 % too, fp32
// K = 5-7 every mode 0-5 %, bf16 K = 6-7 the fused round by 2 % (3B).  At K = 4
// the fused round gains 1 % but the statistics-only mode and the update with
// statistics lose 3-9 % (the update without them and the reset alone 10-23 %),
// and below K = 4 the statistics-only mode needs more waves, so those keep 768.
// Even multiples of 256 are the slowest.  Every mode of a given (k, replica type) uses the same
// grid, so the statistics of a standalone and of a fused call are summed in the
// same order, bit for bit.
// round_grid = false: a kernel with no statistics to keep in step with the
// round's modes (the reset alone, AdamW's gradient-norm pass), which keeps three
// per compute unit at every K.
int blocks_for(const autoloco_ctx* ctx, int64_t n, int32_t dtype, int k, bool bf16p = false,
               bool round_grid = true) {
    const int64_t v = dtype == AUTOLOCO_BF16 ? 8 : 4;
    const int64_t nvec = n / v;
    int per_cu = (bf16p ? ctx->occupancy_bf16p : ctx->occupancy)[dtype == AUTOLOCO_BF16 ? 1 : 0][k];
    if (per_cu > 3) per_cu = 3;
    // one workgroup per CU for the round's modes from K = 5 (fp32) or 6 (bf16
    // replicas), where the modes are as fast or faster than at three
    if (round_grid && k >= (dtype == AUTOLOCO_BF16 ? 6 : 5)) per_cu = 1;
    if (per_cu < 1) per_cu = 1;
    int limit = ctx->grid_limit > 0 ? ctx->grid_limit : ctx->num_cus * per_cu;
    if (limit > kMaxBlocks) limit = kMaxBlocks;
    int64_t want = (nvec + kBlock - 1) / kBlock;
    if (want < 1) want = 1;
    return static_cast<int>(want < limit ? want : limit);
}

// Workgroups per worker of the AdamW update: about two per compute unit in
// total, split evenly over the workers' grid rows (measured at 1.1B, K = 8 on
// MI355X: 512 workgroups 2-3 % faster than 768, 1,024 or 2,048).
int adamw_blocks(const autoloco_ctx* ctx, int64_t n, int k) {
    int limit = ctx->grid_limit > 0 ? ctx->grid_limit : ctx->num_cus * 2;
    if (limit > kMaxBlocks) limit = kMaxBlocks;
    int per = (limit + k - 1) / k;
    const int64_t want = (n / 4 + kBlock - 1) / kBlock;
    if (want < per) per = static_cast<int>(want);
    return per < 1 ? 1 : per;
}

struct Range {
    uintptr_t lo, hi;
    const char* name;
};

// Largest element count a call accepts: far beyond any device's memory, small
// enough that no byte count or address computed from it overflows.
constexpr int64_t kMaxN = int64_t(1) << 56;
const char* const kBadN = "n outside 0..2^56";

// Checks pointers, sizes, alignment and overlap.  need_momentum: the call
// reads and writes the momentum buffer.
int validate(autoloco_ctx* ctx, const autoloco_buffers* b, bool need_momentum) {
    if (ctx == nullptr) return AUTOLOCO_E_INVALID;
    if (b == nullptr) return fail(ctx, AUTOLOCO_E_INVALID, "null buffers");
    if (b->n < 0 || b->n > kMaxN) return fail(ctx, AUTOLOCO_E_INVALID, kBadN);
    if (b->k < 1 || b->k > AUTOLOCO_MAX_K) return fail(ctx, AUTOLOCO_E_INVALID, "k outside 1..16");
    if (b->replica_dtype != AUTOLOCO_F32 && b->replica_dtype != AUTOLOCO_BF16)
        return fail(ctx, AUTOLOCO_E_INVALID, "unknown replica dtype");
    if (b->n == 0) return AUTOLOCO_OK;
    Range r[AUTOLOCO_MAX_K + 2];
    int nr = 0;
    const uintptr_t fbytes = static_cast<uintptr_t>(b->n) * 4u;
    const uintptr_t rbytes = static_cast<uintptr_t>(b->n) * replica_size(b->replica_dtype);
    if (b->theta == nullptr) return fail(ctx, AUTOLOCO_E_INVALID, "null theta");
    r[nr++] = {reinterpret_cast<uintptr_t>(b->theta), reinterpret_cast<uintptr_t>(b->theta) + fbytes, "theta"};
    if (need_momentum) {
        if (b->momentum == nullptr) return fail(ctx, AUTOLOCO_E_INVALID, "null momentum");
        r[nr++] = {reinterpret_cast<uintptr_t>(b->momentum), reinterpret_cast<uintptr_t>(b->momentum) + fbytes,
                   "momentum"};
    }
    for (int k = 0; k < b->k; ++k) {
        if (b->replicas[k] == nullptr) return fail(ctx, AUTOLOCO_E_INVALID, "null replica " + std::to_string(k));
        const uintptr_t p = reinterpret_cast<uintptr_t>(b->replicas[k]);
        r[nr++] = {p, p + rbytes, "replica"};
    }
    for (int i = 0; i < nr; ++i)
        if (r[i].lo % 16 != 0) return fail(ctx, AUTOLOCO_E_ALIGN, std::string(r[i].name) + " not 16-byte aligned");
    for (int i = 0; i < nr; ++i)
        for (int j = i + 1; j < nr; ++j)
            if (r[i].lo < r[j].hi && r[j].lo < r[i].hi)
                return fail(ctx, AUTOLOCO_E_ALIAS, std::string(r[i].name) + " overlaps " + r[j].name);
    for (int i = 0; i < nr; ++i) {
        const int st = check_device_ptr(ctx, r[i].lo, r[i].name);
        if (st != AUTOLOCO_OK) return st;
    }
    return AUTOLOCO_OK;
}

void finish_stats(const double* sums, int k, double eps, autoloco_stats* out) {
    std::memset(out, 0, sizeof(*out));
    out->k = k;
    double ts = 0.0, tq = 0.0;
    for (int i = 0; i < k; ++i) {
        out->sq_norm[i] = sums[i];
        out->sq_dev[i] = sums[k + i];
        ts += sums[i];
        tq += sums[k + i];
    }
    out->sq_mean = sums[2 * k];
    out->D = ts / k;
    out->C = k * out->sq_mean / (out->D + eps);
    out->disagreement = tq / k;
    bool fin = std::isfinite(out->sq_mean) && std::isfinite(out->D) && std::isfinite(out->C) &&
               std::isfinite(out->disagreement);
    for (int i = 0; i < k; ++i) fin = fin && std::isfinite(out->sq_norm[i]) && std::isfinite(out->sq_dev[i]);
    out->finite = fin ? 1 : 0;
}

RoundLauncher launcher(int32_t dtype, int mode) {
    static const RoundLauncher f32[MODE_COUNT] = {launch_round_f32_m0, launch_round_f32_m1, launch_round_f32_m2,
                                                  launch_round_f32_m3, launch_round_f32_m4, launch_round_f32_m5,
                                                  launch_round_f32_m6, launch_round_f32_m7, launch_round_f32_m8};
    static const RoundLauncher bf16[MODE_COUNT] = {launch_round_bf16_m0, launch_round_bf16_m1,
                                                   launch_round_bf16_m2, launch_round_bf16_m3,
                                                   launch_round_bf16_m4, launch_round_bf16_m5,
                                                   launch_round_bf16_m6, launch_round_bf16_m7,
                                                   launch_round_bf16_m8};
    return dtype == AUTOLOCO_BF16 ? bf16[mode] : f32[mode];
}

RoundArgs make_args(autoloco_ctx* ctx, const autoloco_buffers* b) {
    RoundArgs a;
    std::memset(&a, 0, sizeof(a));
    a.theta = b->theta;
    a.momentum = b->momentum;
    for (int k = 0; k < b->k; ++k) a.replicas[k] = b->replicas[k];
    a.n = b->n;
    a.mu = 0.f;
    a.eta = 0.f;
    a.scale = 1.f;
    a.inv_k = 1.0f / static_cast<float>(b->k);
    a.partials = ctx->partials;
    return a;
}

// Timing of a call's device work.  The previous timing is dropped before the
// start event of a new launch is recorded, so a call that fails after that
// point leaves no timing (E_STATE) rather than a start and stop of two calls.
int timer_start(autoloco_ctx* c) {
    c->timed_valid = false;
    if (!c->timing) return AUTOLOCO_OK;
    const hipError_t e = hipEventRecord(c->ev_start, c->stream);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventRecord");
    return AUTOLOCO_OK;
}

int timer_stop(autoloco_ctx* c, bool adamw = false, bool norm_ran = false) {
    if (!c->timing) return AUTOLOCO_OK;
    const hipError_t e = hipEventRecord(c->ev_stop, c->stream);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventRecord");
    c->timed_valid = true;
    c->adamw_timed = adamw;
    c->adamw_norm_ran = norm_ran;
    return AUTOLOCO_OK;
}

// Brings the count sums of the last reduction to host_sums and waits for them:
// with a device view of host_sums the reduction kernel already wrote them there
// (coherent host memory, visible once the stream has finished), else a copy.
int sums_to_host(autoloco_ctx* c, size_t count) {
    hipError_t e;
    if (c->host_sums_dev == nullptr &&
        (e = hipMemcpyAsync(c->host_sums, c->sums, sizeof(double) * count, hipMemcpyDeviceToHost, c->stream)) !=
            hipSuccess)
        return hip_fail(c, e, "hipMemcpyAsync");
    if ((e = hipStreamSynchronize(c->stream)) != hipSuccess) return hip_fail(c, e, "hipStreamSynchronize");
    return AUTOLOCO_OK;
}

// Launches one round kernel (timed if requested); with stats, waits for the
// sums and fills *out.
int run_round(autoloco_ctx* ctx, const autoloco_buffers* b, const RoundArgs& a, int mode, bool stats,
              double eps, autoloco_stats* out) {
    const int blocks = blocks_for(ctx, b->n, b->replica_dtype, b->k, mode >= MODE_P_UPDATE);
    int ts = timer_start(ctx);
    if (ts != AUTOLOCO_OK) return ts;
    hipError_t e = launcher(b->replica_dtype, mode)(b->k, blocks, ctx->stream, a);
    if (e != hipSuccess) return hip_fail(ctx, e, "kernel launch");
    if (stats && (e = launch_finish_sums(2 * b->k + 1, kBlock, blocks, ctx->partials, ctx->sums, ctx->stream,
                                         ctx->host_sums_dev)) != hipSuccess)
        return hip_fail(ctx, e, "reduction launch");
    if ((ts = timer_stop(ctx)) != AUTOLOCO_OK) return ts;
    if (stats) {
        if ((ts = sums_to_host(ctx, 2 * b->k + 1)) != AUTOLOCO_OK) return ts;
        finish_stats(ctx->host_sums, b->k, eps, out);
    }
    ctx->err.clear();
    return AUTOLOCO_OK;
}


// Checks the AdamW buffers: sizes, pointers, alignment and overlap.
int validate_adamw(autoloco_ctx* ctx, const autoloco_adamw_buffers* b, bool* copy) {
    if (ctx == nullptr) return AUTOLOCO_E_INVALID;
    if (b == nullptr) return fail(ctx, AUTOLOCO_E_INVALID, "null buffers");
    if (b->n < 0 || b->n > kMaxN) return fail(ctx, AUTOLOCO_E_INVALID, kBadN);
    if (b->k < 1 || b->k > AUTOLOCO_MAX_K) return fail(ctx, AUTOLOCO_E_INVALID, "k outside 1..16");
    int ncopy = 0;
    for (int k = 0; k < b->k; ++k) ncopy += b->model_bf16[k] != nullptr;
    if (ncopy != 0 && ncopy != b->k) return fail(ctx, AUTOLOCO_E_INVALID, "model_bf16 set for some workers only");
    *copy = ncopy != 0;
    if (b->n == 0) return AUTOLOCO_OK;
    std::vector<Range> r;
    const uintptr_t fbytes = static_cast<uintptr_t>(b->n) * 4u;
    for (int k = 0; k < b->k; ++k) {
        const void* ptrs[5] = {b->params[k], b->exp_avg[k], b->exp_avg_sq[k], b->grads[k], b->model_bf16[k]};
        static const char* names[5] = {"params", "exp_avg", "exp_avg_sq", "grads", "model_bf16"};
        for (int j = 0; j < 5; ++j) {
            if (j == 4 && !*copy) continue;
            if (ptrs[j] == nullptr) return fail(ctx, AUTOLOCO_E_INVALID, std::string("null ") + names[j]);
            const uintptr_t lo = reinterpret_cast<uintptr_t>(ptrs[j]);
            r.push_back({lo, lo + (j == 4 ? fbytes / 2 : fbytes), names[j]});
        }
    }
    for (const Range& x : r)
        if (x.lo % 16 != 0) return fail(ctx, AUTOLOCO_E_ALIGN, std::string(x.name) + " not 16-byte aligned");
    for (size_t i = 0; i < r.size(); ++i)
        for (size_t j = i + 1; j < r.size(); ++j)
            if (r[i].lo < r[j].hi && r[j].lo < r[i].hi)
                return fail(ctx, AUTOLOCO_E_ALIAS, std::string(r[i].name) + " overlaps " + r[j].name);
    for (const Range& x : r) {
        const int st = check_device_ptr(ctx, x.lo, x.name);
        if (st != AUTOLOCO_OK) return st;
    }
    return AUTOLOCO_OK;
}

double adamw_clip(double norm_sq, double max_norm) {
    if (max_norm == 0.0) return 1.0;
    const double c = max_norm / (std::sqrt(norm_sq) + 1e-6);
    return c > 1.0 ? 1.0 : c;
}

void finish_adamw(const double* sums, int k, double max_norm, autoloco_adamw_stats* out) {
    std::memset(out, 0, sizeof(*out));
    out->k = k;
    bool fin = true;
    for (int i = 0; i < k; ++i) {
        out->grad_norm[i] = std::sqrt(sums[i]);
        out->clip_coef[i] = adamw_clip(sums[i], max_norm);
        fin = fin && std::isfinite(out->grad_norm[i]);
    }
    out->finite = fin ? 1 : 0;
}


// Checks alignment and pairwise overlap of a list of ranges.
int check_ranges(autoloco_ctx* ctx, const std::vector<Range>& r) {
    for (const Range& x : r) {
        if (x.lo == 0) return fail(ctx, AUTOLOCO_E_INVALID, std::string("null ") + x.name);
        if (x.lo % 16 != 0) return fail(ctx, AUTOLOCO_E_ALIGN, std::string(x.name) + " not 16-byte aligned");
    }
    for (size_t i = 0; i < r.size(); ++i)
        for (size_t j = i + 1; j < r.size(); ++j)
            if (r[i].lo < r[j].hi && r[j].lo < r[i].hi)
                return fail(ctx, AUTOLOCO_E_ALIAS, std::string(r[i].name) + " overlaps " + r[j].name);
    for (const Range& x : r) {
        const int st = check_device_ptr(ctx, x.lo, x.name);
        if (st != AUTOLOCO_OK) return st;
    }
    return AUTOLOCO_OK;
}

// Launches a kernel of `blocks` workgroups that leaves one float64 partial sum
// per workgroup, then the reduction of those into ctx->sums[0]; with out,
// waits for it and stores it.
template <typename Launch>
int run_one_sum(autoloco_ctx* c, Launch launch, int blocks, double* out) {
    int ts = timer_start(c);
    if (ts != AUTOLOCO_OK) return ts;
    hipError_t e;
    if ((e = launch()) != hipSuccess) return hip_fail(c, e, "kernel launch");
    if ((e = launch_finish_sums(1, kBlock, blocks, c->partials, c->sums, c->stream, c->host_sums_dev)) != hipSuccess)
        return hip_fail(c, e, "reduction launch");
    if ((ts = timer_stop(c)) != AUTOLOCO_OK) return ts;
    if (out != nullptr) {
        if ((ts = sums_to_host(c, 1)) != AUTOLOCO_OK) return ts;
        *out = c->host_sums[0];
    }
    c->err.clear();
    return AUTOLOCO_OK;
}

// Workgroups of the per-GPU share kernels (two quads of 4 parameters per lane
// per window): the payload kernel two per CU, the shard step three (measured on
// MI355X with both kernels loading both runs before any store: payload 1.1B
// 1.93 ms at 512 against 1.98 at 768; shard step 3B K = 8 2.27 ms at 768 against
// 2.40 at 512, 2.31 at 1,024, and equal at 1.1B).
int blocks8(const autoloco_ctx* ctx, int64_t n, int per_cu = 2) {
    int limit = ctx->grid_limit > 0 ? ctx->grid_limit : ctx->num_cus * per_cu;
    if (limit > kMaxBlocks) limit = kMaxBlocks;
    int64_t want = (n / 8 + kBlock - 1) / kBlock;
    if (want < 1) want = 1;
    return static_cast<int>(want < limit ? want : limit);
}

// Outer coefficients a kernel can use: finite, with rho > 0.
int check_coeffs(autoloco_ctx* c, const autoloco_outer_coeffs* co) {
    if (!std::isfinite(co->mu) || !std::isfinite(co->eta_out) || !std::isfinite(co->rho) || !(co->rho > 0.0))
        return fail(c, AUTOLOCO_E_INVALID, "coefficients must be finite with rho > 0");
    return AUTOLOCO_OK;
}

// Checks shared by the outer-step calls, in this order: buffers, coefficients
// present, flags, the statistics output and eps (with FUSE_STATS), coefficient
// values.  Sets *stats and *reset from the flags.
int validate_step(autoloco_ctx* c, const autoloco_buffers* b, const autoloco_outer_coeffs* co, uint32_t flags,
                  double eps, const autoloco_stats* out, bool* stats, bool* reset) {
    int st = validate(c, b, true);
    if (st != AUTOLOCO_OK) return st;
    if (co == nullptr) return fail(c, AUTOLOCO_E_INVALID, "null coefficients");
    if ((flags & ~(AUTOLOCO_FUSE_STATS | AUTOLOCO_FUSE_RESET)) != 0) return fail(c, AUTOLOCO_E_INVALID, "unknown flags");
    *stats = (flags & AUTOLOCO_FUSE_STATS) != 0;
    *reset = (flags & AUTOLOCO_FUSE_RESET) != 0;
    if (*stats && out == nullptr) return fail(c, AUTOLOCO_E_INVALID, "FUSE_STATS needs a stats output");
    // C = K ||mean||^2 / (D + eps) with eps > 0 (eq. adaptive-h-core-diagnostics), so D = 0 gives C = 0
    if (*stats && !(eps > 0.0 && std::isfinite(eps))) return fail(c, AUTOLOCO_E_INVALID, "eps must be finite and > 0");
    return check_coeffs(c, co);
}

// The corrected step's scalars in a round kernel's arguments (fp32; 1/rho when normalising).
void set_step(RoundArgs& a, const autoloco_outer_coeffs* co) {
    a.mu = static_cast<float>(co->mu);
    a.eta = static_cast<float>(co->eta_out);
    a.scale = co->normalize ? static_cast<float>(1.0 / co->rho) : 1.0f;
}

void zero_stats(int k, double eps, autoloco_stats* out) {
    double z[kMaxSums] = {0};
    finish_stats(z, k, eps, out);
}

// ---------------------------------------------- outer step without allocation
constexpr int kStaticDevices = 64;

// Per device, set up on its first call: scratch's device address and the
// tables the launch shape is computed from (those of a context).
struct StaticDevice {
    bool ready = false;
    double* scratch_ptr = nullptr;   // scratch's device address on this device
    int num_cus = 0;
    int occupancy[2][AUTOLOCO_MAX_K + 1] = {};
};
StaticDevice g_static[kStaticDevices];
std::mutex g_static_mu;

// With `device` current.
int static_device(int device, StaticDevice** out) {
    std::lock_guard<std::mutex> lock(g_static_mu);
    StaticDevice& d = g_static[device];
    if (!d.ready) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
            (void)hipGetLastError();
            return AUTOLOCO_E_DEVICE;
        }
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess)
            return AUTOLOCO_E_DEVICE;
        d.scratch_ptr = static_cast<double*>(p);
        d.num_cus = cus > 0 ? cus : 1;
        for (int k = 1; k <= AUTOLOCO_MAX_K; ++k) {
            d.occupancy[0][k] = occupancy_round_f32_m4(k);
            d.occupancy[1][k] = occupancy_round_bf16_m4(k);
        }
        d.ready = true;
    }
    *out = &d;
    return AUTOLOCO_OK;
}

}  // namespace

extern "C" {

int autoloco_outer_step_static(int device, void* stream, const autoloco_buffers* b, const autoloco_outer_coeffs* co,
                               uint32_t flags, double eps, autoloco_stats* out) {
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || device < 0 || device >= count || device >= kStaticDevices)
        return AUTOLOCO_E_INVALID;
    DeviceGuard g(device);
    if (!g.ok) return AUTOLOCO_E_DEVICE;
    StaticDevice* sd = nullptr;
    int st = static_device(device, &sd);
    if (st != AUTOLOCO_OK) return st;
    // a context on the stack over the static scratch: the same validation,
    // launch shape and kernels as autoloco_outer_step, nothing allocated
    autoloco_ctx c;
    c.device = device;
    c.stream = static_cast<hipStream_t>(stream);
    c.num_cus = sd->num_cus;
    std::memcpy(c.occupancy, sd->occupancy, sizeof(c.occupancy));
    c.partials = sd->scratch_ptr;
    c.sums = sd->scratch_ptr + kStaticBlocks * kMaxSums;
    double host_sums[kMaxSums];
    c.host_sums = host_sums;
    bool stats = false, reset = false;
    st = validate_step(&c, b, co, flags, eps, out, &stats, &reset);
    if (st != AUTOLOCO_OK) return st;
    if (b->n == 0) {
        if (stats) zero_stats(b->k, eps, out);
        return AUTOLOCO_OK;
    }
    if (blocks_for(&c, b->n, b->replica_dtype, b->k) > kStaticBlocks) return AUTOLOCO_E_INVALID;
    RoundArgs a = make_args(&c, b);
    set_step(a, co);
    const int mode = stats ? (reset ? MODE_UPDATE_STATS_RESET : MODE_UPDATE_STATS)
                           : (reset ? MODE_UPDATE_RESET : MODE_UPDATE);
    return run_round(&c, b, a, mode, stats, eps, out);
}

int autoloco_create(int device, void* stream, autoloco_ctx** out) {
    if (out == nullptr) return AUTOLOCO_E_INVALID;
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || device < 0 || device >= count) return AUTOLOCO_E_INVALID;
    DeviceGuard g(device);
    if (!g.ok) return AUTOLOCO_E_DEVICE;
    auto* c = new (std::nothrow) autoloco_ctx;
    if (c == nullptr) return AUTOLOCO_E_NOMEM;
    c->device = device;
    c->stream = static_cast<hipStream_t>(stream);
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, device) != hipSuccess) {
        delete c;
        return AUTOLOCO_E_DEVICE;
    }
    c->num_cus = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 1;
    for (int k = 1; k <= AUTOLOCO_MAX_K; ++k) {
        c->occupancy[0][k] = occupancy_round_f32_m4(k);
        c->occupancy[1][k] = occupancy_round_bf16_m4(k);
        c->occupancy_int8[0][k] = occupancy_int8_f32_s1r1(k);
        c->occupancy_int8[1][k] = occupancy_int8_bf16_s1r1(k);
        c->occupancy_bf16p[0][k] = occupancy_round_f32_m8(k);
        c->occupancy_bf16p[1][k] = occupancy_round_bf16_m8(k);
    }
    bool ok = hipMalloc(&c->partials, sizeof(double) * kMaxSums * kMaxBlocks) == hipSuccess &&
              hipMalloc(&c->sums, sizeof(double) * kMaxSums) == hipSuccess &&
              hipHostMalloc(&c->host_sums, sizeof(double) * kMaxSums, hipHostMallocMapped | hipHostMallocCoherent) ==
                  hipSuccess;
    // the reduction writes the sums to host_sums through its device view; without
    // one, they are copied
    if (ok && hipHostGetDevicePointer(reinterpret_cast<void**>(&c->host_sums_dev), c->host_sums, 0) != hipSuccess) {
        c->host_sums_dev = nullptr;
        (void)hipGetLastError();
    }
    ok = ok && hipMemset(c->sums, 0, sizeof(double) * kMaxSums) == hipSuccess;
    ok = ok && hipEventCreate(&c->ev_start) == hipSuccess && hipEventCreate(&c->ev_stop) == hipSuccess &&
         hipEventCreate(&c->ev_mid) == hipSuccess;
    ok = ok && hipDeviceSynchronize() == hipSuccess;
    if (!ok) {
        autoloco_destroy(c);
        return AUTOLOCO_E_NOMEM;
    }
    *out = c;
    return AUTOLOCO_OK;
}

void autoloco_destroy(autoloco_ctx* c) {
    if (c == nullptr) return;
    {
        DeviceGuard g(c->device);
        (void)hipStreamSynchronize(c->stream);
        if (c->partials) (void)hipFree(c->partials);
        if (c->sums) (void)hipFree(c->sums);
        if (c->host_sums) (void)hipHostFree(c->host_sums);
        if (c->ev_start) (void)hipEventDestroy(c->ev_start);
        if (c->ev_stop) (void)hipEventDestroy(c->ev_stop);
        if (c->ev_mid) (void)hipEventDestroy(c->ev_mid);
    }
    delete c;
}

const char* autoloco_last_error(const autoloco_ctx* c) { return c == nullptr ? "null context" : c->err.c_str(); }

int autoloco_set_timing(autoloco_ctx* c, int enable) {
    if (c == nullptr) return AUTOLOCO_E_INVALID;
    c->timing = enable != 0;
    c->timed_valid = false;
    return AUTOLOCO_OK;
}

int autoloco_last_kernel_ms(autoloco_ctx* c, float* ms) {
    if (c == nullptr || ms == nullptr) return AUTOLOCO_E_INVALID;
    if (!c->timed_valid) return fail(c, AUTOLOCO_E_STATE, "no timed launch yet");
    DeviceGuard g(c->device);
    hipError_t e = hipEventSynchronize(c->ev_stop);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventSynchronize");
    e = hipEventElapsedTime(ms, c->ev_start, c->ev_stop);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventElapsedTime");
    return AUTOLOCO_OK;
}

int autoloco_set_grid_limit(autoloco_ctx* c, int max_blocks) {
    if (c == nullptr) return AUTOLOCO_E_INVALID;
    if (max_blocks < 0 || max_blocks > kMaxBlocks)
        return fail(c, AUTOLOCO_E_INVALID, "grid limit outside 0..16384");
    c->grid_limit = max_blocks;
    return AUTOLOCO_OK;
}

int autoloco_launch_shape(const autoloco_ctx* c, int64_t n, int32_t k, int32_t dtype, int32_t* blocks,
                          int32_t* threads) {
    if (c == nullptr || blocks == nullptr || threads == nullptr || n < 0 || n > kMaxN) return AUTOLOCO_E_INVALID;
    if (dtype != AUTOLOCO_F32 && dtype != AUTOLOCO_BF16) return AUTOLOCO_E_INVALID;
    if (k < 1 || k > AUTOLOCO_MAX_K) return AUTOLOCO_E_INVALID;
    *blocks = blocks_for(c, n, dtype, k);
    *threads = kBlock;
    return AUTOLOCO_OK;
}

int autoloco_round_stats(autoloco_ctx* c, const autoloco_buffers* b, double eps, autoloco_stats* out) {
    int st = validate(c, b, false);
    if (st != AUTOLOCO_OK) return st;
    if (out == nullptr) return fail(c, AUTOLOCO_E_INVALID, "null stats output");
    if (!(eps > 0.0 && std::isfinite(eps))) return fail(c, AUTOLOCO_E_INVALID, "eps must be finite and > 0");
    if (b->n == 0) {
        zero_stats(b->k, eps, out);
        return AUTOLOCO_OK;
    }
    DeviceGuard g(c->device);
    if (!g.ok) return fail(c, AUTOLOCO_E_DEVICE, "hipSetDevice failed");
    RoundArgs a = make_args(c, b);
    return run_round(c, b, a, MODE_STATS, true, eps, out);
}

int autoloco_outer_step(autoloco_ctx* c, const autoloco_buffers* b, const autoloco_outer_coeffs* co,
                        uint32_t flags, double eps, autoloco_stats* out) {
    bool stats = false, reset = false;
    const int st = validate_step(c, b, co, flags, eps, out, &stats, &reset);
    if (st != AUTOLOCO_OK) return st;
    if (b->n == 0) {
        if (stats) zero_stats(b->k, eps, out);
        return AUTOLOCO_OK;
    }
    DeviceGuard g(c->device);
    if (!g.ok) return fail(c, AUTOLOCO_E_DEVICE, "hipSetDevice failed");
    RoundArgs a = make_args(c, b);
    set_step(a, co);
    const int mode = stats ? (reset ? MODE_UPDATE_STATS_RESET : MODE_UPDATE_STATS)
                           : (reset ? MODE_UPDATE_RESET : MODE_UPDATE);
    return run_round(c, b, a, mode, stats, eps, out);
}

int autoloco_outer_step_bf16(autoloco_ctx* c, const autoloco_buffers* b, const autoloco_outer_coeffs* co,
                             uint32_t flags, double eps, autoloco_stats* out, uint16_t* mean_bf16) {
    bool stats = false, reset = false;
    const int st = validate_step(c, b, co, flags, eps, out, &stats, &reset);
    if (st != AUTOLOCO_OK) return st;
    if (b->n == 0) {
        if (stats) zero_stats(b->k, eps, out);
        return AUTOLOCO_OK;
    }
    if (mean_bf16 != nullptr) {
        const uintptr_t lo = reinterpret_cast<uintptr_t>(mean_bf16), hi = lo + static_cast<uintptr_t>(b->n) * 2u;
        if (lo % 16 != 0) return fail(c, AUTOLOCO_E_ALIGN, "mean_bf16 not 16-byte aligned");
        const uintptr_t fbytes = static_cast<uintptr_t>(b->n) * 4u;
        const uintptr_t rbytes = static_cast<uintptr_t>(b->n) * replica_size(b->replica_dtype);
        auto hit = [&](const void* p, uintptr_t len) {
            const uintptr_t q = reinterpret_cast<uintptr_t>(p);
            return lo < q + len && q < hi;
        };
        bool alias = hit(b->theta, fbytes) || hit(b->momentum, fbytes);
        for (int k = 0; k < b->k; ++k) alias = alias || hit(b->replicas[k], rbytes);
        if (alias) return fail(c, AUTOLOCO_E_ALIAS, "mean_bf16 overlaps a round buffer");
        const int ds = check_device_ptr(c, lo, "mean_bf16");
        if (ds != AUTOLOCO_OK) return ds;
    }
    DeviceGuard g(c->device);
    if (!g.ok) return fail(c, AUTOLOCO_E_DEVICE, "hipSetDevice failed");
    RoundArgs a = make_args(c, b);
    set_step(a, co);
    a.payload = mean_bf16;
    a.inv_k64 = 1.0 / static_cast<double>(b->k);
    const int mode = stats ? (reset ? MODE_P_UPDATE_STATS_RESET : MODE_P_UPDATE_STATS)
                           : (reset ? MODE_P_UPDATE_RESET : MODE_P_UPDATE);
    return run_round(c, b, a, mode, stats, eps, out);
}

int autoloco_outer_step_int8(autoloco_ctx* c, const autoloco_buffers* b, const autoloco_outer_coeffs* co,
                             uint32_t flags, double eps, autoloco_stats* out, int8_t* codes, float* scales) {
    bool stats = false, reset = false;
    const int st = validate_step(c, b, co, flags, eps, out, &stats, &reset);
    if (st != AUTOLOCO_OK) return st;
    if ((codes == nullptr) != (scales == nullptr))
        return fail(c, AUTOLOCO_E_INVALID, "pass both payload buffers or neither");
    if (b->n == 0) {
        if (stats) zero_stats(b->k, eps, out);
        return AUTOLOCO_OK;
    }
    const int64_t nblocks = (b->n + kCodecBlock - 1) / kCodecBlock;
    if (codes != nullptr) {
        const uintptr_t cp = reinterpret_cast<uintptr_t>(codes), sp = reinterpret_cast<uintptr_t>(scales);
        if (cp % 16 != 0 || sp % 16 != 0) return fail(c, AUTOLOCO_E_ALIGN, "payload buffers not 16-byte aligned");
        const uintptr_t c_hi = cp + static_cast<uintptr_t>(b->n), s_hi = sp + static_cast<uintptr_t>(nblocks) * 4u;
        if (cp < s_hi && sp < c_hi) return fail(c, AUTOLOCO_E_ALIAS, "payload buffers overlap");
        const uintptr_t fb = static_cast<uintptr_t>(b->n) * 4u, rb = static_cast<uintptr_t>(b->n) * replica_size(b->replica_dtype);
        uintptr_t lo[AUTOLOCO_MAX_K + 2], hi[AUTOLOCO_MAX_K + 2];
        int nr = 0;
        lo[nr] = reinterpret_cast<uintptr_t>(b->theta); hi[nr] = lo[nr] + fb; ++nr;
        lo[nr] = reinterpret_cast<uintptr_t>(b->momentum); hi[nr] = lo[nr] + fb; ++nr;
        for (int k = 0; k < b->k; ++k) {
            lo[nr] = reinterpret_cast<uintptr_t>(b->replicas[k]);
            hi[nr] = lo[nr] + rb;
            ++nr;
        }
        for (int i = 0; i < nr; ++i)
            if ((cp < hi[i] && lo[i] < c_hi) || (sp < hi[i] && lo[i] < s_hi))
                return fail(c, AUTOLOCO_E_ALIAS, "payload buffers overlap a round buffer");
        int ds = check_device_ptr(c, cp, "mean_codes");
        if (ds == AUTOLOCO_OK) ds = check_device_ptr(c, sp, "mean_scales");
        if (ds != AUTOLOCO_OK) return ds;
    }
    DeviceGuard g(c->device);
    if (!g.ok) return fail(c, AUTOLOCO_E_DEVICE, "hipSetDevice failed");
    Int8Args a;
    std::memset(&a, 0, sizeof(a));
    a.theta = b->theta;
    a.momentum = b->momentum;
    for (int k = 0; k < b->k; ++k) a.replicas[k] = b->replicas[k];
    a.n = b->n;
    a.mu = static_cast<float>(co->mu);
    a.eta = static_cast<float>(co->eta_out);
    a.scale = co->normalize ? static_cast<float>(1.0 / co->rho) : 1.0f;
    a.inv_k = 1.0 / static_cast<double>(b->k);
    a.mean_codes = codes;
    a.mean_scales = scales;
    a.partials = c->partials;
    const int rt = b->replica_dtype == AUTOLOCO_BF16 ? 1 : 0;
    int per_cu = c->occupancy_int8[rt][b->k];
    if (per_cu < 1) per_cu = 1;
    int limit = c->grid_limit > 0 ? c->grid_limit : c->num_cus * per_cu;
    if (limit > kMaxBlocks) limit = kMaxBlocks;
    const int blocks = static_cast<int>(nblocks < limit ? nblocks : limit);
    static const Int8Launcher table[2][2][2] = {
        {{launch_int8_f32_s0r0, launch_int8_f32_s0r1}, {launch_int8_f32_s1r0, launch_int8_f32_s1r1}},
        {{launch_int8_bf16_s0r0, launch_int8_bf16_s0r1}, {launch_int8_bf16_s1r0, launch_int8_bf16_s1r1}}};
    int ts = timer_start(c);
    if (ts != AUTOLOCO_OK) return ts;
    hipError_t e = table[rt][stats ? 1 : 0][reset ? 1 : 0](b->k, blocks, c->stream, a);
    if (e != hipSuccess) return hip_fail(c, e, "kernel launch");
    if (stats && (e = launch_finish_sums(2 * b->k + 1, kInt8Threads, blocks, c->partials, c->sums, c->stream,
                                         c->host_sums_dev)) != hipSuccess)
        return hip_fail(c, e, "reduction launch");
    if ((ts = timer_stop(c)) != AUTOLOCO_OK) return ts;
    if (stats) {
        if ((ts = sums_to_host(c, 2 * b->k + 1)) != AUTOLOCO_OK) return ts;
        finish_stats(c->host_sums, b->k, eps, out);
    }
    c->err.clear();
    return AUTOLOCO_OK;
}

int autoloco_broadcast_reset(autoloco_ctx* c, const autoloco_buffers* b) {
    int st = validate(c, b, false);
    if (st != AUTOLOCO_OK) return st;
    if (b->n == 0) return AUTOLOCO_OK;
    DeviceGuard g(c->device);
    if (!g.ok) return fail(c, AUTOLOCO_E_DEVICE, "hipSetDevice failed");
    RoundArgs a = make_args(c, b);
    const int blocks = blocks_for(c, b->n, b->replica_dtype, b->k, false, false);
    int ts = timer_start(c);
    if (ts != AUTOLOCO_OK) return ts;
    hipError_t e = launch_reset(b->replica_dtype == AUTOLOCO_BF16 ? RT_BF16 : RT_F32, b->k, blocks, c->stream, a);
    if (e != hipSuccess) return hip_fail(c, e, "kernel launch");
    if ((ts = timer_stop(c)) != AUTOLOCO_OK) return ts;
    c->err.clear();
    return AUTOLOCO_OK;
}

int autoloco_traffic_reference(autoloco_ctx* c, const autoloco_buffers* b) {
    int st = validate(c, b, true);
    if (st != AUTOLOCO_OK) return st;
    if (b->n == 0) return AUTOLOCO_OK;
    DeviceGuard g(c->device);
    if (!g.ok) return fail(c, AUTOLOCO_E_DEVICE, "hipSetDevice failed");
    RoundArgs a = make_args(c, b);
    const int blocks = blocks_for(c, b->n, b->replica_dtype, b->k);
    int ts = timer_start(c);
    if (ts != AUTOLOCO_OK) return ts;
    hipError_t e = launch_traffic(b->replica_dtype == AUTOLOCO_BF16 ? RT_BF16 : RT_F32, b->k, blocks, c->stream, a, 0u);
    if (e != hipSuccess) return hip_fail(c, e, "kernel launch");
    if ((ts = timer_stop(c)) != AUTOLOCO_OK) return ts;
    c->err.clear();
    return AUTOLOCO_OK;
}

int autoloco_traffic_probe(autoloco_ctx* c, int64_t n, const autoloco_probe_stream* streams, int32_t count,
                           int32_t shape, int32_t blocks, double* bytes) {
    if (c == nullptr) return AUTOLOCO_E_INVALID;
    if (streams == nullptr) return fail(c, AUTOLOCO_E_INVALID, "null streams");
    if (n < 0 || n > kMaxN) return fail(c, AUTOLOCO_E_INVALID, kBadN);
    if (shape < AUTOLOCO_PROBE_RUN1 || shape > AUTOLOCO_PROBE_RUN8)
        return fail(c, AUTOLOCO_E_INVALID, "unknown probe shape");
    if (count < 1 || count > kProbeMaxStreams) return fail(c, AUTOLOCO_E_INVALID, "stream count outside 1..18");
    if (blocks < 0 || blocks > kMaxBlocks) return fail(c, AUTOLOCO_E_INVALID, "blocks outside 0..16384");
    // classes in order: 4-byte in place, 4-byte read, 2-byte read, 2-byte written, 4-byte written
    int cls_count[5] = {0, 0, 0, 0, 0};
    int last = 0;
    std::vector<Range> r;
    for (int s = 0; s < count; ++s) {
        const autoloco_probe_stream& x = streams[s];
        const bool rd = x.access == AUTOLOCO_PROBE_READ || x.access == (AUTOLOCO_PROBE_READ | AUTOLOCO_PROBE_WRITE);
        const bool wr = x.access == AUTOLOCO_PROBE_WRITE || x.access == (AUTOLOCO_PROBE_READ | AUTOLOCO_PROBE_WRITE);
        if (!rd && !wr) return fail(c, AUTOLOCO_E_INVALID, "access must be read, write or both");
        int cls;
        if (x.elem_bytes == 4)
            cls = rd && wr ? 0 : rd ? 1 : 4;
        else if (x.elem_bytes == 2 && !(rd && wr))
            cls = rd ? 2 : 3;
        else
            return fail(c, AUTOLOCO_E_INVALID, "streams are 4-byte, or 2-byte read only or written only");
        if (cls < last)
            return fail(c, AUTOLOCO_E_INVALID, "streams must come in class order: 4-byte in place, 4-byte read, "
                                               "2-byte read, 2-byte written, 4-byte written");
        last = cls;
        ++cls_count[cls];
        const uintptr_t lo = reinterpret_cast<uintptr_t>(x.ptr);
        r.push_back({lo, lo + static_cast<uintptr_t>(n) * static_cast<uintptr_t>(x.elem_bytes), "probe stream"});
    }
    ProbePattern p;
    p.shape = shape == AUTOLOCO_PROBE_SERIAL ? PROBE_SERIAL : shape == AUTOLOCO_PROBE_TILE ? PROBE_TILE
            : shape == AUTOLOCO_PROBE_PHASED ? PROBE_PHASED : PROBE_RUN;
    p.r = shape == AUTOLOCO_PROBE_RUN2 ? 2 : shape == AUTOLOCO_PROBE_RUN8 ? 8 : 1;
    p.a = cls_count[0];
    p.b = cls_count[1];
    p.c = cls_count[2];
    p.d = cls_count[3];
    p.e = cls_count[4];
    const bool phased = p.shape == PROBE_PHASED;
    if (phased ? !(p.a == kPhaseStreams && count == kPhaseStreams) : !probe_available(p))
        return fail(c, AUTOLOCO_E_INVALID, "no probe instance for this pattern and shape");
    const int nb = blocks > 0 ? blocks : c->num_cus;   // default: one workgroup per compute unit
    if (phased && nb > probe_phased_occupancy() * c->num_cus)
        return fail(c, AUTOLOCO_E_INVALID, "phased probe: more workgroups than can be resident at once");
    if (n == 0) {
        if (bytes) *bytes = 0.0;
        return AUTOLOCO_OK;
    }
    const int st = check_ranges(c, r);
    if (st != AUTOLOCO_OK) return st;
    DeviceGuard g(c->device);
    if (!g.ok) return fail(c, AUTOLOCO_E_DEVICE, "hipSetDevice failed");
    ProbeArgs a;
    std::memset(&a, 0, sizeof(a));
    for (int s = 0; s < count; ++s) a.ptr[s] = streams[s].ptr;
    a.n = n;
    a.sentinel = 0x9E3779B9u;
    a.sink = reinterpret_cast<uint32_t*>(c->partials);
    // elements the shape moves per stream: whole runs of 4, whole tiles, or
    // whole rounds of tiles over the grid
    const int64_t tile = 4 * kProbeTileQuads * kBlock;
    const int64_t ptile = 4 * static_cast<int64_t>(kPhaseLdsRuns + kPhaseRegRuns) * kBlock;
    const int64_t moved = p.shape == PROBE_RUN ? n / 4 * 4 : phased ? n / (ptile * nb) * (ptile * nb) : n / tile * tile;
    double b = 0.0;
    for (int s = 0; s < count; ++s)
        b += static_cast<double>(moved) * streams[s].elem_bytes * (streams[s].access == 3 ? 2 : 1);
    uint32_t* sync = reinterpret_cast<uint32_t*>(c->partials);   // the phased shape's barrier words
    hipError_t e;
    if (phased && (e = hipMemsetAsync(sync, 0, 2 * sizeof(uint32_t), c->stream)) != hipSuccess)
        return hip_fail(c, e, "hipMemsetAsync");
    int ts = timer_start(c);
    if (ts != AUTOLOCO_OK) return ts;
    e = phased ? launch_probe_phased(nb, c->stream, a, sync) : launch_probe(p, nb, c->stream, a);
    if (e != hipSuccess) return hip_fail(c, e, "kernel launch");
    if ((ts = timer_stop(c)) != AUTOLOCO_OK) return ts;
    if (phased) {
        uint32_t words[2] = {0, 0};
        if ((e = hipMemcpyAsync(words, sync, sizeof(words), hipMemcpyDeviceToHost, c->stream)) != hipSuccess)
            return hip_fail(c, e, "hipMemcpyAsync");
        if ((e = hipStreamSynchronize(c->stream)) != hipSuccess) return hip_fail(c, e, "hipStreamSynchronize");
        if (words[1] != 0) return fail(c, AUTOLOCO_E_STATE, "phased probe: a grid barrier gave up waiting");
    }
    if (bytes) *bytes = b;
    c->err.clear();
    return AUTOLOCO_OK;
}

const char* autoloco_build_id(void) { return AUTOLOCO_BUILD_ID; }

int autoloco_alloc_spread(autoloco_ctx* c, int32_t count, size_t bytes, void** out, int32_t* spread) {
    if (c == nullptr) return AUTOLOCO_E_INVALID;
    if (out == nullptr || count < 1 || count > 64 || bytes == 0)
        return fail(c, AUTOLOCO_E_INVALID, "alloc_spread: need out, 1 <= count <= 64, bytes > 0");
    DeviceGuard g(c->device);
    if (!g.ok) return fail(c, AUTOLOCO_E_DEVICE, "hipSetDevice failed");
    const size_t gran = size_t(2) << 20;
    const size_t slot = (bytes + gran - 1) / gran * gran;
    size_t free_b = 0, total_b = 0;
    if (hipMemGetInfo(&free_b, &total_b) != hipSuccess) return fail(c, AUTOLOCO_E_DEVICE, "hipMemGetInfo failed");
    size_t reserve = total_b / 64;
    if (reserve < (size_t(2) << 30)) reserve = size_t(2) << 30;
    size_t want = free_b > reserve ? (free_b - reserve) / slot : 0;
    if (want > 1024) want = 1024;
    if (spread) *spread = 0;
    if (want < size_t(2) * count) {
        // not enough room to spread: plain allocations
        for (int i = 0; i < count; ++i) {
            if (hipMalloc(&out[i], slot) != hipSuccess) {
                for (int j = 0; j < i; ++j) (void)hipFree(out[j]);
                return fail(c, AUTOLOCO_E_NOMEM, "alloc_spread: hipMalloc failed");
            }
        }
        return AUTOLOCO_OK;
    }
    // Fill the free memory with equal slots in allocation order, keep an even
    // selection of them, and return the others.
    std::vector<void*> slots;
    slots.reserve(want);
    for (size_t i = 0; i < want; ++i) {
        void* p = nullptr;
        if (hipMalloc(&p, slot) != hipSuccess) break;
        slots.push_back(p);
    }
    (void)hipGetLastError();  // a failed probe allocation is expected near the end
    const size_t m = slots.size();
    if (m < size_t(count)) {
        for (void* p : slots) (void)hipFree(p);
        return fail(c, AUTOLOCO_E_NOMEM, "alloc_spread: not enough device memory");
    }
    std::vector<char> keep(m, 0);
    for (int i = 0; i < count; ++i) {
        const size_t idx = count == 1 ? m / 2 : (size_t)((double)i * (double)(m - 1) / (double)(count - 1) + 0.5);
        keep[idx] = 1;
        out[i] = slots[idx];
    }
    for (size_t i = 0; i < m; ++i)
        if (!keep[i]) (void)hipFree(slots[i]);
    if (spread) *spread = m >= size_t(2) * count ? 1 : 0;
    c->err.clear();
    return AUTOLOCO_OK;
}

int autoloco_free(autoloco_ctx* c, void* ptr) {
    if (c == nullptr) return AUTOLOCO_E_INVALID;
    if (ptr == nullptr) return AUTOLOCO_OK;
    DeviceGuard g(c->device);
    const hipError_t e = hipFree(ptr);
    if (e != hipSuccess) return hip_fail(c, e, "hipFree");
    return AUTOLOCO_OK;
}

int autoloco_rank_payload(autoloco_ctx* c, int64_t n, const float* theta, const void* replica, int32_t dtype,
                          uint16_t* payload, double* sq_norm) {
    if (c == nullptr) return AUTOLOCO_E_INVALID;
    if (n < 0 || n > kMaxN) return fail(c, AUTOLOCO_E_INVALID, kBadN);
    if (dtype != AUTOLOCO_F32 && dtype != AUTOLOCO_BF16) return fail(c, AUTOLOCO_E_INVALID, "unknown replica dtype");
    if (n == 0) {
        if (sq_norm != nullptr) *sq_norm = 0.0;
        return AUTOLOCO_OK;
    }
    const uintptr_t un = static_cast<uintptr_t>(n);
    std::vector<Range> r = {{reinterpret_cast<uintptr_t>(theta), reinterpret_cast<uintptr_t>(theta) + 4 * un, "theta"},
                            {reinterpret_cast<uintptr_t>(replica),
                             reinterpret_cast<uintptr_t>(replica) + un * replica_size(dtype), "replica"},
                            {reinterpret_cast<uintptr_t>(payload), reinterpret_cast<uintptr_t>(payload) + 2 * un,
                             "payload"}};
    int st = check_ranges(c, r);
    if (st != AUTOLOCO_OK) return st;
    DeviceGuard g(c->device);
    if (!g.ok) return fail(c, AUTOLOCO_E_DEVICE, "hipSetDevice failed");
    RankPayloadArgs a;
    a.theta = theta;
    a.replica = replica;
    a.payload = payload;
    a.n = n;
    a.partials = c->partials;
    const int blocks = blocks8(c, n);
    const int rt = dtype == AUTOLOCO_BF16 ? RT_BF16 : RT_F32;
    return run_one_sum(c, [&] { return launch_rank_payload(rt, blocks, c->stream, a); }, blocks, sq_norm);
}

int autoloco_shard_step(autoloco_ctx* c, const autoloco_shard_buffers* b, const autoloco_outer_coeffs* co,
                        uint16_t* mean_bf16, double* sq_mean) {
    if (c == nullptr) return AUTOLOCO_E_INVALID;
    if (b == nullptr || co == nullptr) return fail(c, AUTOLOCO_E_INVALID, "null buffers or coefficients");
    if (b->n < 0 || b->n > kMaxN) return fail(c, AUTOLOCO_E_INVALID, kBadN);
    if (b->k < 1 || b->k > AUTOLOCO_MAX_K) return fail(c, AUTOLOCO_E_INVALID, "k outside 1..16");
    const int cs = check_coeffs(c, co);
    if (cs != AUTOLOCO_OK) return cs;
    if (b->n == 0) {
        if (sq_mean != nullptr) *sq_mean = 0.0;
        return AUTOLOCO_OK;
    }
    const uintptr_t un = static_cast<uintptr_t>(b->n);
    std::vector<Range> r = {
        {reinterpret_cast<uintptr_t>(b->theta), reinterpret_cast<uintptr_t>(b->theta) + 4 * un, "theta"},
        {reinterpret_cast<uintptr_t>(b->momentum), reinterpret_cast<uintptr_t>(b->momentum) + 4 * un, "momentum"}};
    for (int k = 0; k < b->k; ++k)
        r.push_back({reinterpret_cast<uintptr_t>(b->payloads[k]), reinterpret_cast<uintptr_t>(b->payloads[k]) + 2 * un,
                     "payload"});
    if (mean_bf16 != nullptr)
        r.push_back({reinterpret_cast<uintptr_t>(mean_bf16), reinterpret_cast<uintptr_t>(mean_bf16) + 2 * un,
                     "mean_bf16"});
    int st = check_ranges(c, r);
    if (st != AUTOLOCO_OK) return st;
    DeviceGuard g(c->device);
    if (!g.ok) return fail(c, AUTOLOCO_E_DEVICE, "hipSetDevice failed");
    ShardArgs a;
    std::memset(&a, 0, sizeof(a));
    a.theta = b->theta;
    a.momentum = b->momentum;
    for (int k = 0; k < b->k; ++k) a.payloads[k] = b->payloads[k];
    a.mean_out = mean_bf16;
    a.n = b->n;
    a.mu = static_cast<float>(co->mu);
    a.eta = static_cast<float>(co->eta_out);
    a.scale = co->normalize ? static_cast<float>(1.0 / co->rho) : 1.0f;
    a.inv_k64 = 1.0 / static_cast<double>(b->k);
    a.partials = c->partials;
    const int blocks = blocks8(c, b->n, 3);
    const int k = b->k;
    return run_one_sum(c, [&] { return launch_shard_step(k, blocks, c->stream, a); }, blocks, sq_mean);
}

int autoloco_inner_adamw(autoloco_ctx* c, const autoloco_adamw_buffers* b, const autoloco_adamw_coeffs* co,
                         autoloco_adamw_stats* out) {
    bool copy = false;
    int st = validate_adamw(c, b, &copy);
    if (st != AUTOLOCO_OK) return st;
    if (co == nullptr) return fail(c, AUTOLOCO_E_INVALID, "null coefficients");
    if (co->step < 1) return fail(c, AUTOLOCO_E_INVALID, "step counts from 1");
    const double nonneg[4] = {co->lr, co->eps, co->weight_decay, co->max_grad_norm};
    for (double x : nonneg)
        if (!(std::isfinite(x) && x >= 0.0))
            return fail(c, AUTOLOCO_E_INVALID, "lr, eps, weight_decay and max_grad_norm must be finite and >= 0");
    if (!(co->beta1 >= 0.0 && co->beta1 < 1.0 && co->beta2 >= 0.0 && co->beta2 < 1.0))
        return fail(c, AUTOLOCO_E_INVALID, "betas must lie in [0, 1)");
    const bool clip = co->max_grad_norm > 0.0;
    if (b->n == 0) {
        if (out != nullptr) {
            double z[AUTOLOCO_MAX_K] = {0};
            finish_adamw(z, b->k, co->max_grad_norm, out);
        }
        return AUTOLOCO_OK;
    }
    DeviceGuard g(c->device);
    if (!g.ok) return fail(c, AUTOLOCO_E_DEVICE, "hipSetDevice failed");
    const bool norm_pass = clip || out != nullptr;
    int ts = timer_start(c);
    if (ts != AUTOLOCO_OK) return ts;
    hipError_t e;
    if (norm_pass) {
        GradNormArgs na;
        std::memset(&na, 0, sizeof(na));
        for (int k = 0; k < b->k; ++k) na.grads[k] = b->grads[k];
        na.n = b->n;
        na.partials = c->partials;
        const int nblocks = blocks_for(c, b->n, AUTOLOCO_F32, b->k, false, false);
        e = launch_grad_norm(b->k, nblocks, c->stream, na);
        if (e != hipSuccess) return hip_fail(c, e, "gradient norm launch");
        e = launch_finish_sums(b->k, kBlock, nblocks, c->partials, c->sums, c->stream, c->host_sums_dev);
        if (e != hipSuccess) return hip_fail(c, e, "reduction launch");
    }
    if (c->timing && (e = hipEventRecord(c->ev_mid, c->stream)) != hipSuccess) return hip_fail(c, e, "hipEventRecord");
    AdamWArgs a;
    std::memset(&a, 0, sizeof(a));
    for (int k = 0; k < b->k; ++k) {
        a.params[k] = b->params[k];
        a.exp_avg[k] = b->exp_avg[k];
        a.exp_avg_sq[k] = b->exp_avg_sq[k];
        a.grads[k] = b->grads[k];
        a.copy[k] = static_cast<uint16_t*>(b->model_bf16[k]);
    }
    a.n = b->n;
    a.norm_sq = clip ? c->sums : nullptr;
    a.max_norm = co->max_grad_norm;
    a.decay = static_cast<float>(1.0 - co->lr * co->weight_decay);
    a.beta1 = static_cast<float>(co->beta1);
    a.beta2 = static_cast<float>(co->beta2);
    a.omb1 = static_cast<float>(1.0 - co->beta1);
    a.omb2 = static_cast<float>(1.0 - co->beta2);
    const double t = static_cast<double>(co->step);
    a.step_size = static_cast<float>(co->lr / (1.0 - std::pow(co->beta1, t)));
    a.inv_sqrt_bc2 = static_cast<float>(1.0 / std::sqrt(1.0 - std::pow(co->beta2, t)));
    a.eps = static_cast<float>(co->eps);
    e = launch_adamw(copy, false, b->k, adamw_blocks(c, b->n, b->k), c->stream, a);
    if (e != hipSuccess) return hip_fail(c, e, "AdamW launch");
    if ((ts = timer_stop(c, true, norm_pass)) != AUTOLOCO_OK) return ts;
    if (out != nullptr) {
        if ((ts = sums_to_host(c, b->k)) != AUTOLOCO_OK) return ts;
        finish_adamw(c->host_sums, b->k, co->max_grad_norm, out);
    }
    c->err.clear();
    return AUTOLOCO_OK;
}

int autoloco_adamw_traffic_reference(autoloco_ctx* c, const autoloco_adamw_buffers* b) {
    bool copy = false;
    int st = validate_adamw(c, b, &copy);
    if (st != AUTOLOCO_OK) return st;
    if (b->n == 0) return AUTOLOCO_OK;
    DeviceGuard g(c->device);
    if (!g.ok) return fail(c, AUTOLOCO_E_DEVICE, "hipSetDevice failed");
    AdamWArgs a;
    std::memset(&a, 0, sizeof(a));
    for (int k = 0; k < b->k; ++k) {
        a.params[k] = b->params[k];
        a.exp_avg[k] = b->exp_avg[k];
        a.exp_avg_sq[k] = b->exp_avg_sq[k];
        a.grads[k] = b->grads[k];
        a.copy[k] = static_cast<uint16_t*>(b->model_bf16[k]);
    }
    a.n = b->n;
    a.mask = 0u;
    int ts = timer_start(c);
    if (ts != AUTOLOCO_OK) return ts;
    const hipError_t e = launch_adamw(copy, true, b->k, adamw_blocks(c, b->n, b->k), c->stream, a);
    if (e != hipSuccess) return hip_fail(c, e, "AdamW traffic reference launch");
    if ((ts = timer_stop(c)) != AUTOLOCO_OK) return ts;
    c->err.clear();
    return AUTOLOCO_OK;
}

int autoloco_last_adamw_ms(autoloco_ctx* c, float* norm_ms, float* update_ms) {
    if (c == nullptr || norm_ms == nullptr || update_ms == nullptr) return AUTOLOCO_E_INVALID;
    if (!c->timed_valid || !c->adamw_timed) return fail(c, AUTOLOCO_E_STATE, "no timed AdamW step yet");
    DeviceGuard g(c->device);
    hipError_t e = hipEventSynchronize(c->ev_stop);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventSynchronize");
    *norm_ms = 0.0f;
    if (c->adamw_norm_ran && (e = hipEventElapsedTime(norm_ms, c->ev_start, c->ev_mid)) != hipSuccess)
        return hip_fail(c, e, "hipEventElapsedTime");
    if ((e = hipEventElapsedTime(update_ms, c->ev_mid, c->ev_stop)) != hipSuccess)
        return hip_fail(c, e, "hipEventElapsedTime");
    return AUTOLOCO_OK;
}

}  // extern "C"

// ------------------------------------------------------------ reset launcher
namespace autoloco {
namespace {
// Windows of 256 quads per workgroup and iteration.  fp32 replicas: 8 from
// three replicas on, where the longer contiguous writes per replica are 3-10 %
// faster than one window on MI355X (1.1B: K = 8 6.20-6.28 ms against 6.64-6.85,
// K = 6 4.83-4.88 against 5.37-5.53), one below (a copy at K = 1, which runs no
// faster with longer spans).  bf16 replicas: two windows (a 4 KB run per
// replica), faster than 4 to 16 at every K (3B, K = 8: 10.5 ms against 10.6-11.1;
// K = 3: 5.1 against 5.5-6.1).
template <int K>
hipError_t reset_k(int rt, int blocks, hipStream_t s, const RoundArgs& a) {
    if (rt == RT_BF16)
        hipLaunchKernelGGL((reset_kernel<K, RT_BF16, 2>), dim3(blocks), dim3(kBlock), 0, s, a);
    else if constexpr (K >= 3)
        hipLaunchKernelGGL((reset_kernel<K, RT_F32, 8>), dim3(blocks), dim3(kBlock), 0, s, a);
    else
        hipLaunchKernelGGL((reset_kernel<K, RT_F32, 1>), dim3(blocks), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}
}  // namespace

hipError_t launch_reset(int rt, int k, int blocks, hipStream_t s, const RoundArgs& a) {
    switch (k) {
        case 1: return reset_k<1>(rt, blocks, s, a);
        case 2: return reset_k<2>(rt, blocks, s, a);
        case 3: return reset_k<3>(rt, blocks, s, a);
        case 4: return reset_k<4>(rt, blocks, s, a);
        case 5: return reset_k<5>(rt, blocks, s, a);
        case 6: return reset_k<6>(rt, blocks, s, a);
        case 7: return reset_k<7>(rt, blocks, s, a);
        case 8: return reset_k<8>(rt, blocks, s, a);
        case 9: return reset_k<9>(rt, blocks, s, a);
        case 10: return reset_k<10>(rt, blocks, s, a);
        case 11: return reset_k<11>(rt, blocks, s, a);
        case 12: return reset_k<12>(rt, blocks, s, a);
        case 13: return reset_k<13>(rt, blocks, s, a);
        case 14: return reset_k<14>(rt, blocks, s, a);
        case 15: return reset_k<15>(rt, blocks, s, a);
        case 16: return reset_k<16>(rt, blocks, s, a);
        default: return hipErrorInvalidValue;
    }
}
}  // namespace autoloco

// -------------------------------------------------------- traffic launcher
namespace autoloco {
namespace {
template <int K>
hipError_t traffic_k(int rt, int blocks, hipStream_t s, const RoundArgs& a, uint32_t mask) {
    if (rt == RT_BF16)
        hipLaunchKernelGGL((traffic_kernel<K, RT_BF16>), dim3(blocks), dim3(kBlock), 0, s, a, mask);
    else
        hipLaunchKernelGGL((traffic_kernel<K, RT_F32>), dim3(blocks), dim3(kBlock), 0, s, a, mask);
    return hipGetLastError();
}
}  // namespace

hipError_t launch_traffic(int rt, int k, int blocks, hipStream_t s, const RoundArgs& a, uint32_t mask) {
    switch (k) {
        case 1: return traffic_k<1>(rt, blocks, s, a, mask);
        case 2: return traffic_k<2>(rt, blocks, s, a, mask);
        case 3: return traffic_k<3>(rt, blocks, s, a, mask);
        case 4: return traffic_k<4>(rt, blocks, s, a, mask);
        case 5: return traffic_k<5>(rt, blocks, s, a, mask);
        case 6: return traffic_k<6>(rt, blocks, s, a, mask);
        case 7: return traffic_k<7>(rt, blocks, s, a, mask);
        case 8: return traffic_k<8>(rt, blocks, s, a, mask);
        case 9: return traffic_k<9>(rt, blocks, s, a, mask);
        case 10: return traffic_k<10>(rt, blocks, s, a, mask);
        case 11: return traffic_k<11>(rt, blocks, s, a, mask);
        case 12: return traffic_k<12>(rt, blocks, s, a, mask);
        case 13: return traffic_k<13>(rt, blocks, s, a, mask);
        case 14: return traffic_k<14>(rt, blocks, s, a, mask);
        case 15: return traffic_k<15>(rt, blocks, s, a, mask);
        case 16: return traffic_k<16>(rt, blocks, s, a, mask);
        default: return hipErrorInvalidValue;
    }
}
}  // namespace autoloco
