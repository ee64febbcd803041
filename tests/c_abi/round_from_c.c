/* One fused synchronisation round driven from plain C through the library's
 * C ABI: device memory from hipMalloc, no Python and no torch.
 *
 * usage: round_from_c DIR N K
 *   reads DIR/theta.f32, DIR/momentum.f32, DIR/replica<k>.f32 (raw little-endian fp32, N each),
 *   takes the outer coefficients from the library's schedule preview and correction (H^step = 750
 *   against H^ref = 500 at step 20,000), runs autoloco_outer_step with statistics and reset, and
 *   writes DIR/theta_out.f32, DIR/momentum_out.f32, DIR/replica0_out.f32 and DIR/stats.txt
 *   (D, C, disagreement, sq_mean and the per-worker sums as %.17g), then asks the controller for its
 *   first interval and appends it.  Exit status 0 on success. */
#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "autoloco.h"

static int read_f32(const char* dir, const char* name, float* dst, long n) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE* f = fopen(path, "rb");
    if (!f) return -1;
    const size_t got = fread(dst, sizeof(float), (size_t)n, f);
    fclose(f);
    return got == (size_t)n ? 0 : -1;
}

static int write_f32(const char* dir, const char* name, const float* src, long n) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE* f = fopen(path, "wb");
    if (!f) return -1;
    const size_t put = fwrite(src, sizeof(float), (size_t)n, f);
    fclose(f);
    return put == (size_t)n ? 0 : -1;
}

#define HIP_OK(x)                                                          \
    do {                                                                   \
        if ((x) != hipSuccess) {                                           \
            fprintf(stderr, "%s failed at line %d\n", #x, __LINE__);       \
            return 1;                                                      \
        }                                                                  \
    } while (0)

int main(int argc, char** argv) {
    if (argc != 4) {
        fprintf(stderr, "usage: %s DIR N K\n", argv[0]);
        return 2;
    }
    const char* dir = argv[1];
    const long n = atol(argv[2]);
    const int k = atoi(argv[3]);
    if (n <= 0 || k < 1 || k > AUTOLOCO_MAX_K) return 2;
    const size_t bytes = (size_t)n * sizeof(float);
    float* host = (float*)malloc(bytes);
    if (!host) return 1;

    autoloco_buffers b;
    memset(&b, 0, sizeof b);
    b.n = n;
    b.k = k;
    b.replica_dtype = AUTOLOCO_F32;
    HIP_OK(hipMalloc((void**)&b.theta, bytes));
    HIP_OK(hipMalloc((void**)&b.momentum, bytes));
    for (int i = 0; i < k; ++i) HIP_OK(hipMalloc(&b.replicas[i], bytes));

    if (read_f32(dir, "theta.f32", host, n)) return 3;
    HIP_OK(hipMemcpy(b.theta, host, bytes, hipMemcpyHostToDevice));
    if (read_f32(dir, "momentum.f32", host, n)) return 3;
    HIP_OK(hipMemcpy(b.momentum, host, bytes, hipMemcpyHostToDevice));
    for (int i = 0; i < k; ++i) {
        char name[64];
        snprintf(name, sizeof name, "replica%d.f32", i);
        if (read_f32(dir, name, host, n)) return 3;
        HIP_OK(hipMemcpy(b.replicas[i], host, bytes, hipMemcpyHostToDevice));
    }

    /* host side: coefficients from the schedule preview and the correction */
    autoloco_controller_cfg cc;
    autoloco_controller_default_cfg(&cc);
    const double lam = autoloco_lr_mass(&cc.sched, 20000, 750);
    const double lam_b = autoloco_lr_mass(&cc.sched, 20000, 500);
    autoloco_outer_coeffs co;
    if (autoloco_outer_correction(&cc.outer, lam, lam_b, &co) != AUTOLOCO_OK) return 4;

    autoloco_ctx* ctx = NULL;
    if (autoloco_create(0, NULL, &ctx) != AUTOLOCO_OK) return 5;
    autoloco_stats st;
    const int rc = autoloco_outer_step(ctx, &b, &co, AUTOLOCO_FUSE_STATS | AUTOLOCO_FUSE_RESET, 1e-12, &st);
    if (rc != AUTOLOCO_OK) {
        fprintf(stderr, "autoloco_outer_step: %s (%s)\n", autoloco_status_string(rc), autoloco_last_error(ctx));
        return 6;
    }

    HIP_OK(hipMemcpy(host, b.theta, bytes, hipMemcpyDeviceToHost));
    if (write_f32(dir, "theta_out.f32", host, n)) return 7;
    HIP_OK(hipMemcpy(host, b.momentum, bytes, hipMemcpyDeviceToHost));
    if (write_f32(dir, "momentum_out.f32", host, n)) return 7;
    HIP_OK(hipMemcpy(host, b.replicas[0], bytes, hipMemcpyDeviceToHost));
    if (write_f32(dir, "replica0_out.f32", host, n)) return 7;

    /* the controller's first interval */
    autoloco_controller* ctl = NULL;
    if (autoloco_controller_create(&cc, &ctl) != AUTOLOCO_OK) return 8;
    autoloco_decision dec;
    if (autoloco_select_interval(ctl, NULL, &dec) != AUTOLOCO_OK) return 8;

    char path[4096];
    snprintf(path, sizeof path, "%s/stats.txt", dir);
    FILE* f = fopen(path, "w");
    if (!f) return 7;
    fprintf(f, "D %.17g\nC %.17g\ndisagreement %.17g\nsq_mean %.17g\nfinite %d\n", st.D, st.C, st.disagreement,
            st.sq_mean, st.finite);
    for (int i = 0; i < k; ++i) fprintf(f, "sq_norm%d %.17g\nsq_dev%d %.17g\n", i, st.sq_norm[i], i, st.sq_dev[i]);
    fprintf(f, "mu %.17g\neta_out %.17g\nrho %.17g\n", co.mu, co.eta_out, co.rho);
    fprintf(f, "first_h_step %lld\nfirst_h_ref %lld\n", (long long)dec.h_step, (long long)dec.h_ref);
    fclose(f);

    autoloco_controller_destroy(ctl);
    autoloco_destroy(ctx);
    for (int i = 0; i < k; ++i) HIP_OK(hipFree(b.replicas[i]));
    HIP_OK(hipFree(b.theta));
    HIP_OK(hipFree(b.momentum));
    free(host);
    return 0;
}
