// Host-side scalar routines of the AutoLoCo round: the inner learning-rate
// schedule, learning-rate masses and the Outer Optimizer Correction.
//
//   Lambda = sum_{h=1..H} eta(s_t + h - 1)        (App. B.2, eq. app-outer-correction-lr-masses)
//   rho    = max(Lambda / (Lambda_base + eps), 1)  (eq. outer-correction-ratio)
//   mu     = clip(mu_base^rho, mu_min, mu_max), kappa = min(rho, kappa_max)
//   eta    = eta_base * kappa * (1 - mu) / (1 - mu_base)   (eq. adjusted-outer-learning-rate)
//
// Built without floating-point contraction so that a decision taken from these
// values does not depend on the compiler.
#include <cmath>
#include <limits>

#include "autoloco.h"

extern "C" const char* autoloco_status_string(int status) {
    switch (status) {
        case AUTOLOCO_OK: return "ok";
        case AUTOLOCO_E_INVALID: return "invalid argument";
        case AUTOLOCO_E_ALIGN: return "device pointer not 16-byte aligned";
        case AUTOLOCO_E_ALIAS: return "device buffers overlap";
        case AUTOLOCO_E_DEVICE: return "HIP runtime error";
        case AUTOLOCO_E_NOMEM: return "out of memory";
        case AUTOLOCO_E_STATE: return "call out of order";
        default: return "unknown status";
    }
}

extern "C" double autoloco_inner_lr(const autoloco_schedule* s, int64_t step) {
    if (s == nullptr || step < 0) return std::numeric_limits<double>::quiet_NaN();
    if (step < s->warmup) return s->peak * static_cast<double>(step + 1) / static_cast<double>(s->warmup);
    const int64_t span = s->total - s->warmup;
    double frac = span > 0 ? static_cast<double>(step - s->warmup) / static_cast<double>(span) : 1.0;
    if (frac > 1.0) frac = 1.0;
    return s->min_lr + (s->peak - s->min_lr) * 0.5 * (1.0 + std::cos(M_PI * frac));
}

extern "C" double autoloco_lr_mass(const autoloco_schedule* s, int64_t start_step, int64_t steps) {
    if (s == nullptr || start_step < 0 || steps < 0) return std::numeric_limits<double>::quiet_NaN();
    double total = 0.0;
    for (int64_t h = 1; h <= steps; ++h) total += autoloco_inner_lr(s, start_step + h - 1);
    return total;
}

extern "C" int autoloco_outer_correction(const autoloco_outer_cfg* cfg, double lambda_sel,
                                         double lambda_base, autoloco_outer_coeffs* out) {
    if (cfg == nullptr || out == nullptr) return AUTOLOCO_E_INVALID;
    if (!std::isfinite(lambda_sel) || !std::isfinite(lambda_base)) return AUTOLOCO_E_INVALID;
    if (!(cfg->mu_base > 0.0 && cfg->mu_base < 1.0) || !(cfg->mu_min <= cfg->mu_max) ||
        !(cfg->kappa_max >= 1.0) || !(cfg->eps >= 0.0))
        return AUTOLOCO_E_INVALID;
    double rho = lambda_sel / (lambda_base + cfg->eps);
    if (!(rho > 1.0)) rho = 1.0;
    double mu = std::pow(cfg->mu_base, rho);
    if (mu < cfg->mu_min) mu = cfg->mu_min;
    if (mu > cfg->mu_max) mu = cfg->mu_max;
    const double kappa = rho < cfg->kappa_max ? rho : cfg->kappa_max;
    out->mu = mu;
    out->kappa = kappa;
    out->rho = rho;
    out->eta_out = cfg->eta_base * kappa * ((1.0 - mu) / (1.0 - cfg->mu_base));
    out->normalize = cfg->normalize ? 1 : 0;
    return AUTOLOCO_OK;
}
