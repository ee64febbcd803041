// Adaptive interval controller and token mapper of AutoLoCo (host, scalar).
//
// Sec. "Adaptive Interval Selection": the residuals of the completed
// interval against the accepted-horizon reference profile
//   xi  = Lambda_done / (Lambda_ref + eps)                     (eq. adaptive-h-lr-mass)
//   r_D = log(sqrt(D) / (sqrt(D_ref) xi + eps) + eps),
//   r_C = -log(C / (C_ref + eps) + eps)                        (eq. adaptive-h-core-residuals)
//   z   = max([r_D - c_D]_+ / s_D, [r_C - c_C]_+ / s_C)        (eq. adaptive-h-core-deviation)
// with c the median and s the MAD scale of the stored residual histories;
// z is classified by Table "Interval assessments".  App. A gives the phases:
// recipe horizon through the warm-up, two reference intervals (geometric
// mean), three variability intervals, monitoring, candidate search (longest
// admissible horizon within 1.15x the accepted LR exposure, or the geometric
// midpoint under a rejected-horizon bound), candidate evaluation, and
// reductions by 1.20 / 1.50 followed by one initialising, three variability
// and one monitoring interval.  The token mapper (eq.
// adaptive-h-token-mapping) turns token-equivalent horizons into executable
// steps with M_base (median token mass of the first three intervals) and an
// EMA of tokens per step.
//
// Where the paper leaves a detail open the controller takes one reading:
//   robust scale max(1.4826 MAD, 1e-3), an empty history contributing 0;
//   log-space EMA coefficient 0.9 for D_ref and C_ref (skipped for values <= 0);
//   reductions snap to the admissible multiple nearest H/divisor strictly
//   below the accepted H, ties to the lower one; the geometric midpoint picks
//   the admissible horizon strictly inside the bound nearest sqrt(H_acc H_rej),
//   ties lower; two consecutive severe-or-invalid intervals fall back to
//   H_min; a non-finite statistic takes the severe reduction path outside the
//   candidate phases and rejects inside them, and is ignored during warm-up;
//   the bound keeps the previewed LR mass of the rejected interval and retires
//   when a preview at the bound is at most 0.90 of it; mapped step horizons
//   round half up to a multiple of q_H (at least q_H); the last interval is
//   truncated to the remaining budget.
//
// Everything is IEEE double without contraction, so two runs on the same
// inputs take the same decisions bit for bit.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <new>

#include "autoloco.h"

namespace {

constexpr int kMaxList = 16;
constexpr uint32_t kMagic = 0x4c4f434fu;  // "LOCO"
constexpr uint32_t kVersion = 1;

struct State {
    uint32_t magic;
    uint32_t version;
    autoloco_controller_cfg cfg;
    int32_t phase;
    int32_t started;
    int64_t start;   // first step of the interval in flight
    int64_t h_cur;   // its token-equivalent horizon
    int64_t h_step;  // its executed steps
    int64_t h_acc;   // accepted token-equivalent horizon
    int64_t h_cand;  // candidate under evaluation
    double lambda_sel;
    int32_t n_boot;
    int32_t n_hist;
    double boot_d[kMaxList], boot_c[kMaxList], boot_l[kMaxList];
    double d_ref, c_ref, l_ref;
    double hist_d[kMaxList], hist_c[kMaxList];  // oldest first
    int32_t var_count, mod_streak, bad_streak, bound_active;
    int64_t h_rej;
    double l_rej;
    int32_t n_msamples, have_m_base;
    double m_samples[kMaxList];
    double m_base;
    int32_t have_n_hat, pad_;
    double n_hat;
    int64_t interval;
};

double median_of(const double* xs, int n) {
    double tmp[kMaxList];
    for (int i = 0; i < n; ++i) tmp[i] = xs[i];
    std::sort(tmp, tmp + n);
    if (n % 2 == 1) return tmp[n / 2];
    return (tmp[n / 2 - 1] + tmp[n / 2]) / 2;
}

double lr_mass_of(const State& s, int64_t start, int64_t steps) {
    return autoloco_lr_mass(&s.cfg.sched, start, steps);
}

int64_t map_steps(const State& s, int64_t h_tok) {
    if (!s.have_m_base || !s.have_n_hat) return h_tok;
    const double x = s.m_base * static_cast<double>(h_tok) /
                     (static_cast<double>(s.cfg.h_base) * (s.n_hat + s.cfg.eps));
    const int64_t q = s.cfg.q_h;
    int64_t h = static_cast<int64_t>(std::floor(x / static_cast<double>(q) + 0.5)) * q;
    return h > q ? h : q;
}

int64_t ref_steps(const State& s) {
    if (!s.have_m_base || !s.have_n_hat) return s.cfg.h_base;
    return map_steps(s, s.cfg.h_base);
}

int64_t adm_lo(const State& s) { return (s.cfg.h_min + s.cfg.q_h - 1) / s.cfg.q_h; }
int64_t adm_hi(const State& s) { return s.cfg.h_max / s.cfg.q_h; }

double z_of(const State& s, const double* hist, int n, double r) {
    if (n == 0) return 0.0;
    const double c = median_of(hist, n);
    double dev_abs[kMaxList];
    for (int i = 0; i < n; ++i) dev_abs[i] = std::fabs(hist[i] - c);
    const double mad = median_of(dev_abs, n);
    double sc = s.cfg.mad_scale * mad;
    if (sc < s.cfg.scale_floor) sc = s.cfg.scale_floor;
    double dev = r - c;
    if (dev < 0.0) dev = 0.0;
    return dev / sc;
}

int classify(const State& s, double z) {
    if (std::isnan(z)) return AUTOLOCO_ASSESS_INVALID;
    if (z < s.cfg.thr_cand) return AUTOLOCO_ASSESS_SUPPORTED;
    if (z < s.cfg.thr_mod) return AUTOLOCO_ASSESS_CONSISTENT;
    if (z < s.cfg.thr_sev) return AUTOLOCO_ASSESS_MODERATE;
    return AUTOLOCO_ASSESS_SEVERE;
}

void push_residuals(State& s, double rd, double rc) {
    if (s.n_hist == s.cfg.hist_max) {
        for (int i = 1; i < s.n_hist; ++i) {
            s.hist_d[i - 1] = s.hist_d[i];
            s.hist_c[i - 1] = s.hist_c[i];
        }
        --s.n_hist;
    }
    s.hist_d[s.n_hist] = rd;
    s.hist_c[s.n_hist] = rc;
    ++s.n_hist;
}

void set_reference(State& s, double d, double c, double lam) {
    s.d_ref = d;
    s.c_ref = c;
    s.l_ref = lam;
    s.n_hist = 0;
    s.var_count = 0;
    s.phase = AUTOLOCO_PHASE_VAR;
}

void ema_reference(State& s, double d, double c, double lam) {
    const double a = s.cfg.ref_ema;
    if (d > 0.0 && s.d_ref > 0.0) s.d_ref = std::exp(a * std::log(s.d_ref) + (1.0 - a) * std::log(d));
    if (c > 0.0 && s.c_ref > 0.0) s.c_ref = std::exp(a * std::log(s.c_ref) + (1.0 - a) * std::log(c));
    s.l_ref = lam;
}

int64_t snap_below(const State& s, double x, int64_t h_cur) {
    int64_t best = -1;
    for (int64_t m = adm_lo(s); m <= adm_hi(s); ++m) {
        const int64_t h = m * s.cfg.q_h;
        if (h >= h_cur) continue;
        if (best < 0 || std::fabs(static_cast<double>(h) - x) < std::fabs(static_cast<double>(best) - x))
            best = h;
    }
    return best < 0 ? h_cur : best;
}

void reduce(State& s, double factor) {
    int64_t h_new;
    if (s.bad_streak >= s.cfg.fallback_count)
        h_new = s.cfg.h_min;
    else
        h_new = snap_below(s, static_cast<double>(s.h_acc) / factor, s.h_acc);
    s.h_acc = h_new;
    s.mod_streak = 0;
    s.n_boot = 0;
    s.phase = AUTOLOCO_PHASE_INIT;
}

void reject(State& s) {
    s.bound_active = 1;
    s.h_rej = s.h_cur;
    s.l_rej = s.lambda_sel;
    s.phase = AUTOLOCO_PHASE_INIT;
}

// Returns the candidate horizon, or -1 when there is none.
int64_t candidate(State& s, int64_t start) {
    if (s.bound_active) {
        if (lr_mass_of(s, start, map_steps(s, s.h_rej)) <= s.cfg.retire_frac * s.l_rej) s.bound_active = 0;
    }
    int64_t best = -1;
    if (s.bound_active) {
        const double g = std::sqrt(static_cast<double>(s.h_acc * s.h_rej));
        for (int64_t m = adm_lo(s); m <= adm_hi(s); ++m) {
            const int64_t h = m * s.cfg.q_h;
            if (h > s.h_acc && h < s.h_rej) {
                if (best < 0 || std::fabs(static_cast<double>(h) - g) < std::fabs(static_cast<double>(best) - g))
                    best = h;
            }
        }
        return best;
    }
    const double l_acc = lr_mass_of(s, start, map_steps(s, s.h_acc));
    for (int64_t m = adm_lo(s); m <= adm_hi(s); ++m) {
        const int64_t h = m * s.cfg.q_h;
        if (h > s.h_acc && lr_mass_of(s, start, map_steps(s, h)) <= s.cfg.cand_exposure * l_acc) best = h;
    }
    return best;
}

// Processes the observation of the interval in flight; returns its assessment.
int observe(State& s, const autoloco_observation& o, double* z_out) {
    const autoloco_controller_cfg& cfg = s.cfg;
    *z_out = std::numeric_limits<double>::quiet_NaN();
    if (o.h_step_done > 0 && std::isfinite(o.tokens)) {
        const double n_bar = o.tokens / static_cast<double>(o.h_step_done);
        if (!s.have_n_hat) {
            s.n_hat = n_bar;
            s.have_n_hat = 1;
        } else {
            s.n_hat = cfg.beta_tok * s.n_hat + (1.0 - cfg.beta_tok) * n_bar;
        }
        if (s.n_msamples < cfg.n_mapper_boot) {
            s.m_samples[s.n_msamples++] = o.tokens;
            if (s.n_msamples == cfg.n_mapper_boot) {
                s.m_base = median_of(s.m_samples, s.n_msamples);
                s.have_m_base = 1;
            }
        }
    }

    const int64_t end = s.start + s.h_step;
    if (s.phase == AUTOLOCO_PHASE_WARMUP) {
        if (end < cfg.sched.warmup) return AUTOLOCO_ASSESS_NONE;
        s.phase = AUTOLOCO_PHASE_REF_BOOT;
    }

    const bool finite = o.finite != 0 && std::isfinite(o.D) && std::isfinite(o.C) &&
                        std::isfinite(o.lambda_done) && o.D >= 0.0 && o.C >= 0.0;
    const bool in_cand = s.phase == AUTOLOCO_PHASE_CAND1 || s.phase == AUTOLOCO_PHASE_CAND2;
    if (!finite) {
        ++s.bad_streak;
        s.mod_streak = 0;
        if (in_cand)
            reject(s);
        else
            reduce(s, cfg.red_severe);
        return AUTOLOCO_ASSESS_INVALID;
    }

    const int ph = s.phase;
    if (ph == AUTOLOCO_PHASE_REF_BOOT) {
        s.bad_streak = 0;
        s.boot_d[s.n_boot] = o.D;
        s.boot_c[s.n_boot] = o.C;
        s.boot_l[s.n_boot] = o.lambda_done;
        ++s.n_boot;
        if (s.n_boot >= cfg.n_ref_boot) {
            double pd = 1.0, pc = 1.0;
            for (int i = 0; i < s.n_boot; ++i) {
                pd *= s.boot_d[i];
                pc *= s.boot_c[i];
            }
            double dr, cr;
            if (s.n_boot == 2) {
                dr = std::sqrt(pd);
                cr = std::sqrt(pc);
            } else {
                dr = std::pow(pd, 1.0 / s.n_boot);
                cr = std::pow(pc, 1.0 / s.n_boot);
            }
            set_reference(s, dr, cr, s.boot_l[s.n_boot - 1]);
            s.n_boot = 0;
        }
        return AUTOLOCO_ASSESS_NONE;
    }
    if (ph == AUTOLOCO_PHASE_INIT) {
        s.bad_streak = 0;
        set_reference(s, o.D, o.C, o.lambda_done);
        return AUTOLOCO_ASSESS_NONE;
    }

    const double eps = cfg.eps;
    const double xi = o.lambda_done / (s.l_ref + eps);
    const double rd = std::log(std::sqrt(o.D) / (std::sqrt(s.d_ref) * xi + eps) + eps);
    const double rc = -std::log(o.C / (s.c_ref + eps) + eps);

    if (ph == AUTOLOCO_PHASE_VAR) {
        s.bad_streak = 0;
        push_residuals(s, rd, rc);
        if (++s.var_count >= cfg.n_var) s.phase = AUTOLOCO_PHASE_MONITOR;
        return AUTOLOCO_ASSESS_NONE;
    }

    const double zd = z_of(s, s.hist_d, s.n_hist, rd);
    const double zc = z_of(s, s.hist_c, s.n_hist, rc);
    const double z = zd > zc ? zd : zc;
    *z_out = z;
    const int a = classify(s, z);
    if (a == AUTOLOCO_ASSESS_INVALID) {
        ++s.bad_streak;
        s.mod_streak = 0;
        if (in_cand)
            reject(s);
        else
            reduce(s, cfg.red_severe);
        return a;
    }

    if (ph == AUTOLOCO_PHASE_MONITOR) {
        if (a == AUTOLOCO_ASSESS_SUPPORTED || a == AUTOLOCO_ASSESS_CONSISTENT) {
            push_residuals(s, rd, rc);
            ema_reference(s, o.D, o.C, o.lambda_done);
            s.mod_streak = 0;
            s.bad_streak = 0;
            if (a == AUTOLOCO_ASSESS_SUPPORTED) {
                const int64_t c = candidate(s, end);
                if (c >= 0) {
                    s.h_cand = c;
                    s.phase = AUTOLOCO_PHASE_CAND1;
                }
            }
        } else if (a == AUTOLOCO_ASSESS_MODERATE) {
            ++s.mod_streak;
            s.bad_streak = 0;
            if (s.mod_streak >= cfg.moderate_confirm) reduce(s, cfg.red_moderate);
        } else {
            ++s.bad_streak;
            s.mod_streak = 0;
            reduce(s, cfg.red_severe);
        }
        return a;
    }

    // candidate phases
    s.bad_streak = 0;
    const bool adopt = a == AUTOLOCO_ASSESS_SUPPORTED ||
                       (a == AUTOLOCO_ASSESS_CONSISTENT && ph == AUTOLOCO_PHASE_CAND2);
    if (adopt) {
        s.h_acc = s.h_cur;
        s.mod_streak = 0;
        set_reference(s, o.D, o.C, o.lambda_done);
    } else if (a == AUTOLOCO_ASSESS_CONSISTENT) {
        s.phase = AUTOLOCO_PHASE_CAND2;
    } else {
        reject(s);
    }
    return a;
}

bool cfg_valid(const autoloco_controller_cfg& c) {
    if (c.q_h <= 0 || c.h_min <= 0 || c.h_min > c.h_max || c.h_base <= 0 || c.budget_steps < 0) return false;
    if ((c.h_min + c.q_h - 1) / c.q_h * c.q_h > c.h_max) return false;  // no admissible horizon
    if (c.n_mapper_boot < 1 || c.n_mapper_boot > kMaxList) return false;
    if (c.n_ref_boot < 1 || c.n_ref_boot > kMaxList) return false;
    if (c.hist_max < 1 || c.hist_max > kMaxList) return false;
    if (c.n_var < 0 || c.moderate_confirm < 1 || c.fallback_count < 1) return false;
    if (!(c.eps > 0.0) || !(c.beta_tok >= 0.0 && c.beta_tok <= 1.0)) return false;
    if (!(c.thr_cand <= c.thr_mod && c.thr_mod <= c.thr_sev)) return false;
    if (!(c.red_moderate > 1.0) || !(c.red_severe > 1.0)) return false;
    if (!(c.scale_floor > 0.0)) return false;
    if (c.sched.warmup < 0 || c.sched.total < c.sched.warmup) return false;
    autoloco_outer_coeffs probe;
    return autoloco_outer_correction(&c.outer, 1.0, 1.0, &probe) == AUTOLOCO_OK;
}

}  // namespace

struct autoloco_controller {
    State s;
};

extern "C" void autoloco_controller_default_cfg(autoloco_controller_cfg* c) {
    if (c == nullptr) return;
    std::memset(c, 0, sizeof(*c));
    c->h_base = 500;
    c->h_min = 250;
    c->h_max = 750;
    c->q_h = 50;
    c->budget_steps = 50000;
    c->beta_tok = 0.9;
    c->eps = 1e-12;
    c->thr_cand = 1.5;
    c->thr_mod = 2.5;
    c->thr_sev = 4.0;
    c->cand_exposure = 1.15;
    c->retire_frac = 0.90;
    c->red_moderate = 1.20;
    c->red_severe = 1.50;
    c->ref_ema = 0.9;
    c->mad_scale = 1.4826;
    c->scale_floor = 1e-3;
    c->n_mapper_boot = 3;
    c->n_ref_boot = 2;
    c->n_var = 3;
    c->hist_max = 16;
    c->moderate_confirm = 2;
    c->fallback_count = 2;
    c->sched.peak = 4e-4;
    c->sched.min_lr = 0.0;
    c->sched.warmup = 1000;
    c->sched.total = 50000;
    c->outer.eta_base = 0.7;
    c->outer.mu_base = 0.9;
    c->outer.mu_min = 0.45;
    c->outer.mu_max = 0.90;
    c->outer.kappa_max = 1.6;
    c->outer.eps = 1e-12;
    c->outer.normalize = 0;
}

extern "C" int autoloco_controller_create(const autoloco_controller_cfg* cfg, autoloco_controller** out) {
    if (cfg == nullptr || out == nullptr) return AUTOLOCO_E_INVALID;
    if (!cfg_valid(*cfg)) return AUTOLOCO_E_INVALID;
    auto* c = new (std::nothrow) autoloco_controller;
    if (c == nullptr) return AUTOLOCO_E_NOMEM;
    std::memset(&c->s, 0, sizeof(State));
    State& s = c->s;
    s.magic = kMagic;
    s.version = kVersion;
    s.cfg = *cfg;
    s.phase = AUTOLOCO_PHASE_WARMUP;
    s.h_cur = cfg->h_base;
    s.h_acc = cfg->h_base;
    *out = c;
    return AUTOLOCO_OK;
}

extern "C" void autoloco_controller_destroy(autoloco_controller* c) { delete c; }

extern "C" int autoloco_select_interval(autoloco_controller* c, const autoloco_observation* obs,
                                        autoloco_decision* next) {
    if (c == nullptr || next == nullptr) return AUTOLOCO_E_INVALID;
    State& s = c->s;
    if (s.phase == AUTOLOCO_PHASE_DONE) return AUTOLOCO_E_STATE;
    double z = std::numeric_limits<double>::quiet_NaN();
    int a = AUTOLOCO_ASSESS_NONE;
    int64_t start;
    if (!s.started) {
        if (obs != nullptr) return AUTOLOCO_E_INVALID;
        s.started = 1;
        start = 0;
    } else {
        if (obs == nullptr) return AUTOLOCO_E_INVALID;
        a = observe(s, *obs, &z);
        start = s.start + s.h_step;
    }
    autoloco_decision d;
    std::memset(&d, 0, sizeof(d));
    d.z_max = z;
    d.assessment = a;
    d.start_step = start;
    if (start >= s.cfg.budget_steps) {
        s.phase = AUTOLOCO_PHASE_DONE;
        d.phase = AUTOLOCO_PHASE_DONE;
        d.done = 1;
        autoloco_outer_correction(&s.cfg.outer, 0.0, 0.0, &d.coeffs);
        *next = d;
        return AUTOLOCO_OK;
    }
    const int64_t h_tok = (s.phase == AUTOLOCO_PHASE_CAND1 || s.phase == AUTOLOCO_PHASE_CAND2) ? s.h_cand : s.h_acc;
    int64_t h_step = map_steps(s, h_tok);
    const int64_t h_ref = ref_steps(s);
    if (start + h_step > s.cfg.budget_steps) h_step = s.cfg.budget_steps - start;
    const double lam = lr_mass_of(s, start, h_step);
    const double lam_b = lr_mass_of(s, start, h_ref);
    autoloco_outer_correction(&s.cfg.outer, lam, lam_b, &d.coeffs);
    s.start = start;
    s.h_cur = h_tok;
    s.h_step = h_step;
    s.lambda_sel = lam;
    ++s.interval;
    d.h_tok = h_tok;
    d.h_step = h_step;
    d.h_ref = h_ref;
    d.lambda_sel = lam;
    d.lambda_base = lam_b;
    d.phase = s.phase;
    *next = d;
    return AUTOLOCO_OK;
}

extern "C" int autoloco_controller_reference(const autoloco_controller* c, double* d_ref, double* c_ref,
                                             double* lambda_ref) {
    if (c == nullptr || d_ref == nullptr || c_ref == nullptr || lambda_ref == nullptr) return AUTOLOCO_E_INVALID;
    *d_ref = c->s.d_ref;
    *c_ref = c->s.c_ref;
    *lambda_ref = c->s.l_ref;
    return AUTOLOCO_OK;
}

extern "C" int autoloco_controller_save(const autoloco_controller* c, void* buf, size_t* len) {
    if (c == nullptr || len == nullptr) return AUTOLOCO_E_INVALID;
    if (buf == nullptr) {
        *len = sizeof(State);
        return AUTOLOCO_OK;
    }
    if (*len < sizeof(State)) return AUTOLOCO_E_INVALID;
    std::memcpy(buf, &c->s, sizeof(State));
    *len = sizeof(State);
    return AUTOLOCO_OK;
}

extern "C" int autoloco_controller_load(autoloco_controller* c, const void* buf, size_t len) {
    if (c == nullptr || buf == nullptr || len != sizeof(State)) return AUTOLOCO_E_INVALID;
    State tmp;
    std::memcpy(&tmp, buf, sizeof(State));
    if (tmp.magic != kMagic || tmp.version != kVersion || !cfg_valid(tmp.cfg)) return AUTOLOCO_E_INVALID;
    // every count within the array it indexes (a reference interval is stored at
    // boot[n_boot] before n_boot reaches n_ref_boot), every horizon within the
    // configuration's bounds
    const autoloco_controller_cfg& g = tmp.cfg;
    auto horizon_ok = [&](int64_t h) { return h == g.h_base || (h >= g.h_min && h <= g.h_max); };
    if (tmp.n_hist < 0 || tmp.n_hist > g.hist_max || tmp.n_boot < 0 || tmp.n_boot >= g.n_ref_boot ||
        tmp.n_msamples < 0 || tmp.n_msamples > g.n_mapper_boot || tmp.phase < 0 || tmp.phase > AUTOLOCO_PHASE_DONE)
        return AUTOLOCO_E_INVALID;
    if (!horizon_ok(tmp.h_acc) || !horizon_ok(tmp.h_cur) || tmp.h_step < 0 || tmp.start < 0 ||
        tmp.start > g.budget_steps || tmp.var_count < 0 || tmp.mod_streak < 0 || tmp.bad_streak < 0 ||
        tmp.interval < 0)
        return AUTOLOCO_E_INVALID;
    if ((tmp.phase == AUTOLOCO_PHASE_CAND1 || tmp.phase == AUTOLOCO_PHASE_CAND2) && !horizon_ok(tmp.h_cand))
        return AUTOLOCO_E_INVALID;
    if (tmp.bound_active && !horizon_ok(tmp.h_rej)) return AUTOLOCO_E_INVALID;
    c->s = tmp;
    return AUTOLOCO_OK;
}
