"""Hand-derived pins of the interval controller's reference update, robust
scale and minimum-horizon fallback, as scripted observation sequences.

Each scenario feeds an OracleController explicit observations (D, C, the
completed interval's learning-rate mass and token count) and checks its
decisions and reference state against values worked out by hand from the
paper's definitions:

  * App. A.1: the two diagnostic references follow a log-space exponential
    moving average, D_ref' = exp(a ln D_ref + (1 - a) ln D) (a = 0.9), updated
    only by increase-supporting or reference-consistent intervals at the
    accepted horizon;
  * eq. adaptive-h-core-deviation: z_max = max([r_D - c_D]_+ / s_D,
    [r_C - c_C]_+ / s_C) with c the median of the residual history and s its
    median-absolute-deviation scale (1.4826 * MAD, floored at 1e-3), with
    histories of odd and even length;
  * App. A.3 "Reducing the horizon": repeated severe or invalid observations
    fall back to H_min (two in a row), a single one reduces by 1.50.

Every expected value below is a literal or a short expression of literals:
the medians and MADs of the histories are worked out by hand in the comments,
never by calling a median routine.  The observations are built from the
controller's current reference (as a trainer's statistics would sit relative
to it), so that each residual takes the value the scenario names.

Both the oracle tests and the C++ replay use these scenarios.
"""
import math
from typing import Callable, List, Tuple

from oracle.controller import Assessment, ControllerConfig, Decision, Observation, OracleController

TOK = float(1 << 20)     # tokens per executed step (constant density)
LAM = 1.0                # learning-rate mass reported for every completed interval
SCALE = 1.4826           # MAD consistency factor


def stable(h: int) -> ControllerConfig:
    # H_max = H_base = the accepted horizon: monitoring never proposes a candidate
    return ControllerConfig(h_base=h, h_min=250, h_max=h)


class Script:
    """Runs one controller through explicit observations; keeps every decision
    and observation so the sequence can be replayed into another controller."""

    def __init__(self, cfg: ControllerConfig):
        self.cfg = cfg
        self.ctl = OracleController(cfg)
        self.decisions: List[Decision] = [self.ctl.select_interval(None)]
        self.observations: List[Observation] = []

    @property
    def last(self) -> Decision:
        return self.decisions[-1]

    def feed(self, D: float, C: float, finite: bool = True, lam: float = LAM) -> Decision:
        h = self.last.h_step
        obs = Observation(D, C, lam, TOK * h, h, finite)
        self.observations.append(obs)
        self.decisions.append(self.ctl.select_interval(obs))
        return self.decisions[-1]

    def at(self, x: float, y: float) -> Decision:
        """An interval whose residuals are r_D = x and r_C = y against the current
        reference (eq. adaptive-h-core-residuals): sqrt(D) = sqrt(D_ref) xi e^x,
        C = C_ref e^-y, with xi = Lambda_done / (Lambda_ref + eps)."""
        c = self.ctl
        xi = LAM / (c.l_ref + self.cfg.eps)
        return self.feed(c.d_ref * xi * xi * math.exp(2.0 * x), c.c_ref * math.exp(-y))

    def bootstrap(self, d: float, c: float) -> None:
        """Warm-up interval(s), then two reference intervals at (d, c): the first
        intervals of a run whose last step reaches step 1,000 or later boot the
        reference (App. A.1)."""
        while self.ctl.phase == 0:           # WARMUP
            self.feed(d, c)
        self.feed(d, c)                      # second reference interval


def run_ema() -> Tuple[Script, List[Tuple[str, float, float]]]:
    """Log-space EMA of the references (App. A.1).  Returns the script and a
    list of (what, got, want) to compare."""
    s = Script(stable(500))
    d0, c0 = 2.0 ** -6, 4.0                  # reference = geometric mean of two equal intervals
    s.bootstrap(d0, c0)
    checks = [("D_ref after bootstrap", s.ctl.d_ref, d0), ("C_ref after bootstrap", s.ctl.c_ref, c0)]
    for _ in range(3):                       # three variability intervals on the profile
        s.at(0.0, 0.0)
    # A monitoring interval far off the profile on the favourable side: D 1024x
    # below it and C 1024x above it.  Both residuals are negative, so z = 0 and
    # the interval is increase-supporting; it updates the references:
    #   D_ref' = exp(0.9 ln D_ref + 0.1 ln(D_ref xi^2 / 1024)) = D_ref xi^0.2 / 2
    #   C_ref' = exp(0.9 ln 4 + 0.1 ln 4096) = 4 * 1024^0.1 = 8
    xi = LAM / (s.ctl.l_ref + s.cfg.eps)
    dec = s.feed(d0 * xi * xi / 1024.0, c0 * 1024.0)
    checks += [("z of the favourable interval", dec.z_max, 0.0),
               ("assessment of the favourable interval", dec.assessment, Assessment.SUPPORTED),
               ("D_ref after the EMA", s.ctl.d_ref, 2.0 ** -7 * xi ** 0.2),
               ("C_ref after the EMA", s.ctl.c_ref, 8.0),
               ("Lambda_ref after the EMA", s.ctl.l_ref, LAM)]
    # The next interval sits exactly on the updated profile: both residuals 0.
    dec = s.feed(2.0 ** -7 * xi ** 0.2 * xi * xi, 8.0)
    checks += [("z on the updated profile", dec.z_max, 0.0),
               ("assessment on the updated profile", dec.assessment, Assessment.SUPPORTED)]
    # Twice the learning-rate mass of the reference interval (xi = 2): four
    # times the reference drift energy is on the profile (r_D = 0, z = 0).
    xi2 = 2.0 * LAM / (s.ctl.l_ref + s.cfg.eps)
    dec = s.feed(s.ctl.d_ref * xi2 * xi2, s.ctl.c_ref, lam=2.0 * LAM)
    checks += [("z at twice the learning-rate mass", dec.z_max, 0.0),
               ("assessment at twice the learning-rate mass", dec.assessment, Assessment.SUPPORTED),
               ("Lambda_ref follows the accepted interval", s.ctl.l_ref, 2.0 * LAM)]
    # A moderate deviation does not move the references (only supporting or
    # consistent intervals update them).  Every residual in the histories is
    # 0 up to rounding except the favourable interval's (r_D = -ln 32,
    # r_C = -ln 1024): median 0, MAD 0, so s = 1e-3 (the floor), and r_C =
    # 0.003 gives z = 3.0.
    d_before, c_before = s.ctl.d_ref, s.ctl.c_ref
    dec = s.at(0.0, 0.003)
    checks += [("z of the moderate interval", dec.z_max, 3.0),
               ("assessment of the moderate interval", dec.assessment, Assessment.MODERATE),
               ("D_ref kept by a moderate interval", s.ctl.d_ref, d_before),
               ("C_ref kept by a moderate interval", s.ctl.c_ref, c_before)]
    # The same on the drift side (r_D = 0.003: z = 3.0 at the floor), the second
    # moderate interval in a row: the horizon drops by 1.20, 500 / 1.2 = 416.7 ->
    # 400 (nearest admissible multiple of 50 strictly below 500).
    dec = s.at(0.003, 0.0)
    checks += [("z of the drift-side moderate interval", dec.z_max, 3.0),
               ("assessment of the drift-side moderate interval", dec.assessment, Assessment.MODERATE),
               ("horizon after two moderate intervals", dec.h_tok, 400)]
    return s, checks


def run_mad() -> Tuple[Script, List[Tuple[str, float, float]]]:
    """Median / MAD scale of z_max (eq. adaptive-h-core-deviation) over
    histories of 3 to 6 residuals, landing in each class of Table "Interval
    assessments"."""
    s = Script(stable(500))
    s.bootstrap(2.0 ** -6, 4.0)
    # variability intervals: r_D = 0, 0.004, -0.004; r_C = 0, 0.01, -0.01
    for x, y in ((0.0, 0.0), (0.004, 0.01), (-0.004, -0.01)):
        s.at(x, y)
    checks = []
    # (1) 3 entries.  D: {-.004, 0, .004}: median 0, |dev| {0, .004, .004}: MAD .004.
    #     r_D = .008 -> z_D = .008 / (1.4826 * .004) = 1.349 (supported); r_C = 0 -> z_C = 0.
    dec = s.at(0.008, 0.0)
    checks += [("z, 3 entries", dec.z_max, 0.008 / (SCALE * 0.004)),
               ("class, 3 entries", dec.assessment, Assessment.SUPPORTED)]
    # (2) 4 entries.  D: {-.004, 0, .004, .008}: median .002; C: {-.01, 0, 0, .01}:
    #     median 0, |dev| {0, 0, .01, .01}: MAD (0 + .01) / 2 = .005.
    #     r_D = -.008 (below the centre, z_D = 0); r_C = .015 -> z_C = .015 / (1.4826 * .005) = 2.023.
    dec = s.at(-0.008, 0.015)
    checks += [("z, 4 entries", dec.z_max, 0.015 / (SCALE * 0.005)),
               ("class, 4 entries", dec.assessment, Assessment.CONSISTENT)]
    # (3) 5 entries.  D: {-.008, -.004, 0, .004, .008}: median 0, MAD .004;
    #     C: {-.01, 0, 0, .01, .015}: median 0, |dev| {0, 0, .01, .01, .015}: MAD .01.
    #     r_D = 3 * 1.4826 * .004 -> z_D = 3 (moderate); r_C = .01 -> z_C = .6745.
    dec = s.at(3 * SCALE * 0.004, 0.01)
    checks += [("z, 5 entries (moderate)", dec.z_max, 3.0),
               ("class, 5 entries (moderate)", dec.assessment, Assessment.MODERATE)]
    # a moderate interval is not added to the history: still 5 entries.
    #     r_D = 0 -> 0; r_C = 1.4826 * .01 -> z_C = 1 (supported), added.
    dec = s.at(0.0, SCALE * 0.01)
    checks += [("z, 5 entries (supported)", dec.z_max, 1.0),
               ("class, 5 entries (supported)", dec.assessment, Assessment.SUPPORTED)]
    # (4) 6 entries.  D: {-.008, -.004, 0, 0, .004, .008}: median 0, |dev| {0, 0,
    #     .004, .004, .008, .008}: MAD .004.  C: {-.01, 0, 0, .01, .014826, .015}:
    #     median (0 + .01) / 2 = .005, |dev| {.005, .005, .005, .009826, .01, .015}:
    #     MAD (.005 + .009826) / 2 = .007413.
    #     r_C = .005 + 4.5 * 1.4826 * .007413 -> z_C = 4.5 (severe); r_D = 0.
    mad_c = (0.005 + (SCALE * 0.01 - 0.005)) / 2.0
    dec = s.at(0.0, 0.005 + 4.5 * SCALE * mad_c)
    checks += [("z, 6 entries (severe)", dec.z_max, 4.5),
               ("class, 6 entries (severe)", dec.assessment, Assessment.SEVERE),
               ("horizon after the severe interval (500 / 1.5 -> 350)", dec.h_tok, 350)]
    return s, checks


def run_fallback(kind: str) -> Tuple[Script, List[Tuple[str, float, float]]]:
    """H_min fallback (App. A.3) at H_base = H_max = 750, H_min = 250, q_H = 50.
    A single severe or invalid interval reduces 750 / 1.5 = 500; a second one in
    a row (the next interval, which would otherwise initialise the new
    reference) falls back to 250, where a plain reduction would give 500 / 1.5
    = 333.3 -> 350.  A severe interval after a completed re-estimation is not
    in a streak: 350."""
    s = Script(stable(750))
    s.bootstrap(2.0 ** -6, 4.0)
    for _ in range(3):
        s.at(0.0, 0.0)
    nan = float("nan")
    checks = []
    if kind == "invalid-invalid":
        d1 = s.feed(nan, 4.0, finite=False)
        d2 = s.feed(nan, 4.0, finite=False)
        checks += [("first invalid", d1.assessment, Assessment.INVALID), ("after one", d1.h_tok, 500),
                   ("second invalid", d2.assessment, Assessment.INVALID), ("after two", d2.h_tok, 250)]
    elif kind == "severe-invalid":
        d1 = s.at(0.0, 0.005)               # MAD 0: s = 1e-3, z = 5 -> severe
        d2 = s.feed(nan, 4.0, finite=False)
        checks += [("severe", d1.assessment, Assessment.SEVERE), ("after one", d1.h_tok, 500),
                   ("then invalid", d2.assessment, Assessment.INVALID), ("after two", d2.h_tok, 250)]
    elif kind == "severe-later-severe":
        d1 = s.at(0.0, 0.005)
        checks += [("severe", d1.assessment, Assessment.SEVERE), ("after one", d1.h_tok, 500)]
        s.at(0.0, 0.0)                      # initialises the reference at 500
        for _ in range(3):
            s.at(0.0, 0.0)                  # variability
        d2 = s.at(0.0, 0.005)
        checks += [("severe again", d2.assessment, Assessment.SEVERE),
                   ("not a streak: 500 / 1.5 -> 350", d2.h_tok, 350)]
    else:
        raise ValueError(kind)
    return s, checks


SCENARIOS: List[Tuple[str, Callable]] = [
    ("ema", run_ema),
    ("mad", run_mad),
    ("fallback-invalid-invalid", lambda: run_fallback("invalid-invalid")),
    ("fallback-severe-invalid", lambda: run_fallback("severe-invalid")),
    ("fallback-severe-later-severe", lambda: run_fallback("severe-later-severe")),
]


def failures(checks, rel: float = 1e-9, abs_tol: float = 1e-7) -> List[str]:
    """The checks whose got differs from want (integers and classes exactly)."""
    bad = []
    for what, got, want in checks:
        if isinstance(want, float):
            ok = math.isclose(got, want, rel_tol=rel, abs_tol=abs_tol) if math.isfinite(want) else got == want
        else:
            ok = got == want
        if not ok:
            bad.append(f"{what}: got {got!r}, want {want!r}")
    return bad
