"""Reference oracle for the AutoLoCo synchronisation round — TEST INFRASTRUCTURE.

A plain, slow, CPU-only evaluation of what one synchronisation round computes,
written from the paper (arxiv 2609.36662, "AutoLoCo: Communication Efficient
Distributed LLM Training via Adaptive Synchronization") in float64 and exact
rational arithmetic.  It exists to check the GPU library against; it is not
part of the library.

Only the test suite, the smoke check of the package entry file and the CPU
baseline leg of the benchmark may import or run anything in this package.  It
shares no code with the HIP/C++ library: it includes no header of it, loads no
binary of it and reuses none of its constants or helpers.

Modules
  round       — pseudo-gradients, their mean, local-drift energy D and
                aggregation coherence C (Sec. "Adaptive Interval Selection",
                eq. adaptive-h-core-diagnostics; App. C.1), the corrected
                Nesterov outer step (eq. autoloco-corrected-nesterov) and the
                replica reset (Alg. "AutoLoCo outer interval").
  exact       — the same round in ``fractions.Fraction`` arithmetic for tiny
                inputs (brute-force pin of ``round``).
  correction  — the inner learning-rate schedule, learning-rate masses and the
                Outer Optimizer Correction (eqs. outer-correction-ratio,
                normalized-pseudo-gradient, adjusted-outer-learning-rate;
                App. B.2-B.4).
  controller  — the adaptive interval controller and token mapper (Sec.
                "Adaptive Interval Selection"; App. A).
  int8_codec  — the INT8 blockwise pseudo-gradient codec and the round that
                averages through it (App. G.1).
  bf16_payload — the round whose worker average travels as BF16
                pseudo-gradients (the payload of the paper's main runs).
  adamw       — one inner AdamW step of every worker with its own
                gradient-norm clipping (Table "Training settings"; App. G.1).

Parity unpinned (no value printed by the paper and no closed form fixes them;
each is one reading of a point the paper leaves open):
  * the constants 1.4826 (MAD consistency factor) and 1e-3 (scale floor) of
    z_max's robust scale,
  * the coefficient 0.9 of the log-space EMA of the reference diagnostics,
  * tie-breaking of reductions and geometric midpoints,
  * the count 2 of severe/invalid intervals that triggers the H_min fallback,
  * the rejected-horizon bound beyond its printed constants.
The forms around those constants (the median/MAD scale over odd and even
histories, the log-space EMA and which intervals update it, the fallback after
a streak versus a single reduction) are pinned by hand-derived scenarios in the
test suite, and the controller as a whole by the executed interval sequence the
paper prints for its C4 run (App. F.2).
"""
