"""AutoLoCo synchronisation round on AMD Instinct MI355X (gfx950).

The round (pseudo-gradients, their mean, the D/C diagnostics, the corrected
Nesterov outer step and the replica reset), and the workers' inner AdamW
step between rounds, run in hand-written HIP kernels
behind the C ABI of include/autoloco.h; the interval controller and the outer
correction are host C++ behind the same ABI.  This package is the thin Python
binding (same names as the C calls) and the in-tree build.
"""
from ._lib import (  # noqa: F401
    BF16, F32, FUSE_RESET, FUSE_STATS, MAX_K, AutolocoError, Context, Controller,
    autoloco_alloc_spread, autoloco_broadcast_reset, autoloco_controller_create, autoloco_free, autoloco_controller_load,
    autoloco_controller_reference, autoloco_controller_save, autoloco_create, autoloco_destroy,
    autoloco_inner_lr, autoloco_last_error, autoloco_last_kernel_ms, autoloco_launch_shape,
    autoloco_lr_mass, autoloco_outer_correction, autoloco_outer_step, autoloco_outer_step_bf16, autoloco_outer_step_int8, autoloco_round_stats,
    autoloco_select_interval, autoloco_set_grid_limit, autoloco_set_timing, default_controller_cfg,
    lib, make_buffers, make_coeffs, make_observation, make_outer_cfg, make_schedule, spread_tensors,
    autoloco_inner_adamw, autoloco_last_adamw_ms, autoloco_adamw_traffic_reference, autoloco_rank_payload, autoloco_shard_step, make_adamw_buffers, make_adamw_coeffs,
    autoloco_traffic_reference, autoloco_traffic_probe, autoloco_build_id, autoloco_outer_step_static,
    PROBE_READ, PROBE_WRITE, PROBE_RUN1, PROBE_RUN2, PROBE_SERIAL, PROBE_TILE, PROBE_PHASED, PROBE_RUN8,
)
