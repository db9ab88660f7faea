"""GNMR controller pass on AMD Instinct MI355X (gfx950).

The controller pass (per-unit gradient L2 norms, GNMR / Delta-GNMR state
update, budgeted Top_maxO selection with lock counters) runs in hand-written
HIP kernels behind the C ABI of include/gnmr.h (libgnmr.so).  This package is
the thin Python binding over that ABI.
"""
from .binding import (GNMR_BF16, GNMR_BUDGET_ACTIVE, GNMR_BUDGET_ADMITTED,  # noqa: F401
                      GNMR_BUDGET_STATIC, GNMR_FMT_BF16, GNMR_FMT_E2M1, GNMR_FMT_E3M2,
                      GNMR_FMT_E4M3, GNMR_FMT_E5M2, GNMR_FMT_INT8, Actuator, gnmr_actuate,
                      gnmr_actuate_matrix,
                      gnmr_actuator_create, gnmr_actuator_destroy, gnmr_actuator_info,
                      GNMR_F32, Controller, GnmrError,
                      gnmr_destroy, gnmr_device_outputs, gnmr_get_state, gnmr_info,
                      gnmr_init, gnmr_last_error, gnmr_profile_read, gnmr_query,
                      gnmr_set_profiling, gnmr_set_state, gnmr_state_size, gnmr_step,
                      gnmr_step_from_norms, gnmr_sumsq, gnmr_sumsq_noalloc, gnmr_wgrad_num_tiles,
                      gnmr_wgrad_sumsq, gnmr_wgrad_sumsq_batched, gnmr_bind_partials, gnmr_step_from_partials,
                      load_library)
