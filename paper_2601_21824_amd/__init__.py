"""MI355X-native deterministic FlashAttention backward (DASH schedules).

The computation lives in libdash.so (HIP kernels for gfx950 behind the C ABI
in include/dash.h); ``binding`` is its ctypes wrapper and ``synth`` draws the
seeded synthetic inputs.
"""
from . import binding  # noqa: F401
from .binding import (DashError, attn_bwd, attn_fwd, dash_attn_bwd, dash_attn_fwd,  # noqa: F401
                      dash_bwd_check, dash_bwd_workspace_size, dash_last_error,
                      dash_bwd_placement, dash_mfma_peak, dash_release_workspace, dash_resolve_schedule,
                      dash_schedule_table)
