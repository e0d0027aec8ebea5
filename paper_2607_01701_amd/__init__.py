"""libt2vattn: packed variable-length bidirectional attention (forward and backward)
for AMD MI355X (gfx950), behind a C ABI (include/t2vattn.h).

The binding below only marshals arguments; all computation is in the HIP library.
"""
from ._lib import (  # noqa: F401
    ORDER_LONGEST_FIRST, ORDER_NATURAL, T2VError, attn_bwd, attn_fwd, t2v_attn_bwd, t2v_attn_fwd,
    t2v_build_worklist, t2v_kernel_times, t2v_last_error, t2v_timing_enable, t2v_plan_makespan, t2v_release_cache, t2v_version,
    use_checked_library,
)
from .autograd import varlen_attention  # noqa: F401
