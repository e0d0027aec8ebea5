"""Float64 CPU oracle (test infrastructure only).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this package. The product path (the HIP library and its binding) never does.
"""
from .varlen_attention import attention, head_forward_backward, key_rows, key_rows_torch, query_rows  # noqa: F401
