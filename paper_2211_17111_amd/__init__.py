"""BEVPoolv2 view-transform path for AMD Instinct MI355X (gfx950).

HIP kernels behind the C ABI of include/bevpool.h, with a thin ctypes
binding (``paper_2211_17111_amd.bevpool``).
"""

from .bevpool import (  # noqa: F401
    BEVPOOL_F16,
    BEVPOOL_F32,
    BevpoolError,
    Plan,
    Schedule,
    backward,
    backward_scheduled,
    bev_pool,
    bevpool_backward,
    bevpool_backward_scheduled,
    bevpool_backward_workspace_size,
    bevpool_forward,
    bevpool_forward_scheduled,
    bevpool_forward_scheduled_workspace_size,
    bevpool_forward_workspace_size,
    bevpool_last_error,
    bevpool_prepare,
    bevpool_prepare_workspace_size,
    bevpool_schedule,
    bevpool_schedule_size,
    bevpool_strerror,
    bevpool_version,
    declared_symbols,
    forward,
    forward_scheduled,
    forward_scheduled_workspace,
    load_library,
    prepare,
    schedule,
)
