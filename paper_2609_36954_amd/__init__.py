"""MI355X-native datapath executor of Purlin (arXiv 2609.36954).

``purlin``     ctypes binding of the C-ABI library libpurlin.so (HIP kernels
               for gfx950); loads the library on first use and raises if it
               is missing.
``workloads``  seeded synthetic inputs shaped like the paper's workloads.
``build``      compiles libpurlin.so in-tree.
"""

from .purlin import (  # noqa: F401
    DESC_DTYPE,
    DTYPES,
    OPS,
    Plan,
    Policy,
    PurlinError,
    lib,
    purlin_exec,
    purlin_exec_v,
    purlin_pack,
    purlin_pack_workspace_size,
    purlin_plan,
    purlin_plan_rooted,
    purlin_plan_v,
    purlin_status_string,
    purlin_unpack,
    purlin_version,
)
