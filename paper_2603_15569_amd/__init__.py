"""libm3: the Mamba-3 SSM layer's prefill scan and decode step on MI355X.

The compute path is the HIP library libm3.so (C ABI in include/m3.h); this
package holds its sources (csrc/), the build script, the ctypes binding (m3)
and the seeded workload generators (inputs).
"""
from . import inputs  # noqa: F401
from .m3 import (M3Dims, M3Error, lib, scan_fwd, step, workspace_bytes)  # noqa: F401
