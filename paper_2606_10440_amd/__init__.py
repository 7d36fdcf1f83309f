"""MI355X-native line-granularity network simulator (HIP kernels behind a C ABI).

``paper_2606_10440_amd.sim`` is the ctypes binding of ``libsimgpu.so``;
``paper_2606_10440_amd.build`` compiles it for gfx950.
"""
from . import sim  # noqa: F401
from .sim import Simulator, SimError  # noqa: F401
