"""MI355X-native pipelined-offloading OPT decoder (PIPO, arXiv 2504.03664).

The compute path lives in ``libpipo.so`` (HIP kernels for gfx950 behind the
C ABI of ``include/pipo.h``); ``binding`` exposes that ABI under the same
names and ``model`` lays weights out in pinned host memory.
"""
from . import binding  # noqa: F401
from .model import Decoder, HostWeights, c_policy, c_shape  # noqa: F401
