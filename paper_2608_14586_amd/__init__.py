"""MI355X-native GPU-resident prefix of block-layer partitioned VLA inference.

The compute path is the HIP library ``libvlaprefix.so`` (gfx950 kernels plus a
C ABI, see include/vla_prefix.h); ``binding`` marshals arguments to it.
"""
from . import binding  # noqa: F401
from .binding import Boundary, Context, VlaError, stack_cfg  # noqa: F401
