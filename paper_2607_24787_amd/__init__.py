"""MI355X (gfx950) SpecPrefetch offloaded-MoE decode hot path.

``spp`` is the ctypes binding of the C ABI (include/spp.h) implemented by
libspp.so (HIP kernels + native runtime); ``model`` assembles a synthetic
stack on the device with PyTorch used only for memory and streams.
"""
from . import spp  # noqa: F401
