"""MI355X-native data-parallel optimizer update (SlideDP's hot path):
aggregate R ranks' BF16 gradients, clip by the global L2 norm, mixed-precision
AdamW on FP32 master/moments, BF16 re-emit -- hand-written HIP for gfx950
behind the C ABI in include/sdp.h.  ``sdp`` is the ctypes binding."""
from . import sdp  # noqa: F401  (raises ImportError if libsdp.so is not built)

__all__ = ["sdp"]
