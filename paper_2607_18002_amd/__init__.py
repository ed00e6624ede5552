"""MI355X-native (gfx950) routed-expert MoE hot path with an adaptive
persistent kernel: top-k gating, permutation, the SwiGLU expert FFN run as
one persistent kernel with a device tile scheduler, and the weighted combine.

The compute lives in libmoe_apk.so (HIP); `ops` is a thin binding of its C ABI
and `pipeline` owns device buffers for a set of operations.  Importing this
package does not load the library; the first call does, and fails loudly if
the library has not been built.
"""
from ._lib import (  # noqa: F401
    MOE_BF16,
    MOE_DECODE,
    MOE_F32,
    MOE_FP8_E4M3,
    MOE_PREFILL,
    MoEError,
    load_library,
)

__all__ = ["load_library", "MoEError", "MOE_BF16", "MOE_F32", "MOE_FP8_E4M3", "MOE_PREFILL", "MOE_DECODE"]
