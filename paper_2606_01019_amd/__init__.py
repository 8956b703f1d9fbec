"""MI355X (gfx950) verification step of Hybrid Verified Decoding.

The work runs in libhvd.so (C ABI in include/hvd.h, HIP kernels in csrc/);
this package holds the build script and a thin ctypes binding.
"""

from .hvd import (  # noqa: F401
    EXPORTS,
    Config,
    HvdError,
    KVCache,
    Model,
    load_library,
    measure_mfma_peak,
    tensor_names,
)
