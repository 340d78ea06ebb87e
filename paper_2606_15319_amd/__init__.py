"""MI355X-native AR-DiT chunk-denoise block: HIP kernels behind a C ABI.

The compute lives in libardit.so (include/ardit.h); ``ardit`` is its ctypes
binding and ``layout`` the host view of its page and text layouts."""
from . import layout  # noqa: F401


def load():
    """Import the binding (raises if libardit.so has not been built)."""
    from . import ardit
    return ardit
