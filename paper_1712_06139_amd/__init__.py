"""Request batching for model serving on one MI355X (gfx950).

The batching path of TensorFlow-Serving's inter-request batching (paper
section 2.2.1) as a HIP library (librbatch.so, C ABI in include/rb.h) with a
thin ctypes binding in `rb`. Loading fails loudly when the library is not
built: there is no fallback path.
"""
from . import rb  # noqa: F401
