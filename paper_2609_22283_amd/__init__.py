"""MI355X-native packed causal-context DiT step (streaming video diffusion).

Thin ctypes binding over ``libstreamctx.so`` (C ABI in include/streamctx.h).
Every computation runs in the library's HIP kernels or its C++ host core;
this module only marshals arguments.  PyTorch supplies device memory and
streams.  Loading fails loudly when the library has not been built: there is
no fallback path.
"""
from .binding import *  # noqa: F401,F403
from .binding import __all__  # noqa: F401
