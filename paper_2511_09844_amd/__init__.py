"""MI355X (gfx950) SD^2 speculative-decoding round: C-ABI library libsd2.so + thin binding.

Every step of the round runs in the library's HIP kernels; this package only
marshals arguments (PyTorch supplies device memory and the stream).  Importing
the binding fails loudly when libsd2.so has not been built.
"""
from .build import build, SO  # noqa: F401
