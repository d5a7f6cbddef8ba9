"""MI355X (gfx950) implementation of DFlow's per-round block-diffusion
speculative decoding step behind the C ABI declared in include/dflow.h.

Every computation runs in the HIP kernels of libdflow.so; the Python layer
marshals arguments, allocates device memory through PyTorch and sequences
the four round calls.
"""
from .runtime import DFlowError, Runtime, library_path, load_library  # noqa: F401
