"""ADT-Tree draft-then-verify hot path on MI355X (gfx950): HIP kernels behind a C ABI
(include/adt.h, libadt.so) and a thin ctypes binding.  PyTorch supplies device memory and
streams only."""
from . import abi  # noqa: F401

__all__ = ["abi", "build", "runtime"]
