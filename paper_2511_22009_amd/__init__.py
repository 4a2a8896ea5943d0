"""Stream-batched rectified-flow step on MI355X (gfx950): Python binding of
libstreamflow.so. Every computation runs in the library's HIP kernels; this package
marshals arguments (torch tensors provide device memory and streams)."""
from .binding import (Buffer, Cond, KernelClass, Model, SFError, Precision, lib_path, load_library,
                      library_symbols)

__all__ = ["Buffer", "Cond", "KernelClass", "Model", "SFError", "Precision", "lib_path", "load_library",
           "library_symbols"]
