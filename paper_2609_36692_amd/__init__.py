"""NormPre optimizer step (arXiv 2609.36692) for AMD MI355X (gfx950).

The compute path is libnormpre.so (hand-written HIP kernels behind the C ABI of
include/normpre.h); ``normpre`` is its ctypes binding and ``workloads`` draws
seeded synthetic inputs.  Importing the package does not load the library.
"""
__all__ = ["normpre", "workloads"]
