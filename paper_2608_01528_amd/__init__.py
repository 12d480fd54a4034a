"""Gram-Space matrix-space operators on MI355X (gfx950).

The compute lives in the HIP library built from csrc/ (C-ABI declared in
include/gramspace.h); `gramspace` is its thin ctypes binding.  Importing the
package does not load the library: `paper_2608_01528_amd.gramspace` does, and
fails loudly when it has not been built.
"""
__all__ = ["gramspace", "workloads"]
