"""Warp-specialised tiled GEMM for AMD MI355X (gfx950).

C = A B with producer (data-movement) wavefronts filling a multi-stage LDS
ring and consumer (MFMA) wavefronts draining it, after the kernel structure
modelled in "A Performance Model for Warp Specialization Kernels"
(arXiv 2506.11209, Section 1.3 and Algorithm 1).

The compute path is the C-ABI library ``libwsgemm.so`` (``include/ws_gemm.h``);
``paper_2506_11209_amd.wsgemm`` is its ctypes binding.  Importing this package
does not load the library; importing ``paper_2506_11209_amd.wsgemm`` does, and
raises if it has not been built.
"""

__all__ = ["inputs", "workloads"]
