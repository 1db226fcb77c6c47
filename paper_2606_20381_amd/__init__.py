"""UFP4 hot path on MI355X: fused block-16 RHT + 4-bit block-scaled quantization and block-scaled 4-bit GEMMs
(arXiv 2606.20381), as a HIP library (libufp4.so, C ABI in include/ufp4.h) with a thin ctypes binding.

Submodules: ``ufp4`` (the binding), ``workloads`` (seeded synthetic layers), ``build`` (hipcc build).
The binding loads the library lazily; importing the package does not touch the GPU.
"""

__version__ = "0.1.0"
