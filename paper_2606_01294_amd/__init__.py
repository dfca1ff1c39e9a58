"""MI355X (gfx950) Curvature-Conditioned Query: chunkwise CCQ-GLA / CCQ-GDN kernels.

The compute lives in libccq.so (HIP kernels behind the C ABI of include/ccq.h);
``paper_2606_01294_amd.ccq`` is its ctypes binding and
``paper_2606_01294_amd.inputs`` the seeded input generator.
"""
__version__ = "0.1.0"
