"""MI355X (gfx950) block-diffusion denoising step: HIP kernels behind a C ABI.

The native library ``libbd.so`` (see ``include/bd.h``) is loaded by
``paper_2609_33887_amd.bd``; build it with ``python -m paper_2609_33887_amd.build``.
"""
__all__ = ["bd"]
