"""Confidence-modulated speculative decoding, logit pass, on MI355X (gfx950).

The compute path is ``libcmsd.so`` (HIP kernels behind include/cmsd.h); the
``cmsd`` submodule is its ctypes binding.  Build with
``python -m paper_2508_15371_amd.build``.
"""
__all__ = ["cmsd"]
