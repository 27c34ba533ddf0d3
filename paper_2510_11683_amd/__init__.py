"""MI355X (gfx950) implementation of the BGPO masked-diffusion ELBO head.

The compute path is the HIP library ``libbgpo.so`` built from ``csrc/`` (C ABI
in ``include/bgpo.h``); ``paper_2510_11683_amd.bgpo`` is its ctypes binding and
``paper_2510_11683_amd.build`` compiles it.  Importing the package itself does
not load the library.
"""
__all__ = ["bgpo", "build"]
