"""Bounded-State Restoration (BSR) restore path for MI355X (gfx950).

The product is the HIP library ``libbsr.so`` (C ABI in ``include/bsr.h``);
``paper_2608_17826_amd.bsr`` is its ctypes binding.  Build with
``python -m paper_2608_17826_amd.build``.
"""
