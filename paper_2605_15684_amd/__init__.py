"""SSBA (Shift Sparse Block Attention) forward pass for AMD MI355X (gfx950).

The compute path lives in ``libssba.so`` (HIP kernels behind a C ABI declared
in ``include/ssba.h``); ``paper_2605_15684_amd.ssba`` is the thin torch-facing
binding.  Importing the package does not load the library; importing
``paper_2605_15684_amd.ssba`` does, and fails loudly if it is not built.
"""
__version__ = "0.1.0"
