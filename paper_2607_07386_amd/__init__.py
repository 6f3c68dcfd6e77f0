"""SDM (Sparse Delta Memory, arXiv 2607.07386) hot path on MI355X (gfx950).

The computation lives in ``libsdm.so`` (HIP kernels behind the C ABI of
``include/sdm.h``); :mod:`paper_2607_07386_amd.sdm` is its Python binding.
"""
from . import sdm  # noqa: F401

__all__ = ["sdm"]
