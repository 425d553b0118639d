"""Pattern-sparse 3x3 convolution for AMD MI355X (gfx950).

The compute path is the HIP library ``libpsc.so`` (sources in ``csrc/``,
C ABI in ``include/psc.h``); ``binding`` wraps it for torch tensors.
"""
from . import binding  # noqa: F401

__all__ = ["binding"]
