"""Reduced-precision (4-bit / 8-bit) integer convolution for AMD MI355X (gfx950).

The compute path is ``libqconv.so`` (hand-written HIP kernels behind a C ABI,
declared in ``include/qconv.h``); :mod:`paper_2202_06819_amd.qconv` is its
ctypes binding, :mod:`paper_2202_06819_amd.nets` chains layers,
:mod:`paper_2202_06819_amd.sweep` measures the compiled tile space.
"""
from . import qconv  # noqa: F401
from .qconv import QConvError, conv2d, default_tile, layout, pack, tiles  # noqa: F401

__all__ = ["qconv", "QConvError", "conv2d", "default_tile", "layout", "pack", "tiles"]
