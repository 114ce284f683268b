"""MI355X (gfx950) block-decode step of linear self-speculation (arXiv 2607.05722, Sec. 3.3).

``libnld.so`` (HIP kernels + C ABI, see include/nld.h) does the work;
``paper_2607_05722_amd.runtime`` is its Python binding.  PyTorch is used for
device memory and streams only.
"""
from . import _lib
from .buildlib import build

__all__ = ["_lib", "build"]
