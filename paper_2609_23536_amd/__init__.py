"""MI355X (gfx950) FP8 delayed-scaling linear layer with split backward.

The work is done by libqe.so (HIP kernels for gfx950 + the C ABI declared in
include/qe.h); ``paper_2609_23536_amd.qe`` is a ctypes binding with the same
entry-point names.  Build the library in-tree with
``python -m paper_2609_23536_amd.build``.
"""
from . import qe  # noqa: F401

__all__ = ["qe"]
