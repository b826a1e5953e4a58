"""GNNShap coalition-evaluation path for one AMD Instinct MI355X (gfx950).

The work runs in libgnnshap.so (HIP kernels + host C++, C ABI in
include/gnnshap.h).  ``_lib`` binds the C ABI one function per entry point;
``explainer.Explainer`` drives the four calls with torch-owned device memory.
"""
from . import _lib  # noqa: F401
from ._lib import load, GnnShapError  # noqa: F401


def Explainer(*args, **kwargs):
    from .explainer import Explainer as _E
    return _E(*args, **kwargs)
