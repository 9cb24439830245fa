"""MixFlow-MG meta-gradients on MI355X: HIP kernels behind a C ABI (include/mfmg.h).

``paper_2505_00793_amd._lib`` is the ctypes binding; ``build`` compiles the
library in-tree.  Importing the package does not load the library.
"""
from . import _lib  # noqa: F401
from ._lib import Problem, make_desc, lib, MfmgError  # noqa: F401
