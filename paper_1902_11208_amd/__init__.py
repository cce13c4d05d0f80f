"""Packed four-direction MDLSTM layer for MI355X (gfx950).

The computation lives in libmdlstm.so (C ABI: include/mdlstm.h; HIP kernels:
csrc/). This package is its Python binding; torch supplies device memory and
streams.
"""
from ._lib import LIB_PATH, MdlstmError, lib  # noqa: F401

__all__ = ["LIB_PATH", "MdlstmError", "lib"]
