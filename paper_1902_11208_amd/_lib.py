"""ctypes loader for libmdlstm.so (the C ABI in include/mdlstm.h).

The library is built in-tree by ``python -m paper_1902_11208_amd.build``;
nothing here falls back to another implementation when it is missing.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmdlstm.so")

# names and argument types of every exported entry point
c_i32, c_size, c_void, c_char_p = ctypes.c_int32, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_char_p


class Rect(ctypes.Structure):
    _fields_ = [("y0", c_i32), ("x0", c_i32), ("h", c_i32), ("w", c_i32)]


class LayerDesc(ctypes.Structure):
    _fields_ = [("c_in", c_i32), ("hidden", c_i32), ("dtype", c_i32), ("memory_states", c_i32)]


class HeadDesc(ctypes.Structure):
    _fields_ = [("hidden", c_i32), ("classes", c_i32)]


P_I32 = ctypes.POINTER(c_i32)
P_RECT = ctypes.POINTER(Rect)
P_DESC = ctypes.POINTER(LayerDesc)
P_HEAD = ctypes.POINTER(HeadDesc)
P_VOIDP = ctypes.POINTER(c_void)

SIGNATURES = {
    "mdlstm_pack_workspace_bytes": (c_size, [c_i32]),
    "mdlstm_pack_layout": (c_i32, [c_i32, P_I32, P_I32, c_i32, P_RECT, P_I32, c_void, c_size, c_void, c_size, c_void]),
    "mdlstm_pack_layout_noalloc": (c_i32, [c_i32, P_I32, P_I32, c_i32, P_RECT, P_I32, c_void, c_size, c_void]),
    "mdlstm_pad_layout": (c_i32, [c_i32, P_I32, P_I32, P_RECT, P_RECT, P_I32, P_I32, c_void, c_size, c_void, c_size,
                                  c_void]),
    "mdlstm_pack_data": (c_i32, [c_i32, P_VOIDP, P_RECT, c_i32, c_i32, c_i32, c_i32, c_void, c_void, c_size, c_void]),
    "mdlstm_unpack_data": (c_i32, [c_i32, P_VOIDP, P_RECT, c_i32, c_i32, c_i32, c_i32, c_void, c_void, c_size,
                                   c_void]),
    "mdlstm_workspace_bytes": (c_size, [P_DESC, c_i32, c_i32, c_i32]),
    "mdlstm_forward": (c_i32, [P_DESC, c_i32, c_i32, c_void, c_void, c_i32, P_RECT, c_void, c_void, c_void, c_void,
                               c_void, c_size, c_void]),
    "mdlstm_forward_stepwise": (c_i32, [P_DESC, c_i32, c_i32, c_void, c_void, c_i32, P_RECT, c_void, c_void, c_void,
                                        c_void, c_void, c_size, c_void]),
    "mdlstm_backward": (c_i32, [P_DESC, c_i32, c_i32, c_void, c_void, c_i32, P_RECT, c_void, c_void, c_void, c_void,
                                c_void, c_void, c_void, c_void, c_void, c_void, c_size, c_void]),
    "mdlstm_head_workspace_bytes": (c_size, [P_HEAD, c_i32, P_RECT, P_I32]),
    "mdlstm_head_forward": (c_i32, [P_HEAD, c_i32, c_i32, c_void, c_i32, P_RECT, c_void, c_void, c_void, c_void,
                                    c_size, c_void]),
    "mdlstm_ctc_loss": (c_i32, [P_HEAD, c_i32, P_RECT, P_I32, P_I32, c_void, c_void, c_void, c_void, c_size, c_void]),
    "mdlstm_head_backward": (c_i32, [P_HEAD, c_i32, c_i32, c_i32, P_RECT, c_void, c_void, c_void, c_void, c_void,
                                     c_void, c_size, c_void]),
    "mdlstm_last_error": (c_char_p, []),
    "mdlstm_gradients_fused": (c_i32, [P_DESC]),
    "mdlstm_set_phase_events": (c_i32, [c_i32, P_VOIDP]),
    "mdlstm_blocks_workspace_bytes": (c_size, [c_i32, c_i32, c_i32]),
    "mdlstm_pack_blocks": (c_i32, [c_i32, P_VOIDP, c_i32, c_i32, c_i32, P_RECT, c_i32, c_i32, c_void, c_void, c_size,
                                   c_void]),
    "mdlstm_block_conv_forward": (c_i32, [c_i32, c_i32, c_i32, c_i32, c_i32, P_RECT, c_i32, c_i32, c_void, c_void,
                                          c_void, P_RECT, c_i32, c_i32, c_void, c_void, c_size, c_void]),
    "mdlstm_block_conv_backward": (c_i32, [c_i32, c_i32, c_i32, c_i32, c_i32, P_RECT, c_i32, c_i32, c_void, c_void,
                                           P_RECT, c_i32, c_i32, c_void, c_void, c_void, c_void, c_void, c_void, c_size,
                                           c_void]),
}

STATUS = {0: "OK", 1: "INVALID_ARG", 2: "TOO_WIDE", 3: "BAD_LAYOUT", 4: "WORKSPACE", 5: "UNSUPPORTED", 6: "DEVICE",
          7: "NUMERIC"}


class MdlstmError(RuntimeError):
    def __init__(self, status: int, msg: str):
        self.status = status
        self.code = STATUS.get(status, str(status))
        super().__init__(f"{self.code}: {msg}")


_lib = None


def lib() -> ctypes.CDLL:
    """Load libmdlstm.so once; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_1902_11208_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def check(status: int) -> None:
    if status != 0:
        raise MdlstmError(status, lib().mdlstm_last_error().decode(errors="replace"))
