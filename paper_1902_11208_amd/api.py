"""Python binding of the C ABI: argument marshalling only.

torch provides device memory and the current stream; every step of the
computation runs in libmdlstm.so's HIP kernels.
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from ._lib import LayerDesc, Rect, P_VOIDP, check, lib

F32, BF16 = 0, 1
TORCH_DTYPE = {F32: torch.float32, BF16: torch.bfloat16}


def dtype_code(t: torch.dtype) -> int:
    if t == torch.float32:
        return F32
    if t == torch.bfloat16:
        return BF16
    raise TypeError(f"storage dtype {t} is not float32 or bfloat16")


def _stream(stream=None) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _rect_array(rects) -> ctypes.Array:
    r = np.ascontiguousarray(np.asarray(rects, dtype=np.int32).reshape(-1, 4))
    arr = (Rect * max(1, r.shape[0]))()
    ctypes.memmove(arr, r.ctypes.data, r.nbytes)
    return arr


def _rects_from(arr, n) -> np.ndarray:
    out = np.zeros((n, 4), np.int32)
    if n:
        ctypes.memmove(out.ctypes.data, arr, n * 16)
    return out


def _i32_array(v) -> ctypes.Array:
    a = np.ascontiguousarray(np.asarray(v, dtype=np.int32).reshape(-1))
    arr = (ctypes.c_int32 * max(1, a.size))()
    ctypes.memmove(arr, a.ctypes.data, a.nbytes)
    return arr


def _check_dev(t: torch.Tensor, name: str):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def check_tensor(t, name: str, shape, dtype: torch.dtype, device=None):
    """Reject a tensor whose shape, dtype or device differs from what the C ABI
    will assume: the library sees only pointers, so a wrong buffer would be
    read or written past its end by the kernels."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch.Tensor")
    if tuple(t.shape) != tuple(int(v) for v in shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(int(v) for v in shape)}")
    if t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    _check_dev(t, name)
    if device is not None and t.device != torch.device(device):
        raise ValueError(f"{name} is on {t.device}, expected {device}")


# ---------------------------------------------------------------------------
# Packing
# ---------------------------------------------------------------------------
def pack_workspace_bytes(n: int) -> int:
    return int(lib().mdlstm_pack_workspace_bytes(int(n)))


def pack_layout(heights, widths, canvas_w: int, device="cuda", stream=None):
    """Example packing (placement kernel + mask kernel).
    Returns (rects int32 [n, 4] by original index, canvas_h, mask uint8 [canvas_h, canvas_w])."""
    hs, ws = _i32_array(heights), _i32_array(widths)
    n = len(np.asarray(heights).reshape(-1))
    work = torch.empty(pack_workspace_bytes(n), dtype=torch.uint8, device=device)
    rects = (Rect * max(1, n))()
    ch = ctypes.c_int32(0)
    st = _stream(stream)
    # One call when the sizes are valid: the mask is allocated for the tallest
    # possible canvas (every example on its own row, plus separators) and cut
    # to the placed height. Otherwise the library reports what is wrong.
    h64 = np.asarray(heights, np.int64).reshape(-1)
    w64 = np.asarray(widths, np.int64).reshape(-1)
    max_h = int(np.sum(h64 + 1)) if n else 0
    if n and h64.min() >= 1 and w64.min() >= 1 and w64.max() <= int(canvas_w) and max_h <= 2 ** 21 - 1:
        full = torch.empty((max_h, int(canvas_w)), dtype=torch.uint8, device=device)
        check(lib().mdlstm_pack_layout(n, hs, ws, int(canvas_w), rects, ctypes.byref(ch), _ptr(full), full.numel(),
                                       _ptr(work), work.numel(), st))
        mask = full[:ch.value]
    else:
        check(lib().mdlstm_pack_layout(n, hs, ws, int(canvas_w), rects, ctypes.byref(ch), None, 0, _ptr(work),
                                       work.numel(), st))
        mask = torch.empty((ch.value, int(canvas_w)), dtype=torch.uint8, device=device)
    torch.cuda.current_stream().synchronize() if stream is None else stream.synchronize()
    return _rects_from(rects, n), ch.value, mask


def pack_layout_noalloc(heights, widths, canvas_w: int, mask=None, stream=None):
    """Placement and mask through the allocation-free entry point: the caller
    owns the mask buffer (uint8, at least canvas_h x canvas_w cells, row-major
    from its start; None computes the placement only) and the library uses its
    static device scratch. Returns (rects int32 [n, 4], canvas_h)."""
    n = len(np.asarray(heights).reshape(-1))
    hs, ws = _i32_array(heights), _i32_array(widths)
    if mask is not None:
        if mask.dtype != torch.uint8:
            raise ValueError(f"mask has dtype {mask.dtype}, expected torch.uint8")
        _check_dev(mask, "mask")
    rects = (Rect * max(1, n))()
    ch = ctypes.c_int32(0)
    s = stream if stream is not None else torch.cuda.current_stream()
    check(lib().mdlstm_pack_layout_noalloc(n, hs, ws, int(canvas_w), rects, ctypes.byref(ch), _ptr(mask),
                                           0 if mask is None else mask.numel(), _stream(s)))
    return _rects_from(rects, n), ch.value


def pad_layout(heights, widths, device="cuda", stream=None):
    """Last-minute batch padding layout. Returns (tiles, place, canvas_h, canvas_w, mask)."""
    n = len(np.asarray(heights).reshape(-1))
    hs, ws = _i32_array(heights), _i32_array(widths)
    tiles, place = (Rect * max(1, n))(), (Rect * max(1, n))()
    ch, cw = ctypes.c_int32(0), ctypes.c_int32(0)
    check(lib().mdlstm_pad_layout(n, hs, ws, tiles, place, ctypes.byref(ch), ctypes.byref(cw), None, 0, None, 0, 0))
    mask = torch.empty((ch.value, cw.value), dtype=torch.uint8, device=device)
    work = torch.empty(pack_workspace_bytes(n), dtype=torch.uint8, device=device)
    s = stream if stream is not None else torch.cuda.current_stream()
    check(lib().mdlstm_pad_layout(n, hs, ws, tiles, place, ctypes.byref(ch), ctypes.byref(cw), _ptr(mask),
                                  mask.numel(), _ptr(work), work.numel(), _stream(s)))
    s.synchronize()
    return _rects_from(tiles, n), _rects_from(place, n), ch.value, cw.value, mask


def pack_data(examples, rects, canvas_h: int, canvas_w: int, stream=None, out=None):
    """Scatter HWC example tensors into a zeroed [canvas_h, canvas_w, c] canvas."""
    n = len(examples)
    if n == 0:
        raise ValueError("pack_data needs at least one example to know channels and dtype")
    c = examples[0].shape[2]
    dt = examples[0].dtype
    dev = examples[0].device
    r = np.asarray(rects, np.int32).reshape(-1, 4)
    for k, e in enumerate(examples):
        _check_dev(e, f"example {k}")
        if e.dtype != dt or e.shape != (r[k, 2], r[k, 3], c):
            raise ValueError(f"example {k} has shape {tuple(e.shape)}, rect says {tuple(r[k, 2:])}x{c}")
    if out is not None:
        check_tensor(out, "out", (canvas_h, canvas_w, c), dt, dev)
    canvas = out if out is not None else torch.empty((canvas_h, canvas_w, c), dtype=dt, device=dev)
    ptrs = (ctypes.c_void_p * n)(*[e.data_ptr() for e in examples])
    work = torch.empty(pack_workspace_bytes(n), dtype=torch.uint8, device=dev)
    s = stream if stream is not None else torch.cuda.current_stream()
    check(lib().mdlstm_pack_data(n, ctypes.cast(ptrs, P_VOIDP), _rect_array(r), canvas_h, canvas_w, c,
                                 dtype_code(dt), _ptr(canvas), _ptr(work), work.numel(), _stream(s)))
    s.synchronize()  # the workspace (pointer table) is released on return
    return canvas


def unpack_data(canvas: torch.Tensor, rects, stream=None):
    """Gather per-example HWC tensors out of a canvas."""
    _check_dev(canvas, "canvas")
    r = np.asarray(rects, np.int32).reshape(-1, 4)
    n = r.shape[0]
    ch, cw, c = canvas.shape
    outs = [torch.empty((int(h), int(w), c), dtype=canvas.dtype, device=canvas.device) for _, _, h, w in r]
    if n == 0:
        return outs
    ptrs = (ctypes.c_void_p * n)(*[o.data_ptr() for o in outs])
    work = torch.empty(pack_workspace_bytes(n), dtype=torch.uint8, device=canvas.device)
    s = stream if stream is not None else torch.cuda.current_stream()
    check(lib().mdlstm_unpack_data(n, ctypes.cast(ptrs, P_VOIDP), _rect_array(r), ch, cw, c, dtype_code(canvas.dtype),
                                   _ptr(canvas), _ptr(work), work.numel(), _stream(s)))
    s.synchronize()
    return outs


# ---------------------------------------------------------------------------
# Layer
# ---------------------------------------------------------------------------
def layer_desc(c_in: int, hidden: int, dtype: int, memory_states: int = 0) -> LayerDesc:
    return LayerDesc(int(c_in), int(hidden), int(dtype), int(memory_states))


def workspace_bytes(c_in: int, hidden: int, dtype: int, canvas_h: int, canvas_w: int, n_rects: int) -> int:
    d = layer_desc(c_in, hidden, dtype)
    return int(lib().mdlstm_workspace_bytes(ctypes.byref(d), canvas_h, canvas_w, n_rects))


def gradients_fused(c_in: int, hidden: int, dtype: int) -> bool:
    """Whether one kernel computes both the input and the weight gradients."""
    d = layer_desc(c_in, hidden, dtype)
    r = int(lib().mdlstm_gradients_fused(ctypes.byref(d)))
    if r < 0:
        raise ValueError(f"layer c_in={c_in} hidden={hidden} dtype={dtype} is not supported")
    return bool(r)


class Prepared:
    """Host-side argument bundle for one canvas layout, reused across calls."""

    def __init__(self, c_in: int, hidden: int, dtype: int, canvas_h: int, canvas_w: int, rects, memory_states=0):
        self.desc = layer_desc(c_in, hidden, dtype, memory_states)
        self.canvas_h, self.canvas_w = int(canvas_h), int(canvas_w)
        self.rects_np = np.asarray(rects, np.int32).reshape(-1, 4)
        self.n_rects = int(self.rects_np.shape[0])
        self.rects = _rect_array(self.rects_np)
        self.ws_bytes = int(lib().mdlstm_workspace_bytes(ctypes.byref(self.desc), self.canvas_h, self.canvas_w,
                                                         self.n_rects))


def forward(prep: Prepared, x, mask, wx, u, b, y, workspace, stream=None):
    """Enqueue the forward pass; y and workspace are caller-allocated."""
    check(lib().mdlstm_forward(ctypes.byref(prep.desc), prep.canvas_h, prep.canvas_w, _ptr(x), _ptr(mask),
                               prep.n_rects, prep.rects, _ptr(wx), _ptr(u), _ptr(b), _ptr(y), _ptr(workspace),
                               prep.ws_bytes if workspace is not None else 0, _stream(stream)))


def forward_stepwise(prep: Prepared, x, mask, wx, u, b, y, workspace, stream=None):
    """Forward pass with one wavefront launch per diagonal, replayed from a HIP graph (comparison variant)."""
    check(lib().mdlstm_forward_stepwise(ctypes.byref(prep.desc), prep.canvas_h, prep.canvas_w, _ptr(x), _ptr(mask),
                                        prep.n_rects, prep.rects, _ptr(wx), _ptr(u), _ptr(b), _ptr(y),
                                        _ptr(workspace), prep.ws_bytes if workspace is not None else 0,
                                        _stream(stream)))


def backward(prep: Prepared, x, mask, wx, u, b, y, dy, dx, dwx, du, db, workspace, stream=None):
    """Enqueue the backward pass; all outputs caller-allocated, overwritten."""
    check(lib().mdlstm_backward(ctypes.byref(prep.desc), prep.canvas_h, prep.canvas_w, _ptr(x), _ptr(mask),
                                prep.n_rects, prep.rects, _ptr(wx), _ptr(u), _ptr(b), _ptr(y), _ptr(dy), _ptr(dx),
                                _ptr(dwx), _ptr(du), _ptr(db), _ptr(workspace),
                                prep.ws_bytes if workspace is not None else 0, _stream(stream)))


class MDLSTMLayer:
    """Four-direction MDLSTM layer over a canvas with a fixed layout.

    Owns the workspace and the output/gradient buffers for that layout.
    v [4, 3H, 2H] (optional, fp32): memory-state matrices feeding the input and
    forget gates; the backward then also fills self.dv.
    """

    def __init__(self, wx: torch.Tensor, u: torch.Tensor, b: torch.Tensor, canvas_h: int, canvas_w: int, rects,
                 mask: torch.Tensor, v: torch.Tensor = None):
        if wx.dim() != 3 or u.dim() != 3:
            raise ValueError("wx must be [4, 5H, c_in] and u [4, 5H, 2H]")
        self.dtype = dtype_code(wx.dtype)
        self.hidden = int(u.shape[2]) // 2
        self.c_in = int(wx.shape[2])
        H, td, dev = self.hidden, wx.dtype, wx.device
        check_tensor(wx, "wx", (4, 5 * H, self.c_in), td)
        check_tensor(u, "u", (4, 5 * H, 2 * H), td, dev)
        check_tensor(b, "b", (4, 5 * H), td, dev)
        check_tensor(mask, "mask", (canvas_h, canvas_w), torch.uint8, dev)
        self.memory = v is not None
        if self.memory:
            check_tensor(v, "v", (4, 3 * H, 2 * H), td, dev)
            u = torch.cat([u.reshape(-1), v.reshape(-1)])  # U then V, one buffer
        self.wx, self.u, self.b, self.mask = wx, u, b, mask
        self.prep = Prepared(self.c_in, self.hidden, self.dtype, canvas_h, canvas_w, rects, int(self.memory))
        self.workspace = torch.empty(max(1, self.prep.ws_bytes), dtype=torch.uint8, device=dev)
        self.y = torch.empty((canvas_h, canvas_w, 4 * H), dtype=td, device=dev)
        self.dx = torch.empty((canvas_h, canvas_w, self.c_in), dtype=td, device=dev)
        self.dwx = torch.empty((4, 5 * H, self.c_in), dtype=torch.float32, device=dev)
        nu, nv = 4 * 5 * H * 2 * H, (4 * 3 * H * 2 * H if self.memory else 0)
        self._dgrad = torch.empty(nu + nv, dtype=torch.float32, device=dev)
        self.du = self._dgrad[:nu].view(4, 5 * H, 2 * H)
        self.dv = self._dgrad[nu:].view(4, 3 * H, 2 * H) if self.memory else None
        self.db = torch.empty((4, 5 * H), dtype=torch.float32, device=dev)

    def _check_x(self, x):
        check_tensor(x, "x", (self.prep.canvas_h, self.prep.canvas_w, self.c_in), self.wx.dtype, self.wx.device)

    def forward(self, x: torch.Tensor, stream=None) -> torch.Tensor:
        self._check_x(x)
        self.x = x
        forward(self.prep, x, self.mask, self.wx, self.u, self.b, self.y, self.workspace, stream)
        return self.y

    def forward_stepwise(self, x: torch.Tensor, stream=None) -> torch.Tensor:
        self._check_x(x)
        self.x = x
        forward_stepwise(self.prep, x, self.mask, self.wx, self.u, self.b, self.y, self.workspace, stream)
        return self.y

    def backward(self, dy: torch.Tensor, stream=None):
        if getattr(self, "x", None) is None:
            raise ValueError("backward needs a forward call on this layer first")
        check_tensor(dy, "dy", (self.prep.canvas_h, self.prep.canvas_w, 4 * self.hidden), self.wx.dtype,
                     self.wx.device)
        backward(self.prep, self.x, self.mask, self.wx, self.u, self.b, self.y, dy, self.dx, self.dwx, self._dgrad,
                 self.db, self.workspace, stream)
        if self.memory:
            return self.dx, self.dwx, self.du, self.db, self.dv
        return self.dx, self.dwx, self.du, self.db


# ---------------------------------------------------------------------------
# Stack glue (block reshape, grouped block convolution)
# ---------------------------------------------------------------------------
def blocks_workspace_bytes(n: int, hidden: int = 0, og: int = 0) -> int:
    return int(lib().mdlstm_blocks_workspace_bytes(int(n), int(hidden), int(og)))


def pack_blocks(images, rects, canvas_h: int, canvas_w: int, bh: int, bw: int, out=None, stream=None):
    """Block-reshape fp32 HWC images into their rectangles of a [canvas_h, canvas_w, bh*bw*c] canvas."""
    n = len(images)
    r = np.asarray(rects, np.int32).reshape(-1, 4)
    c = int(images[0].shape[2]) if n else 1
    dev = images[0].device if n else torch.device("cuda")
    for k, im in enumerate(images):
        _check_dev(im, f"image {k}")
        if im.dtype != torch.float32 or tuple(im.shape) != (r[k, 2] * bh, r[k, 3] * bw, c):
            raise ValueError(f"image {k} has shape {tuple(im.shape)}, rect says {r[k, 2] * bh}x{r[k, 3] * bw}x{c}")
    if out is not None:
        check_tensor(out, "out", (canvas_h, canvas_w, bh * bw * c), torch.float32, dev)
    canvas = out if out is not None else torch.empty((canvas_h, canvas_w, bh * bw * c), dtype=torch.float32,
                                                     device=dev)
    ptrs = (ctypes.c_void_p * max(1, n))(*[im.data_ptr() for im in images])
    work = torch.empty(blocks_workspace_bytes(n), dtype=torch.uint8, device=dev)
    s = stream if stream is not None else torch.cuda.current_stream()
    check(lib().mdlstm_pack_blocks(n, ctypes.cast(ptrs, P_VOIDP), c, bh, bw, _rect_array(r), canvas_h, canvas_w,
                                   _ptr(canvas), _ptr(work), work.numel(), _stream(s)))
    s.synchronize()  # the pointer table in the workspace is released on return
    return canvas


class BlockConv:
    """Grouped block convolution + tanh from one packed canvas to the next."""

    def __init__(self, w: torch.Tensor, b: torch.Tensor, in_rects, in_hw, out_rects, out_hw, bh: int = 2,
                 bw: int = 4):
        if w.dim() != 3 or int(w.shape[2]) % (bh * bw):
            raise ValueError("w must be [4, og, bh*bw*hidden]")
        self.og = int(w.shape[1])
        self.hidden = int(w.shape[2]) // (bh * bw)
        check_tensor(w, "w", (4, self.og, bh * bw * self.hidden), torch.float32)
        check_tensor(b, "b", (4, self.og), torch.float32, w.device)
        self.w, self.b = w, b
        self.bh, self.bw = int(bh), int(bw)
        self.in_np = np.asarray(in_rects, np.int32).reshape(-1, 4)
        self.out_np = np.asarray(out_rects, np.int32).reshape(-1, 4)
        self.n = int(self.in_np.shape[0])
        self.in_rects, self.out_rects = _rect_array(self.in_np), _rect_array(self.out_np)
        self.in_h, self.in_w = (int(v) for v in in_hw)
        self.out_h, self.out_w = (int(v) for v in out_hw)
        dev = w.device
        self.work = torch.empty(blocks_workspace_bytes(self.n, self.hidden, self.og), dtype=torch.uint8, device=dev)
        self.out = torch.empty((self.out_h, self.out_w, 4 * self.og), dtype=torch.float32, device=dev)
        self.dy = torch.empty((self.in_h, self.in_w, 4 * self.hidden), dtype=torch.float32, device=dev)
        self.dw = torch.empty_like(w)
        self.db = torch.empty_like(b)

    def forward(self, y: torch.Tensor, stream=None) -> torch.Tensor:
        check_tensor(y, "y", (self.in_h, self.in_w, 4 * self.hidden), torch.float32, self.w.device)
        self.y = y
        check(lib().mdlstm_block_conv_forward(self.n, self.hidden, self.og, self.bh, self.bw, self.in_rects, self.in_h,
                                              self.in_w, _ptr(y), _ptr(self.w), _ptr(self.b), self.out_rects,
                                              self.out_h, self.out_w, _ptr(self.out), _ptr(self.work),
                                              self.work.numel(), _stream(stream)))
        return self.out

    def backward(self, dout: torch.Tensor, stream=None):
        if getattr(self, "y", None) is None:
            raise ValueError("backward needs a forward call on this convolution first")
        check_tensor(dout, "dout", (self.out_h, self.out_w, 4 * self.og), torch.float32, self.w.device)
        check(lib().mdlstm_block_conv_backward(self.n, self.hidden, self.og, self.bh, self.bw, self.in_rects,
                                               self.in_h, self.in_w, _ptr(self.y), _ptr(self.w), self.out_rects,
                                               self.out_h, self.out_w, _ptr(self.out), _ptr(dout), _ptr(self.dy),
                                               _ptr(self.dw), _ptr(self.db), _ptr(self.work), self.work.numel(),
                                               _stream(stream)))
        return self.dy, self.dw, self.db


# ---------------------------------------------------------------------------
# Output layer shared by the directions, row collapse, CTC loss
# ---------------------------------------------------------------------------
class Head:
    """The shared fully-connected output layer over a packed canvas (frames =
    canvas columns of each example, rows and directions summed) and the CTC
    loss of every example. fp32; the workspace is sized for `labels`."""

    def __init__(self, w: torch.Tensor, b: torch.Tensor, rects, canvas_hw, labels):
        from ._lib import HeadDesc

        if w.dim() != 2:
            raise ValueError("w must be [classes, hidden]")
        self.classes, self.hidden = int(w.shape[0]), int(w.shape[1])
        check_tensor(w, "w", (self.classes, self.hidden), torch.float32)
        check_tensor(b, "b", (self.classes,), torch.float32, w.device)
        self.w, self.b = w, b
        self.desc = HeadDesc(self.hidden, self.classes)
        self.rects_np = np.asarray(rects, np.int32).reshape(-1, 4)
        self.n = int(self.rects_np.shape[0])
        self.rects = _rect_array(self.rects_np)
        self.canvas_h, self.canvas_w = (int(v) for v in canvas_hw)
        labels = [np.asarray(l, np.int32).reshape(-1) for l in labels]
        if len(labels) != self.n:
            raise ValueError(f"{len(labels)} label sequences for {self.n} examples")
        self.label_lens = _i32_array([l.size for l in labels])
        self.labels = _i32_array(np.concatenate(labels) if labels else np.zeros(0, np.int32))
        self.frames = int(self.rects_np[:, 3].sum()) if self.n else 0
        nbytes = int(lib().mdlstm_head_workspace_bytes(ctypes.byref(self.desc), self.n, self.rects, self.label_lens))
        dev = w.device
        self.workspace = torch.empty(max(1, nbytes), dtype=torch.uint8, device=dev)
        self.logits = torch.empty((max(1, self.frames), self.classes), dtype=torch.float32, device=dev)
        self.dlogits = torch.empty_like(self.logits)
        self.losses = torch.empty(max(1, self.n), dtype=torch.float32, device=dev)
        self.dy = torch.empty((self.canvas_h, self.canvas_w, 4 * self.hidden), dtype=torch.float32, device=dev)
        self.dw = torch.empty_like(w)
        self.db = torch.empty_like(b)

    def forward(self, y: torch.Tensor, stream=None) -> torch.Tensor:
        """Logits [frames, classes] of the layer's output canvas y."""
        check_tensor(y, "y", (self.canvas_h, self.canvas_w, 4 * self.hidden), torch.float32, self.w.device)
        check(lib().mdlstm_head_forward(ctypes.byref(self.desc), self.canvas_h, self.canvas_w, _ptr(y), self.n,
                                        self.rects, _ptr(self.w), _ptr(self.b), _ptr(self.logits),
                                        _ptr(self.workspace), self.workspace.numel(), _stream(stream)))
        return self.logits[:self.frames]

    def ctc(self, logits=None, stream=None):
        """(losses [n], dlogits [frames, classes]) of the CTC loss."""
        z = self.logits if logits is None else logits
        check_tensor(z, "logits", tuple(self.logits.shape), torch.float32, self.w.device)
        check(lib().mdlstm_ctc_loss(ctypes.byref(self.desc), self.n, self.rects, self.label_lens, self.labels,
                                    _ptr(z), _ptr(self.losses), _ptr(self.dlogits), _ptr(self.workspace),
                                    self.workspace.numel(), _stream(stream)))
        return self.losses[:self.n], self.dlogits[:self.frames]

    def backward(self, dlogits=None, stream=None):
        """(dy canvas, dw, db) from the gradient of the logits (default: the CTC gradient)."""
        g = self.dlogits if dlogits is None else dlogits
        check_tensor(g, "dlogits", tuple(self.dlogits.shape), torch.float32, self.w.device)
        check(lib().mdlstm_head_backward(ctypes.byref(self.desc), self.canvas_h, self.canvas_w, self.n, self.rects,
                                         _ptr(self.w), _ptr(g), _ptr(self.dy), _ptr(self.dw), _ptr(self.db),
                                         _ptr(self.workspace), self.workspace.numel(), _stream(stream)))
        return self.dy, self.dw, self.db
