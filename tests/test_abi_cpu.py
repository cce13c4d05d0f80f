"""The C-ABI library loads, exports every declared entry point, and rejects
bad arguments on the host before any HIP call (runs without a GPU)."""
import ctypes
import os
import re

import pytest

from conftest import ROOT


def _declared():
    src = open(os.path.join(ROOT, "include", "mdlstm.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mdlstm_\w+)\s*\(", src)))


def test_exports_every_declared_symbol(built_lib):
    from paper_1902_11208_amd import _lib

    names = _declared()
    assert "mdlstm_forward" in names and "mdlstm_backward" in names and "mdlstm_pack_layout" in names
    L = ctypes.CDLL(built_lib)
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(_lib.SIGNATURES), "binding signatures out of sync with the header"


FAKE = 0x100000  # never dereferenced: validation fails before any device access


def _lib():
    from paper_1902_11208_amd import _lib

    return _lib


def _call_pack(n, hs, ws, cw, ws_bytes=1 << 20):
    L = _lib()
    rects = (L.Rect * max(1, n))()
    ch = ctypes.c_int32(-1)
    arr_h = (ctypes.c_int32 * max(1, n))(*hs)
    arr_w = (ctypes.c_int32 * max(1, n))(*ws)
    st = L.lib().mdlstm_pack_layout(n, arr_h, arr_w, cw, rects, ctypes.byref(ch), None, 0, FAKE, ws_bytes, None)
    return st, ch.value


def test_pack_layout_errors(built_lib):
    assert _call_pack(-1, [], [], 10)[0] == 1
    assert _call_pack(2, [2, 2], [5, 11], 10)[0] == 2          # TOO_WIDE
    assert b"wide" in _lib().lib().mdlstm_last_error()
    assert _call_pack(1, [0], [3], 10)[0] == 1                 # INVALID_ARG
    assert _call_pack(1, [2], [3], 0)[0] == 1
    assert _call_pack(2, [2, 2], [5, 5], 10, ws_bytes=8)[0] == 4  # WORKSPACE
    st, ch = _call_pack(0, [], [], 10)
    assert st == 0 and ch == 0


def test_phase_events_argument_checks(built_lib):
    """n must be 0 or 8 and the array present; NULL entries are allowed (not
    recorded). Setting and clearing touch no device."""
    L = _lib().lib()
    assert L.mdlstm_set_phase_events(3, (ctypes.c_void_p * 8)()) == 1
    assert L.mdlstm_set_phase_events(8, None) == 1
    assert L.mdlstm_set_phase_events(8, (ctypes.c_void_p * 8)()) == 0
    assert L.mdlstm_set_phase_events(0, None) == 0


def _fwd(desc, ch, cw, rects, ws_bytes=None):
    L = _lib()
    arr = (L.Rect * max(1, len(rects)))(*[L.Rect(*r) for r in rects])
    need = L.lib().mdlstm_workspace_bytes(ctypes.byref(desc), ch, cw, len(rects))
    return L.lib().mdlstm_forward(ctypes.byref(desc), ch, cw, FAKE, FAKE, len(rects), arr, FAKE, FAKE, FAKE, FAKE,
                                  FAKE, need if ws_bytes is None else ws_bytes, None)


@pytest.mark.parametrize("c_in,hidden,dtype,code", [
    (16, 65, 0, 5), (16, 128, 0, 5), (16, 129, 1, 5), (260, 16, 0, 5), (16, 16, 7, 1), (0, 16, 0, 1),
    (16, 0, 0, 1), (16, 40, 0, 5),  # memory-state matrices not built above hidden 32 (set below)
])
def test_forward_rejects_descriptor(built_lib, c_in, hidden, dtype, code):
    d = _lib().LayerDesc(c_in, hidden, dtype, 1 if hidden == 40 else 0)
    assert _fwd(d, 10, 10, [(0, 0, 2, 2)]) == code


def test_padded_shapes_are_sized_and_checked(built_lib):
    """A hidden size or c_in between the built ones is padded inside the
    call: its workspace holds the padded copies on top of the built shape's,
    and its arguments are checked at the layer's own sizes before any HIP
    call."""
    L = _lib()
    ws = L.lib().mdlstm_workspace_bytes
    built = ws(ctypes.byref(L.LayerDesc(16, 16, 0)), 10, 10, 1)
    for c_in, hidden, dtype in ((16, 12, 0), (6, 16, 0), (1, 2, 0), (30, 50, 0), (12, 100, 1), (3, 32, 1)):
        assert ws(ctypes.byref(L.LayerDesc(c_in, hidden, dtype)), 10, 10, 1) > 0, (c_in, hidden, dtype)
    assert ws(ctypes.byref(L.LayerDesc(16, 12, 0)), 10, 10, 1) > built
    assert ws(ctypes.byref(L.LayerDesc(16, 10, 0, 1)), 10, 10, 1) > ws(ctypes.byref(L.LayerDesc(16, 16, 0, 1)), 10,
                                                                        10, 1)
    for d in (L.LayerDesc(16, 12, 0), L.LayerDesc(6, 16, 0), L.LayerDesc(5, 20, 1)):
        assert _fwd(d, 10, 10, [(0, 0, 3, 3), (2, 2, 3, 3)]) == 3      # overlap
        assert _fwd(d, 100, 10, [(0, 0, 65, 3)]) == 5                  # too tall
        need = ws(ctypes.byref(d), 10, 10, 1)
        assert _fwd(d, 10, 10, [(0, 0, 3, 3)], ws_bytes=need - 1) == 4  # the padded copies need room too
        assert _bwd(d, 10, 10, [(0, 0, 3, 3)], ws_bytes=need - 1) == 4
        for nm in ("dwx", "dy", "dx"):
            assert _bwd(d, 10, 10, [(0, 0, 3, 3)], **{nm: None}) == 1, nm
        assert _bwd(d, 10, 10, [(0, 0, 3, 3)], dx=FAKE + 4) == 1


def test_forward_rejects_layouts(built_lib):
    d = _lib().LayerDesc(16, 16, 0)
    assert _fwd(d, 10, 10, [(0, 0, 3, 3), (2, 2, 3, 3)]) == 3       # overlap
    assert _fwd(d, 10, 10, [(0, 8, 3, 3)]) == 3                    # leaves canvas
    assert _fwd(d, 10, 10, [(0, 0, 0, 3)]) == 3                    # empty rect
    assert _fwd(d, 100, 10, [(0, 0, 65, 3)]) == 5                  # too tall for the kernels
    assert _fwd(d, 10, 10, [(0, 0, 3, 3)], ws_bytes=16) == 4       # workspace
    # disjoint rectangles pass the layout checks and stop at the (too small) workspace
    assert _fwd(d, 10, 10, [(0, 0, 3, 3), (4, 0, 3, 3), (0, 4, 3, 6)], ws_bytes=16) == 4
    assert b"workspace" in _lib().lib().mdlstm_last_error()


def test_workspace_bytes_scale():
    L = _lib()
    d = L.LayerDesc(16, 16, 0)
    a = L.lib().mdlstm_workspace_bytes(ctypes.byref(d), 100, 100, 4)
    b = L.lib().mdlstm_workspace_bytes(ctypes.byref(d), 200, 100, 4)
    assert a > 100 * 100 * (20 * 16 + 4 * 16) * 4
    assert b > a
    assert L.lib().mdlstm_workspace_bytes(None, 1, 1, 1) == 0
    # an empty canvas still has a (small) workspace; unsupported shapes and
    # out-of-range canvases report 0 instead of a size
    assert L.lib().mdlstm_workspace_bytes(ctypes.byref(L.LayerDesc(64, 128, 1)), 0, 0, 0) > 0
    assert L.lib().mdlstm_workspace_bytes(ctypes.byref(L.LayerDesc(16, 65, 0)), 10, 10, 1) == 0
    assert L.lib().mdlstm_workspace_bytes(ctypes.byref(L.LayerDesc(16, 1 << 20, 0)), 10, 10, 1) == 0
    assert L.lib().mdlstm_workspace_bytes(ctypes.byref(d), 1 << 22, 10, 1) == 0
    assert L.lib().mdlstm_workspace_bytes(ctypes.byref(d), 10, 10, (1 << 24) + 1) == 0


@pytest.mark.parametrize("which", ["x", "wx", "workspace", "y"])
def test_forward_rejects_misaligned_pointers(built_lib, which):
    L = _lib()
    d = L.LayerDesc(16, 16, 0)
    rects = [(0, 0, 3, 3)]
    arr = (L.Rect * 1)(*[L.Rect(*r) for r in rects])
    need = L.lib().mdlstm_workspace_bytes(ctypes.byref(d), 10, 10, 1)
    ptr = {k: FAKE for k in ("x", "mask", "wx", "u", "b", "y", "workspace")}
    ptr[which] = FAKE + 4  # the alignment check fails before any device access
    st = L.lib().mdlstm_forward(ctypes.byref(d), 10, 10, ptr["x"], ptr["mask"], 1, arr, ptr["wx"], ptr["u"],
                                ptr["b"], ptr["y"], ptr["workspace"], need, None)
    assert st == 1
    assert b"aligned" in L.lib().mdlstm_last_error()


def _conv_fwd(n, hidden, og, bh, bw, in_rects, in_hw, out_rects, out_hw, ws_bytes=None, ptr=FAKE):
    L = _lib()
    ia = (L.Rect * max(1, n))(*[L.Rect(*r) for r in in_rects])
    oa = (L.Rect * max(1, n))(*[L.Rect(*r) for r in out_rects])
    need = L.lib().mdlstm_blocks_workspace_bytes(n, hidden, og)
    return L.lib().mdlstm_block_conv_forward(n, hidden, og, bh, bw, ia, in_hw[0], in_hw[1], ptr, FAKE, FAKE, oa,
                                             out_hw[0], out_hw[1], FAKE, FAKE,
                                             need if ws_bytes is None else ws_bytes, None)


def test_block_conv_rejects_bad_arguments(built_lib):
    ok_in, ok_out = [(0, 0, 4, 8)], [(0, 0, 2, 2)]
    assert _conv_fwd(1, 16, 8, 2, 4, ok_in, (4, 8), ok_out, (2, 2), ws_bytes=16) == 4      # workspace
    assert _conv_fwd(1, 16, 8, 3, 4, [(0, 0, 6, 8)], (6, 8), ok_out, (2, 2)) == 5         # block not built
    assert _conv_fwd(1, 16, 12, 2, 4, ok_in, (4, 8), ok_out, (2, 2)) == 5                 # og not built
    assert _conv_fwd(1, 128, 8, 2, 4, ok_in, (4, 8), ok_out, (2, 2)) == 5                 # hidden not built
    assert _conv_fwd(1, 16, 8, 2, 4, [(0, 0, 4, 4)], (4, 8), ok_out, (2, 2)) == 3         # not bh x bw blocks
    assert _conv_fwd(1, 16, 8, 2, 4, ok_in, (4, 8), [(1, 1, 2, 2)], (2, 2)) == 3          # leaves the canvas
    assert _conv_fwd(2, 16, 8, 2, 4, ok_in * 2, (4, 16), [(0, 0, 2, 2), (0, 1, 2, 2)], (2, 4)) == 3  # overlap
    assert _conv_fwd(1, 16, 8, 2, 4, ok_in, (4, 8), ok_out, (2, 2), ptr=FAKE + 4) == 1    # misaligned
    assert b"aligned" in _lib().lib().mdlstm_last_error()


def test_pack_blocks_rejects_bad_arguments(built_lib):
    L = _lib()
    r = (L.Rect * 1)(L.Rect(0, 0, 2, 2))
    imgs = (ctypes.c_void_p * 1)(FAKE)
    need = L.lib().mdlstm_blocks_workspace_bytes(1, 0, 0)
    f = L.lib().mdlstm_pack_blocks
    assert f(1, ctypes.cast(imgs, L.P_VOIDP), 1, 2, 4, r, 2, 2, FAKE, FAKE, 16, None) == 4     # workspace
    assert f(1, ctypes.cast(imgs, L.P_VOIDP), 1, 2, 4, r, 1, 2, FAKE, FAKE, need, None) == 3   # leaves canvas
    assert f(1, ctypes.cast(imgs, L.P_VOIDP), 0, 2, 4, r, 2, 2, FAKE, FAKE, need, None) == 1   # c < 1


def test_binding_rejects_wrong_tensors():
    """The Python binding checks shape, dtype and device before a pointer
    reaches the C ABI (which cannot know buffer sizes)."""
    import torch

    from paper_1902_11208_amd import api

    t = torch.zeros((4, 6, 8), dtype=torch.float32)
    with pytest.raises(ValueError, match="shape"):
        api.check_tensor(t, "x", (4, 6, 16), torch.float32)
    with pytest.raises(ValueError, match="dtype"):
        api.check_tensor(t.to(torch.bfloat16), "x", (4, 6, 8), torch.float32)
    with pytest.raises(ValueError, match="device tensor"):
        api.check_tensor(t, "x", (4, 6, 8), torch.float32)
    with pytest.raises(ValueError, match="torch.Tensor"):
        api.check_tensor(t.numpy(), "x", (4, 6, 8), torch.float32)
    # a layer built from host tensors is refused before any allocation
    H, C = 4, 8
    with pytest.raises(ValueError):
        api.MDLSTMLayer(torch.zeros(4, 5 * H, C), torch.zeros(4, 5 * H, 2 * H), torch.zeros(4, 5 * H), 2, 3,
                        [[0, 0, 2, 3]], torch.zeros(2, 3, dtype=torch.uint8))
    with pytest.raises(ValueError, match="shape"):
        api.MDLSTMLayer(torch.zeros(4, 5 * H, C), torch.zeros(4, 5 * H, 3 * H), torch.zeros(4, 5 * H), 2, 3,
                        [[0, 0, 2, 3]], torch.zeros(2, 3, dtype=torch.uint8))


def _bwd(desc, ch, cw, rects, ws_bytes=None, **over):
    L = _lib()
    arr = (L.Rect * max(1, len(rects)))(*[L.Rect(*r) for r in rects])
    need = L.lib().mdlstm_workspace_bytes(ctypes.byref(desc), ch, cw, len(rects))
    p = {k: FAKE for k in ("x", "mask", "wx", "u", "b", "y", "dy", "dx", "dwx", "du", "db", "workspace")}
    p.update(over)
    return L.lib().mdlstm_backward(ctypes.byref(desc), ch, cw, p["x"], p["mask"], len(rects), arr, p["wx"], p["u"],
                                   p["b"], p["y"], p["dy"], p["dx"], p["dwx"], p["du"], p["db"], p["workspace"],
                                   need if ws_bytes is None else ws_bytes, None)


def test_backward_rejects_bad_arguments(built_lib):
    """mdlstm_backward validates like mdlstm_forward, plus its gradient buffers,
    before any HIP call."""
    L = _lib()
    ok = L.LayerDesc(16, 16, 0)
    assert _bwd(L.LayerDesc(16, 65, 0), 10, 10, [(0, 0, 2, 2)]) == 5          # hidden above the largest built
    assert _bwd(L.LayerDesc(16, 16, 9), 10, 10, [(0, 0, 2, 2)]) == 1          # dtype
    assert _bwd(ok, 10, 10, [(0, 0, 3, 3), (2, 2, 3, 3)]) == 3                # overlap
    assert _bwd(ok, 10, 10, [(0, 8, 3, 3)]) == 3                              # leaves the canvas
    assert _bwd(ok, 100, 10, [(0, 0, 65, 3)]) == 5                            # too tall
    assert _bwd(ok, 10, 10, [(0, 0, 3, 3)], ws_bytes=16) == 4                 # workspace
    assert _bwd(ok, 10, 10, [(0, 0, 3, 3)], workspace=None) == 1              # no workspace
    for nm in ("dwx", "du", "db", "y", "dy", "dx"):
        assert _bwd(ok, 10, 10, [(0, 0, 3, 3)], **{nm: None}) == 1, nm       # NULL output or input
    for nm in ("dy", "dx", "dwx", "y"):
        assert _bwd(ok, 10, 10, [(0, 0, 3, 3)], **{nm: FAKE + 4}) == 1, nm   # misaligned
        assert b"aligned" in L.lib().mdlstm_last_error()


def test_pack_layout_noalloc_errors(built_lib):
    """The allocation-free placement validates like mdlstm_pack_layout and
    refuses more than MDLSTM_NOALLOC_MAX_N examples, all before any HIP call."""
    L = _lib()
    f = L.lib().mdlstm_pack_layout_noalloc

    def call(n, hs, ws, cw):
        rects = (L.Rect * max(1, n))()
        ch = ctypes.c_int32(-1)
        st = f(n, (ctypes.c_int32 * max(1, n))(*hs), (ctypes.c_int32 * max(1, n))(*ws), cw, rects,
               ctypes.byref(ch), None, 0, None)
        return st, ch.value

    assert call(-1, [], [], 10)[0] == 1
    assert call(2, [2, 2], [5, 11], 10)[0] == 2                    # TOO_WIDE
    assert call(1, [0], [3], 10)[0] == 1                           # INVALID_ARG
    assert call(4097, [1] * 4097, [1] * 4097, 10)[0] == 5          # above the static scratch
    assert b"4096" in L.lib().mdlstm_last_error()
    assert call(0, [], [], 10) == (0, 0)


def test_gradients_fused_query(built_lib):
    L = _lib()
    f = L.lib().mdlstm_gradients_fused
    assert f(ctypes.byref(L.LayerDesc(32, 32, 0))) == 1    # lines: one kernel
    assert f(ctypes.byref(L.LayerDesc(64, 128, 1))) == 0   # bf16 H 128: two kernels
    assert f(ctypes.byref(L.LayerDesc(16, 12, 0))) == f(ctypes.byref(L.LayerDesc(16, 16, 0)))  # padded to H 16
    assert f(ctypes.byref(L.LayerDesc(16, 65, 0))) == -1   # above the largest built
    assert f(None) == -1


def test_head_calls_reject_bad_arguments(built_lib):
    """The output-layer and CTC calls validate sizes, rectangles and labels on
    the host before any HIP call."""
    L = _lib()
    lib = L.lib()
    ok = L.HeadDesc(8, 6)
    rects = (L.Rect * 2)(L.Rect(0, 0, 3, 5), L.Rect(0, 6, 2, 4))
    lens = (ctypes.c_int32 * 2)(2, 1)
    need = lib.mdlstm_head_workspace_bytes(ctypes.byref(ok), 2, rects, lens)
    assert need > lib.mdlstm_head_workspace_bytes(ctypes.byref(ok), 2, rects, None) > 0

    def fwd(desc, ch=4, cw=12, r=rects, ws=need):
        return lib.mdlstm_head_forward(ctypes.byref(desc), ch, cw, FAKE, 2, r, FAKE, FAKE, FAKE, FAKE, ws, None)

    assert fwd(L.HeadDesc(6, 6)) == 5            # hidden not a multiple of 4
    assert fwd(L.HeadDesc(8, 300)) == 5          # too many classes
    assert fwd(ok, ch=2) == 3                    # a rectangle leaves the canvas
    assert fwd(ok, r=(L.Rect * 2)(L.Rect(0, 0, 3, 5), L.Rect(0, 4, 2, 4))) == 3  # overlap
    assert fwd(ok, ws=16) == 4                   # workspace

    def ctc(lens_, labs, ws=need):
        ll = (ctypes.c_int32 * 2)(*lens_)
        lb = (ctypes.c_int32 * max(1, len(labs)))(*labs)
        return lib.mdlstm_ctc_loss(ctypes.byref(ok), 2, rects, ll, lb, FAKE, FAKE, FAKE, FAKE, ws, None)

    assert ctc([2, 1], [1, 0, 3]) == 1           # a label is the blank
    assert ctc([2, 1], [1, 6, 3]) == 1           # a label past the classes
    assert ctc([5, 1], [2, 2, 2, 1, 1, 3]) == 1  # 5 labels + 3 repeats > 5 frames
    assert b"aligned" in lib.mdlstm_last_error()
    assert ctc([1000, 1], [1] * 1001) == 5       # above the labels per example
    assert ctc([2, 1], [1, 2, 3], ws=need - 256) == 4

    def bwd(ws=need, dw=FAKE):
        return lib.mdlstm_head_backward(ctypes.byref(ok), 4, 12, 2, rects, FAKE, FAKE, FAKE, dw, FAKE, FAKE, ws, None)

    assert bwd(dw=None) == 1
    assert bwd(ws=16) == 4
