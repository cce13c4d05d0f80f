"""GPU parity of layers whose hidden size or input width lies between the
built kernel shapes (the paper's network uses 2, 10 and 50 hidden units and
a single-channel input, Section IV): the library pads them with zero
weights to the next built shape, which leaves every result unchanged.

Checked through the C ABI against the float64 oracle at the layer's own
sizes (Y and dX per example, the summed weight gradients; 1e-5 fp32, 2e-2
bf16 in the L2 and max norms), and bit for bit against the built shape
called on explicitly zero-padded weights and inputs."""
import sys

import numpy as np
import pytest

from conftest import rel_err, rel_max

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

RTOL = {"f32": 1e-5, "bf16": 2e-2}


@pytest.fixture(scope="module", autouse=True)
def _need_gpu(built_lib):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _cmp(gpu, ref, dtype, label, memory=False):
    tol = RTOL[dtype]
    worst = {}
    for nm in ("Y", "dX"):
        for k, (g, r) in enumerate(zip(gpu[nm], ref[nm])):
            e, m = rel_err(g, r), rel_max(g, r)
            assert e <= tol and m <= tol, (label, nm, k, e, m)
            worst[nm] = max(worst.get(nm, (0, 0)), (e, m))
    for nm in ("dWx", "dU", "db") + (("dV",) if memory else ()):
        e, m = rel_err(gpu[nm], ref[nm]), rel_max(gpu[nm], ref[nm])
        assert e <= tol and m <= tol, (label, nm, e, m)
        worst[nm] = (e, m)
    _say(f"{label}: worst (L2, max) " + ", ".join(f"{k} ({v[0]:.1e}, {v[1]:.1e})" for k, v in worst.items()))


CASES = [
    # name, heights, widths, canvas_w, c_in, hidden, dtype
    ("H2_C1", [9, 4, 1, 13], [20, 7, 3, 1], 32, 1, 2, "f32"),
    ("H10_C6", [16, 5, 30], [25, 40, 3], 64, 6, 10, "f32"),
    ("H20_C30", [12, 33, 2], [40, 9, 17], 64, 30, 20, "f32"),
    ("H50_C40", [20, 7], [33, 50], 64, 40, 50, "f32"),
    ("H12_C16", [17, 3], [20, 9], 32, 16, 12, "f32"),
    ("H3_C5", [6, 2, 11], [9, 14, 3], 24, 5, 3, "f32"),
    ("bf16_H100_C12", [20, 9], [30, 41], 80, 12, 100, "bf16"),
    ("bf16_H40_C3", [16, 5, 1], [22, 30, 2], 64, 3, 40, "bf16"),
    # H 24 -> 32 with C 5 -> 8: the tiled gradient path with fewer gate rows
    # (160) than a weight-gradient block holds (320)
    ("bf16_H24_C5", [20, 9, 33], [37, 16, 8], 64, 5, 24, "bf16"),
    # wide inputs: the input-gradient kernel with more than four channel tiles
    # (two or four 64-row groups of WxT, stages of 128 and 64 gate rows) and
    # weight-gradient blocks over three and four column blocks
    ("bf16_H64_C96", [17, 6], [23, 40], 64, 96, 64, "bf16"),
    ("bf16_H30_C200", [9, 14, 3], [26, 11, 30], 64, 200, 30, "bf16"),
    ("bf16_H128_C256", [12, 5], [19, 24], 48, 256, 128, "bf16"),
    ("H16_C150", [10, 17], [25, 12], 48, 150, 16, "f32"),
    ("H64_C256", [9, 4], [14, 22], 32, 256, 64, "f32"),
    # a canvas of 16k cells and more: the fp32 input gradient with 64-cell
    # waves (smaller canvases take 16-cell ones)
    ("H64_C256_64x256", [64, 64], [120, 130], 256, 256, 64, "f32"),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_padded_layer_against_oracle(case):
    import gpu_run
    import oracle_run
    from synth.configs import custom_workload

    name, hs, ws, cw, c_in, H, dt = case
    _say(f"case padded {name}: heights={hs} widths={ws} W={cw} C={c_in} H={H} {dt}")
    wl = custom_workload(300 + CASES.index(case), hs, ws, cw, c_in, H, dt)
    xs, params = wl.examples(), wl.params()
    dys = [wl.dy(k) for k in range(wl.n)]
    gpu = gpu_run.run_layer(xs, params, dys, hs, ws, cw, dtype=dt)
    ref = oracle_run.run_layer(xs, params, dys)
    _cmp(gpu, ref, dt, name)


MEM_CASES = [
    ("mem_H10_C6", [16, 5, 30], [25, 40, 3], 64, 6, 10),
    ("mem_H20_C1", [12, 33, 2], [40, 9, 17], 64, 1, 20),
]


@pytest.mark.parametrize("case", MEM_CASES, ids=[c[0] for c in MEM_CASES])
def test_padded_memory_states_against_oracle(case):
    import gpu_run
    import oracle_run
    from synth.configs import custom_workload

    name, hs, ws, cw, c_in, H = case
    _say(f"case padded {name}: heights={hs} widths={ws} W={cw} C={c_in} H={H}, memory-state matrices")
    wl = custom_workload(320 + MEM_CASES.index(case), hs, ws, cw, c_in, H)
    params = (*wl.params(), wl.memory_params())
    xs, dys = wl.examples(), [wl.dy(k) for k in range(wl.n)]
    gpu = gpu_run.run_layer(xs, params, dys, hs, ws, cw)
    ref = oracle_run.run_layer(xs, params, dys)
    _cmp(gpu, ref, "f32", name, memory=True)


def _pad_block(a, axis, blocks, n, m):
    """Zero-pad each of `blocks` consecutive runs of n entries along axis to m."""
    parts = np.split(a, blocks, axis=axis)
    out = []
    for p in parts:
        w = [(0, 0)] * a.ndim
        w[axis] = (0, m - n)
        out.append(np.pad(p, w))
    return np.concatenate(out, axis=axis)


@pytest.mark.parametrize("shape", [(6, 10, 8, 16, "f32"), (1, 2, 4, 4, "f32"), (30, 50, 32, 64, "f32"),
                                   (12, 100, 16, 128, "bf16")], ids=["C6_H10", "C1_H2", "C30_H50", "bf16_C12_H100"])
def test_padding_matches_the_built_shape_bitwise(shape):
    """The padded call computes what the built shape computes on zero-padded
    weights and inputs: same kernels, same operands, identical bits."""
    import gpu_run
    from synth.configs import custom_workload

    C, H, Cp, Hp, dt = shape
    hs, ws, cw = [14, 6, 21], [30, 11, 5], 48
    _say(f"case padding vs built shape: C={C}->{Cp} H={H}->{Hp} {dt}")
    wl = custom_workload(340, hs, ws, cw, C, H, dt)
    xs, (wx, u, b) = wl.examples(), wl.params()
    dys = [wl.dy(k) for k in range(wl.n)]
    a = gpu_run.run_layer(xs, (wx, u, b), dys, hs, ws, cw, dtype=dt)
    wxp = _pad_block(_pad_block(wx, 1, 5, H, Hp), 2, 1, C, Cp)
    up = _pad_block(_pad_block(u, 1, 5, H, Hp), 2, 2, H, Hp)
    bp = _pad_block(b, 1, 5, H, Hp)
    xsp = [_pad_block(x, 2, 1, C, Cp) for x in xs]
    dysp = [_pad_block(d, 2, 4, H, Hp) for d in dys]
    p = gpu_run.run_layer(xsp, (wxp, up, bp), dysp, hs, ws, cw, dtype=dt)

    def take_h(t):  # [.., 4Hp] -> [.., 4H]
        return np.concatenate([t[..., d * Hp:d * Hp + H] for d in range(4)], axis=-1)

    for k in range(wl.n):
        assert np.array_equal(a["Y"][k], take_h(p["Y"][k])), ("Y", k)
        assert np.array_equal(a["dX"][k], p["dX"][k][..., :C]), ("dX", k)
        # the padded hidden units stay at exactly zero
        y = p["Y"][k].reshape(*p["Y"][k].shape[:2], 4, Hp)
        assert not np.any(y[..., H:]), k
    sel = np.concatenate([np.arange(g * Hp, g * Hp + H) for g in range(5)])
    assert np.array_equal(a["dWx"], p["dWx"][:, sel, :C])
    selc = np.concatenate([np.arange(g * Hp, g * Hp + H) for g in range(2)])
    assert np.array_equal(a["dU"], p["dU"][:, sel][:, :, selc])
    assert np.array_equal(a["db"], p["db"][:, sel])


def test_padded_stepwise_forward():
    """The per-diagonal schedule runs padded shapes too."""
    import gpu_run
    import oracle_run
    from paper_1902_11208_amd import api
    from synth.configs import custom_workload

    hs, ws, cw = [9, 17, 4], [21, 6, 30], 48
    _say("case padded stepwise forward: C=6 H=10 f32")
    wl = custom_workload(350, hs, ws, cw, 6, 10)
    xs, params = wl.examples(), wl.params()
    units, place, ch, cw_, mask = gpu_run.layout(hs, ws, cw, "packed")
    wx, u, b = (gpu_run.to_dev(t, "f32") for t in params)
    canvas = api.pack_data([gpu_run.to_dev(x, "f32") for x in xs], place, ch, cw_)
    layer = api.MDLSTMLayer(wx, u, b, ch, cw_, units, mask)
    y = layer.forward_stepwise(canvas)
    got = [gpu_run.to_np(t) for t in api.unpack_data(y, place)]
    torch.cuda.synchronize()
    ref = oracle_run.run_layer(xs, params, None, backward=False)
    for k, (g, r) in enumerate(zip(got, ref["Y"])):
        assert rel_err(g, r) <= 1e-5 and rel_max(g, r) <= 1e-5, k


@pytest.mark.parametrize("shape", [(3, 10), (32, 32)], ids=["C3_H10", "C32_H32"])
def test_padded_empty_layout(shape):
    """No rectangles: Y and dX are zero and the weight gradients are zero (C 32,
    H 32 takes the direct-to-LDS strip kernel, whose strip lists are empty)."""
    from paper_1902_11208_amd import api

    C, H = shape
    _say(f"case padded empty layout: C={C} H={H}, 12x40 canvas, no rectangles")
    dev = "cuda"
    g = torch.Generator().manual_seed(5)
    wx = torch.randn(4, 5 * H, C, generator=g).to(dev)
    u = torch.randn(4, 5 * H, 2 * H, generator=g).to(dev)
    b = torch.randn(4, 5 * H, generator=g).to(dev)
    mask = torch.zeros(12, 40, dtype=torch.uint8, device=dev)
    layer = api.MDLSTMLayer(wx, u, b, 12, 40, np.zeros((0, 4), np.int32), mask)
    y = layer.forward(torch.randn(12, 40, C, generator=g).to(dev))
    dx, dwx, du, db = layer.backward(torch.randn(12, 40, 4 * H, generator=g).to(dev))
    torch.cuda.synchronize()
    for t in (y, dx, dwx, du, db):
        assert not torch.any(t != 0)


def test_strip_lists_with_empty_rows_and_slack():
    """C 32, H 32 (the direct-to-LDS strip kernel): rectangles that leave whole
    canvas rows, row ends and a column band empty, so most strips are skipped
    and the others are spread unevenly over the groups; against the oracle,
    and dX exactly zero on every cell outside the rectangles."""
    import gpu_run
    import oracle_run
    from synth.configs import custom_workload

    hs, ws, cw = [3, 17, 5], [70, 9, 33], 160
    _say(f"case strip lists: heights={hs} widths={ws} W={cw} C=32 H=32 f32")
    wl = custom_workload(360, hs, ws, cw, 32, 32)
    xs, params = wl.examples(), wl.params()
    dys = [wl.dy(k) for k in range(wl.n)]
    gpu = gpu_run.run_layer(xs, params, dys, hs, ws, cw, dtype="f32")
    ref = oracle_run.run_layer(xs, params, dys)
    _cmp(gpu, ref, "f32", "strip lists")
    dxc = gpu_run.to_np(gpu["dx_canvas"])
    mask = gpu["mask"]
    mask = mask.cpu().numpy() if hasattr(mask, "cpu") else np.asarray(mask)
    _say(f"  canvas {dxc.shape[0]}x{dxc.shape[1]}, {int((mask != 0).sum())} cells in rectangles")
    assert not np.any(dxc[mask == 0]), "dX outside the rectangles"
