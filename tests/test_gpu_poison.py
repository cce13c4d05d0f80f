"""Poisoned-workspace debug mode (MDLSTM_POISON_WORKSPACE=1): the forward,
backward and head calls first fill the floating-point workspace sections they
write before reading with NaN. If any kernel read a value it had not
written, NaN would reach the results; with the mode on, every result must
equal, bit for bit, the run without it, and match the float64 oracle."""
import os

import numpy as np
import pytest

from conftest import rel_err, rel_max

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu(built_lib):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _poisoned(fn):
    os.environ["MDLSTM_POISON_WORKSPACE"] = "1"
    try:
        return fn()
    finally:
        del os.environ["MDLSTM_POISON_WORKSPACE"]


def _same(a, b, label):
    for k in a:
        if isinstance(a[k], list):
            for i, (x, y) in enumerate(zip(a[k], b[k])):
                if x is not None:
                    assert np.array_equal(x, y), (label, k, i)
        elif isinstance(a[k], np.ndarray):
            assert np.array_equal(a[k], b[k]), (label, k)


CASES = [
    # name, heights, widths, canvas_w, c_in, hidden, dtype, memory states
    ("f32_H16_ragged", [5, 1, 16, 3], [9, 12, 1, 7], 32, 8, 16, "f32", False),
    ("f32_H32_tall", [48, 64, 17], [9, 5, 30], 64, 32, 32, "f32", False),
    ("f32_H64", [7, 20], [30, 11], 32, 16, 64, "f32", False),
    ("bf16_H128", [9, 30, 2], [40, 12, 7], 48, 64, 128, "bf16", False),
    ("f32_H16_memory", [16, 9, 30], [40, 25, 17], 64, 16, 16, "f32", True),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_layer_results_unchanged_by_poison(case):
    import gpu_run
    import oracle_run
    from synth.configs import custom_workload

    name, hs, ws, cw, c_in, H, dt, mem = case
    print(f"case {name}: heights={hs} widths={ws} W={cw} C={c_in} H={H} {dt}, poisoned workspace", flush=True)
    wl = custom_workload(300 + CASES.index(case), hs, ws, cw, c_in, H, dtype=dt)
    params = (*wl.params(), wl.memory_params()) if mem else wl.params()
    xs, dys = wl.examples(), [wl.dy(k) for k in range(wl.n)]
    plain = gpu_run.run_layer(xs, params, dys, hs, ws, cw, dtype=dt)
    pois = _poisoned(lambda: gpu_run.run_layer(xs, params, dys, hs, ws, cw, dtype=dt))
    _same(plain, pois, name)
    if dt == "f32":
        ref = oracle_run.run_layer(xs, params, dys)
        for k, (g, r) in enumerate(zip(pois["Y"], ref["Y"])):
            assert rel_err(g, r) <= 1e-5 and rel_max(g, r) <= 1e-5, (name, "Y", k)
        for nm in ("dWx", "dU", "db"):
            assert rel_err(pois[nm], ref[nm]) <= 1e-5, (name, nm)


def test_training_step_unchanged_by_poison():
    """Layer, output layer, CTC and back on the word batch."""
    import gpu_run
    from synth import configs

    wl = configs.workload(2)
    xs, params, hp = wl.examples(), wl.params(), wl.head_params()
    labels = [wl.label(k) for k in range(wl.n)]
    print("case: training step on the word batch, poisoned workspaces", flush=True)
    a = gpu_run.run_training_step(xs, params, hp, labels, wl.heights, wl.widths, wl.canvas_w)
    b = _poisoned(lambda: gpu_run.run_training_step(xs, params, hp, labels, wl.heights, wl.widths, wl.canvas_w))
    _same(a, b, "training step")
    assert np.all(np.isfinite(b["loss"]))


def test_stepwise_forward_unchanged_by_poison():
    import gpu_run
    from paper_1902_11208_amd import api
    from synth.configs import custom_workload

    wl = custom_workload(320, [16, 9, 30], [40, 25, 17], 64, 16, 16)
    units, place, ch, cw, mask = gpu_run.layout(wl.heights, wl.widths, wl.canvas_w, "packed")
    x = api.pack_data([gpu_run.to_dev(e, "f32") for e in wl.examples()], place, ch, cw)
    layer = api.MDLSTMLayer(*[gpu_run.to_dev(p, "f32") for p in wl.params()], ch, cw, units, mask)
    print("case: per-diagonal forward, poisoned workspace", flush=True)
    ref = layer.forward(x).clone()
    got = _poisoned(lambda: layer.forward_stepwise(x).clone())
    torch.cuda.synchronize()
    assert torch.equal(ref, got)


def test_poison_reaches_the_workspace():
    """The mode really fills: after a poisoned forward on a canvas with slack
    cells (which no kernel writes), the workspace holds more all-ones words
    than after a plain forward from a zeroed workspace (the rectangle ids of
    cells outside every rectangle are -1, all ones, in both)."""
    import gpu_run
    from paper_1902_11208_amd import api
    from synth.configs import custom_workload

    wl = custom_workload(321, [5, 9], [20, 7], 32, 8, 16)
    units, place, ch, cw, mask = gpu_run.layout(wl.heights, wl.widths, wl.canvas_w, "packed")
    x = api.pack_data([gpu_run.to_dev(e, "f32") for e in wl.examples()], place, ch, cw)
    layer = api.MDLSTMLayer(*[gpu_run.to_dev(p, "f32") for p in wl.params()], ch, cw, units, mask)

    def ones_after(fn):
        layer.workspace.zero_()
        y = fn().clone()
        torch.cuda.synchronize()
        words = layer.workspace[: layer.workspace.numel() // 4 * 4].view(torch.int32)
        return int((words == -1).sum().item()), y

    print("case: poisoned words left at slack cells", flush=True)
    n_plain, y_plain = ones_after(lambda: layer.forward(x))
    n_pois, y_pois = _poisoned(lambda: ones_after(lambda: layer.forward(x)))
    assert torch.equal(y_plain, y_pois)
    assert n_pois > n_plain, (n_pois, n_plain)
