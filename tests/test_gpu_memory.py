"""GPU parity of the layer with memory-state matrices (Appendix A; the input
gate and the two forget gates read both predecessor memory states) against
the float64 oracle, through the C ABI: Y, dX per example and dWx, dU, db, dV,
normwise L2 and max-norm relative error <= 1e-5 (fp32)."""
import numpy as np
import pytest

from conftest import rel_err, rel_max

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TOL = 1e-5


@pytest.fixture(scope="module", autouse=True)
def _need_gpu(built_lib):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _cmp(gpu, ref, label):
    worst = {}
    for nm in ("Y", "dX"):
        for k, (g, r) in enumerate(zip(gpu[nm], ref[nm])):
            e, m = rel_err(g, r), rel_max(g, r)
            assert e <= TOL and m <= TOL, (label, nm, k, e, m)
            worst[nm] = max(worst.get(nm, (0, 0)), (e, m))
    for nm in ("dWx", "dU", "db", "dV"):
        e, m = rel_err(gpu[nm], ref[nm]), rel_max(gpu[nm], ref[nm])
        assert e <= TOL and m <= TOL, (label, nm, e, m)
        worst[nm] = (e, m)
    print(f"{label}: worst (L2, max) " + ", ".join(f"{k} ({v[0]:.1e}, {v[1]:.1e})" for k, v in worst.items()),
          flush=True)


CASES = [
    # name, heights, widths, canvas_w, c_in, hidden
    ("H16_ragged", [5, 1, 16, 3], [9, 12, 1, 7], 32, 8, 16),
    ("H16_tall", [64, 20, 33], [6, 17, 4], 64, 16, 16),
    ("H32_ragged", [7, 30, 1, 2], [20, 5, 9, 1], 48, 16, 32),
    ("H32_tall", [48, 64, 17], [9, 5, 30], 64, 32, 32),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_memory_states_small(case):
    import gpu_run
    import oracle_run
    from synth.configs import custom_workload

    name, hs, ws, cw, c_in, H = case
    print(f"case {name}: heights={hs} widths={ws} W={cw} C={c_in} H={H}, memory-state matrices", flush=True)
    wl = custom_workload(200 + CASES.index(case), hs, ws, cw, c_in, H)
    params = (*wl.params(), wl.memory_params())
    xs, dys = wl.examples(), [wl.dy(k) for k in range(wl.n)]
    gpu = gpu_run.run_layer(xs, params, dys, hs, ws, cw)
    ref = oracle_run.run_layer(xs, params, dys)
    _cmp(gpu, ref, name)


def test_memory_states_masked_holes():
    """Touching rectangles and mask holes: state and memory-state input
    restart at every edge and masked cell."""
    import gpu_run
    from oracle import mdlstm, pack
    from paper_1902_11208_amd import api

    rng = np.random.default_rng(15)
    C, H = 8, 16
    rects = np.array([[0, 0, 5, 7], [0, 7, 5, 4], [5, 0, 3, 11], [8, 2, 2, 2]], np.int32)
    ch, cw = 10, 11
    mask = pack.make_mask(rects, ch, cw)
    mask[1, 1] = mask[3, 8] = mask[6, 5] = 0
    x = rng.standard_normal((ch, cw, C)).astype(np.float32)
    dY = rng.standard_normal((ch, cw, 4 * H)).astype(np.float32)
    params = [rng.uniform(-0.3, 0.3, s).astype(np.float32)
              for s in ((4, 5 * H, C), (4, 5 * H, 2 * H), (4, 5 * H), (4, 3 * H, 2 * H))]
    print("case memory states: masked holes, 4 touching rects", flush=True)
    dev = [gpu_run.to_dev(p, "f32") for p in params]
    layer = api.MDLSTMLayer(*dev[:3], ch, cw, rects, torch.from_numpy(mask).cuda(), v=dev[3])
    y = layer.forward(gpu_run.to_dev(x, "f32"))
    dx, dwx, du, db, dv = layer.backward(gpu_run.to_dev(dY, "f32"))
    torch.cuda.synchronize()
    Yr, caches = mdlstm.units_forward(x, mask, rects, params)
    ref = mdlstm.units_backward(x, mask, rects, params, caches, dY)
    for got, want, nm in zip((y, dx, dwx, du, db, dv), (Yr,) + tuple(ref), ("Y", "dX", "dWx", "dU", "db", "dV")):
        e, m = rel_err(gpu_run.to_np(got), want), rel_max(gpu_run.to_np(got), want)
        print(f"  {nm}: L2 {e:.2e} max {m:.2e}", flush=True)
        assert e <= TOL and m <= TOL, nm
    assert np.all(gpu_run.to_np(y)[mask == 0] == 0)


def test_zero_memory_matrices_match_the_plain_kernels():
    """With V = 0 the memory-state wavefronts (their own kernels) give the
    plain layer's results, computed by the other wavefront kernels."""
    import gpu_run
    from synth.configs import custom_workload

    wl = custom_workload(230, [16, 16, 9, 30], [40, 8, 25, 17], 64, 16, 16)
    xs, dys = wl.examples(), [wl.dy(k) for k in range(wl.n)]
    params = wl.params()
    print("case memory states: V = 0 against the plain kernels", flush=True)
    a = gpu_run.run_layer(xs, params, dys, wl.heights, wl.widths, wl.canvas_w)
    b = gpu_run.run_layer(xs, (*params, np.zeros((4, 48, 32), np.float32)), dys, wl.heights, wl.widths,
                          wl.canvas_w)
    for nm in ("Y", "dX"):
        for g, r in zip(a[nm], b[nm]):
            assert rel_max(g, r) <= 1e-6
    for nm in ("dWx", "dU", "db"):
        assert rel_max(a[nm], b[nm]) <= 1e-6
    assert np.all(b["dV"] == b["dV"])  # finite


@pytest.mark.parametrize("cid", [2, 3])
def test_memory_states_full_batch(cid):
    """The word batch (256 x h16, H 16) and the line batch (64 x h32, H 32)
    with memory-state matrices: every example's Y and dX and the full-batch
    weight gradients, V's included, from one GPU run."""
    import gpu_run
    import oracle_run
    from synth import configs

    wl = configs.workload(cid)
    params = (*wl.params(), wl.memory_params())
    xs, dys = wl.examples(), [wl.dy(k) for k in range(wl.n)]
    print(f"case memory states, workload {cid}: {wl.n} examples, H={wl.hidden}, full batch", flush=True)
    gpu = gpu_run.run_layer(xs, params, dys, wl.heights, wl.widths, wl.canvas_w)
    ref = oracle_run.run_layer(xs, params, dys, workers=oracle_run.default_workers(),
                               progress=f"workload {cid} oracle")
    _cmp(gpu, ref, f"workload {cid} with memory states")
