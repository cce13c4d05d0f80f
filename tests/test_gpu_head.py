"""GPU parity of the shared output layer, the row collapse and the CTC loss
(Section II) against the float64 oracle (oracle/head.py), through the C ABI,
alone and as one training step with the MDLSTM layer on a packed canvas.

Tolerance as for the layer: normwise L2 and max-norm relative error <= 1e-5
per tensor (fp32 storage; the CTC recursion runs in double precision)."""
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


def _check(name, got, want, tol=TOL):
    e, m = rel_err(got, want), rel_max(got, want)
    assert e <= tol and m <= tol, (name, e, m)
    return e, m


def test_head_and_ctc_small():
    """Four examples on one canvas (NaN outside the rectangles, which must not
    be read): a one-frame example, an empty label, a label whose repeats fill
    every frame, and a long one; logits, losses, gradients and the upstream
    gradient of the layer, which is zero outside the rectangles."""
    from oracle import head as ohead
    from paper_1902_11208_amd import api

    rng = np.random.default_rng(21)
    H, K = 8, 6
    hs, ws = [3, 5, 2, 4], [1, 7, 4, 20]
    labels = [np.array([2], np.int32), np.array([], np.int32), np.array([3, 3], np.int32),
              rng.integers(1, K, 9).astype(np.int32)]
    rects, ch, _ = api.pack_layout(hs, ws, 24)
    Y = rng.standard_normal((ch, 24, 4 * H)).astype(np.float32)
    inside = np.zeros((ch, 24), bool)
    for y0, x0, h, w in rects:
        inside[y0:y0 + h, x0:x0 + w] = True
    Y[~inside] = np.nan
    W = rng.uniform(-0.3, 0.3, (K, H)).astype(np.float32)
    b = rng.uniform(-0.3, 0.3, K).astype(np.float32)
    print(f"case: head + CTC on 4 examples {list(zip(hs, ws))}, H={H}, K={K}", flush=True)
    hd = api.Head(torch.from_numpy(W).cuda(), torch.from_numpy(b).cuda(), rects, (ch, 24), labels)
    logits = hd.forward(torch.from_numpy(Y).cuda()).cpu().numpy().astype(np.float64)
    losses, dl = hd.ctc()
    losses, dl = losses.cpu().numpy().astype(np.float64), dl.cpu().numpy().astype(np.float64)
    dy, dw, db = hd.backward()
    torch.cuda.synchronize()
    dy, dw, db = (t.cpu().numpy().astype(np.float64) for t in (dy, dw, db))
    off = np.concatenate([[0], np.cumsum(ws)])
    dW_ref, db_ref = np.zeros((K, H)), np.zeros(K)
    for k, (y0, x0, h, w) in enumerate(rects):
        Yk = Y[y0:y0 + h, x0:x0 + w].astype(np.float64)
        loss, dYk, dWk, dbk, lk, dlk = ohead.head_loss_forward_backward(Yk, W, b, labels[k])
        _check(f"logits[{k}]", logits[off[k]:off[k + 1]], lk)
        assert abs(losses[k] - loss) <= TOL * abs(loss), (k, losses[k], loss)
        _check(f"dlogits[{k}]", dl[off[k]:off[k + 1]], dlk)
        _check(f"dY[{k}]", dy[y0:y0 + h, x0:x0 + w], dYk)
        dW_ref += dWk
        db_ref += dbk
    assert np.all(dy[~inside] == 0)
    _check("dW", dw, dW_ref)
    _check("db", db, db_ref)


def _step_case(wl, label, keep=None):
    import gpu_run
    import oracle_run

    xs, params = wl.examples(), wl.params()
    hp = wl.head_params()
    labels = [wl.label(k) for k in range(wl.n)]
    print(f"case: training step on {label}: {wl.n} examples, H={wl.hidden}, {hp[0].shape[0]} classes", flush=True)
    gpu = gpu_run.run_training_step(xs, params, hp, labels, wl.heights, wl.widths, wl.canvas_w, keep=keep)
    ks = range(wl.n) if keep is None else keep
    ref = oracle_run.run_training_step([xs[k] for k in ks] if keep is not None else xs, params, hp,
                                       [labels[k] for k in ks] if keep is not None else labels,
                                       workers=oracle_run.default_workers(), progress=f"{label} oracle")
    worst = {}
    for i, k in enumerate(ks):
        assert abs(gpu["loss"][k] - ref["loss"][i]) <= TOL * abs(ref["loss"][i]), (k, gpu["loss"][k], ref["loss"][i])
        for nm in ("logits", "dlogits", "dX"):
            em = _check(f"{nm}[{k}]", gpu[nm][k], ref[nm][i])
            worst[nm] = max(worst.get(nm, (0, 0)), em)
    return gpu, ref, worst


def test_training_step_words():
    """The word batch (256 x h16, C_in 16, H 16) in one training step: layer,
    shared output layer over the packed canvas, CTC on synthetic labels, and
    back, against the oracle running each example alone."""
    from synth import configs

    gpu, ref, worst = _step_case(configs.workload(2), "word batch")
    for nm in ("dWfc", "dbfc", "dWx", "dU", "db"):
        worst[nm] = _check(nm, gpu[nm], ref[nm])
    print("  worst (L2, max): " + ", ".join(f"{k} ({v[0]:.1e}, {v[1]:.1e})" for k, v in worst.items()), flush=True)
    total = float(np.sum(gpu["loss"]))
    print(f"  batch loss {total:.6e} (oracle {float(np.sum(ref['loss'])):.6e})", flush=True)


def test_training_step_lines_sampled():
    """The line batch (64 x h32, widths 200-600, C_in 32, H 32): the whole
    batch in one GPU run; losses, logits, dlogits and dX of 8 examples
    (the widest among them) against the oracle."""
    from synth import configs

    wl = configs.workload(3)
    keep = sorted(set(np.random.default_rng(8).choice(wl.n, 7, replace=False).tolist()) | {int(np.argmax(wl.widths))})
    _step_case(wl, "line batch", keep=keep)


def test_head_is_deterministic():
    from paper_1902_11208_amd import api
    from synth import configs

    wl = configs.workload(2)
    rng = np.random.default_rng(4)
    rects, ch, _ = api.pack_layout(wl.heights, wl.widths, wl.canvas_w)
    Y = torch.from_numpy(rng.standard_normal((ch, wl.canvas_w, 4 * wl.hidden)).astype(np.float32)).cuda()
    W, b = (torch.from_numpy(t).cuda() for t in wl.head_params())
    outs = []
    for _ in range(2):
        hd = api.Head(W, b, rects, (ch, wl.canvas_w), [wl.label(k) for k in range(wl.n)])
        hd.forward(Y)
        l, g = hd.ctc()
        dy, dw, db = hd.backward()
        torch.cuda.synchronize()
        outs.append([t.clone() for t in (l, g, dy, dw, db)])
    for a, c in zip(*outs):
        assert torch.equal(a, c)


@pytest.mark.parametrize("L", [40, 128, 250, 500])
def test_ctc_long_labels(L):
    """Label lengths that select each width of the CTC scan (states per lane
    1 to 16), with alignments tight enough that the forward variables span
    far more than the double range within a frame (500 labels in 1010
    frames): losses and gradients against the log-space oracle."""
    from oracle import head as ohead
    from paper_1902_11208_amd import api

    rng = np.random.default_rng(L)
    H, K = 8, 80
    T = 2 * L + 10
    hs, ws = [2, 3], [T, T // 2 + L]
    labels = [rng.integers(1, K, L).astype(np.int32), rng.integers(1, K, L // 2).astype(np.int32)]
    rects, ch, _ = api.pack_layout(hs, ws, max(ws))
    Y = (rng.standard_normal((ch, max(ws), 4 * H)) * 0.3).astype(np.float32)
    W = rng.uniform(-0.3, 0.3, (K, H)).astype(np.float32)
    b = rng.uniform(-0.3, 0.3, K).astype(np.float32)
    print(f"case: CTC with {L} and {L // 2} labels over {ws} frames", flush=True)
    hd = api.Head(torch.from_numpy(W).cuda(), torch.from_numpy(b).cuda(), rects, (ch, max(ws)), labels)
    lg = hd.forward(torch.from_numpy(Y).cuda()).cpu().numpy().astype(np.float64)
    losses, dl = hd.ctc()
    torch.cuda.synchronize()
    losses, dl = losses.cpu().numpy().astype(np.float64), dl.cpu().numpy().astype(np.float64)
    off = np.concatenate([[0], np.cumsum(ws)])
    for k in range(2):
        loss, g = ohead.ctc_loss(lg[off[k]:off[k + 1]], labels[k])
        assert abs(losses[k] - loss) <= TOL * abs(loss), (k, losses[k], loss)
        _check(f"dlogits[{k}]", dl[off[k]:off[k + 1]], g)
