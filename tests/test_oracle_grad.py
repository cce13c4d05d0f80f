"""Pins for the oracle's backward pass: central finite differences of the
forward (itself pinned in test_oracle_cell.py) and the adjoint identity."""
import numpy as np
import pytest

from oracle import mdlstm, pack


def _loss_examples(xs, params, dys):
    return sum(float(np.sum(mdlstm.example_forward(x, params) * dy)) for x, dy in zip(xs, dys))


def _grads_examples(xs, params, dys):
    dxs, acc = [], None
    for x, dy in zip(xs, dys):
        dX, dWx, dU, db = mdlstm.example_backward(x, params, dy)
        dxs.append(dX)
        acc = [dWx, dU, db] if acc is None else [a + g for a, g in zip(acc, (dWx, dU, db))]
    return dxs, acc


def _case(seed=0):
    rng = np.random.default_rng(seed)
    C, H = 2, 2
    params = [rng.uniform(-0.6, 0.6, (4, 5 * H, C)), rng.uniform(-0.6, 0.6, (4, 5 * H, 2 * H)),
              rng.uniform(-0.6, 0.6, (4, 5 * H))]
    xs = [rng.standard_normal((3, 4, C)), rng.standard_normal((2, 5, C))]
    dys = [rng.standard_normal((3, 4, 4 * H)), rng.standard_normal((2, 5, 4 * H))]
    return params, xs, dys


def test_central_differences_all_parameters_and_inputs():
    params, xs, dys = _case()
    dxs, (dWx, dU, db) = _grads_examples(xs, params, dys)
    eps = 1e-6
    analytic = [dWx, dU, db]
    for pi in range(3):
        p = params[pi]
        for idx in np.ndindex(p.shape):
            old = p[idx]
            p[idx] = old + eps
            lp = _loss_examples(xs, params, dys)
            p[idx] = old - eps
            lm = _loss_examples(xs, params, dys)
            p[idx] = old
            num = (lp - lm) / (2 * eps)
            assert abs(num - analytic[pi][idx]) <= 1e-6 * max(1.0, abs(num)), (pi, idx, num, analytic[pi][idx])
    for k, x in enumerate(xs):
        for idx in np.ndindex(x.shape):
            old = x[idx]
            x[idx] = old + eps
            lp = _loss_examples(xs, params, dys)
            x[idx] = old - eps
            lm = _loss_examples(xs, params, dys)
            x[idx] = old
            num = (lp - lm) / (2 * eps)
            assert abs(num - dxs[k][idx]) <= 1e-6 * max(1.0, abs(num)), (k, idx, num, dxs[k][idx])


def test_adjoint_identity():
    # <dY, J v> = <J^T dY, v> for a random direction v over all inputs and parameters
    params, xs, dys = _case(seed=5)
    rng = np.random.default_rng(9)
    vp = [rng.standard_normal(p.shape) for p in params]
    vx = [rng.standard_normal(x.shape) for x in xs]
    dxs, gp = _grads_examples(xs, params, dys)
    rhs = sum(float(np.sum(a * b)) for a, b in zip(gp, vp)) + sum(float(np.sum(a * b)) for a, b in zip(dxs, vx))
    t = 1e-5
    plus = [p + t * v for p, v in zip(params, vp)]
    minus = [p - t * v for p, v in zip(params, vp)]
    lhs = (_loss_examples([x + t * v for x, v in zip(xs, vx)], plus, dys)
           - _loss_examples([x - t * v for x, v in zip(xs, vx)], minus, dys)) / (2 * t)
    assert abs(lhs - rhs) <= 1e-7 * max(1.0, abs(rhs))


def test_masked_canvas_backward_matches_differences():
    # a canvas with scheduling rectangles and holes in the mask: gradients of
    # sum(Y * dY) w.r.t. canvas input and weights, by central differences
    rng = np.random.default_rng(21)
    C, H = 2, 1
    params = [rng.uniform(-0.7, 0.7, (4, 5 * H, C)), rng.uniform(-0.7, 0.7, (4, 5 * H, 2 * H)),
              rng.uniform(-0.7, 0.7, (4, 5 * H))]
    rects = np.array([[0, 0, 3, 3], [0, 4, 2, 2], [3, 0, 2, 6]], np.int32)  # two rects touch (rows 2|3)
    ch, cw = 5, 6
    mask = pack.make_mask(rects, ch, cw)
    mask[1, 1] = 0
    mask[3, 4] = 0
    x = rng.standard_normal((ch, cw, C))
    dY = rng.standard_normal((ch, cw, 4 * H))

    def loss():
        Y, _ = mdlstm.units_forward(x, mask, rects, params)
        return float(np.sum(Y * dY * mask[:, :, None]))

    Y, caches = mdlstm.units_forward(x, mask, rects, params)
    dX, dWx, dU, db = mdlstm.units_backward(x, mask, rects, params, caches, dY)
    eps = 1e-6
    for arr, grad in ((x, dX), (params[0], dWx), (params[1], dU), (params[2], db)):
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + eps
            lp = loss()
            arr[idx] = old - eps
            lm = loss()
            arr[idx] = old
            num = (lp - lm) / (2 * eps)
            assert abs(num - grad[idx]) <= 1e-6 * max(1.0, abs(num)), (idx, num, grad[idx])
    assert np.all(dX[mask == 0] == 0)


@pytest.mark.parametrize("d", range(4))
def test_gradient_flows_only_backwards_along_scan(d):
    # dY at one cell of direction d's block reaches exactly the cells that
    # precede it in direction d's scan (its causal cone) and nothing else
    rng = np.random.default_rng(30 + d)
    C, H, h, w = 1, 1, 4, 5
    params = [rng.uniform(-0.5, 0.5, (4, 5 * H, C)), rng.uniform(-0.5, 0.5, (4, 5 * H, 2 * H)),
              rng.uniform(-0.5, 0.5, (4, 5 * H))]
    x = rng.standard_normal((h, w, C))
    dY = np.zeros((h, w, 4 * H))
    py, px = 2, 2
    dY[py, px, d] = 1.0
    dX = mdlstm.example_backward(x, params, dY)[0][:, :, 0]
    sy, sx = mdlstm._steps(d)
    for yy in range(h):
        for xx in range(w):
            in_cone = (yy - py) * sy <= 0 and (xx - px) * sx <= 0
            assert (dX[yy, xx] != 0) == in_cone, (yy, xx)
