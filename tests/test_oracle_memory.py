"""Pins for the oracle's memory-state matrices (Appendix A: three matrices
per predecessor memory state S1 = c_L and S2 = c_T, read here as feeding the
input gate and the two forget gates): a hand-worked 2x2 grid written out with
scalar math, the scalar and diagonal forms against each other, the plain cell
recovered at V = 0, central finite differences over every parameter (V
included) and input, the adjoint identity, and a masked canvas."""
import numpy as np

from conftest import read_fixture
from oracle import mdlstm, pack


def _params(rng, C, H, scale=0.5):
    return (rng.uniform(-scale, scale, (4, 5 * H, C)), rng.uniform(-scale, scale, (4, 5 * H, 2 * H)),
            rng.uniform(-scale, scale, (4, 5 * H)), rng.uniform(-scale, scale, (4, 3 * H, 2 * H)))


def test_hand_worked_2x2_memory_states():
    rows = read_fixture("cell_2x2_memory.txt")
    assert len(rows) == 4
    x = np.array([[0.0, 1.0], [2.0, 3.0]])[:, :, None]
    wx, u, b, v = np.zeros((4, 5, 1)), np.zeros((4, 5, 2)), np.zeros((4, 5)), np.zeros((4, 3, 2))
    for d in range(4):
        wx[d, 4, 0] = 0.5
        b[d] = [np.log(3.0), -np.log(3.0), 0.0, np.log(4.0), 0.25]
        u[d, 4] = [1.0, -2.0]
        v[d] = [[0.5, -0.25], [1.0, 0.5], [-0.75, 0.25]]  # rows i, f_L, f_T; columns c_L, c_T
    Y, cache = mdlstm.layer_forward(x, wx, u, b, v=v)
    Ys = mdlstm.layer_forward_scalar(x, wx, u, b, v=v)
    for r in rows:
        d = int(r[0])
        vals = np.array(list(map(float, r[1:]))).reshape(2, 2, 2)
        np.testing.assert_allclose(Y[:, :, d], vals[:, :, 0], rtol=0, atol=1e-14)
        np.testing.assert_allclose(Ys[:, :, d], vals[:, :, 0], rtol=0, atol=1e-14)
        c = mdlstm._flip(cache["dirs"][d]["c"], d)[:, :, 0]
        np.testing.assert_allclose(c, vals[:, :, 1], rtol=0, atol=1e-14)


def test_scalar_and_diagonal_forms_agree():
    rng = np.random.default_rng(1)
    C, H = 3, 4
    wx, u, b, v = _params(rng, C, H)
    x = rng.standard_normal((5, 7, C))
    valid = rng.random((5, 7)) > 0.2
    Y, _ = mdlstm.layer_forward(x, wx, u, b, valid=valid, v=v)
    Ys = mdlstm.layer_forward_scalar(x, wx, u, b, valid=valid, v=v)
    np.testing.assert_allclose(Y, Ys, rtol=1e-12, atol=1e-14)
    # the memory states change the result
    Y0, _ = mdlstm.layer_forward(x, wx, u, b, valid=valid)
    assert np.max(np.abs(Y - Y0)) > 1e-3


def test_zero_memory_matrices_are_the_plain_cell():
    rng = np.random.default_rng(2)
    C, H = 2, 3
    wx, u, b, _ = _params(rng, C, H)
    x = rng.standard_normal((4, 6, C))
    dY = rng.standard_normal((4, 6, 4 * H))
    Y0, c0 = mdlstm.layer_forward(x, wx, u, b)
    Yz, cz = mdlstm.layer_forward(x, wx, u, b, v=np.zeros((4, 3 * H, 2 * H)))
    assert np.array_equal(Y0, Yz)
    g0 = mdlstm.layer_backward(c0, dY, wx, u, b)
    gz = mdlstm.layer_backward(cz, dY, wx, u, b, v=np.zeros((4, 3 * H, 2 * H)))
    for a, c in zip(g0, gz[:4]):
        np.testing.assert_allclose(a, c, rtol=1e-13, atol=1e-15)


def _loss(xs, params, dys):
    wx, u, b, v = params
    return sum(float(np.sum(mdlstm.layer_forward(x, wx, u, b, v=v)[0] * dy)) for x, dy in zip(xs, dys))


def test_central_differences_with_memory_states():
    rng = np.random.default_rng(3)
    C, H = 2, 2
    params = list(_params(rng, C, H, 0.6))
    xs = [rng.standard_normal((3, 4, C)), rng.standard_normal((2, 5, C))]
    dys = [rng.standard_normal((3, 4, 4 * H)), rng.standard_normal((2, 5, 4 * H))]
    grads, dxs = None, []
    for x, dy in zip(xs, dys):
        _, cache = mdlstm.layer_forward(x, *params[:3], v=params[3])
        g = mdlstm.layer_backward(cache, dy, *params[:3], v=params[3])
        dxs.append(g[0])
        grads = list(g[1:]) if grads is None else [a + c for a, c in zip(grads, g[1:])]
    eps = 1e-6
    for pi in range(4):
        p = params[pi]
        for idx in np.ndindex(p.shape):
            old = p[idx]
            p[idx] = old + eps
            lp = _loss(xs, params, dys)
            p[idx] = old - eps
            lm = _loss(xs, params, dys)
            p[idx] = old
            num = (lp - lm) / (2 * eps)
            assert abs(num - grads[pi][idx]) <= 1e-6 * max(1.0, abs(num)), (pi, idx, num, grads[pi][idx])
    for k, x in enumerate(xs):
        for idx in np.ndindex(x.shape):
            old = x[idx]
            x[idx] = old + eps
            lp = _loss(xs, params, dys)
            x[idx] = old - eps
            lm = _loss(xs, params, dys)
            x[idx] = old
            num = (lp - lm) / (2 * eps)
            assert abs(num - dxs[k][idx]) <= 1e-6 * max(1.0, abs(num)), (k, idx, num)


def test_adjoint_identity_with_memory_states():
    """<dY, J v> = <J^T dY, v> for a direction v in (x, theta) space, J the
    Jacobian of Y (a linearization by a tiny step)."""
    rng = np.random.default_rng(4)
    C, H = 3, 2
    params = list(_params(rng, C, H, 0.4))
    x = rng.standard_normal((4, 5, C))
    dY = rng.standard_normal((4, 5, 4 * H))
    _, cache = mdlstm.layer_forward(x, *params[:3], v=params[3])
    dX, dWx, dU, db, dV = mdlstm.layer_backward(cache, dY, *params[:3], v=params[3])
    dirs = [rng.standard_normal(t.shape) for t in [x] + params]
    eps = 1e-6
    plus = mdlstm.layer_forward(x + eps * dirs[0], *[p + eps * q for p, q in zip(params[:3], dirs[1:4])],
                                v=params[3] + eps * dirs[4])[0]
    minus = mdlstm.layer_forward(x - eps * dirs[0], *[p - eps * q for p, q in zip(params[:3], dirs[1:4])],
                                 v=params[3] - eps * dirs[4])[0]
    jv = np.sum(dY * (plus - minus)) / (2 * eps)
    jtdy = sum(float(np.sum(g * q)) for g, q in zip((dX, dWx, dU, db, dV), dirs))
    assert abs(jv - jtdy) <= 1e-6 * max(1.0, abs(jv))


def test_masked_canvas_with_memory_states():
    """Touching rectangles and mask holes: the units forms with V restart the
    recurrence (state and memory-state input both zero) at every edge and hole,
    checked by finite differences of the canvas loss."""
    rng = np.random.default_rng(5)
    C, H = 2, 2
    params = list(_params(rng, C, H, 0.5))
    rects = np.array([[0, 0, 3, 4], [0, 4, 3, 2], [3, 1, 2, 5]], np.int32)
    ch, cw = 5, 6
    mask = pack.make_mask(rects, ch, cw)
    mask[1, 1] = mask[4, 3] = 0
    x = rng.standard_normal((ch, cw, C))
    dY = rng.standard_normal((ch, cw, 4 * H))
    Y, caches = mdlstm.units_forward(x, mask, rects, params)
    dX, dWx, dU, db, dV = mdlstm.units_backward(x, mask, rects, params, caches, dY)
    assert np.all(Y[mask == 0] == 0)

    def loss(p):
        return float(np.sum(mdlstm.units_forward(x, mask, rects, p)[0] * dY * mask[:, :, None]))

    eps = 1e-6
    for idx in [(0, 0, 0), (1, 2, 1), (2, 5, 3), (3, 4, 0), (3, 1, 2)]:
        p = [t.copy() for t in params]
        p[3][idx] += eps
        lp = loss(p)
        p[3][idx] -= 2 * eps
        lm = loss(p)
        assert abs((lp - lm) / (2 * eps) - dV[idx]) <= 1e-6, idx
