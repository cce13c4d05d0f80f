"""Pins for the oracle's MDLSTM forward (Section III cell, four directions;
Section V masking). Each pin is independent of the oracle's own code path."""
from math import comb

import numpy as np
import pytest
import torch

from conftest import read_fixture
from oracle import mdlstm, pack


def _rand_params(rng, C, H, scale=0.5):
    return (rng.uniform(-scale, scale, (4, 5 * H, C)), rng.uniform(-scale, scale, (4, 5 * H, 2 * H)),
            rng.uniform(-scale, scale, (4, 5 * H)))


def _dir_c(cache, d):
    """Cell state of direction d, mapped back to the example's own frame."""
    return mdlstm._flip(cache["dirs"][d]["c"], d)


def test_hand_worked_2x2():
    rows = read_fixture("cell_2x2.txt")
    x = np.array([[0.0, 1.0], [2.0, 3.0]])[:, :, None]
    H = 1
    wx = np.zeros((4, 5, 1))
    u = np.zeros((4, 5, 2))
    b = np.zeros((4, 5))
    for d in range(4):
        wx[d, 4, 0] = 0.5
        b[d] = [np.log(3.0), -np.log(3.0), 0.0, np.log(4.0), 0.25]
        u[d, 4] = [1.0, -2.0]  # candidate row: +1 * h_L, -2 * h_T
    Y, cache = mdlstm.layer_forward(x, wx, u, b)
    Ys = mdlstm.layer_forward_scalar(x, wx, u, b)
    for r in rows:
        d = int(r[0])
        vals = np.array(list(map(float, r[1:]))).reshape(2, 2, 2)  # (y, x, [h, c])
        np.testing.assert_allclose(Y[:, :, d * H], vals[:, :, 0], rtol=0, atol=1e-14)
        np.testing.assert_allclose(Ys[:, :, d * H], vals[:, :, 0], rtol=0, atol=1e-14)
        np.testing.assert_allclose(_dir_c(cache, d)[:, :, 0], vals[:, :, 1], rtol=0, atol=1e-14)


def _local_coords(h, w, d):
    """(a, b) = number of steps from the scan origin along y and x, per cell."""
    sy, sx = mdlstm._steps(d)
    yy, xx = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
    a = yy if sy == 1 else h - 1 - yy
    bb = xx if sx == 1 else w - 1 - xx
    return a, bb


@pytest.mark.parametrize("d", range(4))
def test_constant_gate_closed_form(d):
    # U = 0 and Wx = 0: every gate is constant, so c(y, x) is a weighted count
    # of monotone lattice paths back to the scan origin:
    #   c = i g sum_{a<=Y, b<=X} C(a+b, a) f_T^a f_L^b
    rng = np.random.default_rng(d)
    h, w, H = 4, 6, 3
    bias = rng.uniform(-1.5, 1.5, (5 * H,))
    wx = np.zeros((4, 5 * H, 2))
    u = np.zeros((4, 5 * H, 2 * H))
    b = np.tile(bias, (4, 1))
    x = rng.standard_normal((h, w, 2))
    Y, cache = mdlstm.layer_forward(x, wx, u, b)
    sig = lambda z: 1.0 / (1.0 + np.exp(-z))  # noqa: E731
    i, fL, fT, o = (sig(bias[k * H:(k + 1) * H]) for k in range(4))
    g = np.tanh(bias[4 * H:])
    A, B = _local_coords(h, w, d)
    c_exp = np.zeros((h, w, H))
    for yy in range(h):
        for xx in range(w):
            s = sum(comb(p + q, p) * fT ** p * fL ** q for p in range(A[yy, xx] + 1) for q in range(B[yy, xx] + 1))
            c_exp[yy, xx] = i * g * s
    np.testing.assert_allclose(_dir_c(cache, d), c_exp, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(Y[:, :, d * H:(d + 1) * H], o * np.tanh(c_exp), rtol=1e-13, atol=1e-15)


def test_unit_forget_binomial_growth():
    # forget gates saturated at exactly 1 (bias 40): c = i g (C(X+Y+2, X+1) - 1),
    # the unbounded growth of the plain MDLSTM state (Section III)
    h, w, H = 7, 9, 2
    bias = np.concatenate([np.full(H, 0.3), np.full(2 * H, 40.0), np.full(H, -0.2), np.full(H, 0.7)])
    assert 1.0 / (1.0 + np.exp(-40.0)) == 1.0
    wx = np.zeros((4, 5 * H, 1))
    u = np.zeros((4, 5 * H, 2 * H))
    b = np.tile(bias, (4, 1))
    Y, cache = mdlstm.layer_forward(np.zeros((h, w, 1)), wx, u, b)
    ig = 1.0 / (1.0 + np.exp(-0.3))
    g = np.tanh(0.7)
    for d in range(4):
        A, B = _local_coords(h, w, d)
        expect = np.array([[ig * g * (comb(A[y, x] + B[y, x] + 2, B[y, x] + 1) - 1) for x in range(w)]
                           for y in range(h)])
        np.testing.assert_allclose(_dir_c(cache, d)[:, :, 0], expect, rtol=1e-13)
        np.testing.assert_allclose(_dir_c(cache, d)[:, :, 1], expect, rtol=1e-13)


def _torch_lstm(xseq, W, U, B, H, use_top):
    """Run torch.nn.LSTM (float64, CPU) with the MDLSTM gates (i, f, g, o) of the
    predecessor that exists in a 1-row / 1-column example."""
    f_rows = slice(2 * H, 3 * H) if use_top else slice(H, 2 * H)
    ucols = slice(H, 2 * H) if use_top else slice(0, H)
    rows = np.r_[0:H, f_rows.start:f_rows.stop, 4 * H:5 * H, 3 * H:4 * H]  # torch gate order i, f, g, o
    lstm = torch.nn.LSTM(W.shape[1], H, batch_first=True).double()
    with torch.no_grad():
        lstm.weight_ih_l0.copy_(torch.from_numpy(W[rows]))
        lstm.weight_hh_l0.copy_(torch.from_numpy(U[rows][:, ucols]))
        lstm.bias_ih_l0.copy_(torch.from_numpy(B[rows]))
        lstm.bias_hh_l0.zero_()
    xt = torch.from_numpy(np.ascontiguousarray(xseq))[None].requires_grad_(True)
    out, _ = lstm(xt)
    return out[0], xt, lstm


@pytest.mark.parametrize("shape", ["row", "col"])
def test_one_row_and_column_equal_torch_lstm(shape):
    rng = np.random.default_rng(11 if shape == "row" else 12)
    H, C, n = 3, 4, 7
    wx, u, b = _rand_params(rng, C, H)
    x = rng.standard_normal((1, n, C)) if shape == "row" else rng.standard_normal((n, 1, C))
    dY = rng.standard_normal(x.shape[:2] + (4 * H,))
    Y, cache = mdlstm.layer_forward(x, wx, u, b)
    dX, dWx, dU, db = mdlstm.layer_backward(cache, dY, wx, u, b)
    dX_t = np.zeros_like(x)
    for d in range(4):
        sy, sx = mdlstm._steps(d)
        step = sx if shape == "row" else sy
        seq = x.reshape(n, C)[::step]
        out, xt, lstm = _torch_lstm(seq, wx[d], u[d], b[d], H, use_top=(shape == "col"))
        ref = out.detach().numpy()[::step]
        np.testing.assert_allclose(Y[:, :, d * H:(d + 1) * H].reshape(n, H), ref, rtol=1e-12, atol=1e-14)
        # backward through autograd: loss = sum(Y_d * dY_d)
        g = torch.from_numpy(np.ascontiguousarray(dY[:, :, d * H:(d + 1) * H].reshape(n, H)[::step]))
        (out * g).sum().backward()
        dX_t += xt.grad[0].numpy()[::step].reshape(x.shape)
        f_rows = np.r_[2 * H:3 * H] if shape == "col" else np.r_[H:2 * H]
        unused = np.r_[H:2 * H] if shape == "col" else np.r_[2 * H:3 * H]
        rows = np.r_[0:H, f_rows, 4 * H:5 * H, 3 * H:4 * H]
        ucols = slice(H, 2 * H) if shape == "col" else slice(0, H)
        np.testing.assert_allclose(dWx[d][rows], lstm.weight_ih_l0.grad.numpy(), rtol=1e-10, atol=1e-13)
        np.testing.assert_allclose(dU[d][rows][:, ucols], lstm.weight_hh_l0.grad.numpy(), rtol=1e-10, atol=1e-13)
        np.testing.assert_allclose(db[d][rows], lstm.bias_ih_l0.grad.numpy(), rtol=1e-10, atol=1e-13)
        # the forget gate of the missing predecessor and its U columns get nothing
        assert np.all(dWx[d][unused] == 0) and np.all(db[d][unused] == 0)
        other = slice(0, H) if shape == "col" else slice(H, 2 * H)
        assert np.all(dU[d][:, other] == 0)
    np.testing.assert_allclose(dX, dX_t, rtol=1e-10, atol=1e-13)


@pytest.mark.parametrize("seed", range(3))
def test_scalar_equals_diagonal(seed):
    rng = np.random.default_rng(100 + seed)
    h, w, C, H = 3 + seed, 5, 2, 3
    params = _rand_params(rng, C, H)
    x = rng.standard_normal((h, w, C))
    valid = rng.random((h, w)) > 0.2
    np.testing.assert_allclose(mdlstm.layer_forward(x, *params, valid=valid)[0],
                               mdlstm.layer_forward_scalar(x, *params, valid=valid), rtol=1e-13, atol=1e-15)


def test_flip_symmetry():
    # mirroring the example left-right and swapping the parameters of the
    # direction pairs (0,1) and (2,3) mirrors the output and swaps its blocks
    rng = np.random.default_rng(7)
    h, w, C, H = 4, 6, 3, 2
    wx, u, b = _rand_params(rng, C, H)
    x = rng.standard_normal((h, w, C))
    perm = [1, 0, 3, 2]
    Y = mdlstm.layer_forward(x, wx, u, b)[0]
    Yf = mdlstm.layer_forward(x[:, ::-1], wx[perm], u[perm], b[perm])[0]
    blocks = np.concatenate([Y[:, ::-1, p * H:(p + 1) * H] for p in perm], axis=2)
    np.testing.assert_allclose(Yf, blocks, rtol=1e-13, atol=1e-15)


def test_packed_canvas_equals_unpacked():
    # Section V: tiling with separating pixels plus masking gives each example
    # exactly the result it has alone. The canvas is scanned as ONE grid per
    # direction with only the mask blocking state, as the paper computes it.
    rng = np.random.default_rng(3)
    hs, ws, cw = [3, 2, 3, 2, 4], [5, 4, 2, 6, 3], 12
    C, H = 2, 3
    params = _rand_params(rng, C, H)
    ex = [rng.standard_normal((h, w, C)) for h, w in zip(hs, ws)]
    rects, ch = pack.pack_layout(hs, ws, cw)
    canvas = pack.scatter(ex, rects, ch, cw, C)
    mask = pack.make_mask(rects, ch, cw)
    Yc = mdlstm.canvas_scan_forward(canvas, mask, params)
    assert np.all(Yc[mask == 0] == 0)
    for got, e in zip(pack.gather(Yc, rects), ex):
        np.testing.assert_allclose(got, mdlstm.example_forward(e, params), rtol=1e-13, atol=1e-15)
    # scheduling units (rectangles) give the same canvas
    Yu, _ = mdlstm.units_forward(canvas, mask, rects, params)
    np.testing.assert_allclose(Yu, Yc, rtol=1e-13, atol=1e-15)


def test_padded_layout_equals_unpacked():
    # last-minute batch padding: tiles of the batch maximum size, no separators,
    # the mask marks each example's true extent
    rng = np.random.default_rng(4)
    hs, ws = [3, 2, 4], [5, 6, 2]
    C, H = 2, 2
    params = _rand_params(rng, C, H)
    ex = [rng.standard_normal((h, w, C)) for h, w in zip(hs, ws)]
    tiles, place, ch, cw = pack.pad_layout(hs, ws)
    canvas = pack.scatter(ex, place, ch, cw, C)
    mask = pack.make_mask(place, ch, cw)
    Y, _ = mdlstm.units_forward(canvas, mask, tiles, params)
    for got, e in zip(pack.gather(Y, place), ex):
        np.testing.assert_allclose(got, mdlstm.example_forward(e, params), rtol=1e-13, atol=1e-15)
    assert np.all(Y[mask == 0] == 0)
