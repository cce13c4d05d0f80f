"""Four-direction 2D MDLSTM layer, forward and backward — float64 oracle.

Test infrastructure only (see ``oracle/__init__.py``).

The cell (Section III; the paper draws it in Fig. 3a and prints no equations,
so the standard two-predecessor MDLSTM it builds on is written out here):
each cell has two predecessors in the scan direction, the left one L and the
top one T, each handing over a (hidden, state) pair. Five pre-activations are
formed from the cell input and both predecessor hidden states (Section IV-B:
input node, input gate, two forget gates, output gate):

    a   = Wx x + b + U [h_L ; h_T]            (5H rows: i, f_L, f_T, o, g)
    i = sig(a_i), f_L = sig(a_fL), f_T = sig(a_fT), o = sig(a_o), g = tanh(a_g)
    c   = i*g + f_L*c_L + f_T*c_T             (the two forget gates weigh the
                                               two predecessor states)
    h   = o * tanh(c)

A predecessor that lies outside the example or is masked out hands over
zeros (Section V: binary masking blocks the hidden and memory state of
invalid predecessors); a masked cell outputs h = c = 0.

Memory-state matrices (Appendix A: besides the five matrices per predecessor
hidden state, three per predecessor memory state S1 = c_L and S2 = c_T, whose
products are summed with the hidden-state ones). Reading: both memory states
feed the same three gates, the input gate and the two forget gates (the gates
that decide what enters and what stays in the new state), through full
H x H matrices:

    a[i, f_L, f_T] += V [c_L ; c_T]           (V: 3H x 2H, per direction)

The output gate and the cell candidate take no memory state. Passing no V
(the default) is the plain cell above; V = 0 gives the same values.

Four directions (Section III): one MDLSTM per scan origin, outputs stacked
along channels as [Y_0 | Y_1 | Y_2 | Y_3]. Direction 0 scans from the
top-left (L = (y, x-1), T = (y-1, x)), 1 from the top-right (L = (y, x+1),
T = (y-1, x)), 2 from the bottom-left (L = (y, x-1), T = (y+1, x)), 3 from the
bottom-right (L = (y, x+1), T = (y+1, x)).

Two independent forms are provided and checked against each other: a scalar
per-cell loop with explicit predecessor offsets, and a flip-to-direction-0
form that walks anti-diagonals (the order the input-skewing trick of
Section IV-A exposes).
"""
from __future__ import annotations

import numpy as np


def sigmoid(z):
    z = np.asarray(z, dtype=np.float64)
    out = np.empty_like(z)
    pos = z >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-z[pos]))
    ez = np.exp(z[~pos])
    out[~pos] = ez / (1.0 + ez)
    return out


def _steps(d: int):
    """Scan steps (sy, sx) of direction d: +1 means the scan moves down / right."""
    sx = 1 if d in (0, 2) else -1
    sy = 1 if d in (0, 1) else -1
    return sy, sx


def _flip(a, d: int):
    """Map direction d's frame to direction 0's frame (an involution)."""
    if d in (1, 3):
        a = a[:, ::-1]
    if d in (2, 3):
        a = a[::-1]
    return a


# ----------------------------------------------------------------------------
# Scalar form: per-cell loop, explicit predecessor offsets per direction.
# ----------------------------------------------------------------------------

def layer_forward_scalar(x, wx, u, b, valid=None, v=None):
    """x [h, w, C]; wx [4, 5H, C]; u [4, 5H, 2H]; b [4, 5H]; optional memory-state
    matrices v [4, 3H, 2H] -> Y [h, w, 4H]."""
    x = np.asarray(x, np.float64)
    h, w, _ = x.shape
    H = u.shape[2] // 2
    valid = np.ones((h, w), bool) if valid is None else np.asarray(valid, bool)
    Y = np.zeros((h, w, 4 * H))
    zero = np.zeros(H)
    for d in range(4):
        sy, sx = _steps(d)
        W, U, B = (np.asarray(t[d], np.float64) for t in (wx, u, b))
        V = None if v is None else np.asarray(v[d], np.float64)
        hh = np.zeros((h, w, H))
        cc = np.zeros((h, w, H))
        for yy in (range(h) if sy == 1 else range(h - 1, -1, -1)):
            for xx in (range(w) if sx == 1 else range(w - 1, -1, -1)):
                if not valid[yy, xx]:
                    continue
                lx, ty = xx - sx, yy - sy
                hL, cL = (hh[yy, lx], cc[yy, lx]) if 0 <= lx < w else (zero, zero)
                hT, cT = (hh[ty, xx], cc[ty, xx]) if 0 <= ty < h else (zero, zero)
                a = W @ x[yy, xx] + B + U @ np.concatenate([hL, hT])
                if V is not None:
                    a[0:3 * H] += V @ np.concatenate([cL, cT])
                ig = sigmoid(a[0:H])
                fL = sigmoid(a[H:2 * H])
                fT = sigmoid(a[2 * H:3 * H])
                og = sigmoid(a[3 * H:4 * H])
                gg = np.tanh(a[4 * H:5 * H])
                c = ig * gg + fL * cL + fT * cT
                cc[yy, xx] = c
                hh[yy, xx] = og * np.tanh(c)
        Y[:, :, d * H:(d + 1) * H] = hh
    return Y


# ----------------------------------------------------------------------------
# Diagonal form in direction 0's frame.
# ----------------------------------------------------------------------------

def scan_forward(z, valid, U, V=None):
    """Direction-0 scan. z [h, w, 5H] = Wx x + b; valid [h, w] bool; U [5H, 2H];
    V [3H, 2H] memory-state matrices or None.

    Returns a cache dict with h, c, activated gates, and the predecessor
    states actually used (zeros where the predecessor is outside or invalid).
    """
    h, w, G = z.shape
    H = G // 5
    # state arrays with one zero row above and one zero column to the left
    hs = np.zeros((h + 1, w + 1, H))
    cs = np.zeros((h + 1, w + 1, H))
    gates = np.zeros((h, w, 5, H))
    hL = np.zeros((h, w, H))
    hT = np.zeros((h, w, H))
    cL = np.zeros((h, w, H))
    cT = np.zeros((h, w, H))
    for s in range(h + w - 1):
        y = np.arange(max(0, s - w + 1), min(h, s + 1))
        x = s - y
        hl, ht = hs[y + 1, x], hs[y, x + 1]
        cl, ct = cs[y + 1, x], cs[y, x + 1]
        a = z[y, x] + np.concatenate([hl, ht], axis=1) @ U.T
        if V is not None:
            a[:, 0:3 * H] += np.concatenate([cl, ct], axis=1) @ V.T
        ig = sigmoid(a[:, 0:H])
        fL = sigmoid(a[:, H:2 * H])
        fT = sigmoid(a[:, 2 * H:3 * H])
        og = sigmoid(a[:, 3 * H:4 * H])
        gg = np.tanh(a[:, 4 * H:5 * H])
        c = ig * gg + fL * cl + fT * ct
        hn = og * np.tanh(c)
        v = valid[y, x][:, None]
        hs[y + 1, x + 1] = np.where(v, hn, 0.0)
        cs[y + 1, x + 1] = np.where(v, c, 0.0)
        gates[y, x] = np.stack([ig, fL, fT, og, gg], axis=1)
        hL[y, x], hT[y, x], cL[y, x], cT[y, x] = hl, ht, cl, ct
    return {"h": hs[1:, 1:].copy(), "c": cs[1:, 1:].copy(), "gates": gates,
            "hL": hL, "hT": hT, "cL": cL, "cT": cT, "valid": valid}


def scan_backward(cache, dh_out, U, V=None):
    """Reverse-diagonal backward of ``scan_forward``. Returns dz [h, w, 5H]
    (gradient of the pre-activations) for upstream gradient dh_out [h, w, H].
    With memory-state matrices V, a predecessor's state also receives
    V^T da[i, f_L, f_T] (its c_L or c_T half)."""
    gates, c_all, valid = cache["gates"], cache["c"], cache["valid"]
    h, w, _, H = gates.shape
    # accumulators for gradient arriving from successors, with one sink row
    # and column (index 0) for predecessors that lie outside the example
    dh_acc = np.zeros((h + 1, w + 1, H))
    dc_acc = np.zeros((h + 1, w + 1, H))
    dz = np.zeros((h, w, 5 * H))
    for s in range(h + w - 2, -1, -1):
        y = np.arange(max(0, s - w + 1), min(h, s + 1))
        x = s - y
        ig, fL, fT, og, gg = (gates[y, x, k] for k in range(5))
        tc = np.tanh(c_all[y, x])
        v = valid[y, x][:, None]
        dh = np.where(v, dh_out[y, x] + dh_acc[y + 1, x + 1], 0.0)
        dc = np.where(v, dc_acc[y + 1, x + 1] + dh * og * (1.0 - tc * tc), 0.0)
        da = np.concatenate([
            dc * gg * ig * (1.0 - ig),
            dc * cache["cL"][y, x] * fL * (1.0 - fL),
            dc * cache["cT"][y, x] * fT * (1.0 - fT),
            dh * tc * og * (1.0 - og),
            dc * ig * (1.0 - gg * gg),
        ], axis=1)
        dz[y, x] = da
        back = da @ U
        backc = da[:, 0:3 * H] @ V if V is not None else np.zeros((len(y), 2 * H))
        dh_acc[y + 1, x] += back[:, :H]      # to the left predecessor (y, x-1)
        dc_acc[y + 1, x] += dc * fL + backc[:, :H]
        dh_acc[y, x + 1] += back[:, H:]      # to the top predecessor (y-1, x)
        dc_acc[y, x + 1] += dc * fT + backc[:, H:]
    return dz


def layer_forward(x, wx, u, b, valid=None, v=None):
    """Four-direction layer on one example (memory-state matrices v [4, 3H, 2H]
    optional). Returns (Y [h, w, 4H], cache)."""
    x = np.asarray(x, np.float64)
    h, w, _ = x.shape
    H = u.shape[2] // 2
    valid = np.ones((h, w), bool) if valid is None else np.asarray(valid, bool)
    Y = np.zeros((h, w, 4 * H))
    caches = []
    for d in range(4):
        W, U, B = (np.asarray(t[d], np.float64) for t in (wx, u, b))
        V = None if v is None else np.asarray(v[d], np.float64)
        z = _flip(x, d) @ W.T + B
        cd = scan_forward(z, _flip(valid, d), U, V)
        Y[:, :, d * H:(d + 1) * H] = _flip(cd["h"], d)
        caches.append(cd)
    return Y, {"x": x, "dirs": caches, "H": H}


def layer_backward(cache, dY, wx, u, b, v=None):
    """Gradients of sum(Y * dY) for ``layer_forward``: (dX, dWx, dU, db), all
    float64, and dV as a fifth entry when memory-state matrices v were used.
    Weight gradients are sums over every cell (not means)."""
    x = cache["x"]
    H = cache["H"]
    dY = np.asarray(dY, np.float64)
    dX = np.zeros_like(x)
    dWx = np.zeros((4, 5 * H, x.shape[2]))
    dU = np.zeros((4, 5 * H, 2 * H))
    db = np.zeros((4, 5 * H))
    dV = None if v is None else np.zeros((4, 3 * H, 2 * H))
    for d in range(4):
        cd = cache["dirs"][d]
        U = np.asarray(u[d], np.float64)
        V = None if v is None else np.asarray(v[d], np.float64)
        dz = scan_backward(cd, _flip(dY[:, :, d * H:(d + 1) * H], d), U, V)
        xf = _flip(x, d)
        dWx[d] = np.einsum("ywr,ywk->rk", dz, xf)
        db[d] = dz.sum(axis=(0, 1))
        hcat = np.concatenate([cd["hL"], cd["hT"]], axis=2)
        dU[d] = np.einsum("ywr,ywk->rk", dz, hcat)
        if V is not None:
            ccat = np.concatenate([cd["cL"], cd["cT"]], axis=2)
            dV[d] = np.einsum("ywr,ywk->rk", dz[:, :, 0:3 * H], ccat)
        dX += _flip(dz @ np.asarray(wx[d], np.float64), d)
    if v is not None:
        return dX, dWx, dU, db, dV
    return dX, dWx, dU, db


def example_forward(x, params):
    """Y of one example computed alone (all cells valid)."""
    wx, u, b = params
    return layer_forward(x, wx, u, b)[0]


def example_backward(x, params, dY):
    wx, u, b = params
    _, cache = layer_forward(x, wx, u, b)
    return layer_backward(cache, dY, wx, u, b)


# ----------------------------------------------------------------------------
# Canvas forms.
# ----------------------------------------------------------------------------

def canvas_scan_forward(canvas_x, mask, params):
    """The paper's packed computation: one scan over the whole canvas in each
    direction, the binary mask alone blocking state from invalid cells."""
    wx, u, b = params
    return layer_forward(canvas_x, wx, u, b, valid=np.asarray(mask, bool))[0]


def units_forward(canvas_x, mask, rects, params):
    """Canvas forward with scheduling rectangles: the recurrence restarts at
    every rectangle edge and at every masked cell; cells outside every
    rectangle output zero. params: (wx, u, b) or (wx, u, b, v).
    Returns (Y [H_c, W_c, 4H], caches)."""
    wx, u, b = params[:3]
    v = params[3] if len(params) > 3 else None
    canvas_x = np.asarray(canvas_x, np.float64)
    Hc, Wc, _ = canvas_x.shape
    H = u.shape[2] // 2
    mask = np.asarray(mask, bool)
    Y = np.zeros((Hc, Wc, 4 * H))
    caches = []
    for y0, x0, h, w in np.asarray(rects).reshape(-1, 4):
        win = (slice(y0, y0 + h), slice(x0, x0 + w))
        Yr, cr = layer_forward(canvas_x[win], wx, u, b, valid=mask[win], v=v)
        Y[win] = Yr
        caches.append(cr)
    return Y, caches


def units_backward(canvas_x, mask, rects, params, caches, dY):
    """Backward of ``units_forward``: (dX canvas, dWx, dU, db[, dV]); dY is
    ignored where the mask is 0 or outside every rectangle."""
    wx, u, b = params[:3]
    v = params[3] if len(params) > 3 else None
    canvas_x = np.asarray(canvas_x, np.float64)
    H = u.shape[2] // 2
    mask = np.asarray(mask, bool)
    dY = np.asarray(dY, np.float64)
    dX = np.zeros_like(canvas_x)
    dWx = np.zeros((4, 5 * H, canvas_x.shape[2]))
    dU = np.zeros((4, 5 * H, 2 * H))
    db = np.zeros((4, 5 * H))
    dV = None if v is None else np.zeros((4, 3 * H, 2 * H))
    for (y0, x0, h, w), cr in zip(np.asarray(rects).reshape(-1, 4), caches):
        win = (slice(y0, y0 + h), slice(x0, x0 + w))
        g = dY[win] * mask[win][:, :, None]
        grads = layer_backward(cr, g, wx, u, b, v)
        a, bw, cu, cb = grads[:4]
        dX[win] = a * mask[win][:, :, None]
        dWx += bw
        dU += cu
        db += cb
        if v is not None:
            dV += grads[4]
    if v is not None:
        return dX, dWx, dU, db, dV
    return dX, dWx, dU, db
