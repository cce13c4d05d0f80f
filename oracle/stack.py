"""Three-layer MDLSTM stack with block-strided convolutions — float64 oracle.

Test infrastructure only (see ``oracle/__init__.py``).

Section V-B: a block-strided convolution has stride equal to its kernel, so
kernel applications never overlap. Tensor-list chunking cuts every example
into blocks of the stride size and stacks the blocks; the convolution is then
a per-block linear map, and de-chunking reassembles each example. The paper
states the chunked result equals computing each example separately, so this
oracle computes each example separately.

Readings: block sizes are height x width (Fig. 1 caption); a block's channel
index is (dy * bw + dx) * C + c; the convolution between MDLSTM layers has one
group per scan direction (group d reads the bh*bw*H channels of direction d's
block and writes out/4 channels, the groups concatenated in direction order),
followed by tanh.
"""
from __future__ import annotations

import numpy as np

from . import mdlstm


def block_reshape(x, bh: int, bw: int):
    """[h, w, C] -> [h/bh, w/bw, bh*bw*C], channel (dy*bw + dx)*C + c."""
    x = np.asarray(x)
    h, w, C = x.shape
    assert h % bh == 0 and w % bw == 0
    t = x.reshape(h // bh, bh, w // bw, bw, C).transpose(0, 2, 1, 3, 4)
    return t.reshape(h // bh, w // bw, bh * bw * C)


def block_unreshape(t, bh: int, bw: int, C: int):
    """Inverse of ``block_reshape``."""
    hb, wb, _ = t.shape
    return t.reshape(hb, wb, bh, bw, C).transpose(0, 2, 1, 3, 4).reshape(hb * bh, wb * bw, C)


def grouped_block_conv(y, W, bias, bh: int, bw: int):
    """y [h, w, 4H]; W [4, og, bh*bw*H]; bias [4, og] -> tanh output [h/bh, w/bw, 4*og]."""
    y = np.asarray(y, np.float64)
    H = y.shape[2] // 4
    outs = []
    for d in range(4):
        blk = block_reshape(y[:, :, d * H:(d + 1) * H], bh, bw)
        outs.append(blk @ np.asarray(W[d], np.float64).T + np.asarray(bias[d], np.float64))
    return np.tanh(np.concatenate(outs, axis=2))


def grouped_block_conv_backward(y, W, out, dout, bh: int, bw: int):
    """Gradients of sum(out * dout) w.r.t. (y, W, bias)."""
    y = np.asarray(y, np.float64)
    H = y.shape[2] // 4
    og = W.shape[1]
    dpre = np.asarray(dout, np.float64) * (1.0 - out * out)
    dy = np.zeros_like(y)
    dW = np.zeros(W.shape)
    db = np.zeros((4, og))
    for d in range(4):
        blk = block_reshape(y[:, :, d * H:(d + 1) * H], bh, bw)
        g = dpre[:, :, d * og:(d + 1) * og]
        dW[d] = np.einsum("abo,abk->ok", g, blk)
        db[d] = g.sum(axis=(0, 1))
        dblk = g @ np.asarray(W[d], np.float64)
        dy[:, :, d * H:(d + 1) * H] = block_unreshape(dblk, bh, bw, H)
    return dy, dW, db


def stack_forward(image, layers, convs, block=(2, 4)):
    """One example: image [h, w] -> (Y3, cache)."""
    bh, bw = block
    x = block_reshape(np.asarray(image, np.float64)[:, :, None], bh, bw)
    cache = {"x": [x], "lc": [], "y": [], "conv_out": []}
    for li, (wx, u, b) in enumerate(layers):
        Y, lc = mdlstm.layer_forward(x, wx, u, b)
        cache["lc"].append(lc)
        cache["y"].append(Y)
        if li < len(convs):
            W, cb = convs[li]
            x = grouped_block_conv(Y, W, cb, bh, bw)
            cache["conv_out"].append(x)
            cache["x"].append(x)
    return cache["y"][-1], cache


def stack_backward(cache, dY3, layers, convs, block=(2, 4)):
    """Returns ([(dWx, dU, db) per layer], [(dW, db) per conv], d_input_blocks)."""
    bh, bw = block
    g = np.asarray(dY3, np.float64)
    lgrads = [None] * len(layers)
    cgrads = [None] * len(convs)
    for li in range(len(layers) - 1, -1, -1):
        wx, u, b = layers[li]
        dX, dWx, dU, db = mdlstm.layer_backward(cache["lc"][li], g, wx, u, b)
        lgrads[li] = (dWx, dU, db)
        if li > 0:
            W, _ = convs[li - 1]
            g, dW, dcb = grouped_block_conv_backward(cache["y"][li - 1], W, cache["conv_out"][li - 1],
                                                     dX, bh, bw)
            cgrads[li - 1] = (dW, dcb)
        else:
            g = dX
    return lgrads, cgrads, g
