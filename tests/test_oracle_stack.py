"""Pins for the three-layer stack oracle (Section V-B block-strided
convolutions with tensor-list chunking)."""
import numpy as np

from oracle import mdlstm, stack


def test_block_reshape_channel_order():
    # a 2x4 block (height x width) becomes 8 channels in raster order (dy*4 + dx)
    img = np.arange(2 * 8, dtype=np.float64).reshape(2, 8, 1)
    t = stack.block_reshape(img, 2, 4)
    assert t.shape == (1, 2, 8)
    np.testing.assert_array_equal(t[0, 0], [0, 1, 2, 3, 8, 9, 10, 11])
    np.testing.assert_array_equal(t[0, 1], [4, 5, 6, 7, 12, 13, 14, 15])
    x = np.random.default_rng(0).standard_normal((4, 8, 3))
    np.testing.assert_array_equal(stack.block_unreshape(stack.block_reshape(x, 2, 4), 2, 4, 3), x)


def test_chunked_conv_equals_dense_block_conv():
    # the chunked per-block linear map equals a stride-equals-kernel
    # convolution written as an explicit sum over kernel taps
    rng = np.random.default_rng(1)
    H, og, bh, bw = 3, 2, 2, 4
    y = rng.standard_normal((4, 8, 4 * H))
    W = rng.standard_normal((4, og, bh * bw * H))
    bias = rng.standard_normal((4, og))
    out = stack.grouped_block_conv(y, W, bias, bh, bw)
    for d in range(4):
        for o in range(og):
            for a in range(2):
                for c in range(2):
                    s = bias[d, o]
                    for dy in range(bh):
                        for dx in range(bw):
                            for j in range(H):
                                s += W[d, o, (dy * bw + dx) * H + j] * y[a * bh + dy, c * bw + dx, d * H + j]
                    assert abs(out[a, c, d * og + o] - np.tanh(s)) < 1e-12


def _tiny_stack(rng):
    hidden, conv_out, c_in = (2, 2, 2), (8, 8), (8, 8, 8)
    layers = []
    for C, H in zip(c_in, hidden):
        layers.append((rng.uniform(-0.5, 0.5, (4, 5 * H, C)), rng.uniform(-0.5, 0.5, (4, 5 * H, 2 * H)),
                       rng.uniform(-0.5, 0.5, (4, 5 * H))))
    convs = [(rng.uniform(-0.5, 0.5, (4, co // 4, 8 * H)), rng.uniform(-0.5, 0.5, (4, co // 4)))
             for co, H in zip(conv_out, hidden[:2])]
    return layers, convs


def test_stack_gradients_central_differences():
    rng = np.random.default_rng(2)
    layers, convs = _tiny_stack(rng)
    img = rng.uniform(0, 1, (8, 64))
    Y3, cache = stack.stack_forward(img, layers, convs)
    assert Y3.shape == (1, 1, 8)
    dY3 = rng.standard_normal(Y3.shape)
    lgrads, cgrads, _ = stack.stack_backward(cache, dY3, layers, convs)

    def loss():
        return float(np.sum(stack.stack_forward(img, layers, convs)[0] * dY3))

    eps = 1e-6
    picks = []
    for li in range(3):
        for pi in range(3):
            picks.append((layers[li][pi], lgrads[li][pi]))
    for ci in range(2):
        for pi in range(2):
            picks.append((convs[ci][pi], cgrads[ci][pi]))
    sel = np.random.default_rng(3)
    for arr, grad in picks:
        flat = arr.reshape(-1)
        for i in sel.choice(flat.size, size=min(6, flat.size), replace=False):
            old = flat[i]
            flat[i] = old + eps
            lp = loss()
            flat[i] = old - eps
            lm = loss()
            flat[i] = old
            num = (lp - lm) / (2 * eps)
            assert abs(num - grad.reshape(-1)[i]) <= 1e-6 * max(1.0, abs(num))


def test_stack_layer_is_mdlstm_of_conv_output():
    rng = np.random.default_rng(4)
    layers, convs = _tiny_stack(rng)
    img = rng.uniform(0, 1, (16, 128))
    Y3, cache = stack.stack_forward(img, layers, convs)
    x2 = stack.grouped_block_conv(cache["y"][1], *convs[1], 2, 4)
    np.testing.assert_allclose(Y3, mdlstm.example_forward(x2, layers[2]), rtol=1e-14, atol=1e-15)
