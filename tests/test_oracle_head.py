"""Pins of the output-layer and CTC oracle (oracle/head.py) against what the
paper and the mathematics fix, independent of its own code: hand-worked CTC
cases, brute-force enumeration of every frame path, PyTorch's CTC loss in
float64 (a library special case), finite differences and the adjoint
identity, and the shared layer's closed forms."""
import itertools

import numpy as np
import pytest

from conftest import read_fixture
from oracle import head


def _softmax(z):
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def _collapse(path, blank=0):
    out, prev = [], None
    for c in path:
        if c != prev and c != blank:
            out.append(c)
        prev = c
    return tuple(out)


def test_ctc_hand_worked_cases():
    rows = read_fixture("ctc_hand.txt")
    assert len(rows) == 4
    for name, T, K, lab, scores, loss, grad in rows:
        T, K = int(T), int(K)
        label = [] if lab == "-" else [int(v) for v in lab.split(",")]
        z = np.array([float(v) for v in scores.split(",")]).reshape(T, K)
        got_loss, got_grad = head.ctc_loss(z, label)
        assert abs(got_loss - float(loss)) <= 1e-14 * max(1.0, float(loss)), name
        want = np.array([float(v) for v in grad.split(",")]).reshape(T, K)
        assert np.max(np.abs(got_grad - want)) <= 1e-14, name


@pytest.mark.parametrize("T,K,label", [(4, 3, [1]), (4, 3, [1, 1]), (5, 3, [2, 1, 2]), (5, 3, [1, 1, 2]),
                                       (4, 3, []), (5, 4, [3, 3]), (3, 3, [1, 2, 1]), (6, 3, [2, 2, 2])])
def test_ctc_against_brute_force_paths(T, K, label):
    """p(label) summed over all K^T frame paths that collapse to it."""
    rng = np.random.default_rng(T * 100 + K * 10 + len(label))
    z = rng.standard_normal((T, K)) * 1.5
    y = _softmax(z)
    p = 0.0
    occ = np.zeros((T, K))
    for path in itertools.product(range(K), repeat=T):
        if _collapse(path) == tuple(label):
            pp = float(np.prod([y[t, c] for t, c in enumerate(path)]))
            p += pp
            for t, c in enumerate(path):
                occ[t, c] += pp
    loss, grad = head.ctc_loss(z, label)
    assert p > 0
    assert abs(loss - (-np.log(p))) <= 1e-12 * max(1.0, abs(loss))
    assert np.max(np.abs(grad - (y - occ / p))) <= 1e-12


def test_ctc_against_torch_float64():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(3)
    for T, K, L in [(12, 6, 4), (30, 10, 9), (7, 5, 3), (20, 4, 8)]:
        label = rng.integers(1, K, L)
        label[1] = label[0]  # a repeat
        z = rng.standard_normal((T, K))
        zt = torch.tensor(z, dtype=torch.float64, requires_grad=True)
        lp = torch.log_softmax(zt, dim=-1)[:, None, :]
        ref = torch.nn.functional.ctc_loss(lp, torch.tensor(label[None, :]), torch.tensor([T]), torch.tensor([L]),
                                           blank=0, reduction="sum")
        ref.backward()
        loss, grad = head.ctc_loss(z, label)
        assert abs(loss - ref.item()) <= 1e-10 * abs(ref.item())
        assert np.max(np.abs(grad - zt.grad.numpy())) <= 1e-10


def test_ctc_gradient_finite_differences():
    rng = np.random.default_rng(5)
    z = rng.standard_normal((9, 5))
    label = [2, 2, 4, 1]
    _, grad = head.ctc_loss(z, label)
    eps = 1e-6
    for t, k in [(0, 0), (0, 2), (3, 4), (5, 2), (8, 1), (8, 0), (4, 3)]:
        zp, zm = z.copy(), z.copy()
        zp[t, k] += eps
        zm[t, k] -= eps
        fd = (head.ctc_loss(zp, label)[0] - head.ctc_loss(zm, label)[0]) / (2 * eps)
        assert abs(fd - grad[t, k]) <= 1e-7, (t, k)


def test_shared_layer_closed_forms():
    rng = np.random.default_rng(7)
    h, w, H, K = 3, 5, 4, 6
    W, b = rng.standard_normal((K, H)), rng.standard_normal(K)
    # zero hidden states: every frame is the bias counted once per row and direction
    z = head.fc_collapse_forward(np.zeros((h, w, 4 * H)), W, b)
    assert np.array_equal(z, np.broadcast_to(4 * h * b, (w, K)))
    # the layer is shared: permuting the directions changes nothing
    Y = rng.standard_normal((h, w, 4 * H))
    perm = np.concatenate([Y[:, :, d * H:(d + 1) * H] for d in (2, 0, 3, 1)], axis=2)
    assert np.allclose(head.fc_collapse_forward(Y, W, b), head.fc_collapse_forward(perm, W, b), rtol=0, atol=1e-12)
    # one nonzero cell of one direction reaches only its own frame, as W h
    Y1 = np.zeros((h, w, 4 * H))
    Y1[1, 3, 2 * H:3 * H] = rng.standard_normal(H)
    z1 = head.fc_collapse_forward(Y1, W, np.zeros(K))
    assert np.allclose(z1[3], W @ Y1[1, 3, 2 * H:3 * H], rtol=0, atol=1e-12)
    assert np.all(z1[[0, 1, 2, 4]] == 0)


def test_shared_layer_adjoint_and_finite_differences():
    rng = np.random.default_rng(9)
    h, w, H, K = 2, 4, 3, 5
    Y, W, b = rng.standard_normal((h, w, 4 * H)), rng.standard_normal((K, H)), rng.standard_normal(K)
    g = rng.standard_normal((w, K))
    dY, dW, db = head.fc_collapse_backward(Y, W, g)
    # the map Y -> logits is affine: <g, J v> = <J^T g, v>
    v = rng.standard_normal(Y.shape)
    jv = head.fc_collapse_forward(Y + v, W, b) - head.fc_collapse_forward(Y, W, b)
    assert abs(np.sum(g * jv) - np.sum(dY * v)) <= 1e-10
    eps = 1e-6
    for (k, j) in [(0, 0), (4, 2), (2, 1)]:
        Wp, Wm = W.copy(), W.copy()
        Wp[k, j] += eps
        Wm[k, j] -= eps
        fd = (np.sum(g * head.fc_collapse_forward(Y, Wp, b)) - np.sum(g * head.fc_collapse_forward(Y, Wm, b))) / (2 * eps)
        assert abs(fd - dW[k, j]) <= 1e-7
    for k in range(K):
        bp, bm = b.copy(), b.copy()
        bp[k] += eps
        bm[k] -= eps
        fd = (np.sum(g * head.fc_collapse_forward(Y, W, bp)) - np.sum(g * head.fc_collapse_forward(Y, W, bm))) / (2 * eps)
        assert abs(fd - db[k]) <= 1e-7


def test_shared_layer_against_torch_linear():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(11)
    h, w, H, K = 4, 7, 8, 10
    Y, W, b = rng.standard_normal((h, w, 4 * H)), rng.standard_normal((K, H)), rng.standard_normal(K)
    t = torch.tensor(Y).reshape(h, w, 4, H)
    ref = torch.nn.functional.linear(t, torch.tensor(W), torch.tensor(b)).sum(dim=(0, 2)).numpy()
    assert np.allclose(head.fc_collapse_forward(Y, W, b), ref, rtol=1e-13, atol=1e-12)
