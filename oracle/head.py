"""Output layer and CTC loss — float64 oracle. Test infrastructure only (see
``oracle/__init__.py``).

The model ends in a fully-connected layer shared by the four scan directions
(Section II, Overview: the model follows Pham et al. 2014 except that the last
fully-connected layer is shared across directions; Section V-B treats it as a
block-strided layer with 1 x 1 blocks), followed by the connectionist temporal
classification loss (Section II, item 3).

Readings (the paper gives no formula for either step):

* The shared layer maps every cell's hidden vector of every direction with the
  same weights: o_d(y, x) = W h_d(y, x) + b, W [K][H], b [K].
* The four directions' outputs are summed and the image's height is collapsed
  by summing over its rows, as in the model the paper follows, so an example
  of width w yields w frames of K scores:
      logits[t] = sum_y sum_d (W h_d(y, t) + b),   t = 0 .. w - 1.
* Class 0 is the CTC blank; softmax over the K classes per frame; the loss of
  an example is -ln p(label | example) (Graves et al. 2006), and the loss of a
  batch is the sum over its examples.
"""
from __future__ import annotations

import numpy as np


def fc_collapse_forward(Y, W, b):
    """Y [h, w, 4H] (directions stacked, channel d*H + j) -> logits [w, K]."""
    Y = np.asarray(Y, np.float64)
    W = np.asarray(W, np.float64)
    b = np.asarray(b, np.float64)
    h, w, C4 = Y.shape
    H = C4 // 4
    logits = np.zeros((w, W.shape[0]))
    for d in range(4):
        o = Y[:, :, d * H:(d + 1) * H] @ W.T + b  # [h, w, K]: the shared layer on direction d
        logits += o.sum(axis=0)                   # collapse the rows
    return logits


def fc_collapse_backward(Y, W, dlogits):
    """Gradients of sum(logits * dlogits) for ``fc_collapse_forward``:
    (dY [h, w, 4H], dW [K, H], db [K])."""
    Y = np.asarray(Y, np.float64)
    W = np.asarray(W, np.float64)
    dlogits = np.asarray(dlogits, np.float64)
    h, w, C4 = Y.shape
    H = C4 // 4
    dY = np.zeros_like(Y)
    dW = np.zeros_like(W)
    db = np.zeros(W.shape[0])
    for d in range(4):
        # every row y of column t receives dlogits[t]
        dY[:, :, d * H:(d + 1) * H] = np.broadcast_to(dlogits @ W, (h, w, H))
        dW += np.einsum("tk,ytj->kj", dlogits, Y[:, :, d * H:(d + 1) * H])
        db += h * dlogits.sum(axis=0)
    return dY, dW, db


def log_softmax(z):
    z = np.asarray(z, np.float64)
    m = z.max(axis=-1, keepdims=True)
    return z - m - np.log(np.exp(z - m).sum(axis=-1, keepdims=True))


def _lse(*xs):
    """log(sum(exp(x))) of scalars, -inf for an empty sum."""
    m = max(xs)
    if m == -np.inf:
        return -np.inf
    return m + np.log(sum(np.exp(x - m) for x in xs))


def ctc_loss(logits, label, blank: int = 0):
    """CTC loss of one example (Graves et al. 2006) and its gradient.

    logits [T, K] unnormalised frame scores; label: sequence of class indices
    (none equal to the blank). Written from the forward-backward definition in
    log space: the extended label l' puts a blank before, between and after the
    labels (length S = 2L + 1); alpha_t(s) sums the probabilities of the path
    prefixes that end in l'_s at frame t, beta_t(s) those of the suffixes that
    start there (both include frame t's probability of l'_s). A path may stay on
    l'_s, advance by one, or skip a blank between two different labels.

    Returns (loss = -ln p(label | logits), dloss/dlogits [T, K]).
    """
    lp = log_softmax(logits)
    T, K = lp.shape
    lab = [blank]
    for c in label:
        lab += [int(c), blank]
    S = len(lab)
    neg = -np.inf
    alpha = np.full((T, S), neg)
    alpha[0, 0] = lp[0, lab[0]]
    if S > 1:
        alpha[0, 1] = lp[0, lab[1]]
    for t in range(1, T):
        for s in range(S):
            terms = [alpha[t - 1, s]]
            if s >= 1:
                terms.append(alpha[t - 1, s - 1])
            if s >= 2 and lab[s] != blank and lab[s] != lab[s - 2]:
                terms.append(alpha[t - 1, s - 2])
            alpha[t, s] = _lse(*terms) + lp[t, lab[s]]
    beta = np.full((T, S), neg)
    beta[T - 1, S - 1] = lp[T - 1, lab[S - 1]]
    if S > 1:
        beta[T - 1, S - 2] = lp[T - 1, lab[S - 2]]
    for t in range(T - 2, -1, -1):
        for s in range(S):
            terms = [beta[t + 1, s]]
            if s + 1 < S:
                terms.append(beta[t + 1, s + 1])
            if s + 2 < S and lab[s] != blank and lab[s] != lab[s + 2]:
                terms.append(beta[t + 1, s + 2])
            beta[t, s] = _lse(*terms) + lp[t, lab[s]]
    logp = _lse(alpha[T - 1, S - 1], alpha[T - 1, S - 2]) if S > 1 else alpha[T - 1, S - 1]
    # d(-ln p)/d logits[t, k] = softmax[t, k] - sum_{s: l'_s = k} alpha_t(s) beta_t(s) / (y_t(k) p)
    occ = np.zeros((T, K))
    for t in range(T):
        for s in range(S):
            v = alpha[t, s] + beta[t, s] - lp[t, lab[s]] - logp
            if v > neg:
                occ[t, lab[s]] += np.exp(v)
    grad = np.exp(lp) - occ
    return -logp, grad


def head_loss_forward_backward(Y, W, b, label):
    """Shared layer, row collapse and CTC on one example: (loss, dY, dW, db, logits)."""
    logits = fc_collapse_forward(Y, W, b)
    loss, dlogits = ctc_loss(logits, label)
    dY, dW, db = fc_collapse_backward(Y, W, dlogits)
    return loss, dY, dW, db, logits, dlogits
