"""Plain CPU oracle of the exit-head training of Sec. IV-A (Eq. (22), (23)).

TEST INFRASTRUCTURE ONLY, like the rest of this package.

* the prediction of a representation: the argmax of the model's output
  head (ties to the lower vocabulary index);
* consistency labels b_{q,l} = 1(prediction at layer l == full-depth
  prediction)                                          -- Eq. (22)
* the exit head xi = sigmoid(w . h + c), trained by full-batch gradient
  descent on the binary cross-entropy over the calibration set  -- Eq. (23)

Readings: E1 the model output head is the vocabulary matrix the exit heads
of the synthetic workloads are scaled copies of (its argmax is that of any
positive multiple, so the layer's own vocabulary head gives the same
label); the full-depth prediction is that head on the last layer's output.
E2 training is plain full-batch gradient descent with a fixed step size
from a given start (the paper names only the loss): per epoch
w <- w - lr * mean_q (xi_q - b_q) h_q and c <- c - lr * mean_q (xi_q - b_q),
the exact gradient of Eq. (23).  E3 the reported loss of an epoch is Eq. (23)
at the weights the epoch starts from.
"""
from __future__ import annotations

import numpy as np


def head_argmax(W, H):
    """Per row of H [Q, d]: (argmax_v (W H^T)[v], margin to the runner-up)."""
    W = np.asarray(W, dtype=np.float64)
    H = np.asarray(H, dtype=np.float64)
    z = H @ W.T                                   # [Q, V]
    idx = np.argmax(z, axis=1)                    # first maximum: lower index
    top = z[np.arange(len(idx)), idx]
    z2 = z.copy()
    z2[np.arange(len(idx)), idx] = -np.inf
    margin = top - z2.max(axis=1) if z.shape[1] > 1 else np.full(len(idx), np.inf)
    return idx, margin


def consistency_labels(pred_layer, pred_final):
    """Eq. (22)."""
    return (np.asarray(pred_layer) == np.asarray(pred_final)).astype(np.uint8)


def bce_loss(z, y):
    """Eq. (23) from logits z = w . h + c, in the overflow-free form
    mean(max(z, 0) - y z + log(1 + exp(-|z|)))."""
    z = np.asarray(z, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    return float(np.mean(np.maximum(z, 0.0) - y * z + np.log1p(np.exp(-np.abs(z)))))


def train_exit_head(H, y, epochs: int, lr: float, w0=None, c0: float = 0.0):
    """E2: returns (w [d], c, losses [epochs]) after `epochs` descent steps."""
    H = np.asarray(H, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    Q, d = H.shape
    w = np.zeros(d) if w0 is None else np.array(w0, dtype=np.float64)
    c = float(c0)
    losses = []
    for _ in range(epochs):
        z = H @ w + c
        losses.append(bce_loss(z, y))
        p = 1.0 / (1.0 + np.exp(-z))
        r = p - y
        w = w - lr * (r @ H) / Q
        c = c - lr * float(r.mean())
    return w, c, np.array(losses)
