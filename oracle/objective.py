"""The prediction head, the masked BCE loss and the Adam update.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Following the "Prediction and Optimization" subsection:

    a      = H W1 + b1,  hid = ReLU(a)                         (two-layer MLP, E18)
    o      = hid W2 + b2                    (one logit per node)
    p      = sigmoid(o)                     (the predicted probability)
    L_BCE  = -(1/N_m) sum_{labelled i} [y_i log p_i + (1 - y_i) log(1 - p_i)]   (E19)
    L      = L_BCE + lambda_CCA L_CCA                                            (E20)

with y in {0, 1} on the labelled nodes (label -1 marks an unlabelled node).
The BCE of a logit is evaluated as softplus(o) - y o, and its gradient is
dL/do_i = (p_i - y_i) / N_m on labelled rows, 0 elsewhere.  Backward:

    dhid = dL/do W2^T,  da = dhid * 1[a > 0]
    dW2 = hid^T dL/do,  db2 = sum dL/do,  dW1 = H^T da,  db1 = sum da,  dH = da W1^T

Adam (the optimiser the paper names, with its weight decay added to the
gradient, first and second moments with bias correction):

    g = grad + wd * theta;  m = b1 m + (1 - b1) g;  v = b2 v + (1 - b2) g^2
    theta -= lr * (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps)

Everything is float64.
"""
from __future__ import annotations

import numpy as np


def mlp_bce(H, W1, b1, W2, b2, labels):
    """Returns (loss, dH, dW1, db1, dW2, db2, mask) in float64; W2 is [d_h, 1],
    b2 [1]; mask is the ReLU decision of the hidden layer."""
    H = np.asarray(H, dtype=np.float64)
    W1, b1 = np.asarray(W1, dtype=np.float64), np.asarray(b1, dtype=np.float64)
    W2, b2 = np.asarray(W2, dtype=np.float64), np.asarray(b2, dtype=np.float64)
    labels = np.asarray(labels)
    a = H @ W1 + b1
    mask = a > 0
    hid = np.where(mask, a, 0.0)
    o = (hid @ W2 + b2)[:, 0]
    lab = labels >= 0
    n_m = int(lab.sum())
    y = np.where(lab, labels, 0).astype(np.float64)
    if n_m == 0:
        loss = 0.0
        do = np.zeros_like(o)
    else:
        sp = np.logaddexp(0.0, o)                        # softplus(o) = -log(1 - p)
        loss = float(((sp - y * o) * lab).sum() / n_m)
        p = 1.0 / (1.0 + np.exp(-o))
        do = np.where(lab, (p - y) / n_m, 0.0)
    dW2 = hid.T @ do[:, None]
    db2 = np.array([do.sum()])
    da = (do[:, None] * W2[:, 0][None, :]) * mask
    dW1 = H.T @ da
    db1 = da.sum(axis=0)
    dH = da @ W1.T
    return loss, dH, dW1, db1, dW2, db2, mask


def adam_step(theta, grad, m, v, t, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-5):
    """One update of step number t >= 1; returns (theta, m, v), float64."""
    theta = np.asarray(theta, dtype=np.float64)
    g = np.asarray(grad, dtype=np.float64) + weight_decay * theta
    m = beta1 * np.asarray(m, dtype=np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, dtype=np.float64) + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** t)
    vhat = v / (1.0 - beta2 ** t)
    return theta - lr * mhat / (np.sqrt(vhat) + eps), m, v
