"""Cross-subgraph CCA consistency-alignment loss and its gradient.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Follows the "Cross-Subgraph Consistency Alignment" section: each view is
standardised per feature column over the overlap batch B (zero mean,
standard deviation 1/sqrt(|B|)), then

    L_inv = sum_b w_b ||Xh_b - Yh_b||^2        (w = 1 gives the paper's Frobenius form)
    L_dec = ||Xh^T Xh - I||_F^2 + ||Yh^T Yh - I||_F^2
    L     = L_inv + lambda_n L_dec

with Xh = (X - mu) / (sigma sqrt(M)), sigma = sqrt(var + eps), var with
divisor M - ddof.  X = H[overlap] is the local view, Y = H_ref the other
subgraph's view.  The returned gradients are scale * dL/dX and
scale * dL/dY (scale = lambda_CCA of the joint objective).  float64.
"""
from __future__ import annotations

import numpy as np


def standardise(V: np.ndarray, eps: float, ddof: int):
    m = V.shape[0]
    mu = V.mean(axis=0)
    var = ((V - mu) ** 2).sum(axis=0) / (m - ddof)
    sd = np.sqrt(var + eps)
    vt = (V - mu) / sd
    return vt / np.sqrt(m), vt, sd


def standardise_backward(g_hat: np.ndarray, vt: np.ndarray, sd: np.ndarray, ddof: int) -> np.ndarray:
    """Gradient w.r.t. V given the gradient w.r.t. Vh = vt / sqrt(M)."""
    m = g_hat.shape[0]
    g = g_hat / np.sqrt(m)                       # gradient w.r.t. vt
    return (g - g.mean(axis=0) - vt * (g * vt).sum(axis=0) / (m - ddof)) / sd


def loss_and_grad(X, Y, omega=None, lambda_n=2e-4, scale=0.1, eps=1e-5, ddof=0):
    """Returns ((L_inv, L_dec, L), dX, dY) with dX = scale*dL/dX, dY = scale*dL/dY."""
    X = np.asarray(X, dtype=np.float64)
    Y = np.asarray(Y, dtype=np.float64)
    m, d = X.shape
    if m == 0:
        return (0.0, 0.0, 0.0), np.zeros_like(X), np.zeros_like(Y)
    w = np.ones(m) if omega is None else np.asarray(omega, dtype=np.float64)
    xh, xt, sx = standardise(X, eps, ddof)
    yh, yt, sy = standardise(Y, eps, ddof)
    diff = xh - yh
    l_inv = float((w[:, None] * diff ** 2).sum())
    eye = np.eye(d)
    cx = xh.T @ xh - eye
    cy = yh.T @ yh - eye
    l_dec = float((cx ** 2).sum() + (cy ** 2).sum())
    loss = l_inv + lambda_n * l_dec
    gx = 2.0 * w[:, None] * diff + 4.0 * lambda_n * (xh @ cx)
    gy = -2.0 * w[:, None] * diff + 4.0 * lambda_n * (yh @ cy)
    dX = scale * standardise_backward(gx, xt, sx, ddof)
    dY = scale * standardise_backward(gy, yt, sy, ddof)
    return (l_inv, l_dec, loss), dX, dY
