"""The temporal module: attention over the w previous states and a GRU update.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Following the "Temporal Graph Learning" paragraph (E12, E13), per node, with
C = [c_0; ...; c_{w-1}] its w previous states (oldest first, each of width d)
and h its spatial embedding at the current snapshot:

    u_k = tanh(Q c_k)            (Q is d x d, applied to the column vector c_k)
    s_k = r . u_k,  a = softmax_k(s),  Ht = sum_k a_k c_k                      (E12)
    H   = GRU(h, Ht)                                                           (E13)

The GRU is the gated recurrent unit with input h and previous hidden state Ht,
in row-vector form with gate order (reset, update, new):

    g_r = h Wi[0] + bi[0] + Ht Wh[0] + bh[0],  r = sigmoid(g_r)
    g_z = h Wi[1] + bi[1] + Ht Wh[1] + bh[1],  z = sigmoid(g_z)
    gh_n = Ht Wh[2] + bh[2],  n = tanh(h Wi[2] + bi[2] + r * gh_n)
    H = (1 - z) * n + z * Ht

With no earlier state (w = 0) Ht = 0: the GRU starts from a zero hidden state.
Backward by the chain rule (written out in `backward`).  Float64 throughout.
"""
from __future__ import annotations

import numpy as np

PARAM_NAMES = ("Q", "r", "Wi", "bi", "Wh", "bh")


def _sig(x):
    return 1.0 / (1.0 + np.exp(-x))


def forward(h, C, p):
    """h [n, d], C [w, n, d], p dict of Q [d, d], r [d], Wi, Wh [3, d, d],
    bi, bh [3, d].  Returns (H, cache)."""
    h = np.asarray(h, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)
    p = {k: np.asarray(v, dtype=np.float64) for k, v in p.items()}
    u = np.tanh(np.einsum("knj,ij->kni", C, p["Q"]))        # u_k = tanh(Q c_k)
    if C.shape[0] == 0:
        a = np.zeros((h.shape[0], 0))
        Ht = np.zeros_like(h)
    else:
        s = np.einsum("kni,i->nk", u, p["r"])
        s = s - s.max(axis=1, keepdims=True)
        a = np.exp(s)
        a /= a.sum(axis=1, keepdims=True)
        Ht = np.einsum("nk,knd->nd", a, C)
    Wi, Wh, bi, bh = p["Wi"], p["Wh"], p["bi"], p["bh"]
    r = _sig(h @ Wi[0] + bi[0] + Ht @ Wh[0] + bh[0])
    z = _sig(h @ Wi[1] + bi[1] + Ht @ Wh[1] + bh[1])
    ghn = Ht @ Wh[2] + bh[2]
    n = np.tanh(h @ Wi[2] + bi[2] + r * ghn)
    H = (1.0 - z) * n + z * Ht
    return H, dict(u=u, a=a, Ht=Ht, r=r, z=z, n=n, ghn=ghn)


def backward(h, C, p, dH):
    """Returns (dh, dC, grads) for the upstream gradient dH = dL/dH."""
    h = np.asarray(h, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)
    dH = np.asarray(dH, dtype=np.float64)
    p = {k: np.asarray(v, dtype=np.float64) for k, v in p.items()}
    _, c = forward(h, C, p)
    u, a, Ht, r, z, n, ghn = c["u"], c["a"], c["Ht"], c["r"], c["z"], c["n"], c["ghn"]
    Wi, Wh = p["Wi"], p["Wh"]
    # GRU
    dn = dH * (1.0 - z)
    dz = dH * (Ht - n)
    dHt = dH * z
    dpn = dn * (1.0 - n * n)            # through tanh
    dghn = dpn * r
    dr = dpn * ghn
    dpr = dr * r * (1.0 - r)            # through the sigmoids
    dpz = dz * z * (1.0 - z)
    dgi = (dpr, dpz, dpn)
    dgh = (dpr, dpz, dghn)
    g = {k: np.zeros_like(v) for k, v in p.items()}
    dh = np.zeros_like(h)
    for k in range(3):
        dh += dgi[k] @ Wi[k].T
        dHt += dgh[k] @ Wh[k].T
        g["Wi"][k] = h.T @ dgi[k]
        g["bi"][k] = dgi[k].sum(axis=0)
        g["Wh"][k] = Ht.T @ dgh[k]
        g["bh"][k] = dgh[k].sum(axis=0)
    # attention: Ht = sum_k a_k c_k, a = softmax(s), s_k = r . u_k, u_k = tanh(Q c_k)
    dC = a.T[:, :, None] * dHt[None, :, :]                  # a_k dHt
    da = np.einsum("nd,knd->nk", dHt, C)
    ds = a * (da - (a * da).sum(axis=1, keepdims=True))
    g["r"] = np.einsum("nk,kni->i", ds, u)
    dpre = ds.T[:, :, None] * p["r"][None, None, :] * (1.0 - u * u)   # [w, n, d]
    dC += np.einsum("kni,ij->knj", dpre, p["Q"])
    g["Q"] = np.einsum("kni,knj->ij", dpre, C)
    return dh, dC, g
