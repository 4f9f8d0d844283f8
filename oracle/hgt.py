"""One heterogeneous-graph-transformer (attention) layer, forward and backward.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Forward, following the equations of the "Heterogeneous Graph Transformer"
paragraph (E6-E11), for an edge e = (i -> j) of relation r = phi(e), S heads
of width dk = d / S, head slices written x^s:

    K = H W_K[type] + b_K[type],  Q = H W_Q[type] + b_Q[type],
    V = H W_V[type] + b_V[type]                        (per-type Linear maps)
    score^s(e) = (K^s_i W_att[r, s]) . Q^s_j * mu[type(i), r, type(j)] / sqrt(dk)  (E6)
    msg^s(e)   = V^s_i W_msg[r, s]                                                 (E7)
    alpha^s(e) = softmax over the in-edges e' of j (all relations) of score^s(e')  (E8)
    h~_j       = concat_s sum_{e into j} alpha^s(e) msg^s(e)   (0 without in-edges) (E9, E10)
    z_j        = h~_j W_agg[type(j)] + b_agg[type(j)]
    h'_j       = ReLU(z_j) + h_j                                                    (E11)

W_att and W_msg are per relation and head ([R, S, dk, dk]); mu is one scalar per
meta relation (source type, relation, destination type), shared by the heads.
V has its own per-type projection; passing W_V = W_K, b_V = b_K gives the
reading in which the message reuses the key projection.

Backward (chain rule, for G = dL/dh' and mask = 1[z > 0], ReLU'(0) = 0):

    dZ = G * mask ;  dh~ = dZ W_agg^T ;  dW_agg_t = h~_t^T dZ_t ;  db_agg_t = sum dZ_t
    dalpha^s(e) = dh~^s_j . msg^s(e) ;  dmsg^s(e) = alpha^s(e) dh~^s_j
    dscore^s(e) = alpha^s(e) (dalpha^s(e) - sum_{e' into j} alpha^s(e') dalpha^s(e'))
    with kt = K^s_i W_att[r,s] and c = mu / sqrt(dk):
      dkt = dscore c Q^s_j ;  dQ^s_j += dscore c kt ;  dmu += dscore (kt . Q^s_j) / sqrt(dk)
      dK^s_i += dkt W_att[r,s]^T ;  dW_att[r,s] += K^s_i^T dkt
      dV^s_i += dmsg W_msg[r,s]^T ;  dW_msg[r,s] += V^s_i^T dmsg
    dH = G + dK W_K^T + dQ W_Q^T + dV W_V^T (per type); dW_K_t = H_t^T dK_t, db_K_t = sum dK_t, ...

Everything is float64 and vectorised over edges with numpy scatter-adds.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

PARAM_NAMES = ("W_K", "b_K", "W_Q", "b_Q", "W_V", "b_V", "W_att", "W_msg", "mu", "W_agg", "b_agg")


@dataclass
class Params:
    W_K: np.ndarray    # [T, d, d]
    b_K: np.ndarray    # [T, d]
    W_Q: np.ndarray
    b_Q: np.ndarray
    W_V: np.ndarray
    b_V: np.ndarray
    W_att: np.ndarray  # [R, S, dk, dk]
    W_msg: np.ndarray  # [R, S, dk, dk]
    mu: np.ndarray     # [T, R, T]
    W_agg: np.ndarray  # [T, d, d]
    b_agg: np.ndarray  # [T, d]

    def as64(self) -> "Params":
        return Params(*[np.asarray(getattr(self, k), dtype=np.float64) for k in PARAM_NAMES])


def _per_type(H, ntype, W, b):
    out = np.zeros((H.shape[0], W.shape[2]))
    for t in range(W.shape[0]):
        rows = ntype == t
        out[rows] = H[rows] @ W[t] + b[t]
    return out


def _heads(X, S):
    return X.reshape(X.shape[0], S, X.shape[1] // S)


def _edge_tables(src, dst, rel, ntype, p: Params, K, Q, V, S):
    """Per-edge key transform kt, message msg, raw dot (kt . q) and c = mu / sqrt(dk)."""
    E = src.shape[0]
    dk = K.shape[1] // S
    Ki, Vi, Qj = _heads(K, S)[src], _heads(V, S)[src], _heads(Q, S)[dst]
    kt = np.zeros((E, S, dk))
    msg = np.zeros((E, S, dk))
    for r in range(p.W_att.shape[0]):
        m = rel == r
        kt[m] = np.einsum("esd,sdf->esf", Ki[m], p.W_att[r])
        msg[m] = np.einsum("esd,sdf->esf", Vi[m], p.W_msg[r])
    dot = (kt * Qj).sum(-1)                                      # [E, S]
    c = p.mu[ntype[src], rel, ntype[dst]] / np.sqrt(dk)          # [E]
    return Ki, Vi, Qj, kt, msg, dot, c


def _softmax_by_dst(n, dst, score):
    """alpha[e, s] = exp(score[e, s]) / sum over the edges into dst[e]."""
    S = score.shape[1]
    mx = np.full((n, S), -np.inf)
    np.maximum.at(mx, dst, score)
    ex = np.exp(score - mx[dst])
    den = np.zeros((n, S))
    np.add.at(den, dst, ex)
    return ex / den[dst]


def _softmax_backward(n, dst, alpha, dalpha):
    """dscore[e, s] = alpha (dalpha - sum over the edges e' into dst[e] of
    alpha(e') dalpha(e')): the softmax's Jacobian applied per destination."""
    sdot = np.zeros((n, alpha.shape[1]))
    np.add.at(sdot, dst, alpha * dalpha)
    return alpha * (dalpha - sdot[dst])


def forward(n: int, src_l, dst_l, rel_l, ntype_l, H, params: Params, S: int):
    """Returns (H_out, Z, h_tilde, alpha) in float64."""
    src = np.asarray(src_l, dtype=np.int64)
    dst = np.asarray(dst_l, dtype=np.int64)
    rel = np.asarray(rel_l, dtype=np.int64)
    ntype = np.asarray(ntype_l, dtype=np.int64)
    H = np.asarray(H, dtype=np.float64)
    p = params.as64()
    d = H.shape[1]
    K = _per_type(H, ntype, p.W_K, p.b_K)
    Q = _per_type(H, ntype, p.W_Q, p.b_Q)
    V = _per_type(H, ntype, p.W_V, p.b_V)
    _, _, _, _, msg, dot, c = _edge_tables(src, dst, rel, ntype, p, K, Q, V, S)
    alpha = _softmax_by_dst(n, dst, dot * c[:, None])
    ht = np.zeros((n, S, d // S))
    np.add.at(ht, dst, alpha[:, :, None] * msg)
    ht = ht.reshape(n, d)
    Z = _per_type(ht, ntype, p.W_agg, p.b_agg)
    return np.maximum(Z, 0.0) + H, Z, ht, alpha


def backward(n: int, src_l, dst_l, rel_l, ntype_l, H, params: Params, S: int, G, mask=None):
    """Returns (dH, grads) with grads a Params of float64 gradients.  ``mask``
    (bool [n, d]) overrides the ReLU decision 1[z > 0]."""
    src = np.asarray(src_l, dtype=np.int64)
    dst = np.asarray(dst_l, dtype=np.int64)
    rel = np.asarray(rel_l, dtype=np.int64)
    ntype = np.asarray(ntype_l, dtype=np.int64)
    H = np.asarray(H, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    p = params.as64()
    d = H.shape[1]
    dk = d // S
    T = p.W_K.shape[0]
    K = _per_type(H, ntype, p.W_K, p.b_K)
    Q = _per_type(H, ntype, p.W_Q, p.b_Q)
    V = _per_type(H, ntype, p.W_V, p.b_V)
    Ki, Vi, Qj, kt, msg, dot, c = _edge_tables(src, dst, rel, ntype, p, K, Q, V, S)
    alpha = _softmax_by_dst(n, dst, dot * c[:, None])
    ht = np.zeros((n, S, dk))
    np.add.at(ht, dst, alpha[:, :, None] * msg)
    ht = ht.reshape(n, d)
    Z = _per_type(ht, ntype, p.W_agg, p.b_agg)
    if mask is None:
        mask = Z > 0
    dZ = G * mask
    g = Params(*[np.zeros_like(getattr(p, k)) for k in PARAM_NAMES])
    dht = np.zeros((n, d))
    for t in range(T):
        rows = ntype == t
        g.W_agg[t] = ht[rows].T @ dZ[rows]
        g.b_agg[t] = dZ[rows].sum(axis=0)
        dht[rows] = dZ[rows] @ p.W_agg[t].T
    dht_j = _heads(dht, S)[dst]                                   # [E, S, dk]
    dalpha = (dht_j * msg).sum(-1)                                # [E, S]
    dmsg = alpha[:, :, None] * dht_j
    dscore = _softmax_backward(n, dst, alpha, dalpha)
    dkt = (dscore * c[:, None])[:, :, None] * Qj
    dQ = np.zeros((n, S, dk))
    np.add.at(dQ, dst, (dscore * c[:, None])[:, :, None] * kt)
    np.add.at(g.mu, (ntype[src], rel, ntype[dst]), (dscore * dot).sum(-1) / np.sqrt(dk))
    dK = np.zeros((n, S, dk))
    dV = np.zeros((n, S, dk))
    for r in range(p.W_att.shape[0]):
        m = rel == r
        np.add.at(dK, src[m], np.einsum("esf,sdf->esd", dkt[m], p.W_att[r]))
        np.add.at(dV, src[m], np.einsum("esf,sdf->esd", dmsg[m], p.W_msg[r]))
        g.W_att[r] = np.einsum("esd,esf->sdf", Ki[m], dkt[m])
        g.W_msg[r] = np.einsum("esd,esf->sdf", Vi[m], dmsg[m])
    dK, dQ, dV = dK.reshape(n, d), dQ.reshape(n, d), dV.reshape(n, d)
    dH = G.copy()
    for t in range(T):
        rows = ntype == t
        for dX, W, dW, db in ((dK, p.W_K, g.W_K, g.b_K), (dQ, p.W_Q, g.W_Q, g.b_Q), (dV, p.W_V, g.W_V, g.b_V)):
            dW[t] = H[rows].T @ dX[rows]
            db[t] = dX[rows].sum(axis=0)
            dH[rows] += dX[rows] @ W[t].T
    return dH, g
