"""One relation-typed mean-aggregation layer, forward and backward.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Forward (the message / aggregation / update equations of the "Heterogeneous
Graph Transformer" paragraph in their reduced form: a relation-typed linear
message h_i W_r, mean aggregation over each relation's in-neighbours, the
per-type linear update, sigma = ReLU and the residual connection):

    m_{j,r} = (1/|N_r(j)|) * sum_{i in N_r(j)} h_i          (0 if N_r(j) is empty)
    z_j     = sum_r m_{j,r} W_r + h_j W_self[type(j)] + b[type(j)]
    h'_j    = ReLU(z_j) + h_j

|N_r(j)| counts in-edges of relation r, duplicates and self-loops included.
The per-type aggregation transform of the update equation is folded into W_r
(a product of two linear maps is one linear map).

With edge weights w_ij (the weighted edges of the problem formulation) each
message is multiplied by its edge's weight and the normaliser stays the
in-edge count:  m_{j,r} = (1/|N_r(j)|) * sum_{i in N_r(j)} w_ij h_i.

Backward, for an upstream gradient G = dL/dh' and mask = 1[z > 0]
(ReLU'(0) = 0):

    dZ        = G * mask
    dH        = G + dZ W_self[type]^T + sum_r A_r^T (dZ W_r^T)
    dW_r      = (A_r H)^T dZ
    dW_self_t = H_t^T dZ_t ,   db_t = sum_{j of type t} dZ_j

with A_r the row-normalised (mean) adjacency of relation r.  Everything is
float64; the sparse products are scipy's.
"""
from __future__ import annotations

import numpy as np
import scipy.sparse as sp


def mean_adjacency(n: int, src_l, dst_l, rel_l, r: int, edge_w=None) -> sp.csr_matrix:
    """A_r[j, i] = (sum of w over the edges i->j of relation r) / |N_r(j)|,
    float64 (w = 1 without weights)."""
    m = np.asarray(rel_l) == r
    s = np.asarray(src_l, dtype=np.int64)[m]
    t = np.asarray(dst_l, dtype=np.int64)[m]
    ones = np.ones(s.shape[0])
    w = ones if edge_w is None else np.asarray(edge_w, dtype=np.float64)[m]
    a = sp.coo_matrix((w, (t, s)), shape=(n, n)).tocsr()  # sums duplicates
    deg = np.bincount(t, minlength=n).astype(np.float64)   # the edge count
    inv = np.divide(1.0, deg, out=np.zeros_like(deg), where=deg > 0)
    return sp.diags(inv) @ a


def forward(n: int, src_l, dst_l, rel_l, ntype_l, H, w_rel, w_self, bias, edge_w=None):
    """Returns (H_out, Z) in float64."""
    H = np.asarray(H, dtype=np.float64)
    w_rel = np.asarray(w_rel, dtype=np.float64)
    w_self = np.asarray(w_self, dtype=np.float64)
    bias = np.asarray(bias, dtype=np.float64)
    ntype_l = np.asarray(ntype_l, dtype=np.int64)
    Z = np.zeros((n, w_self.shape[2]))
    for r in range(w_rel.shape[0]):
        Z += (mean_adjacency(n, src_l, dst_l, rel_l, r, edge_w) @ H) @ w_rel[r]
    for t in range(w_self.shape[0]):
        rows = ntype_l == t
        Z[rows] += H[rows] @ w_self[t] + bias[t]
    return np.maximum(Z, 0.0) + H, Z


def backward(n: int, src_l, dst_l, rel_l, ntype_l, H, w_rel, w_self, bias, G, mask=None, edge_w=None):
    """Returns (dH, dW_rel, dW_self, dbias) in float64.  ``mask`` (bool [n, d])
    overrides the ReLU decision 1[z > 0]; by default it is recomputed."""
    H = np.asarray(H, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    w_rel = np.asarray(w_rel, dtype=np.float64)
    w_self = np.asarray(w_self, dtype=np.float64)
    ntype_l = np.asarray(ntype_l, dtype=np.int64)
    if mask is None:
        _, Z = forward(n, src_l, dst_l, rel_l, ntype_l, H, w_rel, w_self, bias, edge_w)
        mask = Z > 0
    dZ = G * mask
    dH = G.copy()
    dW_rel = np.zeros_like(w_rel)
    for r in range(w_rel.shape[0]):
        a = mean_adjacency(n, src_l, dst_l, rel_l, r, edge_w)
        dW_rel[r] = (a @ H).T @ dZ
        dH += a.T @ (dZ @ w_rel[r].T)
    dW_self = np.zeros_like(w_self)
    dbias = np.zeros((w_self.shape[0], w_self.shape[2]))
    for t in range(w_self.shape[0]):
        rows = ntype_l == t
        dW_self[t] = H[rows].T @ dZ[rows]
        dbias[t] = dZ[rows].sum(axis=0)
        dH[rows] += dZ[rows] @ w_self[t].T
    return dH, dW_rel, dW_self, dbias
