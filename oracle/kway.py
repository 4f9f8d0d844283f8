"""K overlapping subgraphs of one graph and their joint training step.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Algorithm 1 on K workers, run one after another: the node set is split into
K blocks by a partition `part` (the random-hash partition is an input); each
worker k builds its overlapping subgraph G~_k (oracle.select.build) and maps
the features of its nodes to H_k with the L shared layers; MeanAgg averages
the copies of every node over the subgraphs that hold it (the inference /
MeanAgg step of Algorithm 1 and the averaging of overlapping nodes in
"Prediction and Optimization"); the prediction head with the masked BCE acts
on the averaged embeddings; and every worker aligns its overlap nodes with
their home copies (the embedding of the same node in the subgraph of its own
partition block) through the CCA loss, the home copies taken as constants:

    H[v]    = (1 / cnt[v]) sum_{k : v in G~_k} H_k[v],   cnt[v] = #{k : v in G~_k}
    L_total = L_BCE(MLP(H)) + lambda_CCA sum_k L_CCA(H_k[C_k], H_home(C_k))

Backward: dH_k[v] = dH[v] / cnt[v] + lambda_CCA dL_CCA,k/dX on the overlap
rows; the layer gradients of the K workers are summed (what the gradient
all-reduce of the data-parallel training computes).  float64.
"""
from __future__ import annotations

import numpy as np

from . import align, layer, objective, select


def mean_agg(n_nodes: int, l2gs, Hs):
    """(H [n_nodes, d], cnt [n_nodes]) from the K subgraphs' rows."""
    d = np.asarray(Hs[0]).shape[1]
    H = np.zeros((n_nodes, d))
    cnt = np.zeros(n_nodes, dtype=np.int64)
    for l2g, Hk in zip(l2gs, Hs):
        l2g = np.asarray(l2g, dtype=np.int64)
        H[l2g] += np.asarray(Hk, dtype=np.float64)      # l2g is injective within a subgraph
        cnt[l2g] += 1
    nz = cnt > 0
    H[nz] /= cnt[nz, None]
    return H, cnt


def mean_agg_backward(l2gs, cnt, dH):
    """dH_k = dH[l2g_k] / cnt[l2g_k] for every subgraph."""
    dH = np.asarray(dH, dtype=np.float64)
    return [dH[np.asarray(l2g, dtype=np.int64)] / cnt[np.asarray(l2g, dtype=np.int64), None] for l2g in l2gs]


def home_rows(subs, part, sub_k):
    """Home copies of the overlap nodes of subgraph sub_k: for node v, the row
    of v in the subgraph of partition part[v] (where v is a base node)."""
    og = subs[sub_k].local2global[subs[sub_k].overlap].astype(np.int64)
    home = np.asarray(part, dtype=np.int64)[og]
    return home, np.array([subs[h].global2local[v] for h, v in zip(home, og)], dtype=np.int64)


def run_kway(graph_arrays: dict, K: int, build_args: dict, feats_global, weights: list, head: dict,
             labels_global, lambda_n=2e-4, scale=0.1, eps=1e-5, ddof=0, frozen_home=None, masks=None):
    """One step over the K subgraphs.  `frozen_home` (list of K arrays) replaces
    the home copies (finite-difference checks hold them fixed, as the
    gradient does).  `masks[k][l]` (optional) gives the ReLU decisions of
    layer l in subgraph k for the backward (otherwise Z > 0).  Returns a dict."""
    part = graph_arrays["part"]
    subs = [select.build(**graph_arrays, k=k, **build_args) for k in range(K)]
    x = np.asarray(feats_global, dtype=np.float64)
    hs = []
    for sb in subs:
        h = [x[sb.local2global]]
        for w in weights:
            h.append(layer.forward(sb.n_sub, sb.src_l, sb.dst_l, sb.rel_l, sb.ntype_l, h[-1], w.w_rel, w.w_self,
                                   w.bias)[0])
        hs.append(h)
    n = x.shape[0]
    H, cnt = mean_agg(n, [sb.local2global for sb in subs], [h[-1] for h in hs])
    bce, dH, dW1, db1, dW2, db2, _ = objective.mlp_bce(H, head["W1"], head["b1"], head["W2"], head["b2"],
                                                       labels_global)
    dHk = mean_agg_backward([sb.local2global for sb in subs], cnt, dH)
    losses, homes = [], []
    for k, sb in enumerate(subs):
        home, rows = home_rows(subs, part, k)
        Y = (np.stack([hs[h][-1][r] for h, r in zip(home, rows)]) if rows.size else np.zeros((0, x.shape[1])))
        if frozen_home is not None:
            Y = frozen_home[k]
        homes.append(Y)
        lk, dX, _ = align.loss_and_grad(hs[k][-1][sb.overlap], Y, None, lambda_n, scale, eps, ddof)
        losses.append(lk)
        dHk[k][sb.overlap] += dX
    grads = None
    for k, sb in enumerate(subs):
        g = dHk[k]
        for li in reversed(range(len(weights))):
            w = weights[li]
            mk = None if masks is None else masks[k][li]
            g, dwr, dws, db = layer.backward(sb.n_sub, sb.src_l, sb.dst_l, sb.rel_l, sb.ntype_l, hs[k][li], w.w_rel,
                                             w.w_self, w.bias, g, mask=mk)
            if grads is None:
                grads = [None] * len(weights)
            gk = (dwr, dws, db)
            grads[li] = gk if grads[li] is None else tuple(a + b for a, b in zip(grads[li], gk))
    total = bce + scale * sum(l[2] for l in losses)
    return dict(subs=subs, h=hs, H=H, cnt=cnt, bce=bce, losses=losses, total=total, homes=homes,
                head_grads=dict(W1=dW1, b1=db1, W2=dW2, b2=db2), layer_grads=grads, dHk=dHk)
