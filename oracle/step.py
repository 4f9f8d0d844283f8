"""One whole step of the hot path on the CPU: build, L layers forward, the
alignment loss on the overlap rows, L layers backward.  Layers are the
mean-aggregation layer (weights with w_rel / w_self / bias) or the attention
layer (weights as a dict of the oracle.hgt parameter names, with `heads`).
`run_sequence` is the same over the snapshots of one subgraph with the
temporal module between the spatial layers and the losses.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Used by the smoke
check and the benchmark's CPU-baseline leg.
"""
from __future__ import annotations

import numpy as np

from . import align, hgt, layer, objective, select, temporal


def run(graph_arrays: dict, build_args: dict, feats_global: np.ndarray, weights: list,
        h_ref: np.ndarray, g_ext: np.ndarray, omega=None, lambda_n=2e-4, scale=0.1,
        eps=1e-5, ddof=0, heads=None, head=None, labels_global=None, masks=None):
    """With `head` (dict W1, b1, W2, b2) and labels (global order), the
    upstream gradient is the prediction head's dL_BCE/dH instead of g_ext, and
    the result also holds the BCE loss and the head's gradients.  `masks[l]`
    (optional) gives the ReLU decisions of layer l for the backward (a caller
    whose pre-activations were decided in another precision passes its own);
    otherwise they are Z > 0."""
    sub = select.build(**graph_arrays, **build_args)
    edges = (sub.n_sub, sub.src_l, sub.dst_l, sub.rel_l, sub.ntype_l)
    h = [np.asarray(feats_global, dtype=np.float64)[sub.local2global]]
    for w in weights:
        if isinstance(w, dict):
            out = hgt.forward(*edges, h[-1], hgt.Params(*[w[n] for n in hgt.PARAM_NAMES]), heads)[0]
        else:
            out, _ = layer.forward(*edges, h[-1], w.w_rel, w.w_self, w.bias)
        h.append(out)
    losses, dX, _ = align.loss_and_grad(h[-1][sub.overlap], h_ref[: sub.overlap.shape[0]],
                                        omega, lambda_n, scale, eps, ddof)
    head_out = None
    if head is not None:
        lab = np.asarray(labels_global)[sub.local2global]
        bce, g, dW1, db1, dW2, db2, _ = objective.mlp_bce(h[-1], head["W1"], head["b1"], head["W2"], head["b2"], lab)
        head_out = dict(loss=bce, W1=dW1, b1=db1, W2=dW2, b2=db2)
    else:
        g = np.asarray(g_ext, dtype=np.float64)[: sub.n_sub].copy()
    g[sub.overlap] += dX
    grads = []
    for li in reversed(range(len(weights))):
        w = weights[li]
        mk = None if masks is None else masks[li]
        if isinstance(w, dict):
            g, gp = hgt.backward(*edges, h[li], hgt.Params(*[w[n] for n in hgt.PARAM_NAMES]), heads, g, mask=mk)
            grads.append({n: getattr(gp, n) for n in hgt.PARAM_NAMES})
            continue
        g, dwr, dws, db = layer.backward(*edges, h[li], w.w_rel, w.w_self, w.bias, g, mask=mk)
        grads.append((dwr, dws, db))
    if head is not None:
        return sub, h, losses, g, grads[::-1], head_out
    return sub, h, losses, g, grads[::-1]


def run_sequence(graph_arrays: dict, build_args: dict, edge_ts, cuts, feats_global: np.ndarray, weights: list,
                 heads: int, tparams: dict, window: int, h_ref: np.ndarray, head: dict, labels_global,
                 omega=None, lambda_n=2e-4, scale=0.1, eps=1e-5, ddof=0, masks=None):
    """T snapshots of one overlapping subgraph (snapshot t keeps the edges
    with timestamp <= cuts[t]; all share the node set).  Per snapshot the
    attention layers map the features to the spatial embedding h^t and the
    temporal module (E12, E13) gives S^t = GRU(h^t, attention over the
    min(t, window) previous S); the prediction head with masked BCE and the
    alignment act on the last S.  The backward runs through every snapshot
    (the gradient of S^j collects the contributions of every later snapshot
    whose context holds it); weights shared over the snapshots get the sum of
    their per-snapshot gradients.  `masks[t][l]` (optional) gives the ReLU
    decisions of layer l at snapshot t for the backward (a caller whose
    pre-activations were decided in another precision passes its own);
    otherwise they are Z > 0.  Returns a dict."""
    subs = [select.build(**graph_arrays, **build_args, edge_ts=edge_ts, t_cut=c) for c in cuts]
    T = len(subs)
    sub0 = subs[0]
    x = np.asarray(feats_global, dtype=np.float64)[sub0.local2global]
    params = [hgt.Params(*[w[n] for n in hgt.PARAM_NAMES]) for w in weights]
    edges = [(sb.n_sub, sb.src_l, sb.dst_l, sb.rel_l, sb.ntype_l) for sb in subs]
    hs, S = [], []
    for t in range(T):
        h = [x]
        for p in params:
            h.append(hgt.forward(*edges[t], h[-1], p, heads)[0])
        hs.append(h)
        ctx = S[max(0, t - window):t]
        Cs = np.stack(ctx) if ctx else np.zeros((0,) + x.shape)
        S.append(temporal.forward(h[-1], Cs, tparams)[0])
    lab = np.asarray(labels_global)[sub0.local2global]
    bce, g, dW1, db1, dW2, db2, _ = objective.mlp_bce(S[-1], head["W1"], head["b1"], head["W2"], head["b2"], lab)
    losses, dX, _ = align.loss_and_grad(S[-1][sub0.overlap], h_ref[: sub0.overlap.shape[0]], omega, lambda_n,
                                        scale, eps, ddof)
    g[sub0.overlap] += dX
    dS = [np.zeros_like(x) for _ in range(T)]
    dS[-1] = g
    tgrads = {k: np.zeros_like(np.asarray(v, dtype=np.float64)) for k, v in tparams.items()}
    lgrads = [{n: 0.0 for n in hgt.PARAM_NAMES} for _ in weights]
    dx = np.zeros_like(x)
    for t in reversed(range(T)):
        idx = list(range(max(0, t - window), t))
        Cs = np.stack([S[j] for j in idx]) if idx else np.zeros((0,) + x.shape)
        dh, dC, gt = temporal.backward(hs[t][-1], Cs, tparams, dS[t])
        for k, j in enumerate(idx):
            dS[j] = dS[j] + dC[k]
        for k in tgrads:
            tgrads[k] = tgrads[k] + gt[k]
        gg = dh
        for li in reversed(range(len(weights))):
            mk = None if masks is None else masks[t][li]
            gg, gp = hgt.backward(*edges[t], hs[t][li], params[li], heads, gg, mask=mk)
            for n in hgt.PARAM_NAMES:
                lgrads[li][n] = lgrads[li][n] + getattr(gp, n)
        dx += gg
    return dict(subs=subs, h=hs, S=S, losses=losses, bce=bce,
                head_grads=dict(W1=dW1, b1=db1, W2=dW2, b2=db2), temporal_grads=tgrads, layer_grads=lgrads,
                dS=dS, dx=dx)
