"""One whole step of the hot path on the CPU: build, L layers forward, the
alignment loss on the overlap rows, L layers backward.  Layers are the
mean-aggregation layer (weights with w_rel / w_self / bias) or the attention
layer (weights as a dict of the oracle.hgt parameter names, with `heads`).

TEST INFRASTRUCTURE ONLY (see the package docstring).  Used by the smoke
check and the benchmark's CPU-baseline leg.
"""
from __future__ import annotations

import numpy as np

from . import align, hgt, layer, objective, select


def run(graph_arrays: dict, build_args: dict, feats_global: np.ndarray, weights: list,
        h_ref: np.ndarray, g_ext: np.ndarray, omega=None, lambda_n=2e-4, scale=0.1,
        eps=1e-5, ddof=0, heads=None, head=None, labels_global=None):
    """With `head` (dict W1, b1, W2, b2) and labels (global order), the
    upstream gradient is the prediction head's dL_BCE/dH instead of g_ext, and
    the result also holds the BCE loss and the head's gradients."""
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
        if isinstance(w, dict):
            g, gp = hgt.backward(*edges, h[li], hgt.Params(*[w[n] for n in hgt.PARAM_NAMES]), heads, g)
            grads.append({n: getattr(gp, n) for n in hgt.PARAM_NAMES})
            continue
        g, dwr, dws, db = layer.backward(*edges, h[li], w.w_rel, w.w_self, w.bias, g)
        grads.append((dwr, dws, db))
    if head is not None:
        return sub, h, losses, g, grads[::-1], head_out
    return sub, h, losses, g, grads[::-1]
