"""One training step of the hot path through the C ABI: subgraph build,
L layers forward, the CCA alignment on the overlap rows, L layers backward.

This module only allocates buffers (torch) and sequences library calls; all
arithmetic runs in libhg.so.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np
import torch

from . import api, synth


@dataclass
class StepInputs:
    wl: synth.Workload
    graph: dict                 # device tensors src, dst, rel, ntype, part
    k: int
    sub: api.Subgraph
    build_ws: torch.Tensor
    h0: torch.Tensor            # [n_sub, d] features in local order
    weights: List[tuple]        # per layer (w_rel, w_self, bias) device float32
    weights_np: list
    href: torch.Tensor          # [m_sel, d]
    gext: torch.Tensor          # [n_sub, d]
    omega: Optional[torch.Tensor]
    feats_np: np.ndarray
    href_np: np.ndarray
    gext_np: np.ndarray
    # preallocated per-step buffers
    H: List[torch.Tensor] = field(default_factory=list)
    saved: List[torch.Tensor] = field(default_factory=list)
    dH: List[torch.Tensor] = field(default_factory=list)
    g: Optional[torch.Tensor] = None        # upstream gradient of the last layer (G_ext + the alignment's)
    grads: List[tuple] = field(default_factory=list)
    fwd_ws: Optional[torch.Tensor] = None
    bwd_ws: Optional[torch.Tensor] = None
    align_ws: Optional[torch.Tensor] = None
    loss: Optional[torch.Tensor] = None
    hgt_saved: List[torch.Tensor] = field(default_factory=list)
    # full objective (prediction head, masked BCE, Adam)
    labels: Optional[torch.Tensor] = None
    labels_np: Optional[np.ndarray] = None
    label_rows: Optional[torch.Tensor] = None  # rows with a label, ascending (only they go through the head)
    head: Optional[dict] = None
    head_np: Optional[dict] = None
    head_grads: Optional[dict] = None
    head_ws: Optional[torch.Tensor] = None
    loss_bce: Optional[torch.Tensor] = None
    adam: list = field(default_factory=list)   # (param, grad, m, v) for every trained tensor
    t: int = 0


@dataclass
class StepResult:
    loss: torch.Tensor
    dH0: torch.Tensor
    grads: List[tuple]


def _dev(x, device):
    return torch.from_numpy(np.ascontiguousarray(x)).to(device)


def _label_rows(labels: torch.Tensor) -> torch.Tensor:
    """Rows with a label (>= 0), ascending int32: fixed by the input labels,
    computed once at set-up."""
    return torch.nonzero(labels >= 0).flatten().to(torch.int32).contiguous()


def make_inputs(wl: synth.Workload, g: synth.Graph, device="cuda", feats: Optional[np.ndarray] = None
                ) -> StepInputs:
    cfg, mc = wl.graph, wl.model
    d = mc.d
    gd = {k: _dev(getattr(g, k), device) for k in ("src", "dst", "rel", "ntype", "part")}
    sub = api.hg_build_csr(gd["src"], gd["dst"], gd["rel"], gd["ntype"], gd["part"], g.k, cfg.n_rel,
                           g.n_ntype, cfg.budget, key=cfg.key, theta=cfg.theta, seed=cfg.seed,
                           want_eid=False)
    build_ws = sub.arrays["ws"]
    feats = synth.features(mc.seed, g.n_nodes, d) if feats is None else feats
    fdt = torch.bfloat16 if mc.dtype == "bf16" else torch.float32
    if mc.dtype == "bf16":
        feats = synth.round_bf16(feats)
    l2g = sub.view("local2global").long()
    h0 = _dev(feats, device).index_select(0, l2g).to(fdt).contiguous()
    if mc.kind == "hgt":
        weights_np = [synth.hgt_weights(mc.seed, li, cfg.n_rel, g.n_ntype, d, mc.heads, mc.bias_range)
                      for li in range(mc.n_layers)]
        weights = [{n: _dev(v, device) for n, v in w.items()} for w in weights_np]
    else:
        weights_np = [synth.layer_weights(mc.seed, li, cfg.n_rel, g.n_ntype, d, mc.bias_range)
                      for li in range(mc.n_layers)]
        weights = [(_dev(w.w_rel, device), _dev(w.w_self, device), _dev(w.bias, device)) for w in weights_np]
    m = sub.m_sel
    href_np = synth.reference_embeddings(mc.seed, max(m, 1), d)
    gext_np = synth.upstream_grad(mc.seed, max(sub.n_sub, 1), d)
    if mc.dtype == "bf16":
        href_np, gext_np = synth.round_bf16(href_np), synth.round_bf16(gext_np)
    omega = None
    if mc.weighted_align and m > 0:
        orel = sub.view("overlap_rel").cpu().numpy()
        omega = _dev(synth.align_weights(orel, g.rel, cfg.n_rel), device)
    inp = StepInputs(wl, gd, g.k, sub, build_ws, h0, weights, weights_np,
                     _dev(href_np[:m], device).to(fdt), _dev(gext_np[: sub.n_sub], device).to(fdt),
                     omega, feats, href_np, gext_np)
    ns = sub.n_sub
    f32 = dict(dtype=torch.float32, device=device)
    act = dict(dtype=fdt, device=device)
    inp.H = [h0] + [torch.empty((ns, d), **act) for _ in range(mc.n_layers)]
    inp.saved = [torch.empty((max(ns, 1), d // 32), dtype=torch.int32, device=device)
                 for _ in range(mc.n_layers)]
    inp.dH = [torch.empty((ns, d), **act) for _ in range(2)]
    # g holds G_ext outside the overlap rows for good; every step's alignment
    # writes its overlap rows as G_ext + its gradient
    inp.g = inp.gext.clone() if mc.objective != "bce" else torch.empty((ns, d), **act)
    if mc.kind == "hgt":
        inp.grads = [{n: torch.empty_like(v) for n, v in w.items()} for w in weights]
        inp.hgt_saved = [api._ws(api.hg_hgt_saved_size(sub, d, mc.heads), device) for _ in range(mc.n_layers)]
        inp.fwd_ws = api._ws(api.hg_hgt_fwd_workspace_size(sub, d, mc.heads), device)
        inp.bwd_ws = api._ws(api.hg_hgt_bwd_workspace_size(sub, d, mc.heads), device)
    else:
        inp.grads = [(torch.empty_like(w[0]), torch.empty_like(w[1]), torch.empty_like(w[2])) for w in weights]
        inp.fwd_ws = api._ws(api.hg_layer_fwd_workspace_size(sub, d, fdt), device)
        inp.bwd_ws = api._ws(api.hg_layer_bwd_workspace_size(sub, d, fdt), device)
    inp.align_ws = api._ws(api.hg_align_workspace_size(m, d), device)
    inp.loss = torch.empty(3, **f32)
    if mc.objective == "bce":
        inp.labels_np = synth.labels(mc.seed, g.ntype)
        inp.labels = _dev(inp.labels_np, device).index_select(0, l2g).contiguous()
        inp.label_rows = _label_rows(inp.labels)
        inp.head_np = synth.head_weights(mc.seed, d)
        inp.head = {k: _dev(v, device) for k, v in inp.head_np.items()}
        inp.head_grads = {k: torch.empty_like(v) for k, v in inp.head.items()}
        inp.head_ws = api._ws(api.hg_mlp_bce_workspace_size(ns, d), device)
        inp.loss_bce = torch.empty(1, **f32)
        pairs = []
        for li, w in enumerate(inp.weights):
            gw = inp.grads[li]
            if isinstance(w, dict):
                pairs += [(w[k], gw[k]) for k in w]
            else:
                pairs += list(zip(w, gw))
        pairs += [(inp.head[k], inp.head_grads[k]) for k in inp.head]
        inp.adam = [(p, gr, torch.zeros_like(p), torch.zeros_like(p)) for p, gr in pairs]
    return inp


def run_step(inp: StepInputs, rebuild: bool = True) -> StepResult:
    cfg, mc = inp.wl.graph, inp.wl.model
    gd = inp.graph
    if rebuild:
        api.hg_build_csr(gd["src"], gd["dst"], gd["rel"], gd["ntype"], gd["part"], inp.k, cfg.n_rel, 2,
                         cfg.budget, key=cfg.key, theta=cfg.theta, seed=cfg.seed, ws=inp.build_ws,
                         out=inp.sub)
    sub = inp.sub
    hgt = mc.kind == "hgt"
    for li in range(mc.n_layers):
        if hgt:
            api.hg_hgt_fwd(sub, inp.H[li], inp.weights[li], mc.heads, H_out=inp.H[li + 1], mask=inp.saved[li],
                           saved=inp.hgt_saved[li], ws=inp.fwd_ws)
            continue
        w_rel, w_self, bias = inp.weights[li]
        api.hg_layer_fwd(sub, inp.H[li], w_rel, w_self, bias, H_out=inp.H[li + 1], saved=inp.saved[li],
                         ws=inp.fwd_ws)
    g = inp.g
    overlap = sub.view("overlap")
    base = None
    if mc.objective == "bce":
        # dL_BCE/dH of the prediction head on the labelled rows (overwrites g)
        api.hg_mlp_bce_fwd_bwd(inp.H[-1], inp.head["W1"], inp.head["b1"], inp.head["W2"], inp.head["b2"],
                               inp.labels, dH=g, grads=inp.head_grads, loss=inp.loss_bce, ws=inp.head_ws,
                               rows=inp.label_rows)
    else:
        base = inp.gext
    api.hg_align_loss_fwd_bwd(inp.H[-1], overlap, inp.href, g, w=inp.omega, lambda_n=mc.lambda_n,
                              scale=mc.lambda_cca, eps=mc.eps, ddof=mc.ddof, loss3=inp.loss,
                              ws=inp.align_ws, dH_base=base)
    gin, nxt = g, 0
    for li in reversed(range(mc.n_layers)):
        if hgt:
            api.hg_hgt_bwd(sub, inp.H[li], inp.weights[li], mc.heads, inp.saved[li], inp.hgt_saved[li], gin,
                           dH_in=inp.dH[nxt], grads=inp.grads[li], ws=inp.bwd_ws)
        else:
            w_rel, w_self, _ = inp.weights[li]
            gw = inp.grads[li]
            api.hg_layer_bwd(sub, inp.H[li], w_rel, w_self, inp.saved[li], gin, dH_in=inp.dH[nxt],
                             dW_rel=gw[0], dW_self=gw[1], dbias=gw[2], ws=inp.bwd_ws)
        gin, nxt = inp.dH[nxt], 1 - nxt
    if mc.objective == "bce":
        inp.t += 1
        for p, gr, m1, m2 in inp.adam:
            api.hg_adam_step(p, gr, m1, m2, inp.t, lr=mc.lr, weight_decay=mc.weight_decay)
    return StepResult(inp.loss, gin, inp.grads)


# ---- multi-snapshot step (attention layers + temporal module) ---------------

@dataclass
class SeqInputs:
    wl: synth.Workload
    graph: dict                 # device tensors src, dst, rel, ntype, part, ts
    k: int
    cuts: List[int]
    subs: List[api.Subgraph]    # one per snapshot; all share local ids and overlap
    build_ws: torch.Tensor
    h0: torch.Tensor            # [n_sub, d] features in local order (shared by the snapshots)
    weights: List[dict]
    weights_np: List[dict]
    tparams: dict
    tparams_np: dict
    head: dict
    head_np: dict
    labels: torch.Tensor
    labels_np: np.ndarray
    label_rows: torch.Tensor
    href: torch.Tensor
    href_np: np.ndarray
    feats_np: np.ndarray
    ts_np: np.ndarray
    H: List[torch.Tensor] = field(default_factory=list)       # layer activations of the latest snapshot run
    masks: List[torch.Tensor] = field(default_factory=list)   # its ReLU masks
    Hs: List[List[torch.Tensor]] = field(default_factory=list)     # Hs[t][l]: every snapshot's activations
    ms: List[List[torch.Tensor]] = field(default_factory=list)     # ms[t][l]: their masks
    saved: List[List[torch.Tensor]] = field(default_factory=list)  # saved[t][l]: lean attention intermediates
    S: List[torch.Tensor] = field(default_factory=list)       # temporal states, one per snapshot
    dS: List[torch.Tensor] = field(default_factory=list)
    dH: List[torch.Tensor] = field(default_factory=list)      # ping-pong gradient buffers
    grads: List[dict] = field(default_factory=list)
    tgrads: Optional[dict] = None
    head_grads: Optional[dict] = None
    fwd_ws: Optional[torch.Tensor] = None
    bwd_ws: Optional[torch.Tensor] = None
    t_ws: Optional[torch.Tensor] = None
    align_ws: Optional[torch.Tensor] = None
    head_ws: Optional[torch.Tensor] = None
    loss: Optional[torch.Tensor] = None
    loss_bce: Optional[torch.Tensor] = None
    adam: list = field(default_factory=list)
    t: int = 0

    @property
    def edges_per_pass(self) -> int:
        """Edges of all snapshots (one pass of a layer over every snapshot)."""
        return sum(s.e_sub for s in self.subs)


def _build_snapshots(inp_graph, g_k, cfg, cuts, ws=None, subs=None):
    out = []
    for i, c in enumerate(cuts):
        sub = api.hg_build_csr(inp_graph["src"], inp_graph["dst"], inp_graph["rel"], inp_graph["ntype"],
                               inp_graph["part"], g_k, cfg.n_rel, 2, cfg.budget, key=cfg.key, theta=cfg.theta,
                               seed=cfg.seed, want_eid=False, ws=ws, out=None if subs is None else subs[i],
                               edge_ts=inp_graph["ts"], t_cut=c)
        if ws is None:
            ws = sub.arrays["ws"]
        out.append(sub)
    return out, ws


def make_seq_inputs(wl: synth.Workload, g: synth.Graph, device="cuda") -> SeqInputs:
    cfg, mc = wl.graph, wl.model
    d, T = mc.d, mc.snapshots
    ts_np = synth.edge_times(cfg.seed, g.n_edges, T)
    cuts = synth.snapshot_cuts(T)
    gd = {k: _dev(getattr(g, k), device) for k in ("src", "dst", "rel", "ntype", "part")}
    gd["ts"] = _dev(ts_np, device)
    subs, build_ws = _build_snapshots(gd, g.k, cfg, cuts)
    sub0 = subs[0]
    feats = synth.features(mc.seed, g.n_nodes, d)
    l2g = sub0.view("local2global").long()
    h0 = _dev(feats, device).index_select(0, l2g).contiguous()
    weights_np = [synth.hgt_weights(mc.seed, li, cfg.n_rel, g.n_ntype, d, mc.heads, mc.bias_range)
                  for li in range(mc.n_layers)]
    weights = [{n: _dev(v, device) for n, v in w.items()} for w in weights_np]
    tparams_np = synth.temporal_weights(mc.seed, d)
    tparams = {k: _dev(v, device) for k, v in tparams_np.items()}
    head_np = synth.head_weights(mc.seed, d)
    head = {k: _dev(v, device) for k, v in head_np.items()}
    labels_np = synth.labels(mc.seed, g.ntype)
    labels = _dev(labels_np, device).index_select(0, l2g).contiguous()
    m = sub0.m_sel
    href_np = synth.reference_embeddings(mc.seed, max(m, 1), d)
    inp = SeqInputs(wl, gd, g.k, cuts, subs, build_ws, h0, weights, weights_np, tparams, tparams_np, head, head_np,
                    labels, labels_np, _label_rows(labels), _dev(href_np[:m], device), href_np, feats, ts_np)
    ns = sub0.n_sub
    f32 = dict(dtype=torch.float32, device=device)
    # every snapshot keeps its activations, masks and lean intermediates (the
    # relation transforms are left out of them and computed again in the
    # backward), so the backward never runs an earlier snapshot's forward again
    inp.Hs = [[h0] + [torch.empty((ns, d), **f32) for _ in range(mc.n_layers)] for _ in range(T)]
    inp.ms = [[torch.empty((max(ns, 1), d // 32), dtype=torch.int32, device=device) for _ in range(mc.n_layers)]
              for _ in range(T)]
    inp.saved = [[api._ws(api.hg_hgt_saved_size(sb, d, mc.heads, lean=True), device) for _ in range(mc.n_layers)]
                 for sb in subs]
    inp.H, inp.masks = inp.Hs[0], inp.ms[0]
    inp.S = [torch.empty((ns, d), **f32) for _ in range(T)]
    inp.dS = [torch.empty((ns, d), **f32) for _ in range(T)]
    inp.dH = [torch.empty((ns, d), **f32) for _ in range(2)]
    inp.grads = [{n: torch.empty_like(v) for n, v in w.items()} for w in weights]
    inp.tgrads = {k: torch.empty_like(v) for k, v in tparams.items()}
    inp.head_grads = {k: torch.empty_like(v) for k, v in head.items()}
    # forward and backward never overlap: one workspace serves both
    inp.fwd_ws = api._ws(max(max(api.hg_hgt_fwd_workspace_size(s, d, mc.heads, lean=True),
                                 api.hg_hgt_bwd_workspace_size(s, d, mc.heads, lean=True)) for s in subs), device)
    inp.bwd_ws = inp.fwd_ws
    inp.t_ws = api._ws(api.hg_temporal_bwd_workspace_size(ns, d, min(mc.window, T - 1)), device)
    inp.align_ws = api._ws(api.hg_align_workspace_size(m, d), device)
    inp.head_ws = api._ws(api.hg_mlp_bce_workspace_size(ns, d), device)
    inp.loss = torch.empty(3, **f32)
    inp.loss_bce = torch.empty(1, **f32)
    pairs = []
    for w, gw in zip(inp.weights, inp.grads):
        pairs += [(w[k], gw[k]) for k in w]
    pairs += [(inp.tparams[k], inp.tgrads[k]) for k in inp.tparams]
    pairs += [(inp.head[k], inp.head_grads[k]) for k in inp.head]
    inp.adam = [(p, gr, torch.zeros_like(p), torch.zeros_like(p)) for p, gr in pairs]
    return inp


def _seq_layers_fwd(inp: SeqInputs, t: int):
    mc = inp.wl.model
    H, m = inp.Hs[t], inp.ms[t]
    for li in range(mc.n_layers):
        api.hg_hgt_fwd(inp.subs[t], H[li], inp.weights[li], mc.heads, H_out=H[li + 1], mask=m[li],
                       saved=inp.saved[t][li], ws=inp.fwd_ws, lean=True)
    inp.H, inp.masks = H, m


def run_seq_step(inp: SeqInputs, rebuild: bool = True, update: bool = True, on_snapshot=None):
    """One step over the snapshots of the subgraph: per snapshot t the
    attention layers give h^t and the temporal module S^t = GRU(h^t,
    attention over the previous min(t, w) states); the head's masked BCE and
    the alignment act on the last state.  The backward runs through every
    snapshot, latest first, from the activations every snapshot kept (the
    attention layers' relation transforms are computed again from their
    kept keys and values), the temporal backward adds each context state's
    gradient into that state's buffer, and the shared weights sum their
    per-snapshot gradients.  Then Adam updates every parameter.
    `on_snapshot(t)`, if given, is called after the forward of snapshot t
    (its layer activations and masks are then in inp.H and inp.masks)."""
    cfg, mc = inp.wl.graph, inp.wl.model
    T, w = len(inp.subs), mc.window
    if rebuild:
        _build_snapshots(inp.graph, inp.k, cfg, inp.cuts, ws=inp.build_ws, subs=inp.subs)
    for t in range(T):
        _seq_layers_fwd(inp, t)
        api.hg_temporal_fwd(inp.Hs[t][-1], inp.S[max(0, t - w):t], inp.tparams, H=inp.S[t])
        if on_snapshot is not None:
            on_snapshot(t)
    g = inp.dS[T - 1]
    api.hg_mlp_bce_fwd_bwd(inp.S[T - 1], inp.head["W1"], inp.head["b1"], inp.head["W2"], inp.head["b2"], inp.labels,
                           dH=g, grads=inp.head_grads, loss=inp.loss_bce, ws=inp.head_ws, rows=inp.label_rows)
    api.hg_align_loss_fwd_bwd(inp.S[T - 1], inp.subs[0].view("overlap"), inp.href, g, lambda_n=mc.lambda_n,
                              scale=mc.lambda_cca, eps=mc.eps, ddof=mc.ddof, loss3=inp.loss, ws=inp.align_ws)
    for j in range(T - 1):
        inp.dS[j].zero_()
    for t in reversed(range(T)):
        H, m = inp.Hs[t], inp.ms[t]
        lo = max(0, t - w)
        acc = t < T - 1
        cur, nxt = 0, 1
        api.hg_temporal_bwd(H[-1], inp.S[lo:t], inp.tparams, inp.dS[t], dh=inp.dH[cur], dstates=inp.dS[lo:t],
                            grads=inp.tgrads, accumulate=acc, ws=inp.t_ws)
        for li in reversed(range(mc.n_layers)):
            api.hg_hgt_bwd(inp.subs[t], H[li], inp.weights[li], mc.heads, m[li], inp.saved[t][li],
                           inp.dH[cur], dH_in=inp.dH[nxt], grads=inp.grads[li], accumulate=acc, ws=inp.bwd_ws,
                           lean=True)
            cur, nxt = nxt, cur
    if update:
        inp.t += 1
        for p, gr, m1, m2 in inp.adam:
            api.hg_adam_step(p, gr, m1, m2, inp.t, lr=mc.lr, weight_decay=mc.weight_decay)
    return inp


# ---- K subgraphs of one graph on one device (Algorithm 1 over K workers) ----

@dataclass
class KwayInputs:
    wl: synth.Workload
    graph: dict                 # device tensors src, dst, rel, ntype, part (the K-way partition)
    part_np: np.ndarray
    subs: List[api.Subgraph]    # subgraph k of partition block k
    build_ws: torch.Tensor      # shared by the K builds (each keeps its own outputs)
    keys: torch.Tensor          # selection key of every node, computed once for the K builds
    keys_ws: torch.Tensor
    weights: List[tuple]        # per layer (w_rel, w_self, bias), shared by the K workers
    weights_np: list
    head: dict
    head_np: dict
    labels: torch.Tensor        # int8 [n_nodes], global order
    labels_np: np.ndarray
    label_rows: torch.Tensor
    feats_np: np.ndarray
    H: List[List[torch.Tensor]] = field(default_factory=list)      # H[k][l]: layer l rows of subgraph k
    saved: List[List[torch.Tensor]] = field(default_factory=list)
    H_agg: Optional[torch.Tensor] = None     # MeanAgg of the K last-layer outputs [n_nodes, d]
    cnt: Optional[torch.Tensor] = None       # copies of every node
    dH_agg: Optional[torch.Tensor] = None
    g: Optional[torch.Tensor] = None         # upstream gradient of one subgraph's last layer
    dH: List[torch.Tensor] = field(default_factory=list)
    Y: Optional[torch.Tensor] = None         # home copies of one subgraph's overlap rows
    grads: List[tuple] = field(default_factory=list)
    head_grads: Optional[dict] = None
    fwd_ws: Optional[torch.Tensor] = None
    bwd_ws: Optional[torch.Tensor] = None
    align_ws: Optional[torch.Tensor] = None
    head_ws: Optional[torch.Tensor] = None
    loss: Optional[torch.Tensor] = None      # [K, 3] alignment losses
    loss_bce: Optional[torch.Tensor] = None
    adam: list = field(default_factory=list)
    t: int = 0

    @property
    def edges_per_pass(self) -> int:
        """Edges of all K subgraphs (one pass of a layer over every worker)."""
        return sum(s.e_sub for s in self.subs)


def _build_parts(gd, cfg, K, keys, ws=None, subs=None):
    out = []
    for k in range(K):
        sub = api.hg_build_csr(gd["src"], gd["dst"], gd["rel"], gd["ntype"], gd["part"], k, cfg.n_rel, 2,
                               cfg.budget, key=cfg.key, theta=cfg.theta, seed=cfg.seed, want_eid=False, ws=ws,
                               out=None if subs is None else subs[k], node_key=keys)
        if ws is None:
            ws = sub.arrays["ws"]
        out.append(sub)
    return out, ws


def make_kway_inputs(wl: synth.Workload, g: synth.Graph, device="cuda") -> KwayInputs:
    cfg, mc = wl.graph, wl.model
    d, K = mc.d, mc.parts
    if mc.kind != "mean" or mc.dtype != "f32" or mc.objective != "bce":
        raise ValueError("the K-subgraph step runs mean layers on float32 rows with the head objective")
    part_np = synth.random_partition(g.n_nodes, K, mc.seed)
    gd = {k: _dev(getattr(g, k), device) for k in ("src", "dst", "rel", "ntype")}
    gd["part"] = _dev(part_np, device)
    keys_ws = api._ws(api.hg_node_keys_workspace_size(g.n_nodes, g.n_edges, cfg.n_rel, cfg.key), device)
    keys = api.hg_node_keys(gd["src"], gd["dst"], gd["rel"], g.n_nodes, cfg.n_rel, cfg.key, ws=keys_ws)
    subs, build_ws = _build_parts(gd, cfg, K, keys)
    feats = synth.features(mc.seed, g.n_nodes, d)
    feats_d = _dev(feats, device)
    weights_np = [synth.layer_weights(mc.seed, li, cfg.n_rel, g.n_ntype, d, mc.bias_range)
                  for li in range(mc.n_layers)]
    weights = [(_dev(w.w_rel, device), _dev(w.w_self, device), _dev(w.bias, device)) for w in weights_np]
    head_np = synth.head_weights(mc.seed, d)
    head = {k: _dev(v, device) for k, v in head_np.items()}
    labels_np = synth.labels(mc.seed, g.ntype)
    labels = _dev(labels_np, device)
    inp = KwayInputs(wl, gd, part_np, subs, build_ws, keys, keys_ws, weights, weights_np, head, head_np,
                     labels, labels_np, _label_rows(labels), feats)
    f32 = dict(dtype=torch.float32, device=device)
    for sb in subs:
        h0 = feats_d.index_select(0, sb.view("local2global").long()).contiguous()
        inp.H.append([h0] + [torch.empty((sb.n_sub, d), **f32) for _ in range(mc.n_layers)])
        inp.saved.append([torch.empty((max(sb.n_sub, 1), d // 32), dtype=torch.int32, device=device)
                          for _ in range(mc.n_layers)])
    del feats_d
    n = g.n_nodes
    ns = max(sb.n_sub for sb in subs)
    m = max(sb.m_sel for sb in subs)
    inp.H_agg = torch.empty((n, d), **f32)
    inp.cnt = torch.empty(n, dtype=torch.int32, device=device)
    inp.dH_agg = torch.empty((n, d), **f32)
    inp.g = torch.empty((ns, d), **f32)
    inp.dH = [torch.empty((ns, d), **f32) for _ in range(2)]
    inp.Y = torch.empty((max(m, 1), d), **f32)
    inp.grads = [(torch.empty_like(w[0]), torch.empty_like(w[1]), torch.empty_like(w[2])) for w in weights]
    inp.head_grads = {k: torch.empty_like(v) for k, v in head.items()}
    inp.fwd_ws = api._ws(max(api.hg_layer_fwd_workspace_size(s, d, torch.float32) for s in subs), device)
    inp.bwd_ws = api._ws(max(api.hg_layer_bwd_workspace_size(s, d, torch.float32) for s in subs), device)
    inp.align_ws = api._ws(api.hg_align_workspace_size(m, d), device)
    inp.head_ws = api._ws(api.hg_mlp_bce_workspace_size(n, d), device)
    inp.loss = torch.empty((K, 3), **f32)
    inp.loss_bce = torch.empty(1, **f32)
    pairs = []
    for w, gw in zip(inp.weights, inp.grads):
        pairs += list(zip(w, gw))
    pairs += [(inp.head[k], inp.head_grads[k]) for k in inp.head]
    inp.adam = [(p, gr, torch.zeros_like(p), torch.zeros_like(p)) for p, gr in pairs]
    return inp


def run_kway_step(inp: KwayInputs, rebuild: bool = True, update: bool = True):
    """One step of Algorithm 1 over the K workers' subgraphs, the workers run
    one after another on this device: each worker's layers map its features
    to H_k; MeanAgg averages every node's copies into H; the head with the
    masked BCE acts on H; every worker aligns its overlap rows with their
    home copies (held constant) through the CCA loss; each worker's backward
    starts from the MeanAgg backward of dL_BCE/dH plus its alignment
    gradient; the shared weights collect the sum of the K workers' gradients
    (what the gradient all-reduce forms); then Adam updates every parameter.
    The node keys of the selection do not depend on the partition block: they
    are computed once and shared by the K builds."""
    cfg, mc = inp.wl.graph, inp.wl.model
    K = len(inp.subs)
    if rebuild:
        gd = inp.graph
        api.hg_node_keys(gd["src"], gd["dst"], gd["rel"], int(gd["ntype"].shape[0]), cfg.n_rel, cfg.key,
                         keys=inp.keys, ws=inp.keys_ws)
        _build_parts(gd, cfg, K, inp.keys, ws=inp.build_ws, subs=inp.subs)
    for k, sb in enumerate(inp.subs):
        for li in range(mc.n_layers):
            w_rel, w_self, bias = inp.weights[li]
            api.hg_layer_fwd(sb, inp.H[k][li], w_rel, w_self, bias, H_out=inp.H[k][li + 1], saved=inp.saved[k][li],
                             ws=inp.fwd_ws)
    g2l = [sb.view("global2local") for sb in inp.subs]
    last = [h[-1] for h in inp.H]
    api.hg_mean_agg_fwd(g2l, last, H=inp.H_agg, cnt=inp.cnt)
    api.hg_mlp_bce_fwd_bwd(inp.H_agg, inp.head["W1"], inp.head["b1"], inp.head["W2"], inp.head["b2"], inp.labels,
                           dH=inp.dH_agg, grads=inp.head_grads, loss=inp.loss_bce, ws=inp.head_ws,
                           rows=inp.label_rows)
    for k, sb in enumerate(inp.subs):
        ns, m = sb.n_sub, sb.m_sel
        l2g = sb.view("local2global")
        overlap = sb.view("overlap")
        g = inp.g[:ns]
        api.hg_mean_agg_bwd(l2g, inp.cnt, inp.dH_agg, dh_part=g)
        Y = inp.Y[:m]
        api.hg_home_gather(overlap, l2g, sb.view("overlap_home"), g2l, last, Y=Y)
        api.hg_align_loss_fwd_bwd(last[k], overlap, Y, g, lambda_n=mc.lambda_n, scale=mc.lambda_cca, eps=mc.eps,
                                  ddof=mc.ddof, loss3=inp.loss[k], ws=inp.align_ws)
        gin, nxt = g, 0
        for li in reversed(range(mc.n_layers)):
            w_rel, w_self, _ = inp.weights[li]
            gw = inp.grads[li]
            api.hg_layer_bwd(sb, inp.H[k][li], w_rel, w_self, inp.saved[k][li], gin, dH_in=inp.dH[nxt][:ns],
                             dW_rel=gw[0], dW_self=gw[1], dbias=gw[2], accumulate=k > 0, ws=inp.bwd_ws)
            gin, nxt = inp.dH[nxt][:ns], 1 - nxt
    if update:
        inp.t += 1
        for p, gr, m1, m2 in inp.adam:
            api.hg_adam_step(p, gr, m1, m2, inp.t, lr=mc.lr, weight_decay=mc.weight_decay)
    return inp
