"""Destination hubs.  The paper's graphs carry the inverse of every relation
(a relation and its reverse, Problem Formulation), so a source hub with
millions of out-edges is also a destination with millions of in-edges.
Destination rows longer than the plan's chunk are split into chunks whose
partial sums (mean layer), softmax states (attention forward) and dQ shares
(attention backward) are merged in chunk order.

Graphs: the 1M-node / 20M-edge workload with the out-edges of its 16 largest
source hubs added reversed as a fifth relation (the largest reversed row
holds about 3.8M in-edges), and the same recipe at a twentieth of the size
for the attention layer (largest row about 190k in-edges).  Checked against
the oracle: the build bit-exact, every output of one mean layer forward and
backward, every output of one attention layer forward and backward; and the
forward's time per edge on the hub graph against the graph without the
reversed relation (no row walked by one wave alone)."""
from dataclasses import replace

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import hgt, layer, select
from paper_2608_02168_amd import api, synth
from tests.helpers import graph_to_dev, pack_mask, parity_err, to_dev, unpack_mask
from tests.test_gpu_build import assert_same

pytestmark = pytest.mark.gpu
TOL = 1e-4
CHUNK = 2048  # destination rows longer than this are split (the library's chunk)


def with_reversed_hubs(g, n_hubs=16):
    """g plus the out-edges of its n_hubs largest sources, reversed, as
    relation n_rel (appended after the original edges)."""
    outdeg = np.bincount(g.src, minlength=g.n_nodes)
    hubs = np.argsort(outdeg, kind="stable")[-n_hubs:]
    m = np.isin(g.src, hubs)
    R = g.cfg.n_rel
    src = np.concatenate([g.src, g.dst[m]]).astype(np.int32)
    dst = np.concatenate([g.dst, g.src[m]]).astype(np.int32)
    rel = np.concatenate([g.rel, np.full(int(m.sum()), R, np.uint8)])
    cfg = replace(g.cfg, name=g.cfg.name + "+reversed hubs", n_rel=R + 1, n_edges=src.shape[0])
    return synth.Graph(cfg, src, dst, rel, g.ntype, g.part, g.k)


def build_both(g):
    cfg = g.cfg
    d = graph_to_dev(g)
    sub = api.hg_build_csr(d["src"], d["dst"], d["rel"], d["ntype"], d["part"], g.k, cfg.n_rel, 2, cfg.budget,
                           key=cfg.key, theta=cfg.theta, seed=cfg.seed, want_eid=True)
    ref = select.build(g.src, g.dst, g.rel, g.ntype, g.part, g.k, cfg.n_rel, 2, cfg.budget, key=cfg.key,
                       theta=cfg.theta, seed=cfg.seed)
    return sub, ref


@pytest.fixture(scope="module")
def medium_hubs():
    g = with_reversed_hubs(synth.make_graph(synth.WORKLOADS["medium"].graph))
    sub, ref = build_both(g)
    yield g, sub, ref
    del sub
    torch.cuda.empty_cache()


def test_hub_graph_build_bit_exact(medium_hubs):
    g, sub, ref = medium_hubs
    indeg = np.diff(ref.csr_ptr[:: g.cfg.n_rel])
    print(f"hub graph: E={g.n_edges} e_sub={sub.e_sub} largest destination row {indeg.max()} "
          f"rows over {CHUNK}: {(indeg > CHUNK).sum()} chunks {int(sub.c.plan_fwd_parts)}", flush=True)
    assert indeg.max() > 1_000_000
    assert int(sub.c.plan_fwd_heavy) == int((indeg > CHUNK).sum())
    assert int(sub.c.plan_fwd_parts) == int(np.sum(-(-indeg[indeg > CHUNK] // CHUNK)))
    assert_same(ref, sub)


def test_hub_graph_mean_layer_every_output(medium_hubs):
    g, sub, ref = medium_hubs
    d, R = 64, g.cfg.n_rel
    H = synth.features(8, g.n_nodes, d)[ref.local2global]
    w = synth.layer_weights(8, 0, R, 2, d, 0.1)
    edges = (sub.n_sub, ref.src_l, ref.dst_l, ref.rel_l, ref.ntype_l)
    Hd, wr, wsf, b = to_dev(H), to_dev(w.w_rel), to_dev(w.w_self), to_dev(w.bias)
    out, saved = api.hg_layer_fwd(sub, Hd, wr, wsf, b)
    exp, Z = layer.forward(*edges, H, w.w_rel, w.w_self, w.bias)
    assert parity_err(out.cpu().numpy(), exp) <= TOL
    gm = unpack_mask(saved.cpu().numpy(), d)
    near = np.abs(Z) <= TOL * np.sqrt(np.mean(Z * Z))
    assert np.array_equal(gm[~near], Z[~near] > 0)
    # the hub destinations themselves
    hubs = np.argsort(np.diff(ref.csr_ptr[:: R]))[-16:]
    assert parity_err(out.cpu().numpy()[hubs], exp[hubs]) <= TOL
    G = np.random.default_rng(9).standard_normal((sub.n_sub, d)).astype(np.float32)
    got = api.hg_layer_bwd(sub, Hd, wr, wsf, to_dev(pack_mask(gm)), to_dev(G))
    want = layer.backward(*edges, H, w.w_rel, w.w_self, w.bias, G, mask=gm)
    for a, e, nm in zip(got, want, ("dH", "dW_rel", "dW_self", "dbias")):
        err = parity_err(a.cpu().numpy(), e)
        assert err <= TOL, (nm, err)


def test_hub_graph_forward_time_per_edge(medium_hubs):
    """The forward aggregation's time per edge on the hub graph stays within
    twice that of the same graph without the reversed relation: the 3.8M-edge
    row is spread over the chip, not walked by one wave."""
    g, sub, _ = medium_hubs
    base = synth.make_graph(synth.WORKLOADS["medium"].graph)
    sub0, _ = build_both(base)
    d = 64
    per_edge = []
    for gg, s in ((base, sub0), (g, sub)):
        H = to_dev(synth.features(8, gg.n_nodes, d)[:s.n_sub])
        w = synth.layer_weights(8, 0, gg.cfg.n_rel, 2, d, 0.1)
        wr, wsf, b = to_dev(w.w_rel), to_dev(w.w_self), to_dev(w.bias)
        api.hg_layer_fwd(s, H, wr, wsf, b)
        torch.cuda.synchronize()
        api.hg_timing_collect()
        api.hg_timing_enable(True)
        for _ in range(3):
            api.hg_layer_fwd(s, H, wr, wsf, b)
        torch.cuda.synchronize()
        api.hg_timing_enable(False)
        kern = api.hg_timing_collect()
        ms = sum(v[1] for k, v in kern.items() if k.startswith("spmm_fwd")) / 3
        per_edge.append(ms / s.e_sub)
        print(f"{gg.cfg.name}: e_sub={s.e_sub} aggregation {ms:.3f} ms "
              f"({ {k: round(v[1] / 3, 3) for k, v in kern.items() if k.startswith('spmm_fwd')} })", flush=True)
    assert per_edge[1] <= 2.0 * per_edge[0], per_edge


def test_hub_graph_attention_layer():
    g = with_reversed_hubs(synth.make_graph(synth.scaled(synth.WORKLOADS["medium"].graph, 0.05)))
    sub, ref = build_both(g)
    indeg = np.diff(ref.csr_ptr[:: g.cfg.n_rel])
    assert indeg.max() > 50 * CHUNK and int(sub.c.plan_fwd_heavy) > 0
    d, heads, R = 64, 4, g.cfg.n_rel
    edges = (ref.n_sub, ref.src_l, ref.dst_l, ref.rel_l, ref.ntype_l)
    X = synth.features(9, g.n_nodes, d)[ref.local2global]
    w = synth.hgt_weights(9, 0, R, 2, d, heads, 0.1)
    p = hgt.Params(*[w[n] for n in hgt.PARAM_NAMES])
    wd = {n: to_dev(v) for n, v in w.items()}
    Xd = to_dev(X)
    out, mask, saved = api.hg_hgt_fwd(sub, Xd, wd, heads)
    _, Z, _, _ = hgt.forward(*edges, X, p, heads)
    exp = np.maximum(Z, 0) + X
    assert parity_err(out.cpu().numpy(), exp) <= TOL
    gm = unpack_mask(mask.cpu().numpy(), d)
    near = np.abs(Z) <= TOL * np.sqrt(np.mean(Z * Z))
    assert np.array_equal(gm[~near], Z[~near] > 0)
    G = synth.upstream_grad(9, ref.n_sub, d)
    dH, grads = api.hg_hgt_bwd(sub, Xd, wd, heads, to_dev(pack_mask(gm)), saved, to_dev(G))
    edH, eg = hgt.backward(*edges, X, p, heads, G, mask=gm)
    errs = {"dH": parity_err(dH.cpu().numpy(), edH)}
    for n in hgt.PARAM_NAMES:
        errs[n] = parity_err(grads[n].cpu().numpy(), getattr(eg, n))
    assert max(errs.values()) <= TOL, errs
