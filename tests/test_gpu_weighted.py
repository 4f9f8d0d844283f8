"""Weighted edges: each message is multiplied by its edge's weight w_ij and
the mean's normaliser stays the in-edge count.  The build carries the weight
of every CSR entry (csr_w) and folds it into csc_scale = w / deg_r(dst);
checked bit-exactly against the oracle's build (through the sort payload, and
through the edge ids when those are asked for too), and the mean layer's
forward and backward against the oracle with the same weights, including
destination rows long enough to be cut into chunks.  The attention layer
refuses a weighted subgraph."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import layer, select
from paper_2608_02168_amd import api, synth
from tests.helpers import graph_to_dev, pack_mask, parity_err, to_dev, unpack_mask
from tests.test_gpu_build import assert_same
from tests.test_gpu_dest_hubs import with_reversed_hubs

pytestmark = pytest.mark.gpu
TOL = 1e-4

CFGS = {
    "tiny": synth.WORKLOADS["tiny"].graph,
    "medium": synth.WORKLOADS["medium"].graph,
    "tiny_hubs": "tiny+reversed hubs",
}


def make(name):
    if name == "tiny_hubs":
        g = with_reversed_hubs(synth.make_graph(synth.scaled(synth.WORKLOADS["medium"].graph, 0.02)), n_hubs=4)
    else:
        g = synth.make_graph(CFGS[name])
    return g, synth.edge_weights(13, g.n_edges)


def build(g, w, want_eid=True):
    cfg = g.cfg
    d = graph_to_dev(g)
    return api.hg_build_csr(d["src"], d["dst"], d["rel"], d["ntype"], d["part"], g.k, cfg.n_rel, 2, cfg.budget,
                            key=cfg.key, theta=cfg.theta, seed=cfg.seed, want_eid=want_eid, edge_w=to_dev(w))


def oracle_build(g, w):
    cfg = g.cfg
    return select.build(g.src, g.dst, g.rel, g.ntype, g.part, g.k, cfg.n_rel, 2, cfg.budget, key=cfg.key,
                        theta=cfg.theta, seed=cfg.seed, edge_w=w)


@pytest.mark.parametrize("name", sorted(CFGS))
def test_weighted_build_bit_exact(name):
    g, w = make(name)
    sub, ref = build(g, w), oracle_build(g, w)
    assert int(sub.c.weighted) == 1
    assert_same(ref, sub)  # csc_scale bits included: w / deg as a float32 quotient
    got = sub.view("csr_w").cpu().numpy()
    assert np.array_equal(got.view(np.uint32), ref.csr_w.view(np.uint32))
    # without edge ids the weights travel through the CSR sort instead
    sub2 = build(g, w, want_eid=False)
    assert np.array_equal(sub2.view("csr_w").cpu().numpy().view(np.uint32), ref.csr_w.view(np.uint32))
    assert np.array_equal(sub2.view("csc_scale").cpu().numpy().view(np.uint32), ref.csc_scale.view(np.uint32))


@pytest.mark.parametrize("name,d", [("tiny", 64), ("tiny", 128), ("tiny_hubs", 64), ("medium", 64)])
def test_weighted_mean_layer(name, d):
    g, w = make(name)
    sub, ref = build(g, w), oracle_build(g, w)
    if name == "tiny_hubs":
        assert int(sub.c.plan_fwd_heavy) > 0  # chunked destination rows carry weights too
    edges = (ref.n_sub, ref.src_l, ref.dst_l, ref.rel_l, ref.ntype_l)
    H = synth.features(17, g.n_nodes, d)[ref.local2global]
    lw = synth.layer_weights(17, 0, g.cfg.n_rel, 2, d, 0.1)
    Hd, wr, wsf, b = to_dev(H), to_dev(lw.w_rel), to_dev(lw.w_self), to_dev(lw.bias)
    out, saved = api.hg_layer_fwd(sub, Hd, wr, wsf, b)
    exp, Z = layer.forward(*edges, H, lw.w_rel, lw.w_self, lw.bias, edge_w=ref.w_l)
    assert parity_err(out.cpu().numpy(), exp) <= TOL
    gm = unpack_mask(saved.cpu().numpy(), d)
    near = np.abs(Z) <= TOL * np.sqrt(np.mean(Z * Z))
    assert np.array_equal(gm[~near], Z[~near] > 0)
    G = synth.upstream_grad(17, ref.n_sub, d)
    got = api.hg_layer_bwd(sub, Hd, wr, wsf, to_dev(pack_mask(gm)), to_dev(G))
    want = layer.backward(*edges, H, lw.w_rel, lw.w_self, lw.bias, G, mask=gm, edge_w=ref.w_l)
    for a, e, nm in zip(got, want, ("dH", "dW_rel", "dW_self", "dbias")):
        err = parity_err(a.cpu().numpy(), e)
        assert err <= TOL, (nm, err)


def test_attention_refuses_weighted_subgraph():
    g, w = make("tiny")
    sub = build(g, w)
    d, heads = 64, 4
    wd = {k: to_dev(v) for k, v in synth.hgt_weights(3, 0, g.cfg.n_rel, 2, d, heads, 0.1).items()}
    with pytest.raises(RuntimeError, match="weights"):
        api.hg_hgt_fwd(sub, to_dev(np.zeros((sub.n_sub, d), np.float32)), wd, heads)
