"""Many relation types: the paper's risk graph has more than 60 risk-event
relations.  The relation transforms Y_r, their gradients dY_r and the
attention layer's per-relation keys and values take one row per active
(source, relation) pair, A rows in all, so their buffers grow with A and not
with n_sub * R.

On a 1M-node / 10M-edge graph with 64 uniform relations (Zipf(1.2) sources,
d = 64): the build bit-exact against the oracle, every output of one mean
layer forward and backward against the oracle (float32 bar 1e-4, the ReLU
decisions checked outside the rounding band and then passed to the oracle),
and the workspaces sized by A.  The attention layer at R = 64 is covered by
the attention tests' rel64 configuration."""
from dataclasses import replace

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import layer, select
from paper_2608_02168_amd import api, synth
from tests.helpers import graph_to_dev, parity_err, to_dev, unpack_mask
from tests.test_gpu_build import assert_same

pytestmark = pytest.mark.gpu
TOL = 1e-4
R = 64

GRAPH = replace(synth.WORKLOADS["medium"].graph, name="rel64", n_edges=10_000_000, n_rel=R, seed=7)


@pytest.fixture(scope="module")
def built():
    g = synth.make_graph(GRAPH)
    d = graph_to_dev(g)
    cfg = GRAPH
    sub = api.hg_build_csr(d["src"], d["dst"], d["rel"], d["ntype"], d["part"], g.k, R, 2, cfg.budget,
                           key=cfg.key, theta=cfg.theta, seed=cfg.seed, want_eid=True)
    del d
    ref = select.build(g.src, g.dst, g.rel, g.ntype, g.part, g.k, R, 2, cfg.budget, key=cfg.key,
                       theta=cfg.theta, seed=cfg.seed)
    yield g, sub, ref
    del sub
    torch.cuda.empty_cache()


def test_rel64_build_bit_exact(built):
    _, sub, ref = built
    print(f"rel64: n_sub={sub.n_sub} e_sub={sub.e_sub} A={sum(sub.n_active())}", flush=True)
    assert_same(ref, sub)


def test_rel64_workspaces_scale_with_active_pairs(built):
    _, sub, _ = built
    d, A, ns = 64, sum(sub.n_active()), sub.n_sub
    assert A < ns * R // 4  # most (node, relation) pairs are empty at R = 64
    assert int(sub.c.plan_slot_rows) == A  # so the transforms take the compact layout
    fwd = api.hg_layer_fwd_workspace_size(sub, d, torch.float32)
    bwd = api.hg_layer_bwd_workspace_size(sub, d, torch.float32)
    # forward: Y (A rows) and Y_self (n_sub rows); backward: dZ (n_sub rows),
    # dY (A rows), split partial rows and split-K scratch
    assert (A + ns) * d * 4 <= fwd <= (A + ns) * d * 4 + (1 << 20)
    assert bwd <= (A + ns) * d * 4 + int(sub.c.plan_partials) * d * 8 + (64 << 20)
    assert bwd < ns * R * d * 4 // 2


@pytest.fixture(scope="module")
def layer_run(built):
    """One mean layer forward and backward on the GPU (float32, d = 64)."""
    g, sub, ref = built
    d = 64
    H = synth.features(5, g.n_nodes, d)[ref.local2global]
    w = synth.layer_weights(5, 0, R, 2, d, 0.1)
    Hd, wr, wsf, b = to_dev(H), to_dev(w.w_rel), to_dev(w.w_self), to_dev(w.bias)
    out, saved = api.hg_layer_fwd(sub, Hd, wr, wsf, b)
    G = np.random.default_rng(11).standard_normal((sub.n_sub, d)).astype(np.float32)
    got = api.hg_layer_bwd(sub, Hd, wr, wsf, saved, to_dev(G))
    res = dict(H=H, w=w, G=G, out=out.cpu().numpy(), mask=unpack_mask(saved.cpu().numpy(), d),
               grads=[x.cpu().numpy() for x in got])
    del Hd, out, saved, got
    torch.cuda.empty_cache()
    return res


def test_rel64_mean_layer_forward(built, layer_run):
    _, sub, ref = built
    r = layer_run
    exp, Z = layer.forward(sub.n_sub, ref.src_l, ref.dst_l, ref.rel_l, ref.ntype_l, r["H"], r["w"].w_rel,
                           r["w"].w_self, r["w"].bias)
    assert parity_err(r["out"], exp) <= TOL
    near = np.abs(Z) <= TOL * np.sqrt(np.mean(Z * Z))
    assert np.array_equal(r["mask"][~near], Z[~near] > 0)


def test_rel64_mean_layer_backward(built, layer_run):
    """Under the GPU's ReLU decisions (checked by the forward test outside
    the rounding band of zero)."""
    _, sub, ref = built
    r = layer_run
    want = layer.backward(sub.n_sub, ref.src_l, ref.dst_l, ref.rel_l, ref.ntype_l, r["H"], r["w"].w_rel,
                          r["w"].w_self, r["w"].bias, r["G"], mask=r["mask"])
    for a, e, nm in zip(r["grads"], want, ("dH", "dW_rel", "dW_self", "dbias")):
        err = parity_err(a, e)
        assert err <= TOL, (nm, err)
