"""K subgraphs of one graph on the GPU through the C ABI against the oracle
(oracle/kway.py): MeanAgg forward and backward on random subgraph maps
(K = 1, 3 and 5, float32 and bfloat16, every width), the home-copy gather
on real subgraph builds (bit-exact: it is a copy), its NaN rows for
inconsistent inputs, and a whole K-worker step (K builds, mean layers,
MeanAgg, head with masked BCE, home-copy alignment, summed weight gradients)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import kway, layer
from paper_2608_02168_amd import api, runner, synth
from tests.helpers import parity_err, to_dev, unpack_mask

pytestmark = pytest.mark.gpu


def random_maps(rng, n, K):
    """K subgraphs over n nodes: every node in its own block's subgraph and in
    a few others; local order = ascending global id (any injective order
    works for these calls)."""
    part = rng.integers(0, K, n)
    extra = rng.random((K, n)) < 0.15
    l2gs, g2ls = [], []
    for k in range(K):
        ids = np.nonzero((part == k) | extra[k])[0].astype(np.int32)
        rng.shuffle(ids)
        g2l = np.full(n, -1, dtype=np.int32)
        g2l[ids] = np.arange(ids.shape[0], dtype=np.int32)
        l2gs.append(ids)
        g2ls.append(g2l)
    return l2gs, g2ls


@pytest.mark.parametrize("K", [1, 3, 5])
@pytest.mark.parametrize("d,dtype", [(64, torch.float32), (128, torch.float32), (256, torch.float32),
                                     (128, torch.bfloat16)])
def test_mean_agg_matches_oracle(K, d, dtype):
    rng = np.random.default_rng(K * 1000 + d)
    n = 3001
    l2gs, g2ls = random_maps(rng, n, K)
    Hs = [rng.normal(0, 1, (l.shape[0], d)).astype(np.float32) for l in l2gs]
    if dtype == torch.bfloat16:
        Hs = [synth.round_bf16(h) for h in Hs]
    H_ref, cnt_ref = kway.mean_agg(n, l2gs, Hs)
    g2l_d = [to_dev(g) for g in g2ls]
    H, cnt = api.hg_mean_agg_fwd(g2l_d, [to_dev(h).to(dtype) for h in Hs])
    torch.cuda.synchronize()
    assert np.array_equal(cnt.cpu().numpy(), cnt_ref)
    tol = 1e-6 if dtype == torch.float32 else 8e-3
    assert parity_err(H.float().cpu().numpy(), H_ref) <= tol
    # backward into every subgraph, then once more accumulated
    dH = rng.normal(0, 1, (n, d)).astype(np.float32)
    if dtype == torch.bfloat16:
        dH = synth.round_bf16(dH)
    want = kway.mean_agg_backward(l2gs, cnt_ref, dH)
    for l2g, w in zip(l2gs, want):
        got = api.hg_mean_agg_bwd(to_dev(l2g), cnt, to_dev(dH).to(dtype))
        assert parity_err(got.float().cpu().numpy(), w) <= tol
        api.hg_mean_agg_bwd(to_dev(l2g), cnt, to_dev(dH).to(dtype), dh_part=got, accumulate=True)
        assert parity_err(got.float().cpu().numpy(), 2 * w) <= tol


def test_mean_agg_node_in_no_subgraph_is_zero():
    n, d = 100, 64
    l2g = np.arange(0, n, 2, dtype=np.int32)
    g2l = np.full(n, -1, dtype=np.int32)
    g2l[l2g] = np.arange(l2g.shape[0], dtype=np.int32)
    h = np.random.default_rng(0).normal(0, 1, (l2g.shape[0], d)).astype(np.float32)
    H, cnt = api.hg_mean_agg_fwd([to_dev(g2l)], [to_dev(h)])
    H, cnt = H.cpu().numpy(), cnt.cpu().numpy()
    assert np.all(H[1::2] == 0) and np.all(cnt[1::2] == 0) and np.all(cnt[::2] == 1)
    assert np.array_equal(H[::2], h)


def small_kway(factor=0.3, budget=None, parts=None):
    from dataclasses import replace
    base = synth.WORKLOADS["tiny_kway"]
    gc = synth.scaled(base.graph, factor)
    if budget is not None:
        gc = replace(gc, budget=budget)
    mc = base.model if parts is None else replace(base.model, parts=parts)
    return synth.Workload(gc, mc, "tiny_kway")


def test_home_gather_bit_exact_on_real_subgraphs():
    wl = small_kway()
    g = synth.make_graph(wl.graph)
    inp = runner.make_kway_inputs(wl, g)
    runner.run_kway_step(inp, update=False)
    torch.cuda.synchronize()
    last = [h[-1] for h in inp.H]
    g2l = [sb.view("global2local") for sb in inp.subs]
    # the oracle's home rows on the GPU subgraphs' own maps
    from types import SimpleNamespace
    osubs = [SimpleNamespace(local2global=sb.view("local2global").cpu().numpy(),
                             global2local=sb.view("global2local").cpu().numpy(),
                             overlap=sb.view("overlap").cpu().numpy()) for sb in inp.subs]
    H_np = [h.cpu().numpy() for h in last]
    total = 0
    for k, sb in enumerate(inp.subs):
        Y = api.hg_home_gather(sb.view("overlap"), sb.view("local2global"), sb.view("overlap_home"), g2l, last)
        home, rows = kway.home_rows(osubs, inp.part_np, k)
        assert np.array_equal(sb.view("overlap_home").cpu().numpy(), home)
        want = np.stack([H_np[h][r] for h, r in zip(home, rows)]) if rows.size else np.zeros((0, wl.model.d))
        assert np.array_equal(Y.cpu().numpy(), want)
        total += rows.size
    assert total > 0


def test_home_gather_poisons_inconsistent_rows():
    n, d = 64, 64
    l2g = np.arange(n, dtype=np.int32)
    g2l0 = l2g.copy()
    g2l1 = np.full(n, -1, dtype=np.int32)          # subgraph 1 holds no node
    h0 = np.ones((n, d), dtype=np.float32)
    overlap = np.array([0, 1, 2, 3], dtype=np.int32)
    home = np.array([0, 1, 7, -1], dtype=np.int32)  # valid, absent node, out of range twice
    Y = api.hg_home_gather(to_dev(overlap), to_dev(l2g), to_dev(home), [to_dev(g2l0), to_dev(g2l1)],
                           [to_dev(h0), to_dev(h0)]).cpu().numpy()
    assert np.all(Y[0] == 1) and np.all(np.isnan(Y[1:]))


@pytest.mark.parametrize("factor,parts,budget", [(0.3, None, None), (0.1, None, None), (0.2, 2, None),
                                                (0.3, 7, 60), (0.2, 3, 0)])
def test_kway_step_matches_oracle(factor, parts, budget):
    """Every size of a 4-way split, a 2-way and a 7-way split (ragged blocks,
    small budget) and a split with no overlap at all (copy counts all 1, no
    alignment term)."""
    wl = small_kway(factor, budget=budget, parts=parts)
    mc, cfg = wl.model, wl.graph
    g = synth.make_graph(cfg)
    inp = runner.make_kway_inputs(wl, g)
    runner.run_kway_step(inp, update=False)
    torch.cuda.synchronize()
    gmasks = [[unpack_mask(inp.saved[k][li][: sb.n_sub].cpu().numpy(), mc.d) for li in range(mc.n_layers)]
              for k, sb in enumerate(inp.subs)]
    out = kway.run_kway(dict(src=g.src, dst=g.dst, rel=g.rel, ntype=g.ntype, part=inp.part_np), mc.parts,
                        dict(n_rel=cfg.n_rel, n_ntype=2, budget=cfg.budget, key=cfg.key, theta=cfg.theta,
                             seed=cfg.seed),
                        inp.feats_np, inp.weights_np, inp.head_np, inp.labels_np, lambda_n=mc.lambda_n,
                        scale=mc.lambda_cca, eps=mc.eps, ddof=mc.ddof, masks=gmasks)
    for k, (sb, osb) in enumerate(zip(inp.subs, out["subs"])):
        assert np.array_equal(sb.view("local2global").cpu().numpy(), osb.local2global)
        assert np.array_equal(sb.view("overlap").cpu().numpy(), osb.overlap)
        assert sb.e_sub == osb.e_sub
        assert osb.overlap.shape[0] > 1 or wl.graph.budget == 0
    assert np.array_equal(inp.cnt.cpu().numpy(), out["cnt"])
    # the GPU's ReLU decisions agree with the oracle's z > 0 outside the
    # rounding band, and the oracle's backward took them (gmasks)
    for k, osb in enumerate(out["subs"]):
        edges = (osb.n_sub, osb.src_l, osb.dst_l, osb.rel_l, osb.ntype_l)
        for li, w in enumerate(inp.weights_np):
            _, Z = layer.forward(*edges, out["h"][k][li], w.w_rel, w.w_self, w.bias)
            near = np.abs(Z) <= 1e-4 * np.sqrt(np.mean(Z * Z))
            assert np.array_equal(gmasks[k][li][~near], Z[~near] > 0), (k, li)
            assert parity_err(inp.H[k][li + 1].cpu().numpy(), out["h"][k][li + 1]) <= 1e-4
    assert parity_err(inp.H_agg.cpu().numpy(), out["H"]) <= 1e-4
    assert abs(float(inp.loss_bce.cpu()[0]) - out["bce"]) <= 1e-4 * abs(out["bce"])
    loss = inp.loss.cpu().numpy()
    for k in range(mc.parts):
        for a, b in zip(loss[k], out["losses"][k]):
            assert abs(a - b) <= 1e-4 * abs(b), (k, a, b)
    for n in ("W1", "b1", "W2", "b2"):
        assert parity_err(inp.head_grads[n].cpu().numpy(), np.asarray(out["head_grads"][n]).reshape(
            inp.head_grads[n].shape)) <= 1e-4, n
    for (a1, a2, a3), (b1, b2, b3) in zip(inp.grads, out["layer_grads"]):
        for a, b, name in ((a1, b1, "dW_rel"), (a2, b2, "dW_self"), (a3, b3, "dbias")):
            assert parity_err(a.cpu().numpy(), b) <= 1e-4, name


def test_kway_step_deterministic():
    wl = small_kway(0.1)
    g = synth.make_graph(wl.graph)
    inp = runner.make_kway_inputs(wl, g)
    runner.run_kway_step(inp, update=False)
    a = [t.clone() for gw in inp.grads for t in gw] + [inp.H_agg.clone(), inp.loss.clone()]
    runner.run_kway_step(inp, update=False)
    b = [t for gw in inp.grads for t in gw] + [inp.H_agg, inp.loss]
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
