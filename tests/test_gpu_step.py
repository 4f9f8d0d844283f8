"""A whole step (build, 2 layers forward, alignment, 2 layers backward) on
the GPU through the C ABI against the oracle's step.  The ReLU decisions of
the layers are taken by the GPU in float32: its saved masks must agree with
the oracle's float64 pre-activations except within rounding of zero, and the
oracle's backward then takes those checked masks, so the chained gradients
are always compared.  The prediction head's hidden decisions are not
returned by the library; its bias is shifted so that no labelled row's
hidden pre-activation lies within rounding of zero."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import step as oracle_step
from oracle import hgt, layer, select
from paper_2608_02168_amd import runner, synth
from tests.helpers import clear_relu_kinks, parity_err, unpack_mask

pytestmark = pytest.mark.gpu


def _check_masks(ref_sub, h, weights_np, gmasks, heads=None):
    """The GPU's ReLU decisions equal the oracle's z > 0 wherever |z| exceeds
    1e-4 rms(z) (float32 rounding of z stays far inside that band)."""
    edges = (ref_sub.n_sub, ref_sub.src_l, ref_sub.dst_l, ref_sub.rel_l, ref_sub.ntype_l)
    for li, w in enumerate(weights_np):
        if isinstance(w, dict):
            Z = hgt.forward(*edges, h[li], hgt.Params(*[w[n] for n in hgt.PARAM_NAMES]), heads)[1]
        else:
            Z = layer.forward(*edges, h[li], w.w_rel, w.w_self, w.bias)[1]
        near = np.abs(Z) <= 1e-4 * np.sqrt(np.mean(Z * Z))
        assert np.array_equal(gmasks[li][~near], Z[~near] > 0), li


def clear_head_kinks(inp, h_last, local2global):
    """Shift the head's hidden bias (device and host copies) so that no
    labelled row's hidden pre-activation is within rounding of zero."""
    a = h_last @ inp.head_np["W1"].astype(np.float64) + inp.head_np["b1"]
    lab = inp.labels_np[local2global] >= 0
    b1 = (inp.head_np["b1"] + clear_relu_kinks(a, lab)).astype(np.float32)
    inp.head_np["b1"] = b1
    inp.head["b1"].copy_(torch.from_numpy(b1))


@pytest.mark.parametrize("name,factor", [("tiny", 0.3), ("tiny", 0.1), ("skew", 0.001), ("tiny_hgt", 0.3)])
def test_step_matches_oracle(name, factor):
    base = synth.WORKLOADS[name]
    wl = synth.Workload(synth.scaled(base.graph, factor), base.model, name)
    g = synth.make_graph(wl.graph)
    inp = runner.make_inputs(wl, g)
    res = runner.run_step(inp)
    torch.cuda.synchronize()
    sub = inp.sub
    m = sub.m_sel
    d = wl.model.d
    gmasks = [unpack_mask(x[: sub.n_sub].cpu().numpy(), d) for x in inp.saved]
    omega = inp.omega.cpu().numpy() if inp.omega is not None else None
    ref_sub, h, losses, dH0, grads = oracle_step.run(
        dict(src=g.src, dst=g.dst, rel=g.rel, ntype=g.ntype, part=g.part),
        dict(k=g.k, n_rel=wl.graph.n_rel, n_ntype=2, budget=wl.graph.budget, theta=wl.graph.theta,
             seed=wl.graph.seed),
        inp.feats_np, inp.weights_np, inp.href_np[:m], inp.gext_np, omega=omega,
        lambda_n=wl.model.lambda_n, scale=wl.model.lambda_cca, eps=wl.model.eps, ddof=wl.model.ddof,
        heads=wl.model.heads, masks=gmasks)
    _check_masks(ref_sub, h, inp.weights_np, gmasks, wl.model.heads)
    for li in range(len(h) - 1):
        assert parity_err(inp.H[li + 1].cpu().numpy(), h[li + 1]) <= 1e-4
    loss = res.loss.cpu().numpy()
    for a, b in zip(loss, losses):
        assert abs(a - b) <= 1e-4 * abs(b)
    assert parity_err(res.dH0.cpu().numpy(), dH0) <= 1e-4
    for gw, rw in zip(res.grads, grads):
        if isinstance(rw, dict):
            for n in rw:
                assert parity_err(gw[n].cpu().numpy(), rw[n]) <= 1e-4, n
            continue
        for a, b in zip(gw, rw):
            assert parity_err(a.cpu().numpy(), b) <= 1e-4


def test_full_objective_step_matches_oracle():
    """The step with the prediction head, masked BCE (replacing the synthetic
    upstream gradient) and one Adam update of every parameter."""
    from oracle import objective
    base = synth.WORKLOADS["tiny_full"]
    wl = synth.Workload(synth.scaled(base.graph, 0.3), base.model, "tiny_full")
    g = synth.make_graph(wl.graph)
    inp = runner.make_inputs(wl, g)
    mc = wl.model
    # the oracle's forward fixes the head's hidden pre-activations before either side runs
    sb = select.build(g.src, g.dst, g.rel, g.ntype, g.part, g.k, wl.graph.n_rel, 2, wl.graph.budget,
                      wl.graph.key, wl.graph.theta, wl.graph.seed)
    x = inp.feats_np[sb.local2global].astype(np.float64)
    for w in inp.weights_np:
        x = layer.forward(sb.n_sub, sb.src_l, sb.dst_l, sb.rel_l, sb.ntype_l, x, w.w_rel, w.w_self, w.bias)[0]
    clear_head_kinks(inp, x, sb.local2global)
    before = [p.detach().cpu().numpy().copy() for p, _, _, _ in inp.adam]
    res = runner.run_step(inp)
    torch.cuda.synchronize()
    m = inp.sub.m_sel
    gmasks = [unpack_mask(x[: inp.sub.n_sub].cpu().numpy(), mc.d) for x in inp.saved]
    ref_sub, h, losses, dH0, grads, head = oracle_step.run(
        dict(src=g.src, dst=g.dst, rel=g.rel, ntype=g.ntype, part=g.part),
        dict(k=g.k, n_rel=wl.graph.n_rel, n_ntype=2, budget=wl.graph.budget, theta=wl.graph.theta,
             seed=wl.graph.seed),
        inp.feats_np, inp.weights_np, inp.href_np[:m], inp.gext_np, lambda_n=mc.lambda_n, scale=mc.lambda_cca,
        eps=mc.eps, ddof=mc.ddof, head=inp.head_np, labels_global=inp.labels_np, masks=gmasks)
    for li in range(len(h) - 1):
        assert parity_err(inp.H[li + 1].cpu().numpy(), h[li + 1]) <= 1e-4
    assert abs(float(inp.loss_bce.cpu()[0]) - head["loss"]) <= 1e-4 * abs(head["loss"])
    for a, b in zip(res.loss.cpu().numpy(), losses):
        assert abs(a - b) <= 1e-4 * abs(b)
    _check_masks(ref_sub, h, inp.weights_np, gmasks)
    assert parity_err(res.dH0.cpu().numpy(), dH0) <= 1e-4
    ref_grads = []
    for gw, rw in zip(res.grads, grads):
        for x, y in zip(gw, rw):
            assert parity_err(x.cpu().numpy(), y) <= 1e-4
            ref_grads.append(y)
    for k in ("W1", "b1", "W2", "b2"):
        assert parity_err(inp.head_grads[k].cpu().numpy(), head[k]) <= 1e-4, k
        ref_grads.append(head[k])
    # one Adam step from zero moments: each coordinate moves by about lr * sign(g + wd theta)
    n_sure = n_all = 0
    for (p, _, _, _), th0, gr in zip(inp.adam, before, ref_grads):
        th0 = th0.astype(np.float64)
        exp, _, _ = objective.adam_step(th0, gr, np.zeros_like(th0), np.zeros_like(th0), 1, lr=mc.lr,
                                        weight_decay=mc.weight_decay)
        got = p.detach().cpu().numpy().astype(np.float64)
        gh = gr + mc.weight_decay * th0
        # the gradients agree within 1e-4 * max(|g|, rms(g)) (asserted above), so
        # the sign the first step follows is settled where |g| exceeds twice that
        sure = np.abs(gh) > 2e-4 * np.sqrt(np.mean(gr * gr))
        ulp = np.spacing(np.abs(exp).astype(np.float32)).astype(np.float64)
        assert np.all(np.abs(got - exp)[sure] <= ulp[sure] + 1e-4 * np.abs(exp - th0)[sure])
        # elsewhere (e.g. the type-1 bias, whose gradient is zero without
        # labelled type-1 rows) the step is still bounded by the learning rate
        assert np.all(np.abs(got - th0) <= 1.001 * mc.lr + np.spacing(np.abs(th0).astype(np.float32)))
        n_sure += int(sure.sum())
        n_all += sure.size
    assert n_sure > 0.8 * n_all
