"""The multi-snapshot step on the GPU (snapshot builds, attention layers and
the temporal module per snapshot, head with masked BCE and the alignment on
the last state, the backward through every snapshot with the activations of
the earlier snapshots computed again, Adam) against the oracle's sequence
step: states, losses and every gradient within 1e-4 of the parity metric.

The ReLU decisions of the layers are taken by the GPU in float32; they must
agree with the oracle's float64 pre-activations except within rounding of
zero, and the oracle's backward then takes the GPU's decisions.  The head's
hidden decisions are not returned by the library: its bias is shifted so
that no labelled row's hidden pre-activation lies within rounding of zero."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import hgt
from oracle import step as oracle_step
from paper_2608_02168_amd import runner, synth
from tests.helpers import clear_relu_kinks, parity_err, unpack_mask

pytestmark = pytest.mark.gpu
TOL = 1e-4


@pytest.mark.parametrize("factor,window", [(0.1, 3), (0.2, 2), (0.1, 1)])
def test_sequence_step_matches_oracle(factor, window):
    base = synth.WORKLOADS["tiny_dyn"]
    from dataclasses import replace
    wl = synth.Workload(synth.scaled(base.graph, factor), replace(base.model, window=window), "tiny_dyn")
    mc = wl.model
    g = synth.make_graph(wl.graph)
    inp = runner.make_seq_inputs(wl, g)
    T, L, d = mc.snapshots, mc.n_layers, mc.d
    cfg = wl.graph
    garr = dict(src=g.src, dst=g.dst, rel=g.rel, ntype=g.ntype, part=g.part)
    bargs = dict(k=g.k, n_rel=cfg.n_rel, n_ntype=2, budget=cfg.budget, key=cfg.key, theta=cfg.theta, seed=cfg.seed)

    def oracle(masks):
        return oracle_step.run_sequence(
            garr, bargs, inp.ts_np, inp.cuts, inp.feats_np, inp.weights_np, mc.heads, inp.tparams_np, window,
            inp.href_np[: inp.subs[0].m_sel], inp.head_np, inp.labels_np, lambda_n=mc.lambda_n,
            scale=mc.lambda_cca, eps=mc.eps, ddof=mc.ddof, masks=masks)

    # the oracle's last state fixes the head's hidden pre-activations before the GPU runs
    pre = oracle(None)
    a = pre["S"][T - 1] @ inp.head_np["W1"].astype(np.float64) + inp.head_np["b1"]
    lab = inp.labels_np[pre["subs"][0].local2global] >= 0
    inp.head_np["b1"] = (inp.head_np["b1"] + clear_relu_kinks(a, lab)).astype(np.float32)
    inp.head["b1"].copy_(torch.from_numpy(inp.head_np["b1"]))
    del pre
    masks, states = [], []

    def grab(t):
        masks.append([unpack_mask(inp.masks[li][: inp.subs[t].n_sub].cpu().numpy(), d) for li in range(L)])
        states.append([x.cpu().numpy().copy() for x in inp.H[1:]])

    runner.run_seq_step(inp, on_snapshot=grab)
    torch.cuda.synchronize()
    print(f"sequence factor={factor} w={window}: e_sub per snapshot {[s.e_sub for s in inp.subs]}", flush=True)
    ref = oracle(masks)
    for t in range(T):
        assert ref["subs"][t].e_sub == inp.subs[t].e_sub
        sb = ref["subs"][t]
        edges = (sb.n_sub, sb.src_l, sb.dst_l, sb.rel_l, sb.ntype_l)
        for li in range(L):
            p = hgt.Params(*[inp.weights_np[li][n] for n in hgt.PARAM_NAMES])
            Z = hgt.forward(*edges, ref["h"][t][li], p, mc.heads)[1]
            near = np.abs(Z) <= 1e-4 * np.sqrt(np.mean(Z * Z))
            assert np.array_equal(masks[t][li][~near], Z[~near] > 0), (t, li)
            assert parity_err(states[t][li], ref["h"][t][li + 1]) <= TOL, (t, li)
    assert parity_err(inp.S[T - 1].cpu().numpy(), ref["S"][T - 1]) <= TOL
    assert abs(float(inp.loss_bce.cpu()[0]) - ref["bce"]) <= 1e-4 * abs(ref["bce"])
    for a, b in zip(inp.loss.cpu().numpy(), ref["losses"]):
        assert abs(a - b) <= 1e-4 * abs(b)
    errs = {}
    for k in ("W1", "b1", "W2", "b2"):
        errs["head " + k] = parity_err(inp.head_grads[k].cpu().numpy(), ref["head_grads"][k])
    for k in inp.tgrads:
        errs["temporal " + k] = parity_err(inp.tgrads[k].cpu().numpy(), ref["temporal_grads"][k])
    for li in range(L):
        for n in hgt.PARAM_NAMES:
            errs[f"layer{li} {n}"] = parity_err(inp.grads[li][n].cpu().numpy(), ref["layer_grads"][li][n])
    worst = sorted(errs.items(), key=lambda kv: -kv[1])[:4]
    assert worst[0][1] <= TOL, worst
