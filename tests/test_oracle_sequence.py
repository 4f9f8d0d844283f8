"""Pins of the oracle's multi-snapshot step (oracle/step.run_sequence): its
gradients against central finite differences of the total objective
J = L_BCE + lambda_CCA L_CCA on a small graph, for a weight of each kind
(attention layers shared over snapshots, temporal module, head) and the
features -- this checks the chaining through time (a state's gradient from
every later snapshot whose context holds it) and the sums over snapshots --
plus the structure of the snapshots (nested, one node set)."""
import numpy as np
import pytest

from oracle import step
from paper_2608_02168_amd import synth

D, HEADS, R = 8, 2, 2


def small_case(seed):
    rng = np.random.default_rng(seed)
    n, e = 36, 170
    src = rng.integers(0, n, e)
    dst = rng.integers(0, n, e)
    rel = rng.integers(0, R, e).astype(np.uint8)
    ntype = (rng.random(n) < 0.3).astype(np.uint8)
    part = rng.integers(0, 3, n).astype(np.int32)
    ts = rng.integers(0, 12, e)
    feats = rng.normal(0, 1, (n, D))
    weights = [synth.hgt_weights(seed, li, R, 2, D, HEADS, bias_range=0.1) for li in range(2)]
    tparams = {k: v.astype(np.float64) for k, v in synth.temporal_weights(seed, D).items()}
    head = {k: v.astype(np.float64) for k, v in synth.head_weights(seed, D).items()}
    head["b1"] = rng.uniform(-0.1, 0.1, D)
    labels = np.where(rng.random(n) < 0.6, rng.integers(0, 2, n), -1)
    href = rng.normal(0, 1, (n, D))
    return dict(graph=dict(src=src, dst=dst, rel=rel, ntype=ntype, part=part),
                build=dict(k=1, n_rel=R, n_ntype=2, budget=6, seed=3), ts=ts, cuts=[3, 7, 11], feats=feats,
                weights=weights, tparams=tparams, head=head, labels=labels, href=href)


def run(c, window=2):
    return step.run_sequence(c["graph"], c["build"], c["ts"], c["cuts"], c["feats"], c["weights"], HEADS,
                             c["tparams"], window, c["href"], c["head"], c["labels"], scale=0.1)


def objective_value(c, window=2):
    out = run(c, window)
    return out["bce"] + 0.1 * out["losses"][2]


@pytest.mark.parametrize("window", [1, 2])
def test_sequence_gradients_match_finite_differences(window):
    c = small_case(5)
    out = run(c, window)
    assert len(out["S"]) == 3
    rng = np.random.default_rng(9)
    checks = []
    for k in ("Q", "r", "Wi", "bh"):
        checks.append((c["tparams"][k], out["temporal_grads"][k], "temporal " + k))
    for li in range(2):
        for k in ("W_att", "W_Q", "mu", "b_agg"):
            c["weights"][li][k] = c["weights"][li][k].astype(np.float64)
            checks.append((c["weights"][li][k], out["layer_grads"][li][k], f"layer{li} {k}"))
    checks.append((c["head"]["W1"], out["head_grads"]["W1"], "head W1"))
    eps = 1e-6
    for arr, grad, name in checks:
        flat = arr.reshape(-1)
        gflat = np.asarray(grad).reshape(-1)
        for idx in rng.choice(flat.size, size=min(4, flat.size), replace=False):
            old = flat[idx]
            flat[idx] = old + eps
            jp = objective_value(c, window)
            flat[idx] = old - eps
            jm = objective_value(c, window)
            flat[idx] = old
            num = (jp - jm) / (2 * eps)
            assert abs(gflat[idx] - num) <= 1e-6 + 1e-5 * abs(num), (name, idx, gflat[idx], num)


def test_feature_gradient_matches_finite_differences():
    c = small_case(6)
    out = run(c)
    l2g = out["subs"][0].local2global
    eps = 1e-6
    rng = np.random.default_rng(1)
    for _ in range(6):
        i = int(rng.integers(0, l2g.shape[0]))
        j = int(rng.integers(0, D))
        old = c["feats"][l2g[i], j]
        c["feats"][l2g[i], j] = old + eps
        jp = objective_value(c)
        c["feats"][l2g[i], j] = old - eps
        jm = objective_value(c)
        c["feats"][l2g[i], j] = old
        num = (jp - jm) / (2 * eps)
        assert abs(out["dx"][i, j] - num) <= 1e-6 + 1e-5 * abs(num)


def test_snapshots_nest_and_share_nodes():
    c = small_case(7)
    out = run(c)
    subs = out["subs"]
    for a, b in zip(subs, subs[1:]):
        assert np.array_equal(a.local2global, b.local2global)
        assert set(a.eid) <= set(b.eid)
    assert subs[-1].e_sub >= subs[0].e_sub
