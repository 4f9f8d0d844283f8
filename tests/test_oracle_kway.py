"""Pins of the K-worker oracle step (oracle/kway.py): MeanAgg against a
per-node loop and its backward as the exact adjoint, the home copies as the
base-node rows of the right subgraph, the copy counts, the one-worker case
against the one-subgraph step, and the gradients of
J = L_BCE(MLP(MeanAgg)) + lambda_CCA sum_k L_CCA,k (home copies held fixed,
as the stop-gradient makes them) against central finite differences."""
import numpy as np
import pytest

from oracle import kway, step
from paper_2608_02168_amd import synth

D, R, K = 4, 2, 3


def small_case(seed, k_parts=K, budget=4):
    rng = np.random.default_rng(seed)
    n, e = 40, 200
    src = rng.integers(0, n, e)
    dst = rng.integers(0, n, e)
    rel = rng.integers(0, R, e).astype(np.uint8)
    ntype = (rng.random(n) < 0.3).astype(np.uint8)
    part = synth.random_partition(n, k_parts, seed)
    feats = rng.normal(0, 1, (n, D))
    weights = []
    for li in range(2):
        w = synth.layer_weights(seed, li, R, 2, D, bias_range=0.1)
        weights.append(synth.LayerWeights(*(a.astype(np.float64) for a in (w.w_rel, w.w_self, w.bias))))
    head = {k: v.astype(np.float64) for k, v in synth.head_weights(seed, D).items()}
    head["b1"] = rng.uniform(-0.1, 0.1, D)
    labels = np.where(rng.random(n) < 0.6, rng.integers(0, 2, n), -1)
    return dict(graph=dict(src=src, dst=dst, rel=rel, ntype=ntype, part=part), K=k_parts,
                build=dict(n_rel=R, n_ntype=2, budget=budget, seed=3), feats=feats, weights=weights, head=head,
                labels=labels)


def run(c, frozen_home=None):
    return kway.run_kway(c["graph"], c["K"], c["build"], c["feats"], c["weights"], c["head"], c["labels"],
                         scale=0.1, frozen_home=frozen_home)


def test_mean_agg_matches_a_per_node_loop():
    rng = np.random.default_rng(0)
    n, d = 30, 3
    l2gs = [rng.permutation(n)[: rng.integers(5, 20)] for _ in range(4)]
    Hs = [rng.normal(0, 1, (len(l), d)) for l in l2gs]
    H, cnt = kway.mean_agg(n, l2gs, Hs)
    for v in range(n):
        rows = [Hk[list(l).index(v)] for l, Hk in zip(l2gs, Hs) if v in l]
        assert cnt[v] == len(rows)
        want = np.mean(rows, axis=0) if rows else np.zeros(d)
        assert np.allclose(H[v], want, rtol=0, atol=1e-15)


def test_mean_agg_backward_is_the_adjoint():
    rng = np.random.default_rng(1)
    n, d = 50, 5
    l2gs = [rng.permutation(n)[: rng.integers(10, 40)] for _ in range(3)]
    Hs = [rng.normal(0, 1, (len(l), d)) for l in l2gs]
    H, cnt = kway.mean_agg(n, l2gs, Hs)
    dH = rng.normal(0, 1, (n, d))
    dHs = kway.mean_agg_backward(l2gs, cnt, dH)
    lhs = float((H * dH).sum())
    rhs = float(sum((a * b).sum() for a, b in zip(Hs, dHs)))
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))


def test_home_rows_and_copy_counts():
    c = small_case(2)
    out = run(c)
    subs, part = out["subs"], c["graph"]["part"]
    n_overlap = np.zeros(part.shape[0], dtype=np.int64)
    for k, sb in enumerate(subs):
        home, rows = kway.home_rows(subs, part, k)
        og = sb.local2global[sb.overlap]
        assert np.all(home != k)
        assert np.array_equal(home, part[og])
        for h, r, v in zip(home, rows, og):
            assert subs[h].local2global[r] == v
        n_overlap[og] += 1
    assert sum(sb.overlap.shape[0] for sb in subs) > 0
    assert np.array_equal(out["cnt"], 1 + n_overlap)
    # every node's base copy sits in its own partition's subgraph
    for v in range(part.shape[0]):
        assert subs[part[v]].global2local[v] >= 0


def test_one_worker_is_the_one_subgraph_step():
    c = small_case(3, k_parts=1)
    out = run(c)
    sub, h, losses, g, grads, head_out = step.run(
        c["graph"], dict(k=0, **c["build"]), c["feats"], c["weights"], np.zeros((0, D)), None,
        scale=0.1, head=c["head"], labels_global=c["labels"])
    assert sub.overlap.shape[0] == 0 and np.all(out["cnt"] == 1)
    assert np.allclose(out["H"][sub.local2global], h[-1], rtol=0, atol=1e-14)
    assert abs(out["bce"] - head_out["loss"]) <= 1e-14
    for (a1, a2, a3), (b1, b2, b3) in zip(out["layer_grads"], grads):
        for a, b in ((a1, b1), (a2, b2), (a3, b3)):
            assert np.allclose(a, b, rtol=1e-12, atol=1e-14)
    assert np.allclose(out["head_grads"]["W1"], head_out["W1"], rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("seed", [4, 5])
def test_kway_gradients_match_finite_differences(seed):
    c = small_case(seed)
    out = run(c)
    assert all(sb.overlap.shape[0] >= 2 for sb in out["subs"])
    homes = out["homes"]

    def objective():
        o = run(c, frozen_home=homes)
        return o["total"]

    rng = np.random.default_rng(seed + 10)
    checks = []
    for li in range(2):
        w = c["weights"][li]
        checks += [(w.w_rel, out["layer_grads"][li][0], f"layer{li} w_rel"),
                   (w.w_self, out["layer_grads"][li][1], f"layer{li} w_self"),
                   (w.bias, out["layer_grads"][li][2], f"layer{li} bias")]
    checks.append((c["head"]["W1"], out["head_grads"]["W1"], "head W1"))
    eps = 1e-6
    for arr, grad, name in checks:
        flat = arr.reshape(-1)
        gflat = np.asarray(grad).reshape(-1)
        for idx in rng.choice(flat.size, size=min(5, flat.size), replace=False):
            old = flat[idx]
            flat[idx] = old + eps
            jp = objective()
            flat[idx] = old - eps
            jm = objective()
            flat[idx] = old
            num = (jp - jm) / (2 * eps)
            assert abs(gflat[idx] - num) <= 1e-7 + 1e-5 * abs(num), (name, idx, gflat[idx], num)


def test_alignment_term_moves_the_gradient():
    # the CCA terms reach the layer gradients: dropping them (scale 0) changes them
    c = small_case(6)
    a = run(c)
    b = kway.run_kway(c["graph"], c["K"], c["build"], c["feats"], c["weights"], c["head"], c["labels"], scale=0.0)
    assert not np.allclose(a["layer_grads"][1][0], b["layer_grads"][1][0])
    assert abs(a["total"] - a["bce"] - 0.1 * sum(l[2] for l in a["losses"])) < 1e-14
