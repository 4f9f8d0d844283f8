"""GPU parity of the prediction head / masked BCE (hg_mlp_bce_fwd_bwd) and of
the Adam update (hg_adam_step) against the oracle (oracle/objective.py,
float64)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import objective
from paper_2608_02168_amd import api
from tests.helpers import parity_err, to_dev

pytestmark = pytest.mark.gpu
TOL = 1e-4


def head_case(seed, n, d):
    rng = np.random.default_rng(seed)
    H = rng.normal(0, 1, (n, d)).astype(np.float32)
    W1 = rng.uniform(-0.2, 0.2, (d, d)).astype(np.float32)
    b1 = rng.uniform(-0.1, 0.1, d).astype(np.float32)
    W2 = rng.uniform(-0.3, 0.3, (d, 1)).astype(np.float32)
    b2 = rng.uniform(-0.1, 0.1, 1).astype(np.float32)
    lab = np.where(rng.random(n) < 0.12, (rng.random(n) < 0.3).astype(np.int8), -1).astype(np.int8)
    return H, W1, b1, W2, b2, lab


# seeds whose hidden pre-activations all lie at least 5e-6 rms from zero, so
# both sides take the same ReLU decisions (checked below on the CPU)
CASES = [(3, 2049, 64), (5, 1537, 128), (7, 64, 64), (8, 300, 128)]


@pytest.mark.parametrize("seed,n,d", CASES)
def test_head_matches_oracle(seed, n, d):
    H, W1, b1, W2, b2, lab = head_case(seed, n, d)
    a = H.astype(np.float64) @ W1 + b1
    assert np.abs(a).min() > 5e-6 * np.sqrt(np.mean(a * a))
    loss, dH, dW1, db1, dW2, db2, _ = objective.mlp_bce(H, W1, b1, W2, b2, lab)
    prob = torch.empty(n, dtype=torch.float32, device="cuda")
    got_loss, got_dH, g = api.hg_mlp_bce_fwd_bwd(to_dev(H), to_dev(W1), to_dev(b1), to_dev(W2), to_dev(b2),
                                                 torch.from_numpy(lab).cuda(), prob=prob)
    torch.cuda.synchronize()
    assert abs(float(got_loss.cpu()[0]) - loss) <= 1e-5 * abs(loss)
    errs = {"dH": parity_err(got_dH.cpu().numpy(), dH), "W1": parity_err(g["W1"].cpu().numpy(), dW1),
            "b1": parity_err(g["b1"].cpu().numpy(), db1), "W2": parity_err(g["W2"].cpu().numpy(), dW2),
            "b2": parity_err(g["b2"].cpu().numpy(), db2)}
    assert max(errs.values()) <= TOL, errs
    o = np.maximum(H.astype(np.float64) @ W1 + b1, 0) @ W2 + b2
    assert parity_err(prob.cpu().numpy(), 1 / (1 + np.exp(-o[:, 0]))) <= TOL


@pytest.mark.parametrize("seed,n,d", CASES)
@pytest.mark.parametrize("superset", [False, True])
def test_head_on_listed_rows_matches_oracle(seed, n, d, superset):
    """Only the listed rows (the labelled ones, or a shuffled superset with
    unlabelled rows among them) go through the head: same loss and
    gradients as the oracle on every row, and dH zero off the list."""
    H, W1, b1, W2, b2, lab = head_case(seed, n, d)
    loss, dH, dW1, db1, dW2, db2, _ = objective.mlp_bce(H, W1, b1, W2, b2, lab)
    rows = np.nonzero(lab >= 0)[0]
    if superset:
        extra = np.random.default_rng(seed).choice(np.nonzero(lab < 0)[0], size=min(37, int((lab < 0).sum())),
                                                   replace=False)
        rows = np.random.default_rng(seed + 1).permutation(np.concatenate([rows, extra]))
    junk = torch.full((n, d), 3.0, dtype=torch.float32, device="cuda")
    got_loss, got_dH, g = api.hg_mlp_bce_fwd_bwd(to_dev(H), to_dev(W1), to_dev(b1), to_dev(W2), to_dev(b2),
                                                 torch.from_numpy(lab).cuda(), dH=junk,
                                                 rows=to_dev(rows.astype(np.int32)))
    torch.cuda.synchronize()
    assert abs(float(got_loss.cpu()[0]) - loss) <= 1e-5 * abs(loss)
    errs = {"dH": parity_err(got_dH.cpu().numpy(), dH), "W1": parity_err(g["W1"].cpu().numpy(), dW1),
            "b1": parity_err(g["b1"].cpu().numpy(), db1), "W2": parity_err(g["W2"].cpu().numpy(), dW2),
            "b2": parity_err(g["b2"].cpu().numpy(), db2)}
    assert max(errs.values()) <= TOL, errs
    off = np.setdiff1d(np.arange(n), rows)
    assert not got_dH.cpu().numpy()[off].any()


def test_head_on_an_empty_list():
    H, W1, b1, W2, b2, lab = head_case(3, 500, 64)
    lab[:] = -1
    rows = torch.zeros(0, dtype=torch.int32, device="cuda")
    loss, dH, g = api.hg_mlp_bce_fwd_bwd(to_dev(H), to_dev(W1), to_dev(b1), to_dev(W2), to_dev(b2),
                                         torch.from_numpy(lab).cuda(), rows=rows)
    torch.cuda.synchronize()
    assert float(loss.cpu()[0]) == 0.0
    assert not dH.cpu().numpy().any() and not g["W1"].cpu().numpy().any() and not g["b2"].cpu().numpy().any()


def test_head_without_labels_and_empty():
    H, W1, b1, W2, b2, lab = head_case(3, 500, 64)
    lab[:] = -1
    loss, dH, g = api.hg_mlp_bce_fwd_bwd(to_dev(H), to_dev(W1), to_dev(b1), to_dev(W2), to_dev(b2),
                                         torch.from_numpy(lab).cuda())
    torch.cuda.synchronize()
    assert float(loss.cpu()[0]) == 0.0
    assert not dH.cpu().numpy().any() and not g["W1"].cpu().numpy().any() and not g["W2"].cpu().numpy().any()
    e = torch.empty((0, 64), dtype=torch.float32, device="cuda")
    loss, dH, g = api.hg_mlp_bce_fwd_bwd(e, to_dev(W1), to_dev(b1), to_dev(W2), to_dev(b2),
                                         torch.empty(0, dtype=torch.int8, device="cuda"))
    torch.cuda.synchronize()
    assert float(loss.cpu()[0]) == 0.0 and not g["W1"].cpu().numpy().any()


def test_head_deterministic():
    H, W1, b1, W2, b2, lab = head_case(5, 1537, 128)
    args = (to_dev(H), to_dev(W1), to_dev(b1), to_dev(W2), to_dev(b2), torch.from_numpy(lab).cuda())
    r = [api.hg_mlp_bce_fwd_bwd(*args) for _ in range(2)]
    torch.cuda.synchronize()
    assert np.array_equal(r[0][1].cpu().numpy(), r[1][1].cpu().numpy())
    for k in ("W1", "b1", "W2", "b2"):
        assert np.array_equal(r[0][2][k].cpu().numpy(), r[1][2][k].cpu().numpy())


@pytest.mark.parametrize("n", [1, 1000, 262145])
def test_adam_matches_oracle(n):
    rng = np.random.default_rng(n)
    theta = rng.normal(0, 1, n).astype(np.float32)
    m = np.zeros(n, np.float32)
    v = np.zeros(n, np.float32)
    tp, mp, vp = to_dev(theta), to_dev(m), to_dev(v)
    th64, m64, v64 = theta.astype(np.float64), m.astype(np.float64), v.astype(np.float64)
    for t in range(1, 4):
        g = rng.normal(0, 1, n).astype(np.float32)
        before = tp.cpu().numpy().astype(np.float64)
        api.hg_adam_step(tp, to_dev(g), mp, vp, t, lr=1e-3, weight_decay=1e-5)
        torch.cuda.synchronize()
        th64, m64, v64 = objective.adam_step(before, g, m64, v64, t)
        # The parameter is stored in float32: the result may differ from the
        # exact update by the final rounding of theta (one ulp) plus a small
        # relative error of the update itself (computed in float32).
        got = tp.cpu().numpy().astype(np.float64)
        ulp = np.spacing(np.abs(th64).astype(np.float32)).astype(np.float64)
        assert np.all(np.abs(got - th64) <= ulp + 1e-5 * np.abs(th64 - before))
        assert parity_err(got - before, th64 - before) <= 1e-3
        assert parity_err(mp.cpu().numpy(), m64) <= TOL and parity_err(vp.cpu().numpy(), v64) <= TOL
