"""Pins of the prediction-head / BCE / Adam oracle (oracle/objective.py):
PyTorch's own CPU routines in float64 (binary_cross_entropy_with_logits with
autograd, torch.optim.Adam with weight decay), central finite differences,
and closed forms (a zero logit costs log 2; Adam's first step moves each
coordinate by lr * g / (|g| + eps))."""
import numpy as np
import pytest

from oracle import objective

torch = pytest.importorskip("torch")


def rand_case(rng, n=40, d=8, dh=6, label_rate=0.5):
    H = rng.normal(0, 1, (n, d))
    W1 = rng.normal(0, 0.6, (d, dh))
    b1 = rng.normal(0, 0.2, dh)
    W2 = rng.normal(0, 0.6, (dh, 1))
    b2 = rng.normal(0, 0.2, 1)
    lab = np.where(rng.random(n) < label_rate, rng.integers(0, 2, n), -1)
    return H, W1, b1, W2, b2, lab


def test_matches_torch_autograd_float64():
    rng = np.random.default_rng(0)
    H, W1, b1, W2, b2, lab = rand_case(rng)
    loss, dH, dW1, db1, dW2, db2, _ = objective.mlp_bce(H, W1, b1, W2, b2, lab)
    t = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True)
         for k, v in dict(H=H, W1=W1, b1=b1, W2=W2, b2=b2).items()}
    hid = torch.relu(t["H"] @ t["W1"] + t["b1"])
    o = (hid @ t["W2"] + t["b2"])[:, 0]
    sel = torch.from_numpy(lab >= 0)
    y = torch.from_numpy(np.where(lab >= 0, lab, 0).astype(np.float64))
    ref = torch.nn.functional.binary_cross_entropy_with_logits(o[sel], y[sel])
    ref.backward()
    assert abs(loss - ref.item()) <= 1e-13 * max(1.0, abs(ref.item()))
    for got, name in ((dH, "H"), (dW1, "W1"), (db1, "b1"), (dW2, "W2"), (db2, "b2")):
        np.testing.assert_allclose(got, t[name].grad.numpy(), rtol=1e-12, atol=1e-14, err_msg=name)


def test_gradients_match_finite_differences():
    rng = np.random.default_rng(1)
    H, W1, b1, W2, b2, lab = rand_case(rng, n=15, d=5, dh=4)
    _, dH, dW1, db1, dW2, db2, mask = objective.mlp_bce(H, W1, b1, W2, b2, lab)
    args = [H, W1, b1, W2, b2]

    def f(xs):
        # the ReLU decisions held fixed (linear on each side of a kink)
        a = xs[0] @ xs[1] + xs[2]
        o = ((a * mask) @ xs[3] + xs[4])[:, 0]
        sel = lab >= 0
        y = np.where(sel, lab, 0)
        return float(((np.logaddexp(0.0, o) - y * o) * sel).sum() / sel.sum())

    eps = 1e-6
    for k, g in enumerate((dH, dW1, db1, dW2, db2)):
        num = np.zeros_like(args[k])
        for idx in np.ndindex(*args[k].shape):
            xp = [x.copy() for x in args]
            xm = [x.copy() for x in args]
            xp[k][idx] += eps
            xm[k][idx] -= eps
            num[idx] = (f(xp) - f(xm)) / (2 * eps)
        np.testing.assert_allclose(g, num, rtol=1e-6, atol=1e-9)


def test_zero_logit_costs_log2_and_no_labels_cost_nothing():
    n, d = 10, 4
    H = np.ones((n, d))
    lab = np.array([0, 1] * 5)
    loss, *_ = objective.mlp_bce(H, np.zeros((d, 3)), np.zeros(3), np.zeros((3, 1)), np.zeros(1), lab)
    assert abs(loss - np.log(2.0)) < 1e-15
    loss, dH, *_ = objective.mlp_bce(H, np.ones((d, 3)), np.zeros(3), np.ones((3, 1)), np.zeros(1),
                                     np.full(n, -1))
    assert loss == 0.0 and not dH.any()


def test_adam_matches_torch_optim():
    rng = np.random.default_rng(2)
    theta0 = rng.normal(0, 1, (7, 5))
    grads = [rng.normal(0, 1, (7, 5)) for _ in range(4)]
    p = torch.tensor(theta0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([p], lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=1e-5)
    theta, m, v = theta0.copy(), np.zeros_like(theta0), np.zeros_like(theta0)
    for t, g in enumerate(grads, start=1):
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        theta, m, v = objective.adam_step(theta, g, m, v, t)
        np.testing.assert_allclose(theta, p.detach().numpy(), rtol=1e-14, atol=1e-15)


def test_adam_first_step_closed_form():
    g = np.array([3.0, -0.5, 1e-4, 0.0])
    theta, _, _ = objective.adam_step(np.zeros(4), g, np.zeros(4), np.zeros(4), 1, lr=0.1, weight_decay=0.0)
    np.testing.assert_allclose(theta, -0.1 * g / (np.abs(g) + 1e-8), rtol=1e-15)
