"""Pins of the oracle's CCA alignment loss (CPU only): closed forms through
np.corrcoef, invariances, zero-loss configurations and finite differences."""
import numpy as np
import pytest

from oracle import align


def _views(seed, m=40, d=5):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((m, d)) * rng.uniform(0.5, 2, d) + rng.uniform(-1, 1, d)
    Y = 0.6 * X + rng.standard_normal((m, d))
    return X, Y


def test_closed_forms_against_corrcoef():
    X, Y = _views(0)
    d = X.shape[1]
    (l_inv, l_dec, loss), _, _ = align.loss_and_grad(X, Y, lambda_n=0.37, eps=0.0, ddof=0)
    rho = np.array([np.corrcoef(X[:, k], Y[:, k])[0, 1] for k in range(d)])
    assert l_inv == pytest.approx(2 * np.sum(1 - rho), rel=1e-12)
    cx, cy = np.corrcoef(X, rowvar=False), np.corrcoef(Y, rowvar=False)
    off = ~np.eye(d, dtype=bool)
    assert l_dec == pytest.approx(np.sum(cx[off] ** 2) + np.sum(cy[off] ** 2), rel=1e-12)
    assert loss == pytest.approx(l_inv + 0.37 * l_dec, rel=1e-14)


def test_ddof1_uses_unbiased_variance():
    X, Y = _views(1)
    m = X.shape[0]
    xh, _, _ = align.standardise(X, 0.0, 1)
    # column norms of Xh are sqrt((M-1)/M) under the unbiased reading
    np.testing.assert_allclose((xh ** 2).sum(0), (m - 1) / m, rtol=1e-12)
    np.testing.assert_allclose(xh.mean(0), 0, atol=1e-15)


def test_identical_views_zero_invariance_and_gradient():
    X, _ = _views(2)
    (l_inv, _, _), dX, _ = align.loss_and_grad(X, X.copy(), lambda_n=0.0)
    assert l_inv == 0.0
    np.testing.assert_allclose(dX, 0, atol=1e-14)
    # positive per-column affine maps of the second view leave it zero (eps = 0)
    Y = X * np.array([2.0, 0.5, 3.0, 1.0, 7.0]) + 4.0
    (l_inv, _, _), dX, _ = align.loss_and_grad(X, Y, lambda_n=0.0, eps=0.0)
    assert abs(l_inv) < 1e-24
    np.testing.assert_allclose(dX, 0, atol=1e-12)


def test_orthonormal_centred_columns_zero_decorrelation():
    rng = np.random.default_rng(3)
    m, d = 50, 6
    A = rng.standard_normal((m, d))
    A -= A.mean(0)
    Q, _ = np.linalg.qr(A)
    X = np.sqrt(m) * Q            # centred, orthogonal columns of variance 1
    (l_inv, l_dec, _), dX, _ = align.loss_and_grad(X, X, lambda_n=1.0, eps=0.0)
    assert l_dec < 1e-24 and l_inv == 0.0
    np.testing.assert_allclose(dX, 0, atol=1e-12)


def test_unit_weights_equal_unweighted():
    X, Y = _views(4)
    a = align.loss_and_grad(X, Y)
    b = align.loss_and_grad(X, Y, omega=np.ones(X.shape[0]))
    assert a[0] == b[0]
    np.testing.assert_array_equal(a[1], b[1])


@pytest.mark.parametrize("ddof,eps,weighted", [(0, 0.0, False), (1, 0.0, False),
                                               (0, 1e-3, True), (1, 1e-3, True)])
def test_gradients_match_finite_differences(ddof, eps, weighted):
    X, Y = _views(5, m=12, d=4)
    w = np.random.default_rng(6).uniform(0.2, 2.0, 12) if weighted else None
    lam, scale = 0.3, 0.7
    _, dX, dY = align.loss_and_grad(X, Y, w, lam, scale, eps, ddof)

    def L(X_, Y_):
        return align.loss_and_grad(X_, Y_, w, lam, 1.0, eps, ddof)[0][2]

    h = 1e-6
    for target, grad in ((0, dX), (1, dY)):
        num = np.zeros_like(grad)
        for idx in np.ndindex(grad.shape):
            P = [X.copy(), Y.copy()]; Mn = [X.copy(), Y.copy()]
            P[target][idx] += h; Mn[target][idx] -= h
            num[idx] = scale * (L(*P) - L(*Mn)) / (2 * h)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-7)


def test_empty_batch():
    (a, b, c), dX, dY = align.loss_and_grad(np.zeros((0, 3)), np.zeros((0, 3)))
    assert a == b == c == 0.0 and dX.shape == (0, 3)
