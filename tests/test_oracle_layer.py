"""Pins of the oracle's relation-typed mean-aggregation layer (CPU only):
dense brute force, the textbook special case, constant features, edge-order
invariance and central finite differences for every gradient."""
import numpy as np
import pytest

from oracle import layer


def _case(seed, n=30, e=120, R=3, T=2, d=6, bias=0.1):
    rng = np.random.default_rng(seed)
    src = rng.integers(0, n, e)
    dst = rng.integers(0, n, e)
    src[:10] = dst[:10]                  # self loops
    src[10:14] = src[14:18]; dst[10:14] = dst[14:18]   # duplicate edges
    rel = rng.integers(0, R, e)
    ntype = np.sort(rng.integers(0, T, n))
    H = rng.standard_normal((n, d))
    w_rel = rng.uniform(-0.6, 0.6, (R, d, d))
    w_self = rng.uniform(-0.6, 0.6, (T, d, d))
    b = rng.uniform(-bias, bias, (T, d))
    return n, src, dst, rel, ntype, H, w_rel, w_self, b


def _dense_forward(n, src, dst, rel, ntype, H, w_rel, w_self, b, ew=None):
    """Dense brute force: per relation the weighted adjacency A[t, s] += w and
    the in-edge count, loops over the destinations."""
    R, d = w_rel.shape[0], H.shape[1]
    Z = np.zeros((n, d))
    ew = np.ones(len(src)) if ew is None else ew
    for r in range(R):
        A = np.zeros((n, n))
        cnt = np.zeros(n)
        for s, t, rr, we in zip(src, dst, rel, ew):
            if rr == r:
                A[t, s] += we
                cnt[t] += 1
        for j in range(n):
            if cnt[j] > 0:
                Z[j] += (A[j] @ H) / cnt[j] @ w_rel[r]
    for j in range(n):
        Z[j] += H[j] @ w_self[ntype[j]] + b[ntype[j]]
    return np.maximum(Z, 0) + H, Z


@pytest.mark.parametrize("seed", range(4))
def test_forward_matches_dense_brute_force(seed):
    c = _case(seed)
    out, Z = layer.forward(*c)
    out2, Z2 = _dense_forward(*c)
    np.testing.assert_allclose(Z, Z2, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(out, out2, rtol=1e-12, atol=1e-12)


def test_textbook_special_case():
    """R=1, T=1, W_self=0, b=0: z = D^-1 A H W (row-normalised adjacency)."""
    rng = np.random.default_rng(5)
    n, d = 25, 4
    src, dst = rng.integers(0, n, 90), rng.integers(0, n, 90)
    H = rng.standard_normal((n, d))
    W = rng.standard_normal((1, d, d))
    A = np.zeros((n, n))
    np.add.at(A, (dst, src), 1.0)
    deg = A.sum(1, keepdims=True)
    Ahat = np.divide(A, deg, out=np.zeros_like(A), where=deg > 0)
    _, Z = layer.forward(n, src, dst, np.zeros(90, int), np.zeros(n, int), H, W,
                         np.zeros((1, d, d)), np.zeros((1, d)))
    np.testing.assert_allclose(Z, Ahat @ H @ W[0], rtol=1e-12, atol=1e-12)


def test_constant_features_mean_is_exact():
    n, src, dst, rel, ntype, H, w_rel, w_self, b = _case(1)
    c = np.linspace(-1, 1, H.shape[1])
    Hc = np.tile(c, (n, 1))
    _, Z = layer.forward(n, src, dst, rel, ntype, Hc, w_rel, w_self, b)
    for j in range(n):
        expect = c @ w_self[ntype[j]] + b[ntype[j]]
        for r in range(w_rel.shape[0]):
            if np.any((dst == j) & (rel == r)):
                expect = expect + c @ w_rel[r]
        np.testing.assert_allclose(Z[j], expect, rtol=1e-13, atol=1e-13)


def test_edge_order_invariance():
    n, src, dst, rel, ntype, H, w_rel, w_self, b = _case(2)
    p = np.random.default_rng(0).permutation(src.shape[0])
    o1, _ = layer.forward(n, src, dst, rel, ntype, H, w_rel, w_self, b)
    o2, _ = layer.forward(n, src[p], dst[p], rel[p], ntype, H, w_rel, w_self, b)
    assert np.max(np.abs(o1 - o2)) <= 1e-12


def test_isolated_nodes_get_only_self_term():
    n, src, dst, rel, ntype, H, w_rel, w_self, b = _case(3)
    iso = np.setdiff1d(np.arange(n), dst)
    _, Z = layer.forward(n, src, dst, rel, ntype, H, w_rel, w_self, b)
    for j in iso:
        np.testing.assert_allclose(Z[j], H[j] @ w_self[ntype[j]] + b[ntype[j]], rtol=1e-13)


@pytest.mark.parametrize("seed", [11, 12])
def test_backward_matches_finite_differences(seed):
    n, src, dst, rel, ntype, H, w_rel, w_self, b = _case(seed, n=14, e=50, R=2, d=4, bias=0.3)
    G = np.random.default_rng(seed + 100).standard_normal(H.shape)
    _, Z = layer.forward(n, src, dst, rel, ntype, H, w_rel, w_self, b)
    assert np.min(np.abs(Z)) > 1e-3, "pick a case away from ReLU kinks"
    dH, dWr, dWs, db = layer.backward(n, src, dst, rel, ntype, H, w_rel, w_self, b, G)

    def loss(H_, wr_, ws_, b_):
        out, _ = layer.forward(n, src, dst, rel, ntype, H_, wr_, ws_, b_)
        return float((out * G).sum())

    h = 1e-6
    args = [H, w_rel, w_self, b]
    for which, grad in enumerate([dH, dWr, dWs, db]):
        num = np.zeros_like(grad)
        it = np.nditer(args[which], flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            plus = [a.copy() for a in args]; minus = [a.copy() for a in args]
            plus[which][idx] += h; minus[which][idx] -= h
            num[idx] = (loss(*plus) - loss(*minus)) / (2 * h)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-6)


def test_backward_explicit_mask_equals_recomputed():
    c = _case(4)
    G = np.random.default_rng(9).standard_normal(c[5].shape)
    _, Z = layer.forward(*c)
    a = layer.backward(*c, G)
    m = layer.backward(*c, G, mask=Z > 0)
    for x, y in zip(a, m):
        np.testing.assert_array_equal(x, y)


def test_adjoint_identity():
    n, src, dst, rel, *_ = _case(6)
    rng = np.random.default_rng(1)
    X, Y = rng.standard_normal((n, 3)), rng.standard_normal((n, 3))
    for r in range(3):
        A = layer.mean_adjacency(n, src, dst, rel, r)
        assert abs(np.sum((A @ X) * Y) - np.sum(X * (A.T @ Y))) < 1e-12


def _weights(seed, e):
    return np.random.default_rng(seed + 50).uniform(0.1, 2.0, e)


@pytest.mark.parametrize("seed", range(3))
def test_weighted_forward_matches_dense_brute_force(seed):
    """Edge weights multiply the messages; the normaliser stays the in-edge
    count."""
    c = _case(seed)
    ew = _weights(seed, len(c[1]))
    out, Z = layer.forward(*c, edge_w=ew)
    out2, Z2 = _dense_forward(*c, ew=ew)
    np.testing.assert_allclose(Z, Z2, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(out, out2, rtol=1e-12, atol=1e-12)


def test_unit_weights_equal_the_unweighted_layer():
    c = _case(3)
    ones = np.ones(len(c[1]))
    np.testing.assert_array_equal(layer.forward(*c)[1], layer.forward(*c, edge_w=ones)[1])
    G = np.random.default_rng(2).standard_normal(c[5].shape)
    for a, b in zip(layer.backward(*c, G), layer.backward(*c, G, edge_w=ones)):
        np.testing.assert_array_equal(a, b)


def test_weights_scale_the_relation_part_linearly():
    """w = c everywhere multiplies z - (self term) by c (closed form)."""
    n, src, dst, rel, ntype, H, w_rel, w_self, b = _case(8)
    zero_self = np.zeros_like(w_self)
    zb = np.zeros_like(b)
    _, Z1 = layer.forward(n, src, dst, rel, ntype, H, w_rel, zero_self, zb)
    _, Zc = layer.forward(n, src, dst, rel, ntype, H, w_rel, zero_self, zb, edge_w=np.full(len(src), 2.5))
    np.testing.assert_allclose(Zc, 2.5 * Z1, rtol=1e-13, atol=1e-13)


def test_weighted_backward_matches_finite_differences():
    n, src, dst, rel, ntype, H, w_rel, w_self, b = _case(21, n=14, e=50, R=2, d=4, bias=0.3)
    ew = _weights(21, len(src))
    G = np.random.default_rng(121).standard_normal(H.shape)
    _, Z = layer.forward(n, src, dst, rel, ntype, H, w_rel, w_self, b, edge_w=ew)
    assert np.min(np.abs(Z)) > 1e-3, "pick a case away from ReLU kinks"
    grads = layer.backward(n, src, dst, rel, ntype, H, w_rel, w_self, b, G, edge_w=ew)

    def loss(H_, wr_, ws_, b_):
        out, _ = layer.forward(n, src, dst, rel, ntype, H_, wr_, ws_, b_, edge_w=ew)
        return float((out * G).sum())

    h = 1e-6
    args = [H, w_rel, w_self, b]
    for which, grad in enumerate(grads):
        num = np.zeros_like(grad)
        it = np.nditer(args[which], flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            plus = [a.copy() for a in args]; minus = [a.copy() for a in args]
            plus[which][idx] += h; minus[which][idx] -= h
            num[idx] = (loss(*plus) - loss(*minus)) / (2 * h)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-6)

