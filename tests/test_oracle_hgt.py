"""Pins of the attention-layer oracle (oracle/hgt.py) against mathematics that
does not go through it: central finite differences of every gradient, the
reduction to the (separately pinned) mean-aggregation layer when the
attention is uniform, invariance to the attention parameters when every node
has one in-edge, invariance to the order of the edges, and a two-edge closed
form.  Planted mistakes (scale dropped, mu indexed the wrong way round,
W_att transposed, softmax grouped by source, the softmax-gradient term
dropped) are each caught by one of these pins."""
import numpy as np
import pytest

from oracle import hgt, layer


def block_diag(W):
    """[S, dk, dk] -> the d x d block-diagonal matrix."""
    S, dk, _ = W.shape
    out = np.zeros((S * dk, S * dk))
    for s in range(S):
        out[s * dk:(s + 1) * dk, s * dk:(s + 1) * dk] = W[s]
    return out


def rand_params(rng, d, S, R, T, scale=0.5):
    dk = d // S
    return hgt.Params(
        W_K=rng.normal(0, scale, (T, d, d)), b_K=rng.normal(0, 0.1, (T, d)),
        W_Q=rng.normal(0, scale, (T, d, d)), b_Q=rng.normal(0, 0.1, (T, d)),
        W_V=rng.normal(0, scale, (T, d, d)), b_V=rng.normal(0, 0.1, (T, d)),
        W_att=rng.normal(0, scale, (R, S, dk, dk)), W_msg=rng.normal(0, scale, (R, S, dk, dk)),
        mu=rng.uniform(0.5, 1.5, (T, R, T)),
        W_agg=rng.normal(0, scale, (T, d, d)), b_agg=rng.normal(0, 0.1, (T, d)))


def rand_graph(rng, n, E, R, T):
    return (rng.integers(0, n, E), rng.integers(0, n, E), rng.integers(0, R, E), rng.integers(0, T, n))


def pin_finite_differences():
    """Every gradient of the backward against central differences of the forward."""
    rng = np.random.default_rng(1)
    n, E, R, T, d, S = 9, 34, 2, 2, 8, 2
    src, dst, rel, nt = rand_graph(rng, n, E, R, T)
    p = rand_params(rng, d, S, R, T)
    H = rng.normal(0, 1, (n, d))
    G = rng.normal(0, 1, (n, d))
    _, Z, _, _ = hgt.forward(n, src, dst, rel, nt, H, p, S)
    mask = Z > 0

    def f(Hx, px):
        # the layer with the ReLU decision held fixed: linear in Z on each side of a kink
        _, Zx, _, _ = hgt.forward(n, src, dst, rel, nt, Hx, px, S)
        return float((G * (Zx * mask + Hx)).sum())

    dH, g = hgt.backward(n, src, dst, rel, nt, H, p, S, G, mask=mask)
    eps = 1e-6
    num = np.zeros_like(H)
    for idx in np.ndindex(*H.shape):
        Hp, Hm = H.copy(), H.copy()
        Hp[idx] += eps
        Hm[idx] -= eps
        num[idx] = (f(Hp, p) - f(Hm, p)) / (2 * eps)
    np.testing.assert_allclose(dH, num, rtol=1e-6, atol=1e-7)
    for name in hgt.PARAM_NAMES:
        P = getattr(p, name)
        num = np.zeros_like(P)
        for idx in np.ndindex(*P.shape):
            old = P[idx]
            P[idx] = old + eps
            fp = f(H, p)
            P[idx] = old - eps
            fm = f(H, p)
            P[idx] = old
            num[idx] = (fp - fm) / (2 * eps)
        np.testing.assert_allclose(getattr(g, name), num, rtol=1e-6, atol=1e-7, err_msg=name)


def test_gradients_match_finite_differences():
    pin_finite_differences()


@pytest.mark.parametrize("zero", ["W_att", "mu"])
def test_uniform_attention_reduces_to_the_mean_layer(zero):
    # With zero scores the softmax is 1/deg(j); for one relation and one node
    # type, and no value bias, the layer is the mean-aggregation layer with the
    # composed weight W_V . W_msg . W_agg and no self term.
    rng = np.random.default_rng(2)
    n, E, d, S = 30, 140, 8, 2
    src, dst, _, _ = rand_graph(rng, n, E, 1, 1)
    rel = np.zeros(E, dtype=np.int64)
    nt = np.zeros(n, dtype=np.int64)
    p = rand_params(rng, d, S, 1, 1)
    p.b_V[:] = 0.0
    setattr(p, zero, np.zeros_like(getattr(p, zero)))
    H = rng.normal(0, 1, (n, d))
    G = rng.normal(0, 1, (n, d))
    w_rel = (p.W_V[0] @ block_diag(p.W_msg[0]) @ p.W_agg[0])[None]
    w_self = np.zeros((1, d, d))
    Ho, Zo, _, alpha = hgt.forward(n, src, dst, rel, nt, H, p, S)
    Hl, Zl = layer.forward(n, src, dst, rel, nt, H, w_rel, w_self, p.b_agg)
    np.testing.assert_allclose(Zo, Zl, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(Ho, Hl, rtol=1e-12, atol=1e-12)
    deg = np.bincount(dst, minlength=n)
    np.testing.assert_allclose(alpha, np.repeat((1.0 / deg[dst])[:, None], S, axis=1), rtol=1e-14)
    dH, _ = hgt.backward(n, src, dst, rel, nt, H, p, S, G)
    dHl, _, _, _ = layer.backward(n, src, dst, rel, nt, H, w_rel, w_self, p.b_agg, G)
    np.testing.assert_allclose(dH, dHl, rtol=1e-11, atol=1e-11)


def test_single_in_edge_ignores_the_attention_parameters():
    # softmax over one edge is 1 whatever the score
    rng = np.random.default_rng(3)
    n, R, T, d, S = 20, 3, 2, 8, 4
    dst = rng.permutation(n)[:15]
    src = rng.integers(0, n, dst.shape[0])
    rel = rng.integers(0, R, dst.shape[0])
    nt = rng.integers(0, T, n)
    p = rand_params(rng, d, S, R, T)
    H = rng.normal(0, 1, (n, d))
    G = rng.normal(0, 1, (n, d))
    Ho, _, _, alpha = hgt.forward(n, src, dst, rel, nt, H, p, S)
    np.testing.assert_array_equal(alpha, np.ones_like(alpha))
    q = rand_params(rng, d, S, R, T)
    for name in ("W_att", "mu", "W_Q", "b_Q", "W_K", "b_K"):
        setattr(p, name, getattr(q, name))
    Ho2, _, _, _ = hgt.forward(n, src, dst, rel, nt, H, p, S)
    np.testing.assert_allclose(Ho2, Ho, rtol=1e-13, atol=1e-13)
    _, g = hgt.backward(n, src, dst, rel, nt, H, p, S, G)
    for name in ("W_att", "mu", "W_Q", "b_Q", "W_K", "b_K"):
        assert np.abs(getattr(g, name)).max() < 1e-12, name


def test_edge_order_does_not_matter():
    rng = np.random.default_rng(4)
    n, E, R, T, d, S = 25, 120, 3, 2, 8, 2
    src, dst, rel, nt = rand_graph(rng, n, E, R, T)
    p = rand_params(rng, d, S, R, T)
    H = rng.normal(0, 1, (n, d))
    G = rng.normal(0, 1, (n, d))
    perm = rng.permutation(E)
    a = hgt.forward(n, src, dst, rel, nt, H, p, S)[0]
    b = hgt.forward(n, src[perm], dst[perm], rel[perm], nt, H, p, S)[0]
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)
    ga = hgt.backward(n, src, dst, rel, nt, H, p, S, G)
    gb = hgt.backward(n, src[perm], dst[perm], rel[perm], nt, H, p, S, G)
    np.testing.assert_allclose(ga[0], gb[0], rtol=1e-11, atol=1e-11)
    for name in hgt.PARAM_NAMES:
        np.testing.assert_allclose(getattr(ga[1], name), getattr(gb[1], name), rtol=1e-11, atol=1e-11)


def test_nodes_without_in_edges_pass_the_residual_and_bias():
    rng = np.random.default_rng(5)
    n, d, S = 6, 8, 2
    src = np.array([0, 1, 2])
    dst = np.array([1, 1, 3])
    rel = np.array([0, 0, 0])
    nt = np.zeros(n, dtype=np.int64)
    p = rand_params(rng, d, S, 1, 1)
    H = rng.normal(0, 1, (n, d))
    Ho, Z, ht, _ = hgt.forward(n, src, dst, rel, nt, H, p, S)
    for j in (0, 2, 4, 5):
        np.testing.assert_array_equal(ht[j], np.zeros(d))
        np.testing.assert_allclose(Z[j], p.b_agg[0], rtol=1e-15)
        np.testing.assert_allclose(Ho[j], np.maximum(p.b_agg[0], 0) + H[j], rtol=1e-15)


def pin_two_in_edges_closed_form():
    # node 0 (type 0) receives from node 1 (type 1, relation 0) and node 2
    # (type 0, relation 1); with identity projections the weights of the two
    # edges are per head a logistic function of the score difference, the
    # scores being h_i^s W_att[r, s] h_0^s^T * mu[type(i), r, type(0)] / sqrt(d / S)
    rng = np.random.default_rng(6)
    n, d, S, R, T = 3, 8, 2, 2, 2
    dk = d // S
    src, dst, rel = np.array([1, 2]), np.array([0, 0]), np.array([0, 1])
    nt = np.array([0, 1, 0])
    eye = np.stack([np.eye(d)] * T)
    z = np.zeros((T, d))
    W_att = rng.normal(0, 0.7, (R, S, dk, dk))
    mu = np.array([[[0.3, 2.0], [1.3, 4.0]], [[0.7, 3.0], [5.0, 6.0]]])  # [T, R, T], all distinct
    W_msg = np.stack([np.stack([np.eye(dk)] * S)] * R)
    p = hgt.Params(W_K=eye, b_K=z, W_Q=eye.copy(), b_Q=z.copy(), W_V=eye.copy(), b_V=z.copy(), W_att=W_att,
                   W_msg=W_msg, mu=mu, W_agg=eye.copy(), b_agg=z.copy())
    H = rng.normal(0, 1, (n, d))
    _, Z, ht, alpha = hgt.forward(n, src, dst, rel, nt, H, p, S)
    for s in range(S):
        sl = slice(s * dk, (s + 1) * dk)
        s1 = H[1, sl] @ W_att[0, s] @ H[0, sl] * mu[1, 0, 0] / np.sqrt(dk)
        s2 = H[2, sl] @ W_att[1, s] @ H[0, sl] * mu[0, 1, 0] / np.sqrt(dk)
        a1 = 1.0 / (1.0 + np.exp(s2 - s1))
        np.testing.assert_allclose(alpha[:, s], [a1, 1 - a1], rtol=1e-13)
        np.testing.assert_allclose(ht[0, sl], a1 * H[1, sl] + (1 - a1) * H[2, sl], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(Z[0], ht[0], rtol=1e-14)


def test_two_in_edges_closed_form():
    pin_two_in_edges_closed_form()


def _mutant_tables(kind):
    """_edge_tables with one plausible mistake planted."""
    orig = hgt._edge_tables

    def tables(src, dst, rel, ntype, p, K, Q, V, S):
        if kind == "W_att transposed":
            p = hgt.Params(*[np.swapaxes(getattr(p, k), -1, -2) if k == "W_att" else getattr(p, k)
                             for k in hgt.PARAM_NAMES])
        Ki, Vi, Qj, kt, msg, dot, c = orig(src, dst, rel, ntype, p, K, Q, V, S)
        dk = K.shape[1] // S
        if kind == "scale dropped":
            c = c * np.sqrt(dk)
        if kind == "mu transposed":
            c = p.mu[ntype[dst], rel, ntype[src]] / np.sqrt(dk)
        return Ki, Vi, Qj, kt, msg, dot, c
    return tables


@pytest.mark.parametrize("kind", ["scale dropped", "mu transposed", "W_att transposed", "softmax by source",
                                  "softmax gradient term dropped"])
def test_planted_mistakes_are_caught(monkeypatch, kind):
    if kind == "softmax by source":
        # the closed form's two edges come from two different sources
        orig = hgt._softmax_by_dst
        monkeypatch.setattr(hgt, "_softmax_by_dst", lambda n, dst, score: orig(n, np.array([1, 2]), score))
        pin = pin_two_in_edges_closed_form
    elif kind == "softmax gradient term dropped":
        monkeypatch.setattr(hgt, "_softmax_backward", lambda n, dst, alpha, dalpha: alpha * dalpha)
        pin = pin_finite_differences
    else:
        monkeypatch.setattr(hgt, "_edge_tables", _mutant_tables(kind))
        pin = pin_two_in_edges_closed_form
    with pytest.raises(AssertionError):
        pin()
