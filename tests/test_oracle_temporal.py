"""Pins of the temporal-module oracle (oracle/temporal.py): PyTorch's CPU
routines in float64 (torch.nn.GRUCell with the same weights, softmax/tanh
attention, autograd for every gradient), central finite differences, and the
special cases a single state (a = 1, Ht = c_0) and Q = 0 (uniform attention,
Ht = mean of the states)."""
import numpy as np
import pytest

from oracle import temporal

torch = pytest.importorskip("torch")


def rand_case(rng, n=12, d=6, w=3, scale=0.5):
    h = rng.normal(0, 1, (n, d))
    C = rng.normal(0, 1, (w, n, d))
    p = dict(Q=rng.normal(0, scale, (d, d)), r=rng.normal(0, 1, d), Wi=rng.normal(0, scale, (3, d, d)),
             bi=rng.normal(0, 0.2, (3, d)), Wh=rng.normal(0, scale, (3, d, d)), bh=rng.normal(0, 0.2, (3, d)))
    return h, C, p


def torch_reference(h, C, p, dH):
    t = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in p.items()}
    th = torch.tensor(h, dtype=torch.float64, requires_grad=True)
    tC = torch.tensor(C, dtype=torch.float64, requires_grad=True)
    if C.shape[0] == 0:
        Ht = None                       # GRUCell's default: a zero hidden state
    else:
        u = torch.tanh(torch.einsum("knj,ij->kni", tC, t["Q"]))
        a = torch.softmax(torch.einsum("kni,i->nk", u, t["r"]), dim=1)
        Ht = torch.einsum("nk,knd->nd", a, tC)
    d = h.shape[1]
    cell = torch.nn.GRUCell(d, d).double()
    with torch.no_grad():
        # torch computes x W_ih^T with rows of W_ih stacked (reset, update, new)
        cell.weight_ih.copy_(torch.cat([torch.tensor(p["Wi"][k].T) for k in range(3)]))
        cell.weight_hh.copy_(torch.cat([torch.tensor(p["Wh"][k].T) for k in range(3)]))
        cell.bias_ih.copy_(torch.tensor(p["bi"].reshape(-1)))
        cell.bias_hh.copy_(torch.tensor(p["bh"].reshape(-1)))
    H = cell(th, Ht)
    (H * torch.tensor(dH)).sum().backward()
    z = torch.zeros_like
    grads = {"Q": t["Q"].grad if t["Q"].grad is not None else z(t["Q"]),
             "r": t["r"].grad if t["r"].grad is not None else z(t["r"]),
             "Wi": torch.stack([g.T for g in cell.weight_ih.grad.chunk(3)]),
             "Wh": torch.stack([g.T for g in cell.weight_hh.grad.chunk(3)]),
             "bi": cell.bias_ih.grad.view(3, d), "bh": cell.bias_hh.grad.view(3, d)}
    dC = tC.grad.numpy() if tC.grad is not None else np.zeros_like(C)
    return H.detach().numpy(), th.grad.numpy(), dC, {k: v.detach().numpy() for k, v in grads.items()}


@pytest.mark.parametrize("w", [0, 1, 3])
def test_matches_torch_gru_cell_and_autograd(w):
    rng = np.random.default_rng(w)
    h, C, p = rand_case(rng, w=w)
    dH = rng.normal(0, 1, h.shape)
    H, _ = temporal.forward(h, C, p)
    dh, dC, g = temporal.backward(h, C, p, dH)
    Hr, dhr, dCr, gr = torch_reference(h, C, p, dH)
    np.testing.assert_allclose(H, Hr, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(dh, dhr, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dC, dCr, rtol=1e-12, atol=1e-13)
    for k in temporal.PARAM_NAMES:
        np.testing.assert_allclose(g[k], gr[k], rtol=1e-12, atol=1e-13, err_msg=k)


def test_gradients_match_finite_differences():
    rng = np.random.default_rng(1)
    h, C, p = rand_case(rng, n=5, d=4, w=3)
    dH = rng.normal(0, 1, h.shape)
    dh, dC, g = temporal.backward(h, C, p, dH)

    def f(hx, Cx, px):
        return float((temporal.forward(hx, Cx, px)[0] * dH).sum())

    eps = 1e-6
    for arr, grad, name in [(h, dh, "h"), (C, dC, "C")] + [(p[k], g[k], k) for k in temporal.PARAM_NAMES]:
        num = np.zeros_like(arr)
        for idx in np.ndindex(*arr.shape):
            old = arr[idx]
            arr[idx] = old + eps
            fp = f(h, C, p)
            arr[idx] = old - eps
            fm = f(h, C, p)
            arr[idx] = old
            num[idx] = (fp - fm) / (2 * eps)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-8, err_msg=name)


def test_single_state_and_uniform_attention():
    rng = np.random.default_rng(2)
    h, C, p = rand_case(rng, w=1)
    _, c = temporal.forward(h, C, p)
    np.testing.assert_array_equal(c["a"], np.ones_like(c["a"]))
    np.testing.assert_array_equal(c["Ht"], C[0])
    h, C, p = rand_case(rng, w=3)
    p["Q"][:] = 0.0
    _, c = temporal.forward(h, C, p)
    np.testing.assert_allclose(c["a"], np.full_like(c["a"], 1.0 / 3.0), rtol=1e-15)
    np.testing.assert_allclose(c["Ht"], C.mean(axis=0), rtol=1e-14, atol=1e-15)
