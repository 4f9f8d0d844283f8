"""GPU parity of the temporal module (hg_temporal_fwd / hg_temporal_bwd)
against the oracle (oracle/temporal.py, float64): every output element by
element, at sizes that span several 16-row tiles and 128-row blocks with a
ragged tail, for every context length 0..4, float32 and bfloat16 storage,
the accumulate and partial-gradient options, and the argument checks."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import temporal
from paper_2608_02168_amd import api, synth
from tests.helpers import parity_err, to_dev

pytestmark = pytest.mark.gpu
TOL = 1e-4
TOL_BF16 = 2e-2
D = 64


def case(seed, n, w, bias_range=0.1):
    p = synth.temporal_weights(seed, D, bias_range)
    h = synth.features(seed, n, D)
    C = synth.context_states(seed, w, n, D)
    dH = synth.upstream_grad(seed, n, D)
    return h, C, p, dH


def oracle(h, C, p, dH):
    Cs = np.stack(C) if C else np.zeros((0, h.shape[0], D))
    H, _ = temporal.forward(h, Cs, p)
    dh, dC, g = temporal.backward(h, Cs, p, dH)
    return H, dh, list(dC), g


def run(h, C, p, dH, dtype=torch.float32, accumulate=False, dC0=None, g0=None, biases=True):
    def dev(x):
        return to_dev(x).to(dtype)
    hd, dHd = dev(h), dev(dH)
    Cd = [dev(c) for c in C]
    W = {k: to_dev(v) for k, v in p.items() if biases or k not in ("bi", "bh")}
    H = api.hg_temporal_fwd(hd, Cd, W)
    dCd = [dev(x) for x in dC0] if dC0 is not None else [torch.zeros_like(hd) for _ in C]
    grads = {k: to_dev(v) for k, v in g0.items()} if g0 is not None else None
    dh, g = api.hg_temporal_bwd(hd, Cd, W, dHd, dstates=dCd, grads=grads, accumulate=accumulate)
    torch.cuda.synchronize()
    return (H.float().cpu().numpy(), dh.float().cpu().numpy(), [x.float().cpu().numpy() for x in dCd],
            {k: v.cpu().numpy() for k, v in g.items()})


def errors(got, ref, w):
    gH, gdh, gdC, gg = got
    H, dh, dC, g = ref
    e = {"H": parity_err(gH, H), "dh": parity_err(gdh, dh)}
    for k in range(w):
        e[f"dC{k}"] = parity_err(gdC[k], dC[k])
    for k in gg:
        e[k] = parity_err(gg[k], g[k])
    return e


@pytest.mark.parametrize("w", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("n", [1, 77, 4099])
def test_parity_f32(w, n):
    h, C, p, dH = case(10 + w, n, w)
    e = errors(run(h, C, p, dH), oracle(h, C, p, dH), w)
    assert len(e) == 2 + w + 6
    assert max(e.values()) <= TOL, e


@pytest.mark.parametrize("w", [0, 3])
def test_parity_bf16(w):
    n = 1500
    h, C, p, dH = case(20 + w, n, w)
    h, dH = synth.round_bf16(h), synth.round_bf16(dH)
    C = [synth.round_bf16(c) for c in C]
    e = errors(run(h, C, p, dH, dtype=torch.bfloat16), oracle(h, C, p, dH), w)
    assert max(e.values()) <= TOL_BF16, e


@pytest.mark.parametrize("accumulate", [False, True])
def test_state_gradients_add_and_weight_gradients_accumulate(accumulate):
    w, n = 3, 999
    h, C, p, dH = case(30, n, w)
    rng = np.random.default_rng(31)
    dC0 = [rng.normal(0, 1, (n, D)).astype(np.float32) for _ in range(w)]
    g0 = {k: rng.normal(0, 1, v.shape).astype(np.float32) for k, v in p.items()}
    H, dh, dC, g = oracle(h, C, p, dH)
    ref = (H, dh, [dC[k] + dC0[k] for k in range(w)],
           {k: g[k] + (g0[k] if accumulate else 0.0) for k in g})
    e = errors(run(h, C, p, dH, accumulate=accumulate, dC0=dC0, g0=g0), ref, w)
    assert max(e.values()) <= TOL, e


def test_without_biases_and_partial_state_gradients():
    w, n = 2, 500
    h, C, p, dH = case(40, n, w, bias_range=0.0)
    H, dh, dC, g = oracle(h, C, p, dH)
    dev = [to_dev(x) for x in C]
    W = {k: to_dev(v) for k, v in p.items() if k not in ("bi", "bh")}
    grads = {k: torch.empty_like(v) for k, v in W.items()}
    d1 = torch.zeros((n, D), device="cuda")
    Hg = api.hg_temporal_fwd(to_dev(h), dev, W)
    dh_g, g_g = api.hg_temporal_bwd(to_dev(h), dev, W, to_dev(dH), dstates=[None, d1], grads=grads)
    torch.cuda.synchronize()
    assert set(g_g) == {"Q", "r", "Wi", "Wh"}
    assert parity_err(Hg.cpu().numpy(), H) <= TOL
    assert parity_err(dh_g.cpu().numpy(), dh) <= TOL
    assert parity_err(d1.cpu().numpy(), dC[1]) <= TOL
    for k in g_g:
        assert parity_err(g_g[k].cpu().numpy(), g[k]) <= TOL, k
    # no state gradients at all
    dh2, g2 = api.hg_temporal_bwd(to_dev(h), dev, W, to_dev(dH), dstates=None)
    torch.cuda.synchronize()
    assert np.array_equal(dh2.cpu().numpy(), dh_g.cpu().numpy())
    assert np.array_equal(g2["Q"].cpu().numpy(), g_g["Q"].cpu().numpy())


def test_deterministic():
    w, n = 3, 3001
    h, C, p, dH = case(50, n, w)
    a = run(h, C, p, dH)
    b = run(h, C, p, dH)
    for x, y in zip(a[:2], b[:2]):
        assert np.array_equal(x, y)
    for x, y in zip(a[2], b[2]):
        assert np.array_equal(x, y)
    for k in a[3]:
        assert np.array_equal(a[3][k], b[3][k]), k


def test_empty_rows():
    p = {k: to_dev(v) for k, v in synth.temporal_weights(1, D).items()}
    e = torch.empty((0, D), device="cuda")
    H = api.hg_temporal_fwd(e, [e, e], p)
    grads = {k: torch.full_like(v, 3.0) for k, v in p.items()}
    dh, g = api.hg_temporal_bwd(e, [e, e], p, e, dstates=[e, e], grads=grads)
    torch.cuda.synchronize()
    assert H.shape == (0, D) and dh.shape == (0, D)
    for k in g:
        assert not g[k].cpu().numpy().any(), k


def test_argument_checks():
    p = {k: to_dev(v) for k, v in synth.temporal_weights(1, D).items()}
    h = torch.zeros((40, D), device="cuda")
    c = torch.zeros((40, D), device="cuda")
    with pytest.raises(api.HgError) as ei:
        api.hg_temporal_fwd(h, [c] * 5, p)
    assert ei.value.status == api.HG_ERR_UNSUPPORTED
    with pytest.raises(api.HgError) as ei:
        api.hg_temporal_fwd(torch.zeros((40, 128), device="cuda"), [], p)
    assert ei.value.status == api.HG_ERR_UNSUPPORTED
    with pytest.raises(api.HgError) as ei:
        api.hg_temporal_fwd(h, [c], p, H=c)
    assert ei.value.status == api.HG_ERR_ARG
    with pytest.raises(api.HgError) as ei:
        api.hg_temporal_bwd(h, [c], p, h, dh=h)
    assert ei.value.status == api.HG_ERR_ARG
    with pytest.raises(api.HgError) as ei:
        api.hg_temporal_bwd(h, [c], p, torch.zeros_like(h), dstates=[c])
    assert ei.value.status == api.HG_ERR_ARG
