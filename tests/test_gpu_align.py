"""GPU parity of hg_align_loss_fwd_bwd against the oracle (float64)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import align
from paper_2608_02168_amd import api, synth
from tests.helpers import parity_err, to_dev

pytestmark = pytest.mark.gpu
TOL = 1e-4


def make(n_rows, m, d, seed):
    rng = np.random.default_rng(seed)
    H = synth.features(seed, n_rows, d) * rng.uniform(0.5, 2.0, d).astype(np.float32) \
        + rng.uniform(-1, 1, d).astype(np.float32)
    ov = np.sort(rng.choice(n_rows, m, replace=False)).astype(np.int32)
    Href = (0.5 * H[ov] + synth.reference_embeddings(seed, m, d)).astype(np.float32)
    return H.astype(np.float32), ov, Href


@pytest.mark.parametrize("d", [64, 128, 256])
@pytest.mark.parametrize("m", [500, 4099])
@pytest.mark.parametrize("weighted,ddof,eps", [(False, 0, 1e-5), (True, 1, 1e-3), (False, 1, 0.0)])
def test_align_parity(d, m, weighted, ddof, eps):
    H, ov, Href = make(9000, m, d, seed=m + d)
    w = np.random.default_rng(1).uniform(0.2, 3.0, m).astype(np.float32) if weighted else None
    lam, scale = 2e-4, 0.1
    (li, ld, L), dX, dY = align.loss_and_grad(H[ov], Href, w, lam, scale, eps, ddof)
    G0 = synth.upstream_grad(9, H.shape[0], d)
    dH = to_dev(G0.copy())
    dHref = torch.empty((m, d), dtype=torch.float32, device="cuda")
    loss = api.hg_align_loss_fwd_bwd(to_dev(H), to_dev(ov), to_dev(Href), dH,
                                     w=None if w is None else to_dev(w), lambda_n=lam, scale=scale,
                                     eps=eps, ddof=ddof, dH_ref=dHref).cpu().numpy()
    for got, exp in zip(loss, (li, ld, L)):
        assert abs(got - exp) <= TOL * abs(exp)
    expect = G0.astype(np.float64)
    expect[ov] += dX
    assert parity_err(dH.cpu().numpy()[ov], expect[ov]) <= TOL
    rest = np.setdiff1d(np.arange(H.shape[0]), ov)
    assert np.array_equal(dH.cpu().numpy()[rest], G0[rest])
    assert parity_err(dHref.cpu().numpy(), dY) <= TOL


@pytest.mark.parametrize("d", [64, 128, 256])
@pytest.mark.parametrize("m", [5, 33, 70000])
def test_align_parity_sizes(d, m):
    """Batches of one 32-row step or less (5, 33 rows) and one of many chunks
    and reduction groups (70000 rows: every level of the Gram pass's
    fixed-order reduction, padding blocks at d = 256).  (At M = ddof + 1 the
    standardisation backward removes every direction but the one eps leaves:
    dX is float32 rounding of a cancellation, so tiny batches start at 5.)"""
    H, ov, Href = make(max(9000, 2 * m), m, d, seed=m + 3 * d)
    w = np.random.default_rng(2).uniform(0.2, 3.0, m).astype(np.float32)
    lam, scale, eps, ddof = 2e-4, 0.1, 1e-5, 1
    (li, ld, L), dX, dY = align.loss_and_grad(H[ov], Href, w, lam, scale, eps, ddof)
    dH = torch.zeros(H.shape, dtype=torch.float32, device="cuda")
    dHref = torch.empty((m, d), dtype=torch.float32, device="cuda")
    loss = api.hg_align_loss_fwd_bwd(to_dev(H), to_dev(ov), to_dev(Href), dH, w=to_dev(w), lambda_n=lam,
                                     scale=scale, eps=eps, ddof=ddof, dH_ref=dHref).cpu().numpy()
    for got, exp in zip(loss, (li, ld, L)):
        assert abs(got - exp) <= TOL * abs(exp)
    assert parity_err(dH.cpu().numpy()[ov], dX) <= TOL
    assert parity_err(dHref.cpu().numpy(), dY) <= TOL


def test_align_identical_views_zero_invariance():
    H, ov, _ = make(3000, 700, 64, seed=3)
    dH = torch.zeros((3000, 64), dtype=torch.float32, device="cuda")
    loss = api.hg_align_loss_fwd_bwd(to_dev(H), to_dev(ov), to_dev(H[ov].copy()), dH,
                                     lambda_n=0.0, scale=1.0, eps=0.0).cpu().numpy()
    assert abs(loss[0]) < 1e-4
    assert float(dH.abs().max()) < 1e-5


def test_align_empty_batch():
    dH = torch.zeros((10, 64), dtype=torch.float32, device="cuda")
    ov = torch.zeros(0, dtype=torch.int32, device="cuda")
    ref = torch.zeros((0, 64), dtype=torch.float32, device="cuda")
    loss = api.hg_align_loss_fwd_bwd(dH, ov, ref, dH).cpu().numpy()
    assert np.array_equal(loss, np.zeros(3, np.float32))


def test_align_deterministic():
    H, ov, Href = make(5000, 2000, 128, seed=11)
    outs = []
    for _ in range(2):
        dH = torch.zeros((5000, 128), dtype=torch.float32, device="cuda")
        loss = api.hg_align_loss_fwd_bwd(to_dev(H), to_dev(ov), to_dev(Href), dH)
        outs.append((loss.cpu(), dH.cpu()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_align_with_base_rows(dtype):
    # dH[overlap] = base[overlap] + scale dX; every other row of dH untouched
    # and base only read -- equal, bit for bit, to adding into a copy of base
    H, ov, Href = make(6000, 1500, 128, seed=21)
    G0 = synth.upstream_grad(4, H.shape[0], 128)
    junk = np.full_like(G0, 7.0)
    base = to_dev(G0).to(dtype)
    dH = to_dev(junk).to(dtype)
    api.hg_align_loss_fwd_bwd(to_dev(H).to(dtype), to_dev(ov), to_dev(Href).to(dtype), dH, dH_base=base)
    ref = to_dev(G0).to(dtype)
    api.hg_align_loss_fwd_bwd(to_dev(H).to(dtype), to_dev(ov), to_dev(Href).to(dtype), ref)
    got, want = dH.float().cpu().numpy(), ref.float().cpu().numpy()
    assert np.array_equal(got[ov], want[ov])
    rest = np.setdiff1d(np.arange(H.shape[0]), ov)
    assert np.all(got[rest] == 7.0)
    assert torch.equal(base, to_dev(G0).to(dtype))
