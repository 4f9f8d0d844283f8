"""The alignment entry point that allocates nothing (its workspace is the
library's static device scratch), called through the C ABI, against the
entry point with a caller workspace: two calls in a row, the second with a
smaller batch (the scratch keeps the first call's contents), with a row
weight, a base, dH_ref and bf16 rows; results bit for bit equal, and within
the parity bar of the oracle."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import align
from paper_2608_02168_amd import api, synth
from tests.helpers import parity_err, to_dev

pytestmark = pytest.mark.gpu


def _case(n, m, d, seed):
    rng = np.random.default_rng(seed)
    H = (synth.features(seed, n, d) * rng.uniform(0.5, 2.0, d).astype(np.float32)).astype(np.float32)
    ov = np.sort(rng.choice(n, m, replace=False)).astype(np.int32)
    Href = (0.5 * H[ov] + synth.reference_embeddings(seed, m, d)).astype(np.float32)
    w = rng.uniform(0.2, 3.0, m).astype(np.float32)
    G0 = synth.upstream_grad(seed + 1, n, d)
    return H, ov, Href, w, G0


@pytest.mark.parametrize("d,dtype", [(128, torch.float32), (64, torch.float32), (256, torch.bfloat16)])
def test_noalloc_matches_workspace_entry_point(d, dtype):
    assert api.hg_align_noalloc_scratch_size() >= api.hg_align_workspace_size(1 << 40, 256)
    for n, m, seed in ((60000, 41000, 1), (9000, 3001, 2)):  # the second call smaller than the first
        H, ov, Href, w, G0 = _case(n, m, d, seed)
        Hd, ovd, Rd, wd = to_dev(H).to(dtype), to_dev(ov), to_dev(Href).to(dtype), to_dev(w)
        base = to_dev(G0).to(dtype)
        out = {}
        for kind in ("workspace", "noalloc"):
            dH = torch.full((n, d), 7.0, dtype=dtype, device="cuda")
            dR = torch.empty((m, d), dtype=dtype, device="cuda")
            loss = torch.empty(3, dtype=torch.float32, device="cuda")
            if kind == "workspace":
                api.hg_align_loss_fwd_bwd(Hd, ovd, Rd, dH, w=wd, ddof=1, dH_ref=dR, loss3=loss, dH_base=base)
            else:
                api.hg_align_loss_fwd_bwd_noalloc(Hd, ovd, Rd, dH, loss, w=wd, ddof=1, dH_ref=dR, dH_base=base)
            torch.cuda.synchronize()
            out[kind] = (loss.cpu(), dH.float().cpu(), dR.float().cpu())
        for a, b in zip(out["workspace"], out["noalloc"]):
            assert torch.equal(a, b)
        # and the oracle, on the rows as stored
        Hs = H if dtype == torch.float32 else synth.round_bf16(H)
        Rs = Href if dtype == torch.float32 else synth.round_bf16(Href)
        (li, ld, L), dX, dY = align.loss_and_grad(Hs[ov], Rs, w, 2e-4, 0.1, 1e-5, 1)
        tol = 1e-4 if dtype == torch.float32 else 2e-2
        loss, dH, dR = out["noalloc"]
        for got, exp in zip(loss.numpy(), (li, ld, L)):
            assert abs(got - exp) <= tol * abs(exp)
        Gs = G0.astype(np.float64) if dtype == torch.float32 else synth.round_bf16(G0).astype(np.float64)
        assert parity_err(dH.numpy()[ov], Gs[ov] + dX) <= tol
        rest = np.setdiff1d(np.arange(n), ov)
        assert np.all(dH.numpy()[rest] == 7.0)
        assert parity_err(dR.numpy(), dY) <= tol


def test_noalloc_rejects_what_the_workspace_call_rejects():
    z = torch.zeros((10, 96), dtype=torch.float32, device="cuda")
    ov = torch.zeros(3, dtype=torch.int32, device="cuda")
    loss = torch.empty(3, dtype=torch.float32, device="cuda")
    with pytest.raises(api.HgError) as e:
        api.hg_align_loss_fwd_bwd_noalloc(z, ov, z[:3], z, loss)
    assert e.value.status == api.HG_ERR_UNSUPPORTED
