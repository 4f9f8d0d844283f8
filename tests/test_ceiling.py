"""The benchmark's memory-ceiling tool (libhg_ceiling.so): exports on the CPU;
on the GPU its group sums match torch's gather-and-sum and its ids stay in
range, so the ceiling it times does the work it claims."""
import ctypes as C

import pytest

from paper_2608_02168_amd import ceiling


def test_ceiling_exports():
    L = C.CDLL(ceiling.LIB_PATH)
    for name in ("hgc_random_rows", "hgc_gather"):
        assert hasattr(L, name)


def test_ceiling_rejects_bad_arguments():
    L = ceiling.lib()
    one = C.c_void_p(1)
    assert L.hgc_random_rows(None, 10, 10, 0, None) == -1
    assert L.hgc_random_rows(one, 10, 0, 0, None) == -1
    assert L.hgc_gather(one, 10, 128, one, 100, 0, one, 1, None) == -1
    assert L.hgc_gather(one, 10, 128, one, 100, 65, one, 1, None) == -1
    assert L.hgc_gather(None, 10, 128, one, 100, 4, one, 1, None) == -1


@pytest.mark.gpu
@pytest.mark.parametrize("d,group,n_idx", [(64, 1, 1000), (128, 14, 14 * 333 + 5), (128, 64, 64 * 50),
                                           (256, 7, 7 * 101)])
def test_ceiling_gather_matches_torch(d, group, n_idx):
    import torch
    n_rows = 5000
    torch.manual_seed(d + group)
    table = torch.randn((n_rows, d), device="cuda")
    idx = torch.empty(n_idx, dtype=torch.int32, device="cuda")
    ceiling.random_rows(idx, n_rows, 99)
    torch.cuda.synchronize()
    assert int(idx.min()) >= 0 and int(idx.max()) < n_rows
    # ids spread over the table (uniform: every decile of rows is hit)
    hist = torch.bincount((idx.long() * 10) // n_rows, minlength=10)
    assert int((hist > 0).sum()) == 10
    ng = n_idx // group
    out = torch.full((ng, d), float("nan"), device="cuda")
    ceiling.gather(table, idx, group, out, True)
    ref = table[idx[: ng * group].long()].view(ng, group, d).sum(1)
    torch.cuda.synchronize()
    assert torch.allclose(out, ref, rtol=1e-5, atol=1e-4)
    # without writes nothing is stored for a finite table
    sink = torch.full((1, d), 7.0, device="cuda")
    ceiling.gather(table, idx, group, sink, False)
    torch.cuda.synchronize()
    assert bool((sink == 7.0).all())
