"""GPU parity of hg_build_csr against the oracle: every integer output
bit-exact (csc_scale bit-exact as a correctly rounded quotient), run-twice
determinism, and the device range check."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import select
from paper_2608_02168_amd import api, synth
from tests.helpers import graph_to_dev

pytestmark = pytest.mark.gpu

CASES = {
    # name: (graph config, key, theta, budget override)
    "tiny": (synth.WORKLOADS["tiny"].graph, 0, select.THETA_NONE, None),
    "tiny_hindex_theta2": (synth.WORKLOADS["tiny"].graph, 1, 2, None),
    "tiny_budget_cut": (synth.WORKLOADS["tiny"].graph, 0, select.THETA_NONE, 137),
    "tiny_hindex_budget_cut": (synth.WORKLOADS["tiny"].graph, 1, select.THETA_NONE, 211),
    "skew_small_theta3": (synth.scaled(synth.WORKLOADS["skew"].graph, 0.002), 0, 3, None),
    "medium_small": (synth.scaled(synth.WORKLOADS["medium"].graph, 0.01), 0, select.THETA_NONE, 900),
}


def run_both(cfg, key, theta, budget, seed=12345, n_ntype=2):
    g = synth.make_graph(cfg)
    budget = cfg.budget if budget is None else budget
    ref = select.build(g.src, g.dst, g.rel, g.ntype, g.part, g.k, cfg.n_rel, n_ntype, budget,
                       key, theta, seed)
    d = graph_to_dev(g)
    sub = api.hg_build_csr(d["src"], d["dst"], d["rel"], d["ntype"], d["part"], g.k, cfg.n_rel,
                           n_ntype, budget, key=key, theta=theta, seed=seed)
    return g, ref, sub


def assert_same(ref, sub):
    assert sub.n_sub == ref.n_sub and sub.e_sub == ref.e_sub
    assert sub.m_sel == ref.overlap.shape[0]
    for name in ("local2global", "global2local", "type_off", "overlap", "overlap_home",
                 "overlap_rel", "csr_ptr", "csr_col", "csr_eid", "csc_ptr", "csc_row"):
        got = sub.view(name).cpu().numpy()
        exp = getattr(ref, name)
        assert got.shape == exp.shape, name
        assert np.array_equal(got, exp.astype(got.dtype)), name
    sc = sub.view("csc_scale").cpu().numpy()
    assert np.array_equal(sc.view(np.uint32), ref.csc_scale.view(np.uint32))
    assert sub.n_active() == list(ref.n_active)
    assert sub.type_off_host() == list(ref.type_off)


@pytest.mark.parametrize("case", sorted(CASES))
def test_build_bit_exact(case):
    cfg, key, theta, budget = CASES[case]
    _, ref, sub = run_both(cfg, key, theta, budget)
    assert_same(ref, sub)


# The CSR/CSC sorts take digits of 9 bits where that saves a pass: keys of
# 9 bits sort in one 9-bit pass, of 18 bits in two, and the CSC sort's last
# pass (which unpacks each entry's destination and scale) then runs with a
# 9-bit digit.  Subgraph sizes n_sub * R that give exactly those key widths.
DIGIT_PLANS = {9: 0.012, 18: 6.0}


@pytest.mark.parametrize("bits", sorted(DIGIT_PLANS))
def test_build_bit_exact_nine_bit_digits(bits):
    cfg = synth.scaled(synth.WORKLOADS["tiny"].graph, DIGIT_PLANS[bits])
    _, ref, sub = run_both(cfg, 0, select.THETA_NONE, None)
    nq = ref.n_sub * cfg.n_rel
    assert (nq - 1).bit_length() == bits, nq
    assert_same(ref, sub)


def test_build_deterministic():
    cfg, key, theta, budget = CASES["tiny_hindex_budget_cut"]
    g, _, a = run_both(cfg, key, theta, budget)
    _, _, b = run_both(cfg, key, theta, budget)
    for name in ("local2global", "overlap", "csr_col", "csc_row", "csc_scale"):
        assert torch.equal(a.view(name), b.view(name))
    # the plan's used part is identical: rebuild both into zeroed plan buffers
    d = graph_to_dev(g)
    plans = []
    for sub in (a, b):
        sub.arrays["plan"].zero_()
        api.hg_build_csr(d["src"], d["dst"], d["rel"], d["ntype"], d["part"], g.k, cfg.n_rel, 2,
                         budget, key=key, theta=theta, seed=12345, out=sub)
        plans.append(sub.arrays["plan"].cpu().numpy())
    assert np.array_equal(plans[0], plans[1])


def test_build_single_type_single_relation_and_ragged():
    rng = np.random.default_rng(4)
    n, e = 1537, 9001
    src = rng.integers(0, n, e).astype(np.int32)
    dst = rng.integers(0, n, e).astype(np.int32)
    rel = np.zeros(e, np.uint8)
    ntype = np.zeros(n, np.uint8)
    part = (rng.random(n) < 0.3).astype(np.int32)
    ref = select.build(src, dst, rel, ntype, part, 1, 1, 1, 77, 0, select.THETA_NONE, 3)
    t = lambda x: torch.from_numpy(x).cuda()
    sub = api.hg_build_csr(t(src), t(dst), t(rel), t(ntype), t(part), 1, 1, 1, 77, seed=3)
    assert_same(ref, sub)


@pytest.mark.parametrize("parts", [0, 3])
def test_build_hub_destinations(parts):
    """Rows (dst, r) with 254, 255, 256 and 1000 in-edges: the mean weight of
    a row past the byte table's range comes from the row pointers."""
    rng = np.random.default_rng(8)
    n, R = 700, 2
    hubs = {3: 254, 10: 255, 11: 256, 20: 1000, 30: 3000}
    src = [rng.integers(0, n, 4000)]
    dst = [rng.integers(0, n, 4000)]
    rel = [rng.integers(0, R, 4000)]
    for h, k in hubs.items():
        src.append(rng.integers(0, n, k))
        dst.append(np.full(k, h))
        rel.append(np.full(k, 1))
    perm = rng.permutation(sum(len(x) for x in src))
    src = np.concatenate(src)[perm].astype(np.int32)
    dst = np.concatenate(dst)[perm].astype(np.int32)
    rel = np.concatenate(rel)[perm].astype(np.uint8)
    ntype = (rng.random(n) < 0.2).astype(np.uint8)
    part = (synth.random_partition(n, 3, 2) if parts else (np.arange(n) >= 600).astype(np.int32))
    part[list(hubs)] = 0
    ref = select.build(src, dst, rel, ntype, part, 0, R, 2, 150, 0, select.THETA_NONE, 5)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()
    sub = api.hg_build_csr(t(src), t(dst), t(rel), t(ntype), t(part), 0, R, 2, 150, seed=5)
    assert_same(ref, sub)
    assert ref.csc_scale.min() < 1.0 / 255


def test_build_no_edges_and_zero_budget():
    n = 100
    z32 = torch.zeros(0, dtype=torch.int32, device="cuda")
    z8 = torch.zeros(0, dtype=torch.uint8, device="cuda")
    ntype = torch.zeros(n, dtype=torch.uint8, device="cuda")
    part = (torch.arange(n, device="cuda") >= 60).to(torch.int32)
    sub = api.hg_build_csr(z32, z32, z8, ntype, part, 0, 2, 1, 0)
    assert sub.n_sub == 60 and sub.e_sub == 0 and sub.m_sel == 0
    assert torch.equal(sub.view("local2global").cpu(), torch.arange(60, dtype=torch.int32))
    assert int(sub.view("csr_ptr").abs().sum()) == 0


def test_build_single_row_needs_no_sort_pass():
    # one node, one relation: every CSR/CSC key is 0 (no radix pass runs)
    src = torch.zeros(7, dtype=torch.int32, device="cuda")
    rel = torch.zeros(7, dtype=torch.uint8, device="cuda")
    ntype = torch.zeros(1, dtype=torch.uint8, device="cuda")
    part = torch.zeros(1, dtype=torch.int32, device="cuda")
    ref = select.build(np.zeros(7, np.int32), np.zeros(7, np.int32), np.zeros(7, np.uint8), np.zeros(1, np.uint8),
                       np.zeros(1, np.int32), 0, 1, 1, 0, 0, select.THETA_NONE, 0)
    sub = api.hg_build_csr(src, src, rel, ntype, part, 0, 1, 1, 0)
    assert_same(ref, sub)


def test_build_range_error_is_reported():
    n = 50
    src = torch.tensor([1, 2, 70], dtype=torch.int32, device="cuda")  # 70 >= n
    dst = torch.tensor([3, 4, 5], dtype=torch.int32, device="cuda")
    rel = torch.zeros(3, dtype=torch.uint8, device="cuda")
    ntype = torch.zeros(n, dtype=torch.uint8, device="cuda")
    part = torch.zeros(n, dtype=torch.int32, device="cuda")
    with pytest.raises(api.HgError) as ei:
        api.hg_build_csr(src, dst, rel, ntype, part, 0, 1, 1, 5)
    assert ei.value.status == api.HG_ERR_RANGE


SNAPSHOT_CASES = {
    "tiny": (synth.WORKLOADS["tiny"].graph, 0, select.THETA_NONE, None),
    "tiny_hindex_budget_cut": (synth.WORKLOADS["tiny"].graph, 1, select.THETA_NONE, 211),
    "skew_small_theta3": (synth.scaled(synth.WORKLOADS["skew"].graph, 0.002), 0, 3, None),
}


@pytest.mark.parametrize("case", sorted(SNAPSHOT_CASES))
@pytest.mark.parametrize("parts", [0, 3])
def test_snapshot_build_bit_exact(case, parts):
    """Each snapshot (edges with timestamp <= cut, node set from every edge)
    matches the oracle's snapshot bit for bit, for every monthly cut plus a
    cut before the first day (no edges) and one inside a month; with the
    configuration's base set (most nodes in the subgraph) and with block 0 of
    a random 3-way partition (a third of them: the membership-bitmap path)."""
    cfg, key, theta, budget = SNAPSHOT_CASES[case]
    budget = cfg.budget if budget is None else budget
    g = synth.make_graph(cfg)
    if parts:
        g.part = synth.random_partition(g.n_nodes, parts, 11)
    ts = synth.edge_times(cfg.seed, g.n_edges)
    d = graph_to_dev(g)
    ts_d = torch.from_numpy(ts).cuda()
    cuts = [-1, 13] + synth.snapshot_cuts(4)
    sub = None
    for cut in cuts:
        ref = select.build(g.src, g.dst, g.rel, g.ntype, g.part, g.k, cfg.n_rel, 2, budget, key, theta, 99,
                           edge_ts=ts, t_cut=cut)
        sub = api.hg_build_csr(d["src"], d["dst"], d["rel"], d["ntype"], d["part"], g.k, cfg.n_rel, 2, budget,
                               key=key, theta=theta, seed=99, edge_ts=ts_d, t_cut=cut, out=sub)
        print(f"snapshot {case} cut={cut}: e_sub={ref.e_sub}", flush=True)
        assert_same(ref, sub)
    assert sub.e_sub == select.build(g.src, g.dst, g.rel, g.ntype, g.part, g.k, cfg.n_rel, 2, budget, key, theta,
                                     99).e_sub


@pytest.mark.parametrize("case", ["tiny", "tiny_hindex_theta2", "skew_small_theta3", "medium_small"])
def test_node_keys_bit_exact(case):
    cfg, key, _, _ = CASES[case]
    g = synth.make_graph(cfg)
    d = graph_to_dev(g)
    got = api.hg_node_keys(d["src"], d["dst"], d["rel"], g.n_nodes, cfg.n_rel, key).cpu().numpy()
    assert np.array_equal(got, select.node_keys(g.n_nodes, g.src, g.dst, key))


@pytest.mark.parametrize("case", sorted(CASES))
def test_build_with_given_keys_bit_exact(case):
    # the keys of the whole graph given to the build (shared by the builds
    # of several blocks) change none of its outputs; a random 3-way
    # partition, block 1
    cfg, key, theta, budget = CASES[case]
    g = synth.make_graph(cfg)
    budget = cfg.budget if budget is None else budget
    part = synth.random_partition(g.n_nodes, 3, 5)
    ref = select.build(g.src, g.dst, g.rel, g.ntype, part, 1, cfg.n_rel, 2, budget, key, theta, 77)
    d = graph_to_dev(g)
    d["part"] = torch.from_numpy(part).cuda()
    keys = api.hg_node_keys(d["src"], d["dst"], d["rel"], g.n_nodes, cfg.n_rel, key)
    sub = api.hg_build_csr(d["src"], d["dst"], d["rel"], d["ntype"], d["part"], 1, cfg.n_rel, 2, budget, key=key,
                           theta=theta, seed=77, node_key=keys)
    assert_same(ref, sub)


def test_node_keys_range_error_and_empty():
    n = 50
    src = torch.tensor([0, 3, n], dtype=torch.int32, device="cuda")
    dst = torch.tensor([1, 2, 4], dtype=torch.int32, device="cuda")
    rel = torch.zeros(3, dtype=torch.uint8, device="cuda")
    for key in (0, 1):
        with pytest.raises(api.HgError) as e:
            api.hg_node_keys(src, dst, rel, n, 1, key)
        assert e.value.status == api.HG_ERR_RANGE
    empty = torch.zeros(0, dtype=torch.int32, device="cuda")
    for key in (0, 1):
        got = api.hg_node_keys(empty, empty, empty.to(torch.uint8), n, 1, key).cpu().numpy()
        assert np.all(got == 0)


@pytest.mark.parametrize("n_rel", [3, 64])
def test_transform_layout_choice(n_rel):
    """The relation transforms take one row per active (source, relation)
    pair (A rows) unless the row-indexed layout (n_sub * R rows) costs at
    most four times that: tiny at R = 3 (A / (n_sub R) = 0.45) keeps the
    row-indexed layout, R = 64 (0.06) the compact one."""
    from dataclasses import replace
    cfg = replace(synth.WORKLOADS["tiny"].graph, n_rel=n_rel)
    g = synth.make_graph(cfg)
    d = graph_to_dev(g)
    sub = api.hg_build_csr(d["src"], d["dst"], d["rel"], d["ntype"], d["part"], g.k, n_rel, 2, cfg.budget)
    A, nq = sum(sub.n_active()), sub.n_sub * n_rel
    assert int(sub.c.plan_slot_rows) == (nq if nq <= 4 * A else A)
    assert (nq <= 4 * A) == (n_rel == 3)



def test_build_beyond_24_bit_destinations():
    """A subgraph of more than 2^24 nodes: a destination no longer fits the
    24 bits the CSC sort packs next to its row degree, so the sort carries the
    scale 1 / deg as a second value instead; the outputs are the same."""
    cfg = synth.GraphConfig("wide", (1 << 24) + 50_000, 3_000_000, 3, 1.2, 50.0, 1 << 24, 40_000, seed=21)
    _, ref, sub = run_both(cfg, 0, select.THETA_NONE, None)
    assert sub.n_sub > (1 << 24)
    assert int(ref.csc_row.max()) >= (1 << 24)
    assert_same(ref, sub)
