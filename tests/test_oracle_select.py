"""Pins of the oracle's overlapping-subgraph construction (CPU only).

Every check compares the oracle with something other than itself: published
SplitMix64 outputs, pure-Python brute force written from the definitions of
the candidate-set, h-index, TopM and union equations, and structural
invariants of CSR/CSC.
"""
import os

import numpy as np
import pytest

from oracle import select, splitmix
from paper_2608_02168_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "splitmix64_vectors.txt")


def test_splitmix64_published_vectors():
    rows = [l.split() for l in open(GOLDEN) if l.strip() and not l.startswith("#")]
    for seed, idx, val in rows:
        seq = splitmix.sequence(int(seed), int(idx) + 1)
        assert int(seq[int(idx)]) == int(val)


def test_tiebreak_is_first_output_of_seeded_state():
    gids = np.array([0, 1, 7, 123456, 2**31 - 1])
    for seed in (0, 42, 2**40 + 3):
        for g in gids:
            assert int(splitmix.tiebreak(seed, np.array([g]))[0]) == \
                int(splitmix.sequence(seed ^ int(g), 1)[0])


def _random_graph(rng, n, e, r, t=2):
    src = rng.integers(0, n, e)
    # a few hubs so degrees and h-indices vary
    hubs = rng.integers(0, n, max(1, n // 10))
    src[: e // 3] = rng.choice(hubs, e // 3)
    rng.shuffle(src)
    dst = rng.integers(0, n, e)
    rel = rng.integers(0, r, e)
    ntype = (rng.random(n) < 0.2).astype(np.int64) if t == 2 else np.zeros(n, np.int64)
    part = rng.integers(0, 3, n)
    return src, dst, rel, ntype, part


def _brute_hindex(n, src, dst):
    outdeg = [0] * n
    for s in src:
        outdeg[s] += 1
    nbrs = [[] for _ in range(n)]
    for s, d in zip(src, dst):
        nbrs[s].append(outdeg[d])
    h = []
    for v in range(n):
        a = sorted(nbrs[v], reverse=True)
        best = 0
        for i, x in enumerate(a, start=1):
            if x >= i:
                best = i
        h.append(best)
    return np.array(h)


def _brute_build(src, dst, rel, ntype, part, k, R, T, budget, key, theta, seed, ts=None, cut=None):
    n, e = len(ntype), len(src)
    base = {v for v in range(n) if part[v] == k}
    cand = {v for v in range(n) if v not in base and any(
        (src[i] == v and dst[i] in base) or (dst[i] == v and src[i] in base) for i in range(e))}
    if key == select.KEY_OUTDEG:
        keys = [sum(1 for s in src if s == v) for v in range(n)]
    else:
        keys = list(_brute_hindex(n, src, dst))
    pool = [v for v in cand if keys[v] <= theta]
    h = {v: int(splitmix.sequence(seed ^ v, 1)[0]) for v in pool}
    chosen = sorted(pool, key=lambda v: (keys[v], h[v], v))[: min(budget, len(pool))]
    nodes = base | set(chosen)
    local = sorted(nodes, key=lambda v: (ntype[v], v))
    g2l = {v: i for i, v in enumerate(local)}
    edges = [(i, g2l[src[i]], g2l[dst[i]], rel[i]) for i in range(e)
             if src[i] in nodes and dst[i] in nodes and (ts is None or ts[i] <= cut)]
    ns = len(local)
    csr_rows = [[] for _ in range(ns * R)]
    csc_rows = [[] for _ in range(ns * R)]
    for eid, s, d, r in edges:
        csr_rows[d * R + r].append((s, eid))
        csc_rows[s * R + r].append((d, eid))
    csc_rows = [sorted(row) for row in csc_rows]  # a CSC row by (destination, edge index)
    base_rel = {}
    for v in chosen:
        first = min(i for i in range(e) if (src[i] == v and dst[i] in base) or (dst[i] == v and src[i] in base))
        base_rel[v] = rel[first]
    return dict(local=local, edges=edges, csr_rows=csr_rows, csc_rows=csc_rows,
                overlap=sorted(g2l[v] for v in chosen), base_rel=base_rel, g2l=g2l)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("key", [select.KEY_OUTDEG, select.KEY_HINDEX])
def test_build_matches_brute_force(seed, key):
    rng = np.random.default_rng(seed)
    n, e, R = 40 + seed * 7, 160 + seed * 30, 1 + seed % 3
    src, dst, rel, ntype, part = _random_graph(rng, n, e, R)
    budget = int(rng.integers(1, 12))
    theta = [select.THETA_NONE, 1, 2, 4][seed % 4]
    sub = select.build(src, dst, rel, ntype, part, 1, R, 2, budget, key, theta, seed=seed * 11)
    bf = _brute_build(list(src), list(dst), list(rel), list(ntype), list(part), 1, R, 2,
                      budget, key, theta, seed * 11)
    assert list(sub.local2global) == bf["local"]
    assert sub.e_sub == len(bf["edges"])
    assert list(sub.eid) == [x[0] for x in bf["edges"]]
    assert list(sub.overlap) == bf["overlap"]
    for i, loc in enumerate(sub.overlap):
        gid = bf["local"][loc]
        assert sub.overlap_rel[i] == bf["base_rel"][gid]
        assert sub.overlap_home[i] == part[gid]
    for row in range(sub.n_sub * R):
        got = list(zip(sub.csr_col[sub.csr_ptr[row]:sub.csr_ptr[row + 1]],
                       sub.csr_eid[sub.csr_ptr[row]:sub.csr_ptr[row + 1]]))
        assert got == bf["csr_rows"][row]
        got = list(sub.csc_row[sub.csc_ptr[row]:sub.csc_ptr[row + 1]])
        assert got == [d for d, _ in bf["csc_rows"][row]]
    # type offsets
    for t in range(2):
        lo, hi = sub.type_off[t], sub.type_off[t + 1]
        assert all(ntype[bf["local"][i]] == t for i in range(lo, hi))
    # csc_scale = 1/deg_r(dst) as an fp32 quotient
    for row in range(sub.n_sub * R):
        r = row % R
        for p in range(sub.csc_ptr[row], sub.csc_ptr[row + 1]):
            d = sub.csc_row[p]
            deg = len(bf["csr_rows"][d * R + r])
            assert sub.csc_scale[p] == np.float32(1.0) / np.float32(deg)


@pytest.mark.parametrize("seed", range(4))
def test_weighted_build_matches_brute_force(seed):
    """Edge weights: every CSR entry carries its edge's weight and every CSC
    entry's scale is w / deg_r(destination), a float32 quotient; the rest of
    the build is the unweighted one."""
    rng = np.random.default_rng(300 + seed)
    n, e, R = 45 + seed * 5, 200 + seed * 25, 1 + seed % 3
    src, dst, rel, ntype, part = _random_graph(rng, n, e, R)
    w = rng.uniform(0.1, 2.0, e).astype(np.float32)
    sub = select.build(src, dst, rel, ntype, part, 1, R, 2, 7, seed=seed, edge_w=w)
    plain = select.build(src, dst, rel, ntype, part, 1, R, 2, 7, seed=seed)
    for name in ("local2global", "csr_ptr", "csr_col", "csr_eid", "csc_ptr", "csc_row"):
        assert np.array_equal(getattr(sub, name), getattr(plain, name)), name
    bf = _brute_build(list(src), list(dst), list(rel), list(ntype), list(part), 1, R, 2, 7,
                      select.KEY_OUTDEG, select.THETA_NONE, seed)
    for row in range(sub.n_sub * R):
        entries = bf["csr_rows"][row]
        got = sub.csr_w[sub.csr_ptr[row]:sub.csr_ptr[row + 1]]
        assert [float(x) for x in got] == [float(w[eid]) for _, eid in entries]
    for row in range(sub.n_sub * R):
        r = row % R
        for p, (d, eid) in zip(range(sub.csc_ptr[row], sub.csc_ptr[row + 1]), bf["csc_rows"][row]):
            deg = len(bf["csr_rows"][d * R + r])
            assert sub.csc_scale[p] == np.float32(w[eid]) / np.float32(deg)


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("cut", [-1, 3, 6, 9])
def test_snapshot_matches_brute_force(seed, cut):
    rng = np.random.default_rng(100 + seed)
    n, e, R = 50 + seed * 5, 220 + seed * 20, 1 + seed % 3
    src, dst, rel, ntype, part = _random_graph(rng, n, e, R)
    ts = rng.integers(0, 10, e)
    key = seed % 2
    sub = select.build(src, dst, rel, ntype, part, 1, R, 2, 6, key, select.THETA_NONE, seed=seed,
                       edge_ts=ts, t_cut=cut)
    bf = _brute_build(list(src), list(dst), list(rel), list(ntype), list(part), 1, R, 2, 6, key,
                      select.THETA_NONE, seed, ts=list(ts), cut=cut)
    assert list(sub.local2global) == bf["local"]
    assert list(sub.overlap) == bf["overlap"]
    assert list(sub.eid) == [x[0] for x in bf["edges"]]
    for row in range(sub.n_sub * R):
        got = list(zip(sub.csr_col[sub.csr_ptr[row]:sub.csr_ptr[row + 1]],
                       sub.csr_eid[sub.csr_ptr[row]:sub.csr_ptr[row + 1]]))
        assert got == bf["csr_rows"][row]
        got = list(sub.csc_row[sub.csc_ptr[row]:sub.csc_ptr[row + 1]])
        assert got == [d for d, _ in bf["csc_rows"][row]]
        r = row % R
        for p in range(sub.csc_ptr[row], sub.csc_ptr[row + 1]):
            deg = len(bf["csr_rows"][sub.csc_row[p] * R + r])
            assert sub.csc_scale[p] == np.float32(1.0) / np.float32(deg)


def test_snapshots_share_nodes_and_nest():
    g = synth.make_graph(synth.WORKLOADS["tiny"].graph)
    ts = synth.edge_times(0, g.n_edges)
    cfg = synth.WORKLOADS["tiny"].graph
    args = (g.src, g.dst, g.rel, g.ntype, g.part, g.k, cfg.n_rel, 2, cfg.budget, cfg.key, cfg.theta, 7)
    full = select.build(*args)
    cuts = synth.snapshot_cuts(4)
    snaps = [select.build(*args, edge_ts=ts, t_cut=c) for c in cuts]
    for a, b in zip(snaps, snaps[1:]):
        assert a.e_sub < b.e_sub
        assert set(a.eid) <= set(b.eid)
    last = snaps[-1]
    assert int(ts.max()) <= cuts[-1]
    for name in ("local2global", "overlap", "overlap_rel", "csr_ptr", "csr_col", "csr_eid", "csc_ptr",
                 "csc_row", "csc_scale"):
        assert np.array_equal(getattr(last, name), getattr(full, name)), name
    for s in snaps:
        assert np.array_equal(s.local2global, full.local2global)
        assert np.array_equal(s.overlap, full.overlap)
        assert np.array_equal(s.eid, full.eid[ts[full.eid] <= cuts[snaps.index(s)]])


def test_hindex_brute_force_and_bounds():
    rng = np.random.default_rng(7)
    for _ in range(5):
        n, e = 60, 400
        src, dst, _, _, _ = _random_graph(rng, n, e, 1)
        h = select.out_hindex(n, src, dst)
        assert np.array_equal(h, _brute_hindex(n, list(src), list(dst)))
        od = select.out_degree(n, src)
        assert np.all(h <= od)


def test_hindex_textbook_examples():
    # node 0 points to nodes with out-degrees 3, 3, 1 -> h = 2 ("two of degree >= 2")
    src = np.array([0, 0, 0, 1, 1, 1, 2, 2, 2, 3])
    dst = np.array([1, 2, 3, 4, 4, 4, 4, 4, 4, 4])
    h = select.out_hindex(5, src, dst)
    assert h[0] == 2
    assert h[1] == 0 and h[4] == 0           # neighbour 4 has out-degree 0
    # star with all leaves of out-degree 5 and 5 leaves: h = 5
    src = np.concatenate([np.zeros(5, int), np.repeat(np.arange(1, 6), 5)])
    dst = np.concatenate([np.arange(1, 6), np.full(25, 6)])
    assert select.out_hindex(7, src, dst)[0] == 5


def test_budget_covers_pool_selects_all_candidates():
    rng = np.random.default_rng(3)
    src, dst, rel, ntype, part = _random_graph(rng, 200, 900, 2)
    cand = select.candidates(part, 0, src, dst)
    sub = select.build(src, dst, rel, ntype, part, 0, 2, 2, budget=10**6)
    assert set(sub.local2global[sub.overlap]) == set(np.nonzero(cand)[0])


def test_invariants_on_synthetic_tiny():
    g = synth.make_graph(synth.scaled(synth.WORKLOADS["tiny"].graph, 0.2))
    sub = select.build(g.src, g.dst, g.rel, g.ntype, g.part, g.k, g.cfg.n_rel, 2,
                       g.cfg.budget)
    R = g.cfg.n_rel
    assert sub.csr_ptr[-1] == sub.e_sub == sub.csc_ptr[-1]
    assert np.all(np.diff(sub.csr_ptr) >= 0) and np.all(np.diff(sub.csc_ptr) >= 0)
    rows_csr = np.repeat(np.arange(sub.n_sub * R), np.diff(sub.csr_ptr))
    rows_csc = np.repeat(np.arange(sub.n_sub * R), np.diff(sub.csc_ptr))
    a = sorted(zip(rows_csr % R, sub.csr_col, rows_csr // R))
    b = sorted(zip(rows_csc % R, rows_csc // R, sub.csc_row))
    assert a == b
    # in-degree per relation equals CSR row length
    for r in range(R):
        m = sub.rel_l == r
        deg = np.bincount(sub.dst_l[m], minlength=sub.n_sub)
        assert np.array_equal(deg, np.diff(sub.csr_ptr)[r::R])
    # overlap nodes are candidates, not in the base, and within budget
    assert sub.overlap.shape[0] <= g.cfg.budget
    assert np.all(g.part[sub.local2global[sub.overlap]] != g.k)
    # global2local inverts local2global
    assert np.array_equal(sub.global2local[sub.local2global], np.arange(sub.n_sub))
    assert (sub.global2local >= 0).sum() == sub.n_sub


def test_empty_and_degenerate():
    # no edges: no candidates, subgraph = base set
    part = np.array([0, 0, 1, 1])
    sub = select.build(np.zeros(0, int), np.zeros(0, int), np.zeros(0, int),
                       np.array([0, 1, 0, 0]), part, 0, 2, 2, budget=5)
    assert sub.n_sub == 2 and sub.e_sub == 0 and sub.overlap.shape[0] == 0
    assert list(sub.local2global) == [0, 1]
    assert list(sub.csr_ptr) == [0] * 5
    # budget 0: no overlap but base-internal edges are kept
    src, dst = np.array([0, 2, 1]), np.array([1, 0, 3])
    sub = select.build(src, dst, np.zeros(3, int), np.zeros(4, int), part, 0, 1, 1, budget=0)
    assert sub.overlap.shape[0] == 0 and sub.e_sub == 1 and sub.eid[0] == 0


def test_planted_mistake_in_hindex_is_caught(monkeypatch):
    """A plausible off-by-one in the oracle's h-index fails the brute-force pin."""
    def wrong(n, src, dst):
        src = np.asarray(src, dtype=np.int64)
        vals = select.out_degree(n, src)[np.asarray(dst, dtype=np.int64)]
        order = np.lexsort((-vals, src))
        s, a = src[order], vals[order]
        first = np.searchsorted(s, s, side="left")
        rank = np.arange(s.shape[0]) - first + 1
        return np.bincount(s, weights=(a > rank), minlength=n).astype(np.int64)
    rng = np.random.default_rng(7)
    src, dst, _, _, _ = _random_graph(rng, 60, 400, 1)
    assert not np.array_equal(wrong(60, src, dst), _brute_hindex(60, list(src), list(dst)))
