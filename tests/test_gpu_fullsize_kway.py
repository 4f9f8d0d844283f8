"""The 4-subgraph step at its full size (10M nodes, 200M edges, random 4-way
partition, budget 800k per block), in the launch configuration bench.py
times (runner.make_kway_inputs / run_kway_step), against what the oracle can
compute at that size:
  * the node keys of the whole graph, bit-exact;
  * the selection, relabel, overlap, home blocks and base-edge relations of
    two of the four blocks, from the oracle's O(E) pieces, bit-exact, and the
    induced edge counts of all four;
  * the copy counts of every node (1 + the number of overlaps that hold it);
  * MeanAgg on sampled nodes, its backward on sampled rows of a subgraph and
    the home copies on sampled overlap rows, each from the GPU's own
    per-subgraph rows, computed one by one."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import kway, select
from paper_2608_02168_amd import api, runner, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def run():
    wl = synth.WORKLOADS["large_kway"]
    g = synth.make_graph(wl.graph)
    inp = runner.make_kway_inputs(wl, g)
    runner.run_kway_step(inp, update=False)
    torch.cuda.synchronize()
    yield wl, g, inp
    del inp
    torch.cuda.empty_cache()


def test_fullsize_kway_keys_and_selection(run):
    wl, g, inp = run
    cfg = wl.graph
    keys = select.node_keys(g.n_nodes, g.src, g.dst, cfg.key)
    assert np.array_equal(inp.keys.cpu().numpy(), keys)
    part = inp.part_np
    for k in (0, 2):
        sub = inp.subs[k]
        cand = select.candidates(part, k, g.src, g.dst)
        sel = select.top_m(cand, keys, cfg.theta, cfg.budget, cfg.seed)
        first = select.base_edge(part, k, g.src, g.dst)
        member = part == k
        member[sel] = True
        ids = np.nonzero(member)[0]
        l2g = ids[np.lexsort((ids, g.ntype[ids]))]
        assert np.array_equal(sub.view("local2global").cpu().numpy(), l2g), k
        g2l = np.full(g.n_nodes, -1, np.int64)
        g2l[l2g] = np.arange(l2g.shape[0])
        ov = sub.view("overlap").cpu().numpy()
        assert np.array_equal(ov, np.sort(g2l[sel])), k
        og = l2g[ov]
        assert np.array_equal(sub.view("overlap_home").cpu().numpy(), part[og]), k
        assert np.array_equal(sub.view("overlap_rel").cpu().numpy(), g.rel[first[og]]), k
        assert sub.e_sub == int(np.count_nonzero(member[g.src] & member[g.dst])), k
    for sub in inp.subs:
        member = np.zeros(g.n_nodes, bool)
        member[sub.view("local2global").cpu().numpy()] = True
        assert sub.e_sub == int(np.count_nonzero(member[g.src] & member[g.dst]))


def test_fullsize_kway_mean_agg_and_home_copies(run):
    wl, g, inp = run
    n, d = g.n_nodes, wl.model.d
    cnt = inp.cnt.cpu().numpy()
    in_overlap = np.zeros(n, np.int64)
    l2gs = [sb.view("local2global").cpu().numpy() for sb in inp.subs]
    g2ls = [sb.view("global2local").cpu().numpy() for sb in inp.subs]
    for sb, l2g in zip(inp.subs, l2gs):
        in_overlap[l2g[sb.view("overlap").cpu().numpy()]] += 1
    assert np.array_equal(cnt, 1 + in_overlap)
    rng = np.random.default_rng(5)
    # sampled nodes, with every node held by three or more subgraphs among them
    multi = np.nonzero(cnt >= 3)[0]
    v = np.unique(np.concatenate([rng.choice(n, 4000, replace=False), multi[:2000]]))
    last = [h[-1] for h in inp.H]
    rows = [(g2l[v] >= 0) for g2l in g2ls]
    acc = np.zeros((v.shape[0], d))
    for k in range(len(inp.subs)):
        r = g2ls[k][v]
        got = last[k][torch.from_numpy(np.where(r >= 0, r, 0)).cuda().long()].cpu().numpy().astype(np.float64)
        acc += np.where(rows[k][:, None], got, 0.0)
    want = acc / cnt[v][:, None]
    H = inp.H_agg[torch.from_numpy(v).cuda().long()].cpu().numpy()
    assert np.max(np.abs(H - want) / np.maximum(np.abs(want), np.sqrt(np.mean(want ** 2)))) <= 1e-6
    # backward into subgraph 1 on sampled rows
    sb = inp.subs[1]
    dh = api.hg_mean_agg_bwd(sb.view("local2global"), inp.cnt, inp.dH_agg)
    i = rng.choice(sb.n_sub, 4000, replace=False)
    gi = l2gs[1][i]
    want = inp.dH_agg[torch.from_numpy(gi).cuda().long()].cpu().numpy().astype(np.float64) / cnt[gi][:, None]
    got = dh[torch.from_numpy(i).cuda().long()].cpu().numpy()
    assert np.max(np.abs(got - want)) <= 1e-6 * max(np.abs(want).max(), 1e-30)
    # home copies of subgraph 3's overlap rows, bit-exact
    sb = inp.subs[3]
    Y = api.hg_home_gather(sb.view("overlap"), sb.view("local2global"), sb.view("overlap_home"),
                           [s.view("global2local") for s in inp.subs], last).cpu().numpy()
    ov = sb.view("overlap").cpu().numpy()
    home = sb.view("overlap_home").cpu().numpy()
    b = rng.choice(ov.shape[0], 4000, replace=False)
    og = l2gs[3][ov[b]]
    for h in range(4):
        sel = home[b] == h
        if not sel.any():
            continue
        r = torch.from_numpy(g2ls[h][og[sel]]).cuda().long()
        assert np.array_equal(Y[b[sel]], last[h][r].cpu().numpy()), h
    assert np.all(inp.part_np[og] == home[b]) and np.all(home[b] != 3)
