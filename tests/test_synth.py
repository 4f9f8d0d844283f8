"""The seeded generator: determinism, shapes and the degree law it claims."""
import numpy as np

from paper_2608_02168_amd import synth


def test_deterministic_and_shaped():
    cfg = synth.scaled(synth.WORKLOADS["tiny"].graph, 0.5)
    a, b = synth.make_graph(cfg), synth.make_graph(cfg)
    for x, y in ((a.src, b.src), (a.dst, b.dst), (a.rel, b.rel), (a.ntype, b.ntype)):
        assert np.array_equal(x, y)
    assert a.src.dtype == np.int32 and a.rel.dtype == np.uint8
    assert a.src.shape == (cfg.n_edges,) and a.ntype.shape == (cfg.n_nodes,)
    assert a.src.max() < cfg.n_nodes and a.rel.max() < cfg.n_rel
    assert a.part.sum() == cfg.n_nodes - cfg.n_base


def test_degree_law_tiny():
    g = synth.make_graph(synth.WORKLOADS["tiny"].graph)
    deg = np.sort(np.bincount(g.src, minlength=g.n_nodes))[::-1]
    # Zipf(1.1) over 10^4 ranks: the top rank holds ~15% of 10^5 edges
    assert 12_000 < deg[0] < 18_500
    # hubs (type 1) are the top 1% by rank, hence by degree in expectation
    assert g.ntype.sum() == 100
    assert np.bincount(g.src, minlength=g.n_nodes)[g.ntype == 1].sum() > 0.5 * g.n_edges


def test_relation_split():
    cfg = synth.scaled(synth.WORKLOADS["skew"].graph, 0.002)
    g = synth.make_graph(cfg)
    share = np.bincount(g.rel, minlength=8) / g.n_edges
    np.testing.assert_allclose(share, np.array(synth.SKEW_SPLIT) / 100, atol=0.01)


def test_features_fixed_chunks():
    x = synth.features(3, 1000, 8)
    y = synth.features(3, 1000, 8)
    assert np.array_equal(x, y) and x.dtype == np.float32
    assert abs(x.mean()) < 0.05 and abs(x.std() - 1) < 0.05


def test_round_bf16_nearest_even():
    x = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, 1.0 + 2**-9, -2.5, 0.0], dtype=np.float32)
    r = synth.round_bf16(x)
    # 1+2^-8 is a tie between 1 and 1+2^-7: even mantissa -> 1
    assert list(r) == [1.0, 1.0, 1.0 + 2**-6, 1.0, -2.5, 0.0]
