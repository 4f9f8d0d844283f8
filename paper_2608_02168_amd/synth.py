"""Seeded synthetic inputs shaped like the paper's user--risk graphs.

This module is shared by the tests, the benchmark and the oracle's callers.
It draws random numbers only: it contains none of the method's arithmetic
(no selection, no aggregation, no loss).  Every array is a pure function of
the configuration and its seeds.

Graph recipe (stands in for the proprietary dataset of the paper's
experimental-setup section, which has two node types, tens of relation
types and a heavy-tailed user--event degree law):

* sources: a shifted rank-Zipf law, P(rank k) = (k + k0)^-s / Z for
  k = 1..N, drawn as a multinomial count per rank, expanded and shuffled so
  edge order is random; ranks map to node ids through a seeded permutation,
  so hubs are scattered over ids;
* destinations: uniform over all nodes;
* relations: uniform, or a fixed categorical split;
* node types: type 1 ("risk event") for the top 1% Zipf ranks, type 0
  ("user") otherwise;
* base partition: part[v] = 0 for the first n_base ids, 1 otherwise;
* features, reference embeddings, upstream gradients: N(0, 1) float32;
* weights: Xavier-uniform U(+-sqrt(6 / (2 d))); biases U(+-bias_range).
"""
from __future__ import annotations

import concurrent.futures as _cf
import os
from dataclasses import dataclass, field, replace
from typing import Optional, Sequence

import numpy as np

# Relation split of the skew-stress workload (percent of edges per relation).
SKEW_SPLIT = (50, 20, 10, 5, 5, 5, 3, 2)


@dataclass(frozen=True)
class GraphConfig:
    name: str
    n_nodes: int
    n_edges: int
    n_rel: int
    zipf_s: float
    zipf_k0: float
    n_base: int
    budget: int
    key: int = 0            # 0 = out-degree, 1 = out-neighbour h-index
    theta: int = 2**31 - 1  # key filter threshold (INT32_MAX = none)
    rel_split: Optional[Sequence[float]] = None
    hub_frac: float = 0.01
    seed: int = 0


@dataclass(frozen=True)
class ModelConfig:
    d: int
    n_layers: int
    dtype: str = "f32"      # "f32" or "bf16" feature storage
    seed: int = 0
    bias_range: float = 0.0
    lambda_n: float = 2e-4
    lambda_cca: float = 0.1
    eps: float = 1e-5
    ddof: int = 0
    weighted_align: bool = False
    kind: str = "mean"      # "mean" (relation-typed mean aggregation) or "hgt" (attention)
    heads: int = 4          # attention heads (kind == "hgt")
    objective: str = "synthetic"  # "synthetic" (seeded upstream gradient) or "bce" (head, BCE, Adam)
    lr: float = 1e-3
    weight_decay: float = 1e-5
    snapshots: int = 1      # T monthly snapshots of the subgraph (> 1: the temporal module runs between them)
    window: int = 3         # temporal window w: previous states each snapshot attends over
    parts: int = 1          # K > 1: K subgraphs of a random K-way partition, MeanAgg and home-copy alignment


@dataclass(frozen=True)
class Workload:
    graph: GraphConfig
    model: ModelConfig
    desc: str = ""


WORKLOADS = {
    "tiny": Workload(
        GraphConfig("tiny", 10_000, 100_000, 3, 1.1, 0.0, 9_500, 500, seed=0),
        ModelConfig(64, 2, seed=0),
        "10k nodes, 100k edges, 3 relations, Zipf(1.1), d=64 fp32, L=2, overlap 500"),
    "medium": Workload(
        GraphConfig("medium", 1_000_000, 20_000_000, 4, 1.2, 0.0, 900_000, 100_000, seed=2),
        ModelConfig(128, 2, seed=2),
        "1M nodes, 20M edges, 4 relations, Zipf(1.2), d=128 fp32, L=2, overlap budget 100k"),
    "large": Workload(
        GraphConfig("large", 10_000_000, 200_000_000, 5, 1.3, 634.0, 9_200_000, 800_000, seed=3),
        ModelConfig(128, 2, seed=3),
        "10M nodes, 200M edges, 5 relations, Zipf(1.3) k0=634 (max degree ~1e5), d=128 fp32, L=2, overlap budget 800k"),
    "large_bf16": Workload(
        GraphConfig("large", 10_000_000, 200_000_000, 5, 1.3, 634.0, 9_200_000, 800_000, seed=3),
        ModelConfig(256, 3, dtype="bf16", seed=4),
        "the 10M/200M graph with bf16 features at d=256, fp32 accumulation, L=3"),
    "large_full": Workload(
        GraphConfig("large", 10_000_000, 200_000_000, 5, 1.3, 634.0, 9_200_000, 800_000, seed=3),
        ModelConfig(128, 2, seed=3, objective="bce"),
        "the 10M/200M graph, mean layers d=128 fp32, L=2, with the prediction head, masked BCE and Adam"),
    "tiny_full": Workload(
        GraphConfig("tiny", 10_000, 100_000, 3, 1.1, 0.0, 9_500, 500, seed=0),
        ModelConfig(64, 2, seed=0, objective="bce"),
        "10k nodes, 100k edges, mean layers d=64, with the prediction head, masked BCE and Adam"),
    "large_hgt": Workload(
        GraphConfig("large", 10_000_000, 200_000_000, 5, 1.3, 634.0, 9_200_000, 800_000, seed=3),
        ModelConfig(64, 2, seed=3, kind="hgt", heads=4),
        "the 10M/200M graph with attention layers (4 heads) at d=64 fp32, L=2"),
    "tiny_hgt": Workload(
        GraphConfig("tiny", 10_000, 100_000, 3, 1.1, 0.0, 9_500, 500, seed=0),
        ModelConfig(64, 2, seed=0, kind="hgt", heads=4),
        "10k nodes, 100k edges, 3 relations, attention layers (4 heads), d=64 fp32, L=2"),
    "large_dyn": Workload(
        GraphConfig("large", 10_000_000, 200_000_000, 5, 1.3, 634.0, 9_200_000, 800_000, seed=3),
        ModelConfig(64, 2, seed=3, kind="hgt", heads=4, objective="bce", snapshots=4, window=3),
        "the 10M/200M graph over 4 monthly snapshots: attention layers (4 heads) at d=64 fp32, L=2, the temporal "
        "module with w=3, the prediction head, masked BCE and Adam"),
    "tiny_dyn": Workload(
        GraphConfig("tiny", 10_000, 100_000, 3, 1.1, 0.0, 9_500, 500, seed=0),
        ModelConfig(64, 2, seed=0, kind="hgt", heads=4, objective="bce", snapshots=4, window=3),
        "10k nodes, 100k edges over 4 monthly snapshots, attention layers, temporal module w=3, head, BCE, Adam"),
    "large_kway": Workload(
        GraphConfig("large", 10_000_000, 200_000_000, 5, 1.3, 634.0, 9_200_000, 800_000, seed=3),
        ModelConfig(128, 2, seed=3, objective="bce", parts=4),
        "the 10M/200M graph split by a random 4-way partition: 4 overlapping subgraphs (overlap budget 800k each), "
        "mean layers d=128 fp32, L=2, MeanAgg, head and masked BCE on the average, alignment of each subgraph's "
        "overlap rows to their home copies, summed weight gradients and Adam"),
    "tiny_kway": Workload(
        GraphConfig("tiny", 10_000, 100_000, 3, 1.1, 0.0, 9_500, 500, seed=0),
        ModelConfig(64, 2, seed=0, objective="bce", parts=4),
        "10k nodes, 100k edges split 4 ways: 4 overlapping subgraphs, mean layers d=64, MeanAgg, head, BCE, "
        "home-copy alignment, Adam"),
    "skew": Workload(
        GraphConfig("skew", 5_000_000, 150_000_000, 8, 1.6, 6339.0, 4_250_000, 750_000,
                    theta=3, rel_split=SKEW_SPLIT, seed=5),
        ModelConfig(64, 2, seed=5, weighted_align=True),
        "5M nodes, 150M edges, 8 relations split 50/20/10/5/5/5/3/2%, Zipf(1.6) k0=6339, degree<=3 overlap, d=64 fp32, L=2"),
}


def random_partition(n: int, k_parts: int, seed: int) -> np.ndarray:
    """Partition block of every node, uniform over [0, k_parts) and
    independent per node (a random hash partition), int32 [n]."""
    return _rng(seed, 7).integers(0, k_parts, size=n, dtype=np.int32)


def scaled(graph: GraphConfig, factor: float, name: str | None = None) -> GraphConfig:
    """The same recipe at a fraction of the node and edge counts."""
    n = max(16, int(round(graph.n_nodes * factor)))
    return replace(graph, name=name or f"{graph.name}@{factor:g}", n_nodes=n,
                   n_edges=max(16, int(round(graph.n_edges * factor))),
                   n_base=int(round(graph.n_base * factor)),
                   budget=max(1, int(round(graph.budget * factor))),
                   zipf_k0=graph.zipf_k0 * factor)


@dataclass
class Graph:
    cfg: GraphConfig
    src: np.ndarray      # int32 [E]
    dst: np.ndarray      # int32 [E]
    rel: np.ndarray      # uint8 [E]
    ntype: np.ndarray    # uint8 [N]
    part: np.ndarray     # int32 [N]
    k: int = 0

    @property
    def n_nodes(self) -> int:
        return int(self.ntype.shape[0])

    @property
    def n_edges(self) -> int:
        return int(self.src.shape[0])

    @property
    def n_ntype(self) -> int:
        return 2


def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream])))


def edge_weights(seed: int, n_edges: int) -> np.ndarray:
    """Positive per-edge message weights w_ij, float32, uniform in [0.1, 2)."""
    return _rng(seed, 31).uniform(0.1, 2.0, n_edges).astype(np.float32)


def make_graph(cfg: GraphConfig) -> Graph:
    """Draw the typed edge list of one configuration (deterministic in cfg)."""
    n, e = cfg.n_nodes, cfg.n_edges
    rng = _rng(cfg.seed, 1)
    ranks = np.arange(1, n + 1, dtype=np.float64)
    p = (ranks + cfg.zipf_k0) ** (-cfg.zipf_s)
    p /= p.sum()
    counts = rng.multinomial(e, p)
    node_of_rank = rng.permutation(n).astype(np.int32)
    src = np.repeat(node_of_rank, counts)
    rng.shuffle(src)
    dst = rng.integers(0, n, size=e, dtype=np.int32)
    if cfg.rel_split is None:
        rel = rng.integers(0, cfg.n_rel, size=e, dtype=np.uint8)
    else:
        q = np.asarray(cfg.rel_split, dtype=np.float64)
        q = q / q.sum()
        rel = rng.choice(cfg.n_rel, size=e, p=q).astype(np.uint8)
    ntype = np.zeros(n, dtype=np.uint8)
    n_hub = int(round(cfg.hub_frac * n))
    ntype[node_of_rank[:n_hub]] = 1
    part = (np.arange(n) >= cfg.n_base).astype(np.int32)
    return Graph(cfg, src.astype(np.int32, copy=False), dst, rel, ntype, part, 0)


def _normal_f32(seed: int, stream: int, shape, chunks: int = 16) -> np.ndarray:
    """N(0,1) float32 array, filled in fixed chunks (thread-count independent)."""
    out = np.empty(int(np.prod(shape)), dtype=np.float32)
    total = out.shape[0]
    if total == 0:
        return out.reshape(shape)
    bounds = np.linspace(0, total, chunks + 1).astype(np.int64)
    seqs = np.random.SeedSequence([seed, stream]).spawn(chunks)

    def fill(i):
        g = np.random.Generator(np.random.PCG64(seqs[i]))
        g.standard_normal(out=out[bounds[i]:bounds[i + 1]], dtype=np.float32)

    workers = min(chunks, max(1, (os.cpu_count() or 1)))
    if total < (1 << 22) or workers == 1:
        for i in range(chunks):
            fill(i)
    else:
        with _cf.ThreadPoolExecutor(workers) as ex:
            list(ex.map(fill, range(chunks)))
    return out.reshape(shape)


def features(seed: int, n_rows: int, d: int) -> np.ndarray:
    """Input node features X ~ N(0,1), float32 [n_rows, d]."""
    return _normal_f32(seed, 11, (n_rows, d))


def reference_embeddings(seed: int, m: int, d: int) -> np.ndarray:
    """Second view of the overlap nodes, N(0,1) float32 [m, d]."""
    return _normal_f32(seed, 12, (m, d))


def upstream_grad(seed: int, n_rows: int, d: int) -> np.ndarray:
    """Gradient arriving at the last layer's output, N(0,1) float32."""
    return _normal_f32(seed, 13, (n_rows, d))


def context_states(seed: int, w: int, n_rows: int, d: int) -> list:
    """w earlier states of every node, oldest first, N(0, 0.5^2) float32
    [n_rows, d] each (a GRU's states lie mostly inside (-1, 1))."""
    out = []
    for k in range(w):
        x = _normal_f32(seed, 20 + k, (n_rows, d))
        x *= np.float32(0.5)
        out.append(x)
    return out


@dataclass
class LayerWeights:
    w_rel: np.ndarray   # float32 [R, d, d]   (row-vector convention: y = x @ W)
    w_self: np.ndarray  # float32 [T, d, d]
    bias: np.ndarray    # float32 [T, d]


def layer_weights(seed: int, layer: int, n_rel: int, n_ntype: int, d: int,
                  bias_range: float = 0.0) -> LayerWeights:
    rng = _rng(seed, 100 + layer)
    a = np.sqrt(6.0 / (2 * d))
    w_rel = rng.uniform(-a, a, size=(n_rel, d, d)).astype(np.float32)
    w_self = rng.uniform(-a, a, size=(n_ntype, d, d)).astype(np.float32)
    if bias_range > 0:
        bias = rng.uniform(-bias_range, bias_range, size=(n_ntype, d)).astype(np.float32)
    else:
        bias = np.zeros((n_ntype, d), dtype=np.float32)
    return LayerWeights(w_rel, w_self, bias)


def hgt_weights(seed: int, layer: int, n_rel: int, n_ntype: int, d: int, heads: int,
                bias_range: float = 0.0, mu_range=(0.5, 1.5)) -> dict:
    """Attention-layer weights: Xavier-uniform d x d projections and per-head
    dk x dk relation matrices, biases U(+-bias_range), mu U(mu_range); float32."""
    rng = _rng(seed, 200 + layer)
    dk = d // heads
    a, ak = np.sqrt(6.0 / (2 * d)), np.sqrt(6.0 / (2 * dk))
    out = {}
    for name in ("W_K", "W_Q", "W_V", "W_agg"):
        out[name] = rng.uniform(-a, a, size=(n_ntype, d, d)).astype(np.float32)
    for name in ("W_att", "W_msg"):
        out[name] = rng.uniform(-ak, ak, size=(n_rel, heads, dk, dk)).astype(np.float32)
    out["mu"] = rng.uniform(mu_range[0], mu_range[1], size=(n_ntype, n_rel, n_ntype)).astype(np.float32)
    for name in ("b_K", "b_Q", "b_V", "b_agg"):
        if bias_range > 0:
            out[name] = rng.uniform(-bias_range, bias_range, size=(n_ntype, d)).astype(np.float32)
        else:
            out[name] = np.zeros((n_ntype, d), dtype=np.float32)
    return out


def labels(seed: int, ntype: np.ndarray, label_rate: float = 0.117, positive_rate: float = 0.1) -> np.ndarray:
    """int8 labels: users (type 0) labelled with probability label_rate, each
    labelled one positive with probability positive_rate; -1 = unlabelled
    (the paper's dataset leaves 88.3% of users unlabelled)."""
    rng = _rng(seed, 300)
    n = ntype.shape[0]
    lab = rng.random(n) < label_rate
    pos = rng.random(n) < positive_rate
    out = np.where(lab & (ntype == 0), pos.astype(np.int8), np.int8(-1)).astype(np.int8)
    return out


def head_weights(seed: int, d: int) -> dict:
    """Prediction head: W1 [d, d], b1 [d], W2 [d, 1], b2 [1], Xavier-uniform and zero biases."""
    rng = _rng(seed, 301)
    a1, a2 = np.sqrt(6.0 / (2 * d)), np.sqrt(6.0 / (d + 1))
    return {"W1": rng.uniform(-a1, a1, size=(d, d)).astype(np.float32),
            "b1": np.zeros(d, dtype=np.float32),
            "W2": rng.uniform(-a2, a2, size=(d, 1)).astype(np.float32),
            "b2": np.zeros(1, dtype=np.float32)}


def temporal_weights(seed: int, d: int, bias_range: float = 0.1) -> dict:
    """Temporal-module weights, float32: Q, Wi, Wh U(+-1/sqrt(d)) (a GRU
    cell's default range), r U(+-1), biases U(+-bias_range) (zeros if 0)."""
    rng = _rng(seed, 400)
    a = 1.0 / np.sqrt(d)
    out = {"Q": rng.uniform(-a, a, size=(d, d)).astype(np.float32),
           "r": rng.uniform(-1.0, 1.0, size=d).astype(np.float32),
           "Wi": rng.uniform(-a, a, size=(3, d, d)).astype(np.float32),
           "Wh": rng.uniform(-a, a, size=(3, d, d)).astype(np.float32)}
    for name in ("bi", "bh"):
        if bias_range > 0:
            out[name] = rng.uniform(-bias_range, bias_range, size=(3, d)).astype(np.float32)
        else:
            out[name] = np.zeros((3, d), dtype=np.float32)
    return out


def round_bf16(x: np.ndarray) -> np.ndarray:
    """float32 -> nearest-even bfloat16 value, returned as float32 (storage rounding)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> 16) & 1
    r = ((u + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)).astype(np.uint32)
    nan = np.isnan(x)
    out = r.view(np.float32).copy()
    out[nan] = np.nan
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already bf16-representable."""
    return (np.ascontiguousarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def align_weights(overlap_rel: np.ndarray, graph_rel: np.ndarray, n_rel: int) -> np.ndarray:
    """Per-overlap-node weights omega_b proportional to 1/p(relation of its base edge),
    normalised to mean 1, where p is the relation's share of all edges."""
    share = np.bincount(graph_rel, minlength=n_rel).astype(np.float64)
    share = np.maximum(share / max(1, share.sum()), 1e-12)
    w = 1.0 / share[overlap_rel.astype(np.int64)]
    if w.size:
        w = w / w.mean()
    return w.astype(np.float32)


# Snapshot calendar: T monthly snapshots of 30 days (the paper's temporal
# window of w = 3 covers the past three months).
DAYS_PER_SNAPSHOT = 30


def edge_times(seed: int, n_edges: int, n_snapshots: int = 4, days: int = DAYS_PER_SNAPSHOT) -> np.ndarray:
    """Day index of every edge, uniform over [0, n_snapshots * days), int32."""
    rng = _rng(seed, 500)
    return rng.integers(0, n_snapshots * days, size=n_edges, dtype=np.int32)


def snapshot_cuts(n_snapshots: int = 4, days: int = DAYS_PER_SNAPSHOT) -> list:
    """Last day of each snapshot: snapshot t holds the edges with day <= cut[t]."""
    return [(t + 1) * days - 1 for t in range(n_snapshots)]
