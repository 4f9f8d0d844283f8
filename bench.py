"""Benchmark of one training step of the hot path on one MI355X.

A step = subgraph build (selection, relabel, CSR/CSC, plan), L layers
forward, the CCA alignment loss + gradient on the overlap rows, L layers
backward -- every step of it in libhg.so's HIP kernels, inputs resident in
HBM before the timed region.

With a K-subgraph workload (large_kway, tiny_kway) a step covers the K
workers one after another: K subgraph builds, L layers forward per
subgraph, MeanAgg, the head with masked BCE on the average, each
subgraph's alignment with its overlap nodes' home copies, L layers backward
per subgraph (weight gradients summed) and one Adam update; the edge count
is the sum of the K subgraphs' edges.

With a multi-snapshot workload (large_dyn, tiny_dyn) a step covers every
snapshot: T snapshot builds, per snapshot L attention layers and the
temporal module, the head with masked BCE and the alignment on the last
state, the backward through every snapshot and one Adam update; the edge
count is then the sum of the snapshots' edges.

Prints one JSON line: value = L * E_sub / t_step in GTEPS (edges x layers
per second, forward + backward of every layer, build and alignment included),
plus the roofline of the dominant kernel (algorithmic bytes per launch /
average launch time from HIP events recorded around each launch on its own
stream) and the oracle timed on the host cores on a bounded sample.

Beside the value: the same steps timed again on the subgraphs already built
(construction done once, before training; `ms_per_step_no_rebuild`), and for
the build and alignment kernel families their time per step and algorithmic
rate (`families`).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3


# kernel families by timing-log name: the subgraph build (keys, selection,
# relabel, CSR/CSC, plan) and the alignment loss + gradient
FAMILIES = {"build": ("build_", "keys_", "radix_", "scan_", "partition_", "fill"),
            "align": ("align_",)}
# algorithmic bytes of the build per input edge: edge compaction plus two
# stable sorts (lower end of the 80-130 B range of the design estimate)
BUILD_BYTES_PER_EDGE = 80

SPARSE_KERNELS = {"mean": ("spmm_fwd", "spmm_bwd"),
                  "hgt": ("hgt_attn_fwd", "hgt_attn_bwd_dst", "hgt_attn_bwd_src")}


def algorithmic_cost(kind: str, info: dict):
    """(bytes, flops) per launch, counted without cache reuse.  E = subgraph
    edges, N = subgraph nodes, A = active (source, relation) rows, s = bytes
    per feature element, d = width, R = relations, T = node types, S = heads."""
    E, N, A, d, s, R = info["E"], info["N"], info["A"], info["d"], info["s"], info["R"]
    T, S = info.get("T", 2), info.get("S", 1)
    if kind == "hgt_attn_fwd":
        # per edge: Kt and Vt rows of the source plus its column id; per node:
        # Q read, h~ written, S log-sum-exps, R+1 row pointers
        return E * (2 * d * s + 4) + N * (2 * d * s + 4 * S + 4 * (R + 1)), 4.0 * E * d
    if kind == "hgt_attn_bwd_dst":
        # per edge: Kt and Vt rows plus the column id; per node: Q, dh~ and h~
        # read, dQ written, S log-sum-exps read and S sums written, R+1 row
        # pointers, R*T partial sums of the mu gradient
        return E * (2 * d * s + 4) + N * (4 * d * s + 8 * S + 4 * (R + 1) + 4 * R * T), 6.0 * E * d
    if kind == "hgt_attn_bwd_src":
        # per edge: Q and dh~ rows of the destination, its id and its S
        # log-sum-exps and S sums; per work item: Kt, Vt read, dKt, dVt
        # written, 16-byte item
        return E * (2 * d * s + 4 + 8 * S) + A * (4 * d * s + 16), 6.0 * E * d
    if kind == "spmm_fwd":
        # per edge: one gathered row of Y plus its 4-byte column id; per node:
        # R+1 row pointers, Y_self and H_in rows read, H_out row and d/8 mask bytes written
        return E * (d * s + 4) + N * (4 * (R + 1) + 3 * d * s + d / 8), 2.0 * E * d
    if kind == "spmm_bwd":
        # per edge: one gathered dZ row, destination id and scale; per work
        # item 16 bytes; per active row one dY row written (float32 for every
        # feature type: dY feeds the float32 GEMMs)
        return E * (d * s + 8) + A * (d * 4 + 16), 2.0 * E * d
    raise KeyError(kind)


def family_rates(kern: dict, steps: int, n_edges: int, builds: int, align_rows: int, d: int, s: int):
    """Per-step time and algorithmic rate of the build and alignment families.
    Build: BUILD_BYTES_PER_EDGE per input edge per build.  Alignment: about
    6*M*d*s bytes (gather both views, write dX, read them again for the
    gradient) and 6*M*d*d flop (two Grams and the gradient product)."""
    out = {}
    for fam, prefixes in FAMILIES.items():
        ms = sum(v[1] for k, v in kern.items() if k.startswith(prefixes)) / steps
        if fam == "build":
            nbytes, flops = BUILD_BYTES_PER_EDGE * n_edges * builds, 0.0
        else:
            nbytes, flops = 6.0 * align_rows * d * s, 6.0 * align_rows * d * d
        ent = {"ms_per_step": round(ms, 3), "algorithmic_bytes_per_step": int(nbytes)}
        if ms > 0:
            gbs = nbytes / (ms * 1e-3) / 1e9
            ent.update({"achieved_GBs": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)})
            if flops:
                tf = flops / (ms * 1e-3) / 1e12
                ent.update({"algorithmic_flop_per_step": int(flops), "achieved_TFLOPs": round(tf, 2),
                            "fp32_mfma_frac": round(tf / FP32_MFMA_PEAK_TFLOPS, 4)})
            t_bound = max(nbytes / (HBM_PEAK_GBS * 1e9), flops / (FP32_MFMA_PEAK_TFLOPS * 1e12)) * 1e3
            ent.update({"bound_ms": round(t_bound, 3), "frac_of_bound": round(t_bound / ms, 4)})
        out[fam] = ent
    return out


def kernel_source_sha(path: str, kernel: str) -> str:
    """SHA-256 (16 hex digits) of a kernel's own source text: from the
    template line before `kernel(` to the closing brace at column 0."""
    import hashlib
    lines = open(path).read().split("\n")
    start = next(i for i, l in enumerate(lines) if f" {kernel}(" in l and "__global__" in l)
    while start > 0 and not lines[start].startswith("template"):
        start -= 1
    end = next(i for i in range(start, len(lines)) if lines[i] == "}")
    return hashlib.sha256("\n".join(lines[start:end + 1]).encode()).hexdigest()[:16]


def counted_traffic(kernel: str, config: str):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary of this workload, or None if the kernel's source has changed since."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{config}_counters.md")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith((" ", "|", "#")):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    src = os.path.join(ROOT, vals.get("source", ""))
    if not os.path.isfile(src) or "traffic_bytes_per_launch" not in vals or "kernel_function" not in vals:
        return None
    if kernel_source_sha(src, vals["kernel_function"]) != vals.get("kernel_source_sha256_16"):
        return None
    return int(vals["traffic_bytes_per_launch"])


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="large",
                    help="tiny | medium | large | large_bf16 | skew | large_hgt | tiny_hgt | large_full | tiny_full | "
                         "large_dyn | tiny_dyn | large_kway | tiny_kway")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=float, default=None,
                    help="fraction of the workload's node/edge counts the oracle runs on "
                         "(default 0.01, 0.001 for attention layers, 0.0005 for snapshot sequences: "
                         "about 10-30 s of CPU work)")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the random-row gather ceiling measurement")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_02168_amd import api, runner, synth

    wl = synth.WORKLOADS[args.config]
    t0 = time.time()
    g = synth.make_graph(wl.graph)
    print(f"[bench] graph {wl.graph.name}: N={g.n_nodes} E={g.n_edges} generated in {time.time() - t0:.1f}s",
          file=sys.stderr, flush=True)
    seq = wl.model.snapshots > 1
    kway = wl.model.parts > 1
    if seq:
        inp = runner.make_seq_inputs(wl, g, device="cuda")
        subs = inp.subs
        step = lambda rebuild=True: runner.run_seq_step(inp, rebuild=rebuild)
    elif kway:
        inp = runner.make_kway_inputs(wl, g, device="cuda")
        subs = inp.subs
        step = lambda rebuild=True: runner.run_kway_step(inp, rebuild=rebuild)
    else:
        inp = runner.make_inputs(wl, g, device="cuda")
        subs = [inp.sub]
        step = lambda rebuild=True: runner.run_step(inp, rebuild=rebuild)
    sub = subs[-1]
    print(f"[bench] subgraph N_s={sub.n_sub} E_s={[s.e_sub for s in subs]} M_sel={sub.m_sel}", file=sys.stderr,
          flush=True)
    L = wl.model.n_layers
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    api.hg_timing_collect()
    api.hg_timing_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    api.hg_timing_enable(False)
    kern = api.hg_timing_collect()
    ms = (t1 - t0) * 1e3 / args.steps
    # the same steps on the subgraphs already built (construction done once,
    # before training): reported beside the step, never as its value
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(args.steps):
        step(rebuild=False)
    torch.cuda.synchronize()
    ms_nb = (time.perf_counter() - t2) * 1e3 / args.steps
    e_pass = sum(s.e_sub for s in subs)
    edges = L * e_pass
    value = edges / (ms * 1e-3) / 1e9

    infos = [dict(E=s.e_sub, N=s.n_sub, A=sum(s.n_active()), d=wl.model.d, s=2 if wl.model.dtype == "bf16" else 4,
                  R=s.n_rel, T=s.n_ntype, S=wl.model.heads) for s in subs]
    info = infos[-1]
    spmm = {k: v for k, v in kern.items() if k in SPARSE_KERNELS[wl.model.kind]}
    dom = max(spmm, key=lambda k: spmm[k][1])
    launches, total_ms = spmm[dom]
    avg_ms = total_ms / launches
    # launches of the dominant kernel per step and layer: one per snapshot
    # (every snapshot keeps its activations for the backward)
    per_snap = [1 for _ in subs]
    step_bytes = L * sum(n * algorithmic_cost(dom, inf)[0] for n, inf in zip(per_snap, infos))
    assert launches == args.steps * L * sum(per_snap), (dom, launches)
    nbytes = step_bytes / (L * sum(per_snap))
    achieved = nbytes / (avg_ms * 1e-3) / 1e9
    traffic = counted_traffic(dom, args.config)
    roofline = {"kernel": dom, "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "traffic_unit": "L2-miss bytes per launch (rocprofv3 TCC_EA0 read requests x 128 B + write requests by size; "
                                "includes Infinity Cache hits)",
                "avg_launch_ms": round(avg_ms, 4), "algorithmic_bytes_per_launch": int(nbytes)}
    if not args.no_ceiling:
        groups = info["E"] / max(info["A"] if dom in ("spmm_bwd", "hgt_attn_bwd_src") else info["N"], 1)
        roofline["ceiling"] = gather_ceiling(info["N"], info["E"], info["d"] * info["s"], groups, achieved)
    layer_ms = sum(v[1] for k, v in kern.items()
                   if k.startswith(("spmm", "gemm_fwd", "gemm_bwd", "relu_grad", "splitk", "hgt_"))) / args.steps
    breakdown = {k: round(v[1] / args.steps, 3) for k, v in sorted(kern.items(), key=lambda kv: -kv[1][1])}
    align_rows = sum(x.m_sel for x in subs) if kway else subs[0].m_sel
    families = family_rates(kern, args.steps, g.n_edges, len(subs), align_rows, info["d"], info["s"])

    cpu = None
    if not args.no_cpu_baseline:
        frac = args.cpu_sample if args.cpu_sample is not None else (
            0.0005 if seq else 0.001 if wl.model.kind == "hgt" else 0.01)
        cpu = (cpu_baseline_sequence(wl, frac) if seq else cpu_baseline_kway(wl, frac) if kway
               else cpu_baseline(wl, frac))

    out = {
        "metric": "GNN layer fwd+bwd edges/sec (GTEPS) + achieved HBM GB/s fraction, 1 GPU",
        "value": round(value, 4), "unit": "GTEPS", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32" if wl.model.dtype == "f32" else "bf16",
        "data": "synthetic",
        "config": {"workload": wl.desc, "name": args.config, "layer": wl.model.kind, "n_nodes": g.n_nodes,
                   "n_edges": g.n_edges, "n_sub": sub.n_sub, "e_sub": sub.e_sub, "m_sel": sub.m_sel,
                   "n_rel": sub.n_rel, "d": wl.model.d, "layers": L,
                   **({"heads": wl.model.heads} if wl.model.kind == "hgt" else {}),
                   **({"snapshots": len(subs), "window": wl.model.window, "e_sub_per_snapshot":
                       [s.e_sub for s in subs]} if seq else {}),
                   **({"parts": len(subs), "n_sub_per_part": [s.n_sub for s in subs],
                       "e_sub_per_part": [s.e_sub for s in subs], "m_sel_per_part": [s.m_sel for s in subs]}
                      if kway else {}),
                   "parallelism": "none (1 GPU)"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "layer_gteps": round(edges / (layer_ms * 1e-3) / 1e9, 4) if layer_ms > 0 else None,
        "ms_per_step_no_rebuild": round(ms_nb, 3),
        "gteps_no_rebuild": round(edges / (ms_nb * 1e-3) / 1e9, 4),
        "families": families,
        "kernel_ms_per_step": breakdown,
    }
    print(json.dumps(out), flush=True)


def gather_ceiling(n_rows, n_idx, row_bytes, group, achieved):
    """What the memory system delivers for the SpMM access pattern at this
    shape: rows of row_bytes fetched through uniform random ids (n_idx of them
    over n_rows rows), summed in groups of `group`, without and with one row
    written per group (csrc/hg_ceiling.hip).  Bytes are counted like the
    kernels' algorithmic bytes: rows + 4-byte ids + written rows."""
    import torch

    from paper_2608_02168_amd import ceiling

    g = int(min(max(round(group), 1), 64))
    dc = row_bytes // 4
    table = torch.randn((n_rows, dc), device="cuda")
    idx = torch.empty(n_idx, dtype=torch.int32, device="cuda")
    ceiling.random_rows(idx, n_rows, 12345)
    out = torch.empty((n_idx // g, dc), device="cuda")
    res = {}
    for write in (False, True):
        ceiling.gather(table, idx, g, out, write)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(3):
            ceiling.gather(table, idx, g, out, write)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 3
        ng = n_idx // g
        nbytes = ng * g * (row_bytes + 4) + (ng * row_bytes if write else 0)
        res["with_writes" if write else "gather_only"] = round(nbytes / (ms * 1e-3) / 1e9, 1)
    del table, idx, out
    torch.cuda.empty_cache()
    return {"pattern": f"uniform random {row_bytes}-byte rows, {n_idx} ids over {n_rows} rows, "
                       f"groups of {g}, one row written per group",
            "gather_only": res["gather_only"], "with_writes": res["with_writes"], "unit": "GB/s",
            "frac": round(achieved / res["gather_only"], 4),
            "frac_with_writes": round(achieved / res["with_writes"], 4)}


def _timed_runs(fn, min_s=10.0):
    """Run fn() until at least min_s seconds of work have been timed (at least
    once); returns (its last result, seconds per run, runs)."""
    runs, total = 0, 0.0
    while True:
        t0 = time.perf_counter()
        out = fn()
        total += time.perf_counter() - t0
        runs += 1
        if total >= min_s:
            return out, total / runs, runs


def cpu_baseline_sequence(wl, frac):
    """The oracle's sequence step (oracle/step.py run_sequence, unchanged) on
    the same recipe at a fraction of the node and edge counts."""
    from threadpoolctl import threadpool_info

    from oracle import step as oracle_step
    from paper_2608_02168_amd import synth

    cfg = synth.scaled(wl.graph, frac)
    g = synth.make_graph(cfg)
    mc = wl.model
    ts = synth.edge_times(cfg.seed, g.n_edges, mc.snapshots)
    cuts = synth.snapshot_cuts(mc.snapshots)
    feats = synth.features(mc.seed, g.n_nodes, mc.d)
    weights = [synth.hgt_weights(mc.seed, li, cfg.n_rel, 2, mc.d, mc.heads, mc.bias_range)
               for li in range(mc.n_layers)]
    out, dt, runs = _timed_runs(lambda: oracle_step.run_sequence(dict(src=g.src, dst=g.dst, rel=g.rel, ntype=g.ntype, part=g.part),
                                   dict(k=g.k, n_rel=cfg.n_rel, n_ntype=2, budget=cfg.budget, key=cfg.key,
                                        theta=cfg.theta, seed=cfg.seed),
                                   ts, cuts, feats, weights, mc.heads, synth.temporal_weights(mc.seed, mc.d),
                                   mc.window, synth.reference_embeddings(mc.seed, max(cfg.budget, 1), mc.d),
                                   synth.head_weights(mc.seed, mc.d), synth.labels(mc.seed, g.ntype),
                                   lambda_n=mc.lambda_n, scale=mc.lambda_cca, eps=mc.eps, ddof=mc.ddof))
    e_pass = sum(s.e_sub for s in out["subs"])
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": round(mc.n_layers * e_pass / dt / 1e9, 6), "unit": "GTEPS", "cores": threads,
            "kind": "oracle",
            "sample": f"same recipe at {frac:g} of the node/edge counts: N={g.n_nodes}, E={g.n_edges}, "
                      f"E_sub per snapshot {[s.e_sub for s in out['subs']]}; one full sequence step ("
                      f"{mc.snapshots} snapshot builds, {mc.n_layers} attention layers and the temporal module "
                      f"per snapshot, head, BCE and alignment, backward through every snapshot) in {dt:.1f}s, mean of {runs} runs; "
                      f"float64; BLAS {threads} threads"}


def cpu_baseline_kway(wl, frac):
    """The oracle's K-worker step (oracle/kway.py run_kway, unchanged) on the
    same recipe at a fraction of the node and edge counts."""
    from threadpoolctl import threadpool_info

    from oracle import kway as oracle_kway
    from paper_2608_02168_amd import synth

    cfg = synth.scaled(wl.graph, frac)
    g = synth.make_graph(cfg)
    mc = wl.model
    part = synth.random_partition(g.n_nodes, mc.parts, mc.seed)
    feats = synth.features(mc.seed, g.n_nodes, mc.d)
    weights = [synth.layer_weights(mc.seed, li, cfg.n_rel, 2, mc.d, mc.bias_range) for li in range(mc.n_layers)]
    out, dt, runs = _timed_runs(lambda: oracle_kway.run_kway(dict(src=g.src, dst=g.dst, rel=g.rel, ntype=g.ntype, part=part), mc.parts,
                               dict(n_rel=cfg.n_rel, n_ntype=2, budget=cfg.budget, key=cfg.key, theta=cfg.theta,
                                    seed=cfg.seed),
                               feats, weights, synth.head_weights(mc.seed, mc.d), synth.labels(mc.seed, g.ntype),
                               lambda_n=mc.lambda_n, scale=mc.lambda_cca, eps=mc.eps, ddof=mc.ddof))
    e_pass = sum(s.e_sub for s in out["subs"])
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": round(mc.n_layers * e_pass / dt / 1e9, 6), "unit": "GTEPS", "cores": threads,
            "kind": "oracle",
            "sample": f"same recipe at {frac:g} of the node/edge counts: N={g.n_nodes}, E={g.n_edges}, "
                      f"E_sub per subgraph {[s.e_sub for s in out['subs']]}; one full K-worker step ("
                      f"{mc.parts} subgraph builds, {mc.n_layers} mean layers fwd+bwd per subgraph, MeanAgg, "
                      f"head, BCE and home-copy alignment) in {dt:.1f}s, mean of {runs} runs; float64; BLAS {threads} threads"}


def cpu_baseline(wl, frac):
    """The oracle (oracle/step.py, unchanged) on the same recipe at a fraction
    of the node and edge counts; reported in the same unit."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import step as oracle_step
    from paper_2608_02168_amd import synth

    cfg = synth.scaled(wl.graph, frac)
    g = synth.make_graph(cfg)
    mc = wl.model
    feats = synth.features(mc.seed, g.n_nodes, mc.d)
    if mc.dtype == "bf16":
        feats = synth.round_bf16(feats)
    if mc.kind == "hgt":
        weights = [synth.hgt_weights(mc.seed, li, cfg.n_rel, 2, mc.d, mc.heads, mc.bias_range)
                   for li in range(mc.n_layers)]
    else:
        weights = [synth.layer_weights(mc.seed, li, cfg.n_rel, 2, mc.d, mc.bias_range) for li in range(mc.n_layers)]
    href = synth.reference_embeddings(mc.seed, max(cfg.budget, 1), mc.d)
    gext = synth.upstream_grad(mc.seed, g.n_nodes, mc.d)
    extra = {}
    if mc.objective == "bce":
        extra = dict(head=synth.head_weights(mc.seed, mc.d), labels_global=synth.labels(mc.seed, g.ntype))
    (sub, *_), dt, runs = _timed_runs(lambda: oracle_step.run(dict(src=g.src, dst=g.dst, rel=g.rel, ntype=g.ntype, part=g.part),
                              dict(k=g.k, n_rel=cfg.n_rel, n_ntype=2, budget=cfg.budget, key=cfg.key,
                                   theta=cfg.theta, seed=cfg.seed),
                              feats, weights, href, gext, lambda_n=mc.lambda_n, scale=mc.lambda_cca,
                              eps=mc.eps, ddof=mc.ddof, heads=mc.heads, **extra))
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": round(mc.n_layers * sub.e_sub / dt / 1e9, 6), "unit": "GTEPS", "cores": threads,
            "kind": "oracle",
            "sample": f"same recipe at {frac:g} of the node/edge counts: N={g.n_nodes}, E={g.n_edges}, "
                      f"E_sub={sub.e_sub}; one full step (build, {mc.n_layers} layers fwd+bwd, alignment"
                      f"{', prediction head and BCE' if mc.objective == 'bce' else ''}) "
                      f"in {dt:.1f}s, mean of {runs} runs; float64; scipy sparse products single-threaded, BLAS {threads} threads"}


if __name__ == "__main__":
    main()
