"""Overlapping-subgraph construction, written out from its definition.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Follows the Methodology section "Risk-Aware Subgraph Construction" and the
construction loop of Algorithm 1:

1. node keys: out-degree, or the h-index of the out-neighbour multiset
   ("h-index filter" paragraph; the bibliometric h-index: the largest h such
   that at least h neighbours have degree >= h);
2. candidate set C_k: nodes outside the base set V_k joined to V_k by an edge
   in either direction (candidate-set equation);
3. the filter key <= theta, then TopM: ascending (key, SplitMix64 tie-break,
   global id), first min(M, |C'_k|) nodes (the budgeted sampling step);
4. the overlapping node set V_k u C_{k,M} (union equation) and its induced
   subgraph G[V~_k], relabelled in (node type, global id) order;
5. per-relation CSR (destination-major) and CSC (source-major) of the induced
   subgraph, entries of a CSR row in ascending original edge index, entries
   of a CSC row in ascending (destination, original edge index), and the CSC
   scale 1/deg_r(destination) as a float32 quotient (w_ij/deg_r(destination)
   for weighted edges, the message weight over the in-edge count, with the
   weight of every CSR entry);
6. optionally one snapshot of it: only the induced edges whose timestamp is at
   most the cut (the node set, fixed by steps 1-4 on every edge, is shared by
   all snapshots).

Readings where the paper is silent are the ones listed in the design notes:
either edge direction for adjacency, out-neighbour h-index with degrees over
all relations, ascending key (long tail first), seeded hash tie-break,
induced subgraph including overlap-overlap edges.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import splitmix

KEY_OUTDEG = 0
KEY_HINDEX = 1
THETA_NONE = 2**31 - 1


def out_degree(n: int, src: np.ndarray) -> np.ndarray:
    """outdeg(v) = number of edges whose source is v (all relations)."""
    return np.bincount(np.asarray(src, dtype=np.int64), minlength=n).astype(np.int64)


def out_hindex(n: int, src: np.ndarray, dst: np.ndarray) -> np.ndarray:
    """h(v) = max h such that at least h out-edges of v reach nodes of
    out-degree >= h (the out-neighbour multiset, duplicates counted)."""
    src = np.asarray(src, dtype=np.int64)
    vals = out_degree(n, src)[np.asarray(dst, dtype=np.int64)]
    # group by source, values descending inside a group: one sort of the key
    # (source, vmax - value), both parts below 2^32
    vmax = np.int64(src.shape[0])
    key = np.sort((src << 32) | (vmax - vals))
    s, a = key >> 32, vmax - (key & np.int64(0xFFFFFFFF))
    start = np.flatnonzero(np.r_[True, s[1:] != s[:-1]]) if s.size else np.zeros(0, np.int64)
    rank = np.arange(s.shape[0]) - np.repeat(start, np.diff(np.r_[start, s.shape[0]])) + 1
    # a is descending inside a group, so "a_i >= i" (1-based i) holds on a
    # prefix whose length is the h-index.
    return np.bincount(s, weights=(a >= rank), minlength=n).astype(np.int64)


def node_keys(n: int, src, dst, key: int) -> np.ndarray:
    if key == KEY_OUTDEG:
        return out_degree(n, src)
    if key == KEY_HINDEX:
        return out_hindex(n, src, dst)
    raise ValueError(f"unknown key {key}")


def candidates(part: np.ndarray, k: int, src, dst) -> np.ndarray:
    """Boolean [N]: v not in V_k and some edge joins v to a node of V_k."""
    in_base = np.asarray(part) == k
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    cand = np.zeros(in_base.shape[0], dtype=bool)
    cand[src[in_base[dst]]] = True
    cand[dst[in_base[src]]] = True
    return cand & ~in_base


def base_edge(part: np.ndarray, k: int, src, dst) -> np.ndarray:
    """For every node outside V_k: the smallest edge index joining it to V_k
    (either direction), or E if there is none."""
    in_base = np.asarray(part) == k
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    e = src.shape[0]
    first = np.full(in_base.shape[0], e, dtype=np.int64)
    idx = np.arange(e, dtype=np.int64)
    m = in_base[dst] & ~in_base[src]
    np.minimum.at(first, src[m], idx[m])
    m = in_base[src] & ~in_base[dst]
    np.minimum.at(first, dst[m], idx[m])
    return first


def top_m(cand: np.ndarray, keys: np.ndarray, theta: int, budget: int, seed: int) -> np.ndarray:
    """Global ids of C_{k,M}: the candidates with key <= theta, ordered by
    (key, tie-break hash, gid) ascending, first min(M, |C'|). Returned ascending."""
    gid = np.nonzero(cand & (keys <= theta))[0]
    h = splitmix.tiebreak(seed, gid)
    order = np.lexsort((gid, h, keys[gid]))
    take = gid[order[: max(0, min(int(budget), gid.shape[0]))]]
    return np.sort(take)


@dataclass
class Subgraph:
    n_sub: int
    e_sub: int
    n_rel: int
    n_ntype: int
    local2global: np.ndarray   # int32 [N_s]
    global2local: np.ndarray   # int32 [N]  (-1 = absent)
    type_off: np.ndarray       # int32 [T+1]
    overlap: np.ndarray        # int32 [M_sel] local ids, ascending
    overlap_home: np.ndarray   # int32 [M_sel] home partition of each overlap node
    overlap_rel: np.ndarray    # uint8 [M_sel] relation of the node's base edge
    src_l: np.ndarray          # int32 [E_s] subgraph edges in original order
    dst_l: np.ndarray
    rel_l: np.ndarray          # uint8 [E_s]
    eid: np.ndarray            # int32 [E_s] original edge index
    csr_ptr: np.ndarray        # int32 [N_s*R+1], row (dst, r) = dst*R + r
    csr_col: np.ndarray        # int32 [E_s] source local id
    csr_eid: np.ndarray        # int32 [E_s]
    csc_ptr: np.ndarray        # int32 [N_s*R+1], row (src, r) = src*R + r
    csc_row: np.ndarray        # int32 [E_s] destination local id
    csc_scale: np.ndarray      # float32 [E_s] 1 / deg_r(destination)
    n_active: np.ndarray       # int64 [R] sources with at least one out-edge of relation r
    ntype_l: np.ndarray        # uint8 [N_s] node type by local id
    w_l: np.ndarray = None     # float32 [E_s] edge weights in original order (weighted graphs)
    csr_w: np.ndarray = None   # float32 [E_s] weight of each CSR entry (weighted graphs)


def build(src, dst, rel, ntype, part, k: int, n_rel: int, n_ntype: int,
          budget: int, key: int = KEY_OUTDEG, theta: int = THETA_NONE,
          seed: int = 0, edge_ts=None, t_cut=None, edge_w=None) -> Subgraph:
    """The overlapping subgraph of partition k.  With edge_ts, one snapshot
    of it: the node set (and everything that decides it) uses every edge, and
    only the induced edges with edge_ts <= t_cut are kept (snapshots are
    taken of the augmented subgraph by filtering its edges on their
    timestamps, end of "Risk-Aware Subgraph Construction")."""
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    rel = np.asarray(rel, dtype=np.int64)
    ntype = np.asarray(ntype, dtype=np.int64)
    part = np.asarray(part, dtype=np.int64)
    n = ntype.shape[0]
    r_count = int(n_rel)

    keys = node_keys(n, src, dst, key)
    cand = candidates(part, k, src, dst)
    sel = top_m(cand, keys, theta, budget, seed)
    first = base_edge(part, k, src, dst)

    member = part == k
    member[sel] = True
    ids = np.nonzero(member)[0]
    local2global = ids[np.lexsort((ids, ntype[ids]))]
    n_sub = local2global.shape[0]
    global2local = np.full(n, -1, dtype=np.int64)
    global2local[local2global] = np.arange(n_sub)
    ntype_l = ntype[local2global]
    type_off = np.concatenate([[0], np.cumsum(np.bincount(ntype_l, minlength=n_ntype))])

    keep = member[src] & member[dst]
    if edge_ts is not None:
        keep &= np.asarray(edge_ts, dtype=np.int64) <= int(t_cut)
    eid = np.nonzero(keep)[0]
    src_l = global2local[src[eid]]
    dst_l = global2local[dst[eid]]
    rel_l = rel[eid]

    nrows = n_sub * r_count
    key_csr = dst_l * r_count + rel_l
    p = np.argsort(key_csr, kind="stable")
    csr_ptr = np.concatenate([[0], np.cumsum(np.bincount(key_csr, minlength=nrows))])
    csr_col = src_l[p]
    csr_eid = eid[p]

    key_csc = src_l * r_count + rel_l
    q = np.lexsort((eid, dst_l, key_csc))   # row, then destination, then edge index
    csc_counts = np.bincount(key_csc, minlength=nrows)
    csc_ptr = np.concatenate([[0], np.cumsum(csc_counts)])
    csc_row = dst_l[q]
    dst_row = csc_row * r_count + rel_l[q]
    deg = (csr_ptr[dst_row + 1] - csr_ptr[dst_row]).astype(np.float32)
    w_l = csr_w = None
    if edge_w is None:
        csc_scale = (np.float32(1.0) / deg).astype(np.float32)
    else:
        w_l = np.asarray(edge_w, dtype=np.float32)[eid]
        csr_w = w_l[p]
        csc_scale = (w_l[q] / deg).astype(np.float32)   # float32 quotient
    n_active = (csc_counts.reshape(n_sub, r_count) > 0).sum(axis=0).astype(np.int64) \
        if n_sub else np.zeros(r_count, dtype=np.int64)

    overlap = np.sort(global2local[sel])
    og = local2global[overlap]
    return Subgraph(
        n_sub=int(n_sub), e_sub=int(eid.shape[0]), n_rel=r_count, n_ntype=int(n_ntype),
        local2global=local2global.astype(np.int32),
        global2local=global2local.astype(np.int32),
        type_off=type_off.astype(np.int32),
        overlap=overlap.astype(np.int32),
        overlap_home=part[og].astype(np.int32),
        overlap_rel=rel[first[og]].astype(np.uint8) if og.size else np.zeros(0, np.uint8),
        src_l=src_l.astype(np.int32), dst_l=dst_l.astype(np.int32),
        rel_l=rel_l.astype(np.uint8), eid=eid.astype(np.int32),
        csr_ptr=csr_ptr.astype(np.int32), csr_col=csr_col.astype(np.int32),
        csr_eid=csr_eid.astype(np.int32),
        csc_ptr=csc_ptr.astype(np.int32), csc_row=csc_row.astype(np.int32),
        csc_scale=csc_scale, n_active=n_active, ntype_l=ntype_l.astype(np.uint8), w_l=w_l, csr_w=csr_w)
