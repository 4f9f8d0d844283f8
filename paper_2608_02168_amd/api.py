"""ctypes binding of libhg.so with the same entry-point names as include/hg.h.

Argument marshalling only: torch tensors provide device memory and the
current stream; every step of the computation runs in the library's HIP
kernels.  If libhg.so is missing this module raises on first use -- there
is no fallback implementation.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass, field
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libhg.so")

HG_OK = 0
HG_ERR_ARG = -1
HG_ERR_RANGE = -2
HG_ERR_CAPACITY = -3
HG_ERR_HIP = -4
HG_ERR_UNSUPPORTED = -5
HG_KEY_OUTDEG = 0
HG_KEY_HINDEX = 1
HG_KEYDIR_OUT = 0
HG_THETA_NONE = 2**31 - 1
HG_DTYPE_F32 = 0
HG_DTYPE_BF16 = 1
HG_MAX_REL = 255
HG_MAX_NTYPE = 255
HG_MAX_PARTS = 64

EXPORTS = [
    "hg_plan_size", "hg_build_csr_workspace_size", "hg_build_csr", "hg_node_keys_workspace_size", "hg_node_keys",
    "hg_layer_saved_size", "hg_layer_fwd_workspace_size", "hg_layer_bwd_workspace_size",
    "hg_layer_fwd", "hg_layer_bwd", "hg_hgt_saved_size", "hg_hgt_fwd_workspace_size",
    "hg_hgt_bwd_workspace_size", "hg_hgt_fwd", "hg_hgt_bwd", "hg_align_workspace_size", "hg_align_loss_fwd_bwd", "hg_align_noalloc_scratch_size",
    "hg_align_loss_fwd_bwd_noalloc",
    "hg_mlp_bce_workspace_size", "hg_mlp_bce_fwd_bwd", "hg_adam_step",
    "hg_temporal_fwd", "hg_temporal_bwd_workspace_size", "hg_temporal_bwd",
    "hg_mean_agg_fwd", "hg_mean_agg_bwd", "hg_home_gather",
    "hg_status_string", "hg_last_error_detail", "hg_timing_enable", "hg_timing_collect",
]


class HgError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: {status_string(status)} ({detail})")
        self.status = status


class GraphDesc(C.Structure):
    _fields_ = [("n_nodes", C.c_int64), ("n_edges", C.c_int64), ("n_rel", C.c_int32),
                ("n_ntype", C.c_int32), ("src", C.c_void_p), ("dst", C.c_void_p),
                ("rel", C.c_void_p), ("ntype", C.c_void_p), ("part", C.c_void_p),
                ("k", C.c_int32), ("edge_w", C.c_void_p), ("edge_ts", C.c_void_p), ("t_cut", C.c_int32),
                ("reserved", C.c_int32)]


class OverlapDesc(C.Structure):
    _fields_ = [("budget_M", C.c_int64), ("key", C.c_int32), ("key_dir", C.c_int32),
                ("theta", C.c_int32), ("reserved", C.c_int32), ("seed", C.c_uint64), ("node_key", C.c_void_p)]


class SubgraphStruct(C.Structure):
    _fields_ = [("local2global", C.c_void_p), ("global2local", C.c_void_p),
                ("type_off", C.c_void_p), ("overlap", C.c_void_p), ("overlap_home", C.c_void_p),
                ("overlap_rel", C.c_void_p), ("csr_ptr", C.c_void_p), ("csr_col", C.c_void_p),
                ("csr_eid", C.c_void_p), ("csc_ptr", C.c_void_p), ("csc_row", C.c_void_p),
                ("csc_scale", C.c_void_p), ("csr_w", C.c_void_p), ("plan", C.c_void_p),
                ("plan_bytes", C.c_size_t),
                ("n_nodes", C.c_int64), ("n_edges", C.c_int64), ("n_sub", C.c_int64),
                ("e_sub", C.c_int64), ("m_sel", C.c_int64), ("n_rel", C.c_int32),
                ("n_ntype", C.c_int32), ("type_off_host", C.c_int64 * (HG_MAX_NTYPE + 1)),
                ("n_active", C.c_int64 * HG_MAX_REL), ("plan_items", C.c_int64),
                ("plan_heavy", C.c_int64), ("plan_partials", C.c_int64),
                ("plan_fwd_heavy", C.c_int64), ("plan_fwd_parts", C.c_int64), ("plan_slot_rows", C.c_int64),
                ("weighted", C.c_int64)]


class LayerDesc(C.Structure):
    _fields_ = [("d_in", C.c_int32), ("d_out", C.c_int32), ("dtype", C.c_int32),
                ("relu", C.c_int32), ("residual", C.c_int32)]


HGT_PARAMS = ("W_K", "b_K", "W_Q", "b_Q", "W_V", "b_V", "W_att", "W_msg", "mu", "W_agg", "b_agg")


class HgtDesc(C.Structure):
    _fields_ = [("d", C.c_int32), ("heads", C.c_int32), ("dtype", C.c_int32), ("relu", C.c_int32),
                ("residual", C.c_int32), ("lean", C.c_int32)]


class HgtWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in HGT_PARAMS]


TEMPORAL_PARAMS = ("Q", "r", "Wi", "bi", "Wh", "bh")


class TemporalWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in TEMPORAL_PARAMS]


_lib = None


def lib() -> C.CDLL:
    """Load libhg.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: run __graft_entry__.build() "
                          "(python -m paper_2608_02168_amd.build)")
    L = C.CDLL(LIB_PATH)
    vp, sz, i64, i32, f32 = C.c_void_p, C.c_size_t, C.c_int64, C.c_int32, C.c_float
    sig = {
        "hg_plan_size": (sz, [i64, i64, i32]),
        "hg_node_keys_workspace_size": (sz, [vp, i32]),
        "hg_node_keys": (C.c_int, [vp, i32, vp, vp, sz, vp]),
        "hg_build_csr_workspace_size": (sz, [vp, vp]),
        "hg_build_csr": (C.c_int, [vp, vp, vp, vp, sz, vp]),
        "hg_layer_saved_size": (sz, [vp, vp]),
        "hg_layer_fwd_workspace_size": (sz, [vp, vp]),
        "hg_layer_bwd_workspace_size": (sz, [vp, vp]),
        "hg_layer_fwd": (C.c_int, [vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "hg_layer_bwd": (C.c_int, [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, i32, vp, sz, vp]),
        "hg_hgt_saved_size": (sz, [vp, vp]),
        "hg_hgt_fwd_workspace_size": (sz, [vp, vp]),
        "hg_hgt_bwd_workspace_size": (sz, [vp, vp]),
        "hg_hgt_fwd": (C.c_int, [vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "hg_hgt_bwd": (C.c_int, [vp, vp, vp, vp, vp, vp, vp, vp, vp, i32, vp, sz, vp]),
        "hg_align_workspace_size": (sz, [i64, i32]),
        "hg_align_loss_fwd_bwd": (C.c_int, [i64, i32, i32, i64, vp, vp, vp, vp, f32, f32, f32,
                                            i32, vp, vp, vp, vp, vp, sz, vp]),
        "hg_align_noalloc_scratch_size": (sz, []),
        "hg_align_loss_fwd_bwd_noalloc": (C.c_int, [i64, i32, i32, i64, vp, vp, vp, vp, f32, f32, f32,
                                                    i32, vp, vp, vp, vp, vp]),
        "hg_mlp_bce_workspace_size": (sz, [i64, i32, i32]),
        "hg_mlp_bce_fwd_bwd": (C.c_int, [i64, i32, i32] + [vp] * 7 + [i64] + [vp] * 8 + [sz, vp]),
        "hg_adam_step": (C.c_int, [i64, vp, vp, vp, vp, i64, f32, f32, f32, f32, f32, vp]),
        "hg_temporal_fwd": (C.c_int, [i64, i32, i32, i32, vp, vp, vp, vp, vp]),
        "hg_temporal_bwd_workspace_size": (sz, [i64, i32, i32]),
        "hg_temporal_bwd": (C.c_int, [i64, i32, i32, i32, vp, vp, vp, vp, vp, vp, i32, vp, vp, sz, vp]),
        "hg_mean_agg_fwd": (C.c_int, [i64, i32, i32, i32, vp, vp, vp, vp, vp]),
        "hg_mean_agg_bwd": (C.c_int, [i64, i32, i32, vp, vp, vp, vp, i32, vp]),
        "hg_home_gather": (C.c_int, [i64, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp]),
        "hg_status_string": (C.c_char_p, [C.c_int]),
        "hg_last_error_detail": (C.c_char_p, []),
        "hg_timing_enable": (C.c_int, [C.c_int]),
        "hg_timing_collect": (C.c_int, [vp, vp, vp, C.c_int]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().hg_status_string(status).decode()


def last_error_detail() -> str:
    return lib().hg_last_error_detail().decode()


def _check(status: int, where: str):
    if status != HG_OK:
        raise HgError(status, where, last_error_detail())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _ws(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(1, int(nbytes)), dtype=torch.uint8, device=device)


@dataclass
class Subgraph:
    """Device arrays of hg_subgraph plus the host counts the build returned."""
    c: SubgraphStruct
    device: torch.device
    arrays: dict = field(default_factory=dict)

    @property
    def n_sub(self) -> int:
        return int(self.c.n_sub)

    @property
    def e_sub(self) -> int:
        return int(self.c.e_sub)

    @property
    def m_sel(self) -> int:
        return int(self.c.m_sel)

    @property
    def n_rel(self) -> int:
        return int(self.c.n_rel)

    @property
    def n_ntype(self) -> int:
        return int(self.c.n_ntype)

    def view(self, name: str) -> torch.Tensor:
        """The valid prefix of one output array."""
        n_ptr = self.n_sub * self.n_rel + 1
        length = {"local2global": self.n_sub, "global2local": int(self.c.n_nodes),
                  "type_off": self.n_ntype + 1, "overlap": self.m_sel,
                  "overlap_home": self.m_sel, "overlap_rel": self.m_sel, "csr_ptr": n_ptr,
                  "csc_ptr": n_ptr, "csr_col": self.e_sub, "csr_eid": self.e_sub,
                  "csc_row": self.e_sub, "csc_scale": self.e_sub, "csr_w": self.e_sub}[name]
        return self.arrays[name][:length]

    def n_active(self):
        return [int(self.c.n_active[r]) for r in range(self.n_rel)]

    def type_off_host(self):
        return [int(self.c.type_off_host[t]) for t in range(self.n_ntype + 1)]


def hg_plan_size(n_nodes: int, n_edges: int, n_rel: int) -> int:
    return int(lib().hg_plan_size(n_nodes, n_edges, n_rel))


def hg_build_csr(src, dst, rel, ntype, part, k: int, n_rel: int, n_ntype: int, budget_M: int,
                 key: int = HG_KEY_OUTDEG, theta: int = HG_THETA_NONE, seed: int = 0,
                 want_eid: bool = True, stream=None, ws: Optional[torch.Tensor] = None,
                 out: Optional[Subgraph] = None, edge_ts=None, t_cut: int = 0, node_key=None,
                 edge_w=None) -> Subgraph:
    """Overlapping-subgraph construction; inputs are device tensors
    (src/dst/part int32, rel/ntype uint8, edge_ts int32 or None, edge_w
    float32 or None).  Synchronous.  ``out`` reuses the arrays of an earlier
    build of the same input sizes.  With edge_ts, the snapshot that keeps the
    induced edges with edge_ts <= t_cut.  node_key: the graph's keys from
    hg_node_keys (same key kind), or None to compute them inside the build.
    edge_w: message weights of the edges (csr_w is then allocated)."""
    dev = ntype.device
    n, e = int(ntype.shape[0]), int(src.shape[0])
    g = GraphDesc(n, e, n_rel, n_ntype, _ptr(src), _ptr(dst), _ptr(rel), _ptr(ntype), _ptr(part),
                  k, _ptr(edge_w), _ptr(edge_ts), int(t_cut), 0)
    o = OverlapDesc(budget_M, key, HG_KEYDIR_OUT, theta, 0, seed, _ptr(node_key))
    L = lib()
    if out is not None:
        if ws is None:
            ws = out.arrays.get("ws")
        if ws is None:
            ws = _ws(int(L.hg_build_csr_workspace_size(C.byref(g), C.byref(o))), dev)
        _check(L.hg_build_csr(C.byref(g), C.byref(o), C.byref(out.c), _ptr(ws), ws.numel(),
                              _stream(stream)), "hg_build_csr")
        return out
    i32 = dict(dtype=torch.int32, device=dev)
    m_cap = max(1, min(budget_M, n))
    nq = n * n_rel + 1
    arrays = {
        "local2global": torch.empty(n, **i32), "global2local": torch.empty(n, **i32),
        "type_off": torch.empty(n_ntype + 1, **i32), "overlap": torch.empty(m_cap, **i32),
        "overlap_home": torch.empty(m_cap, **i32),
        "overlap_rel": torch.empty(m_cap, dtype=torch.uint8, device=dev),
        "csr_ptr": torch.empty(nq, **i32), "csr_col": torch.empty(max(1, e), **i32),
        "csr_eid": torch.empty(max(1, e), **i32) if want_eid else None,
        "csc_ptr": torch.empty(nq, **i32), "csc_row": torch.empty(max(1, e), **i32),
        "csc_scale": torch.empty(max(1, e), dtype=torch.float32, device=dev),
        "csr_w": torch.empty(max(1, e), dtype=torch.float32, device=dev) if edge_w is not None else None,
    }
    plan_bytes = hg_plan_size(n, e, n_rel)
    arrays["plan"] = _ws(plan_bytes, dev)
    s = SubgraphStruct()
    for name in ("local2global", "global2local", "type_off", "overlap", "overlap_home",
                 "overlap_rel", "csr_ptr", "csr_col", "csr_eid", "csc_ptr", "csc_row",
                 "csc_scale", "csr_w", "plan"):
        setattr(s, name, _ptr(arrays[name]))
    s.plan_bytes = plan_bytes
    need = int(L.hg_build_csr_workspace_size(C.byref(g), C.byref(o)))
    if need == 0:
        _check(L.hg_build_csr(C.byref(g), C.byref(o), C.byref(s), None, 0, _stream(stream)),
               "hg_build_csr")
    if ws is None or ws.numel() < need:
        ws = _ws(need, dev)
    _check(L.hg_build_csr(C.byref(g), C.byref(o), C.byref(s), _ptr(ws), ws.numel(),
                          _stream(stream)), "hg_build_csr")
    arrays["ws"] = ws
    return Subgraph(s, dev, arrays)


def _layer_desc(d: int, dtype, relu: bool, residual: bool) -> LayerDesc:
    code = HG_DTYPE_BF16 if dtype == torch.bfloat16 else HG_DTYPE_F32
    return LayerDesc(d, d, code, int(relu), int(residual))


def hg_layer_saved_size(sub: Subgraph, d: int, dtype=torch.float32) -> int:
    desc = _layer_desc(d, dtype, True, True)
    return int(lib().hg_layer_saved_size(C.byref(sub.c), C.byref(desc)))


def hg_layer_fwd_workspace_size(sub: Subgraph, d: int, dtype=torch.float32) -> int:
    desc = _layer_desc(d, dtype, True, True)
    return int(lib().hg_layer_fwd_workspace_size(C.byref(sub.c), C.byref(desc)))


def hg_layer_bwd_workspace_size(sub: Subgraph, d: int, dtype=torch.float32) -> int:
    desc = _layer_desc(d, dtype, True, True)
    return int(lib().hg_layer_bwd_workspace_size(C.byref(sub.c), C.byref(desc)))


def hg_layer_fwd(sub: Subgraph, H_in, W_rel, W_self, bias=None, relu=True, residual=True,
                 H_out=None, saved=None, ws=None, stream=None):
    """Returns (H_out, saved); saved is the ReLU bitmask [n_sub, d/32] int32."""
    d = int(H_in.shape[1])
    desc = _layer_desc(d, H_in.dtype, relu, residual)
    L = lib()
    if H_out is None:
        H_out = torch.empty_like(H_in)
    if saved is None:
        saved = torch.empty((max(1, sub.n_sub), (d + 31) // 32), dtype=torch.int32, device=H_in.device)
    if ws is None:
        need = int(L.hg_layer_fwd_workspace_size(C.byref(sub.c), C.byref(desc)))
        ws = _ws(need, H_in.device)
    _check(L.hg_layer_fwd(C.byref(sub.c), C.byref(desc), _ptr(H_in), _ptr(W_rel), _ptr(W_self),
                          _ptr(bias), _ptr(H_out), _ptr(saved), _ptr(ws), ws.numel(),
                          _stream(stream)), "hg_layer_fwd")
    return H_out, saved


def hg_layer_bwd(sub: Subgraph, H_in, W_rel, W_self, saved, dH_out, relu=True, residual=True,
                 dH_in=None, dW_rel=None, dW_self=None, dbias=None, want_dbias=True, accumulate=False,
                 ws=None, stream=None):
    """Returns (dH_in, dW_rel, dW_self, dbias); with accumulate the weight
    gradients are added into the given buffers."""
    d = int(H_in.shape[1])
    desc = _layer_desc(d, H_in.dtype, relu, residual)
    L = lib()
    dev = H_in.device
    if dH_in is None:
        dH_in = torch.empty_like(H_in)
    if dW_rel is None:
        dW_rel = torch.empty_like(W_rel)
    if dW_self is None:
        dW_self = torch.empty_like(W_self)
    if dbias is None and want_dbias:
        dbias = torch.empty((W_self.shape[0], d), dtype=torch.float32, device=dev)
    if ws is None:
        need = int(L.hg_layer_bwd_workspace_size(C.byref(sub.c), C.byref(desc)))
        ws = _ws(need, dev)
    _check(L.hg_layer_bwd(C.byref(sub.c), C.byref(desc), _ptr(H_in), _ptr(W_rel), _ptr(W_self),
                          _ptr(saved), _ptr(dH_out), _ptr(dH_in), _ptr(dW_rel), _ptr(dW_self),
                          _ptr(dbias), int(bool(accumulate)), _ptr(ws), ws.numel(), _stream(stream)),
           "hg_layer_bwd")
    return dH_in, dW_rel, dW_self, dbias


def _hgt_desc(d: int, heads: int, relu: bool, residual: bool, lean: bool = False) -> HgtDesc:
    return HgtDesc(d, heads, HG_DTYPE_F32, int(relu), int(residual), int(lean))


def _hgt_struct(weights: dict) -> HgtWeights:
    """weights: name -> device float32 tensor (biases may be missing or None)."""
    return HgtWeights(*[_ptr(weights.get(n)) for n in HGT_PARAMS])


def hg_hgt_saved_size(sub: Subgraph, d: int, heads: int, lean: bool = False) -> int:
    desc = _hgt_desc(d, heads, True, True, lean)
    return int(lib().hg_hgt_saved_size(C.byref(sub.c), C.byref(desc)))


def hg_hgt_fwd_workspace_size(sub: Subgraph, d: int, heads: int, lean: bool = False) -> int:
    desc = _hgt_desc(d, heads, True, True, lean)
    return int(lib().hg_hgt_fwd_workspace_size(C.byref(sub.c), C.byref(desc)))


def hg_hgt_bwd_workspace_size(sub: Subgraph, d: int, heads: int, lean: bool = False) -> int:
    desc = _hgt_desc(d, heads, True, True, lean)
    return int(lib().hg_hgt_bwd_workspace_size(C.byref(sub.c), C.byref(desc)))


def hg_hgt_fwd(sub: Subgraph, H_in, weights: dict, heads: int, relu=True, residual=True, H_out=None,
               mask=None, saved=None, ws=None, stream=None, lean=False):
    """Attention layer forward; returns (H_out, mask, saved): mask is the ReLU
    bitmask [n_sub, d/32] int32, saved a uint8 buffer for the backward (lean:
    without the relation transforms, which the backward computes again)."""
    d = int(H_in.shape[1])
    desc = _hgt_desc(d, heads, relu, residual, lean)
    L = lib()
    if H_out is None:
        H_out = torch.empty_like(H_in)
    if mask is None:
        mask = torch.empty((max(1, sub.n_sub), d // 32), dtype=torch.int32, device=H_in.device)
    if saved is None:
        saved = _ws(int(L.hg_hgt_saved_size(C.byref(sub.c), C.byref(desc))), H_in.device)
    if ws is None:
        ws = _ws(int(L.hg_hgt_fwd_workspace_size(C.byref(sub.c), C.byref(desc))), H_in.device)
    W = _hgt_struct(weights)
    _check(L.hg_hgt_fwd(C.byref(sub.c), C.byref(desc), _ptr(H_in), C.byref(W), _ptr(H_out), _ptr(mask),
                        _ptr(saved), _ptr(ws), ws.numel(), _stream(stream)), "hg_hgt_fwd")
    return H_out, mask, saved


def hg_hgt_bwd(sub: Subgraph, H_in, weights: dict, heads: int, mask, saved, dH_out, relu=True, residual=True,
               dH_in=None, grads: Optional[dict] = None, accumulate: bool = False, ws=None, stream=None, lean=False):
    """Attention layer backward; returns (dH_in, grads) with grads a dict of
    the same names as the weights (bias gradients for the biases given),
    overwritten, or added into when accumulate.  lean as in the forward."""
    d = int(H_in.shape[1])
    desc = _hgt_desc(d, heads, relu, residual, lean)
    L = lib()
    if dH_in is None:
        dH_in = torch.empty_like(H_in)
    if grads is None:
        grads = {n: torch.empty_like(w) for n, w in weights.items() if w is not None}
    if ws is None:
        ws = _ws(int(L.hg_hgt_bwd_workspace_size(C.byref(sub.c), C.byref(desc))), H_in.device)
    G = _hgt_struct(grads)
    W = _hgt_struct(weights)
    _check(L.hg_hgt_bwd(C.byref(sub.c), C.byref(desc), _ptr(H_in), C.byref(W), _ptr(mask), _ptr(saved),
                        _ptr(dH_out), _ptr(dH_in), C.byref(G), int(accumulate), _ptr(ws), ws.numel(),
                        _stream(stream)), "hg_hgt_bwd")
    return dH_in, grads


def hg_mlp_bce_workspace_size(n_rows: int, d: int) -> int:
    return int(lib().hg_mlp_bce_workspace_size(n_rows, d, d))


def hg_mlp_bce_fwd_bwd(H, W1, b1, W2, b2, labels, dH=None, grads: Optional[dict] = None, loss=None, prob=None,
                       ws=None, stream=None, rows=None):
    """Prediction head + masked BCE: returns (loss [1], dH, grads) with grads
    {W1, b1, W2, b2}; dH is overwritten with dL_BCE/dH.  rows: int32 list
    of rows holding every labelled one (only those go through the head)."""
    n, d = int(H.shape[0]), int(H.shape[1])
    L = lib()
    if dH is None:
        dH = torch.empty_like(H)
    if grads is None:
        grads = {"W1": torch.empty_like(W1), "b1": torch.empty_like(b1), "W2": torch.empty_like(W2),
                 "b2": torch.empty_like(b2)}
    if loss is None:
        loss = torch.empty(1, dtype=torch.float32, device=H.device)
    if ws is None:
        ws = _ws(int(L.hg_mlp_bce_workspace_size(n, d, d)), H.device)
    n_list = 0 if rows is None else int(rows.shape[0])
    _check(L.hg_mlp_bce_fwd_bwd(n, d, d, _ptr(H), _ptr(W1), _ptr(b1), _ptr(W2), _ptr(b2), _ptr(labels), _ptr(rows),
                                n_list, _ptr(loss),
                                _ptr(prob), _ptr(dH), _ptr(grads["W1"]), _ptr(grads.get("b1")), _ptr(grads["W2"]),
                                _ptr(grads.get("b2")), _ptr(ws), ws.numel(), _stream(stream)), "hg_mlp_bce_fwd_bwd")
    return loss, dH, grads


def hg_adam_step(param, grad, m, v, step: int, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-5,
                 stream=None):
    """In-place Adam update of one float32 tensor."""
    _check(lib().hg_adam_step(param.numel(), _ptr(param), _ptr(grad), _ptr(m), _ptr(v), step, lr, beta1, beta2, eps,
                              weight_decay, _stream(stream)), "hg_adam_step")


def _host_ptrs(tensors):
    """A host array of device pointers (None entries stay NULL)."""
    arr = (C.c_void_p * max(1, len(tensors)))(*[None if t is None else t.data_ptr() for t in tensors])
    return arr


def _dtype_code(t) -> int:
    return HG_DTYPE_BF16 if t.dtype == torch.bfloat16 else HG_DTYPE_F32


def hg_temporal_fwd(h, states, weights: dict, H=None, stream=None):
    """Temporal module forward: h [n, d] and the w context states (oldest
    first, each [n, d], same dtype); returns H."""
    n, d = int(h.shape[0]), int(h.shape[1])
    if H is None:
        H = torch.empty_like(h)
    ctx = _host_ptrs(states)
    W = TemporalWeights(*[_ptr(weights.get(k)) for k in TEMPORAL_PARAMS])
    _check(lib().hg_temporal_fwd(n, d, len(states), _dtype_code(h), _ptr(h), C.cast(ctx, C.c_void_p), C.byref(W),
                                 _ptr(H), _stream(stream)), "hg_temporal_fwd")
    return H


def hg_temporal_bwd_workspace_size(n: int, d: int, w: int) -> int:
    return int(lib().hg_temporal_bwd_workspace_size(n, d, w))


def hg_temporal_bwd(h, states, weights: dict, dH, dh=None, dstates=None, grads: Optional[dict] = None,
                    accumulate: bool = False, ws=None, stream=None):
    """Temporal module backward: returns (dh, grads).  dL/dc_k is ADDED into
    dstates[k] (a list of tensors or None entries; None = no state
    gradients); grads are overwritten, or added into when accumulate."""
    n, d = int(h.shape[0]), int(h.shape[1])
    w = len(states)
    L = lib()
    if dh is None:
        dh = torch.empty_like(h)
    if grads is None:
        grads = {k: torch.empty_like(v) for k, v in weights.items() if v is not None}
    if ws is None:
        ws = _ws(int(L.hg_temporal_bwd_workspace_size(n, d, w)), h.device)
    ctx = _host_ptrs(states)
    darr = None if dstates is None else _host_ptrs(dstates)  # kept alive through the call
    dctx = None if darr is None else C.cast(darr, C.c_void_p)
    W = TemporalWeights(*[_ptr(weights.get(k)) for k in TEMPORAL_PARAMS])
    G = TemporalWeights(*[_ptr(grads.get(k)) for k in TEMPORAL_PARAMS])
    _check(L.hg_temporal_bwd(n, d, w, _dtype_code(h), _ptr(h), C.cast(ctx, C.c_void_p), C.byref(W), _ptr(dH),
                             _ptr(dh), dctx, int(accumulate), C.byref(G), _ptr(ws), ws.numel(), _stream(stream)),
           "hg_temporal_bwd")
    return dh, grads


def hg_node_keys(src, dst, rel, n_nodes: int, n_rel: int, key: int = HG_KEY_OUTDEG, keys=None, ws=None,
                 stream=None):
    """Key of every node (out-degree or out-neighbour h-index), int32
    [n_nodes] on the device.  Synchronous."""
    dev = src.device
    g = GraphDesc(n_nodes, int(src.shape[0]), n_rel, 1, _ptr(src), _ptr(dst), _ptr(rel), None, None, 0, None, None,
                  0, 0)
    L = lib()
    if keys is None:
        keys = torch.empty(n_nodes, dtype=torch.int32, device=dev)
    if ws is None:
        ws = _ws(int(L.hg_node_keys_workspace_size(C.byref(g), key)), dev)
    _check(L.hg_node_keys(C.byref(g), key, _ptr(keys), _ptr(ws), ws.numel(), _stream(stream)), "hg_node_keys")
    return keys


def hg_node_keys_workspace_size(n_nodes: int, n_edges: int, n_rel: int, key: int = HG_KEY_OUTDEG) -> int:
    g = GraphDesc(n_nodes, n_edges, n_rel, 1, None, C.c_void_p(8), C.c_void_p(8), None, None, 0, None, None, 0, 0)
    g.src = C.c_void_p(8)
    return int(lib().hg_node_keys_workspace_size(C.byref(g), key))


def hg_mean_agg_fwd(g2l: list, h_parts: list, H=None, cnt=None, stream=None):
    """MeanAgg over K subgraphs: g2l[k] (int32 [n_nodes]) and h_parts[k]
    ([n_sub_k, d]) of subgraph k; returns (H [n_nodes, d], cnt int32 [n_nodes])."""
    n, d = int(g2l[0].shape[0]), int(h_parts[0].shape[1])
    if H is None:
        H = torch.empty((n, d), dtype=h_parts[0].dtype, device=h_parts[0].device)
    if cnt is None:
        cnt = torch.empty(n, dtype=torch.int32, device=h_parts[0].device)
    ga, ha = _host_ptrs(g2l), _host_ptrs(h_parts)
    _check(lib().hg_mean_agg_fwd(n, d, _dtype_code(h_parts[0]), len(h_parts), C.cast(ga, C.c_void_p),
                                 C.cast(ha, C.c_void_p), _ptr(H), _ptr(cnt), _stream(stream)), "hg_mean_agg_fwd")
    return H, cnt


def hg_mean_agg_bwd(l2g, cnt, dH, dh_part=None, accumulate=False, stream=None):
    """dh_part[i] = dH[l2g[i]] / cnt[l2g[i]] (added into dh_part when accumulate)."""
    n_sub, d = int(l2g.shape[0]), int(dH.shape[1])
    if dh_part is None:
        dh_part = torch.empty((n_sub, d), dtype=dH.dtype, device=dH.device)
    _check(lib().hg_mean_agg_bwd(n_sub, d, _dtype_code(dH), _ptr(l2g), _ptr(cnt), _ptr(dH), _ptr(dh_part),
                                 int(bool(accumulate)), _stream(stream)), "hg_mean_agg_bwd")
    return dh_part


def hg_home_gather(overlap, l2g, home, g2l: list, h_parts: list, Y=None, stream=None):
    """Home copies of one subgraph's overlap rows: Y [m, d]."""
    m, d = int(overlap.shape[0]), int(h_parts[0].shape[1])
    if Y is None:
        Y = torch.empty((m, d), dtype=h_parts[0].dtype, device=h_parts[0].device)
    ga, ha = _host_ptrs(g2l), _host_ptrs(h_parts)
    _check(lib().hg_home_gather(m, d, _dtype_code(h_parts[0]), len(h_parts), _ptr(overlap), _ptr(l2g), _ptr(home),
                                C.cast(ga, C.c_void_p), C.cast(ha, C.c_void_p), _ptr(Y), _stream(stream)),
           "hg_home_gather")
    return Y


def hg_align_workspace_size(M: int, d: int) -> int:
    return int(lib().hg_align_workspace_size(M, d))


def hg_align_loss_fwd_bwd(H, overlap, H_ref, dH, w=None, lambda_n=2e-4, scale=0.1, eps=1e-5,
                          ddof=0, dH_ref=None, loss3=None, ws=None, stream=None, dH_base=None):
    """CCA alignment: returns loss3 (device float32 [3] = L_inv, L_dec, L);
    dH[overlap] = dH_base[overlap] + scale * dL/dX (dH_base = dH when None:
    the gradient is added into dH) and overwrites dH_ref if given."""
    M = int(overlap.shape[0])
    d = int(H.shape[1])
    L = lib()
    code = HG_DTYPE_BF16 if H.dtype == torch.bfloat16 else HG_DTYPE_F32
    if loss3 is None:
        loss3 = torch.empty(3, dtype=torch.float32, device=H.device)
    if ws is None:
        ws = _ws(int(L.hg_align_workspace_size(M, d)), H.device)
    _check(L.hg_align_loss_fwd_bwd(M, d, code, int(H.shape[0]), _ptr(H), _ptr(overlap), _ptr(H_ref),
                                   _ptr(w), lambda_n, scale, eps, ddof, _ptr(loss3), _ptr(dH), _ptr(dH_base),
                                   _ptr(dH_ref), _ptr(ws), ws.numel(), _stream(stream)),
           "hg_align_loss_fwd_bwd")
    return loss3


def hg_align_noalloc_scratch_size() -> int:
    return int(lib().hg_align_noalloc_scratch_size())


def hg_align_loss_fwd_bwd_noalloc(H, overlap, H_ref, dH, loss3, w=None, lambda_n=2e-4, scale=0.1, eps=1e-5,
                                  ddof=0, dH_ref=None, stream=None, dH_base=None):
    """hg_align_loss_fwd_bwd with the library's static scratch instead of a
    workspace: allocates nothing (loss3 is the caller's device float32 [3])."""
    code = HG_DTYPE_BF16 if H.dtype == torch.bfloat16 else HG_DTYPE_F32
    _check(lib().hg_align_loss_fwd_bwd_noalloc(int(overlap.shape[0]), int(H.shape[1]), code, int(H.shape[0]),
                                               _ptr(H), _ptr(overlap), _ptr(H_ref), _ptr(w), lambda_n, scale, eps,
                                               ddof, _ptr(loss3), _ptr(dH), _ptr(dH_base), _ptr(dH_ref),
                                               _stream(stream)),
           "hg_align_loss_fwd_bwd_noalloc")
    return loss3


def hg_timing_enable(on: bool = True):
    _check(lib().hg_timing_enable(int(on)), "hg_timing_enable")


def hg_timing_collect(cap: int = 256) -> dict:
    """{kernel name: (launches, total_ms)} since the last collect."""
    names = (C.c_char * 64 * cap)()
    launches = (C.c_int64 * cap)()
    total = (C.c_double * cap)()
    n = lib().hg_timing_collect(names, launches, total, cap)
    if n < 0:
        _check(n, "hg_timing_collect")
    out = {}
    for i in range(min(n, cap)):
        out[bytes(names[i]).split(b"\0", 1)[0].decode()] = (int(launches[i]), float(total[i]))
    return out
