"""The C ABI on the host: the library loads, exports every symbol the
header declares, and rejects invalid arguments before any device work
(no GPU is needed for any of these)."""
import ctypes as C
import os
import re

import pytest

from paper_2608_02168_amd import api

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "hg.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(api.LIB_PATH):
        pytest.skip("libhg.so not built")
    return api.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hg_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(api.EXPORTS)


def test_status_strings(L):
    for code in (0, -1, -2, -3, -4, -5):
        assert api.status_string(code).startswith("HG_")
    assert "unknown" in api.status_string(7)


def _graph(n=10, e=5, R=2, T=2, **kw):
    fake = C.c_void_p(0x1000)  # never dereferenced: validation fails first
    d = dict(n_nodes=n, n_edges=e, n_rel=R, n_ntype=T, src=fake, dst=fake, rel=fake, ntype=fake,
             part=fake, k=0, edge_w=None)
    d.update(kw)
    return api.GraphDesc(**d)


def _ov(**kw):
    d = dict(budget_M=3, key=0, key_dir=0, theta=api.HG_THETA_NONE, reserved=0, seed=1)
    d.update(kw)
    return api.OverlapDesc(**d)


@pytest.mark.parametrize("gkw,okw,code", [
    (dict(n_nodes=0), {}, api.HG_ERR_ARG),
    (dict(n_edges=-1), {}, api.HG_ERR_ARG),
    (dict(n_edges=2**31), {}, api.HG_ERR_UNSUPPORTED),
    (dict(n_rel=0), {}, api.HG_ERR_UNSUPPORTED),
    (dict(n_rel=256), {}, api.HG_ERR_UNSUPPORTED),
    (dict(n_ntype=0), {}, api.HG_ERR_UNSUPPORTED),
    (dict(n_nodes=2**30, n_rel=4), {}, api.HG_ERR_UNSUPPORTED),
    (dict(src=None), {}, api.HG_ERR_ARG),
    (dict(part=None), {}, api.HG_ERR_ARG),
    ({}, dict(budget_M=-1), api.HG_ERR_ARG),
    ({}, dict(key=7), api.HG_ERR_ARG),
    ({}, dict(key_dir=1), api.HG_ERR_UNSUPPORTED),
    ({}, dict(theta=-3), api.HG_ERR_ARG),
])
def test_build_validation(L, gkw, okw, code):
    g, o = _graph(**gkw), _ov(**okw)
    s = api.SubgraphStruct()
    assert L.hg_build_csr_workspace_size(C.byref(g), C.byref(o)) == 0
    assert L.hg_build_csr(C.byref(g), C.byref(o), C.byref(s), None, 0, None) == code
    assert len(api.last_error_detail()) > 0


def test_weighted_build_needs_the_weight_output(L):
    """Edge weights are accepted, and then the build writes the weight of
    every CSR entry: a missing csr_w output is refused before any device work."""
    fake = C.c_void_p(0x1000)
    g, o = _graph(edge_w=fake), _ov()
    assert L.hg_build_csr_workspace_size(C.byref(g), C.byref(o)) > \
        L.hg_build_csr_workspace_size(C.byref(_graph()), C.byref(o))
    s = api.SubgraphStruct()
    for name in ("local2global", "global2local", "type_off", "overlap", "overlap_home", "overlap_rel", "csr_ptr",
                 "csr_col", "csc_ptr", "csc_row", "csc_scale", "plan"):
        setattr(s, name, fake)
    s.plan_bytes = api.hg_plan_size(10, 5, 2)
    assert L.hg_build_csr(C.byref(g), C.byref(o), C.byref(s), None, 0, None) == api.HG_ERR_ARG
    assert "csr_w" in api.last_error_detail()


def test_build_capacity_checks(L):
    g, o = _graph(), _ov()
    fake = C.c_void_p(0x1000)
    s = api.SubgraphStruct()
    for name in ("local2global", "global2local", "type_off", "overlap", "overlap_home",
                 "overlap_rel", "csr_ptr", "csr_col", "csc_ptr", "csc_row", "csc_scale", "plan"):
        setattr(s, name, fake)
    s.plan_bytes = 1
    assert L.hg_build_csr(C.byref(g), C.byref(o), C.byref(s), fake, 1 << 30, None) == api.HG_ERR_CAPACITY
    assert "plan" in api.last_error_detail()
    s.plan_bytes = api.hg_plan_size(10, 5, 2)
    need = L.hg_build_csr_workspace_size(C.byref(g), C.byref(o))
    assert need > 0
    assert L.hg_build_csr(C.byref(g), C.byref(o), C.byref(s), fake, need - 1, None) == api.HG_ERR_CAPACITY
    s.overlap = None
    assert L.hg_build_csr(C.byref(g), C.byref(o), C.byref(s), fake, need, None) == api.HG_ERR_ARG


def test_plan_size_monotone(L):
    assert api.hg_plan_size(10, 10, 1) > 0
    assert api.hg_plan_size(1000, 10**5, 3) > api.hg_plan_size(1000, 10**4, 3)
    assert L.hg_plan_size(-1, 0, 1) == 0


def _sub(n_sub=10, R=2, T=2):
    s = api.SubgraphStruct()
    fake = C.c_void_p(0x1000)
    s.csr_ptr = s.csc_ptr = s.plan = fake
    s.n_sub, s.n_rel, s.n_ntype = n_sub, R, T
    s.plan_slot_rows = n_sub * R  # the row-indexed layout of the relation transforms
    return s


@pytest.mark.parametrize("desc,code", [
    (dict(d_in=64, d_out=128), api.HG_ERR_UNSUPPORTED),
    (dict(d_in=96, d_out=96), api.HG_ERR_UNSUPPORTED),
    (dict(d_in=96, d_out=96, dtype=1), api.HG_ERR_UNSUPPORTED),
    (dict(d_in=64, d_out=64, dtype=9), api.HG_ERR_ARG),
    (dict(d_in=64, d_out=64, relu=2), api.HG_ERR_ARG),
])
def test_layer_validation(L, desc, code):
    full = dict(d_in=64, d_out=64, dtype=0, relu=1, residual=1)
    full.update(desc)
    ld = api.LayerDesc(**full)
    s = _sub()
    fake = C.c_void_p(0x1000)
    assert L.hg_layer_fwd(C.byref(s), C.byref(ld), fake, fake, fake, None, C.c_void_p(0x2000), fake,
                          fake, 1, None) == code
    assert L.hg_layer_fwd_workspace_size(C.byref(s), C.byref(ld)) == 0


def test_layer_alias_and_null_checks(L):
    ld = api.LayerDesc(64, 64, 0, 1, 1)
    s = _sub()
    fake = C.c_void_p(0x1000)
    assert L.hg_layer_fwd(C.byref(s), C.byref(ld), fake, fake, fake, None, fake, fake, fake, 1,
                          None) == api.HG_ERR_ARG
    assert L.hg_layer_fwd(C.byref(s), C.byref(ld), None, fake, fake, None, C.c_void_p(8), fake, fake,
                          1, None) == api.HG_ERR_ARG
    assert L.hg_layer_bwd(C.byref(s), C.byref(ld), fake, None, fake, fake, fake, fake, fake, fake,
                          None, 0, fake, 1, None) == api.HG_ERR_ARG
    assert L.hg_layer_bwd(C.byref(s), C.byref(ld), fake, fake, fake, fake, fake, fake, fake, fake,
                          None, 2, fake, 1, None) == api.HG_ERR_ARG
    assert L.hg_layer_fwd(None, C.byref(ld), fake, fake, fake, None, fake, fake, fake, 1,
                          None) == api.HG_ERR_ARG


def test_layer_workspace_sizes_scale_with_graph(L):
    ld = api.LayerDesc(128, 128, 0, 1, 1)
    a, b = _sub(n_sub=100), _sub(n_sub=1000)
    assert L.hg_layer_fwd_workspace_size(C.byref(b), C.byref(ld)) > \
        L.hg_layer_fwd_workspace_size(C.byref(a), C.byref(ld))
    assert L.hg_layer_saved_size(C.byref(b), C.byref(ld)) == 1000 * 4 * 4


@pytest.mark.parametrize("args,code", [
    (dict(M=-1), api.HG_ERR_ARG),
    (dict(d=96), api.HG_ERR_UNSUPPORTED),
    (dict(dtype=1, d=96), api.HG_ERR_UNSUPPORTED),
    (dict(d=512), api.HG_ERR_UNSUPPORTED),
    (dict(dtype=7), api.HG_ERR_ARG),
    (dict(dtype=1, d=256, ws_bytes=1), api.HG_ERR_CAPACITY),
    (dict(M=20, n_rows=10), api.HG_ERR_ARG),
    (dict(M=1, ddof=1), api.HG_ERR_ARG),
    (dict(eps=-1.0), api.HG_ERR_ARG),
    (dict(H=None), api.HG_ERR_ARG),
])
def test_align_validation(L, args, code):
    fake = C.c_void_p(0x1000)
    a = dict(M=5, d=64, dtype=0, n_rows=10, H=fake, overlap=fake, H_ref=fake, w=None, lambda_n=2e-4,
             scale=0.1, eps=1e-5, ddof=0, loss3=fake, dH=fake, dH_base=None, dH_ref=None, ws=fake, ws_bytes=1 << 20,
             stream=None)
    a.update(args)
    assert L.hg_align_loss_fwd_bwd(*a.values()) == code
    assert L.hg_align_workspace_size(5, 96) == 0
    assert L.hg_align_workspace_size(5, 64) > 0


def test_temporal_validation(L):
    fake, out = C.c_void_p(0x1000), C.c_void_p(0x2000)
    ctx = (C.c_void_p * 4)(0x3000, 0x4000, 0x5000, 0x6000)
    cp = C.cast(ctx, C.c_void_p)
    W = api.TemporalWeights(fake, fake, fake, None, fake, None)

    def fwd(n=10, d=64, w=2, dtype=0, h=fake, ctxp=cp, Wp=W, H=out):
        return L.hg_temporal_fwd(n, d, w, dtype, h, ctxp, C.byref(Wp), H, None)

    assert fwd(d=128) == api.HG_ERR_UNSUPPORTED
    assert fwd(w=5) == api.HG_ERR_UNSUPPORTED
    assert fwd(dtype=7) == api.HG_ERR_UNSUPPORTED
    assert fwd(n=-1) == api.HG_ERR_ARG
    assert fwd(w=-1) == api.HG_ERR_ARG
    assert fwd(H=C.c_void_p(0x4000)) == api.HG_ERR_ARG          # aliases context state 1
    assert fwd(H=fake) == api.HG_ERR_ARG                         # aliases h
    assert fwd(ctxp=None) == api.HG_ERR_ARG
    assert fwd(Wp=api.TemporalWeights(None, fake, fake, None, fake, None)) == api.HG_ERR_ARG
    assert fwd(n=0) == api.HG_OK                                 # nothing to do, no device work
    G = api.TemporalWeights(fake, fake, fake, None, fake, None)
    dctx = (C.c_void_p * 4)(0x7000, 0x2000, 0, 0)

    def bwd(accumulate=0, Gp=G, dh=C.c_void_p(0x8000), dcp=None, dH=C.c_void_p(0x9000)):
        return L.hg_temporal_bwd(10, 64, 2, 0, fake, cp, C.byref(W), dH, dh, dcp, accumulate, C.byref(Gp),
                                 fake, 1 << 30, None)

    assert bwd(accumulate=2) == api.HG_ERR_ARG
    assert bwd(Gp=api.TemporalWeights(fake, None, fake, None, fake, None)) == api.HG_ERR_ARG
    assert bwd(dh=C.c_void_p(0x9000)) == api.HG_ERR_ARG          # dh aliases dH
    assert bwd(dcp=C.cast(dctx, C.c_void_p), dh=C.c_void_p(0x2000)) == api.HG_ERR_ARG
    assert L.hg_temporal_bwd_workspace_size(10, 128, 1) == 0
    assert L.hg_temporal_bwd_workspace_size(10, 64, 5) == 0
    assert L.hg_temporal_bwd_workspace_size(1000, 64, 3) > L.hg_temporal_bwd_workspace_size(1000, 64, 1) > 0


def test_product_path_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(api, "_lib", None)
    monkeypatch.setattr(api, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        api.lib()


def test_binding_structs_match_the_header(tmp_path):
    """Size and field offsets of every struct of the ABI, as the C compiler
    lays them out from include/hg.h, equal those of the ctypes binding."""
    import shutil
    import subprocess
    if not shutil.which("gcc"):
        pytest.skip("gcc not available")
    structs = {"hg_graph_desc": api.GraphDesc, "hg_overlap_desc": api.OverlapDesc,
               "hg_subgraph": api.SubgraphStruct, "hg_layer_desc": api.LayerDesc, "hg_hgt_desc": api.HgtDesc,
               "hg_hgt_weights": api.HgtWeights, "hg_temporal_weights": api.TemporalWeights}
    lines = ["#include <stdio.h>", "#include <stddef.h>", f'#include "{HEADER}"', "int main(void) {"]
    for cname, py in structs.items():
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in py._fields_:
            lines.append(f'  printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-o", str(exe), str(src)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l.strip()}
    for cname, py in structs.items():
        assert got[(cname, "size")] == C.sizeof(py), cname
        for fname, _ in py._fields_:
            assert got[(cname, fname)] == getattr(py, fname).offset, (cname, fname)


def test_kway_calls_reject_bad_arguments(L):
    fake = C.c_void_p(0x1000)
    arr = (C.c_void_p * 1)(0x1000)
    # K out of range, bad width, bad dtype, null tables: rejected before any device work
    assert L.hg_mean_agg_fwd(10, 64, 0, 0, arr, arr, fake, None, None) == api.HG_ERR_ARG
    assert L.hg_mean_agg_fwd(10, 64, 0, api.HG_MAX_PARTS + 1, arr, arr, fake, None, None) == api.HG_ERR_ARG
    assert L.hg_mean_agg_fwd(10, 96, 0, 1, arr, arr, fake, None, None) == api.HG_ERR_UNSUPPORTED
    assert L.hg_mean_agg_fwd(10, 64, 5, 1, arr, arr, fake, None, None) == api.HG_ERR_ARG
    assert L.hg_mean_agg_fwd(10, 64, 0, 1, None, arr, fake, None, None) == api.HG_ERR_ARG
    nul = (C.c_void_p * 2)(0x1000, None)
    assert L.hg_mean_agg_fwd(10, 64, 0, 2, nul, arr, fake, None, None) == api.HG_ERR_ARG
    assert L.hg_mean_agg_bwd(10, 64, 0, fake, fake, fake, fake, 2, None) == api.HG_ERR_ARG
    assert L.hg_mean_agg_bwd(10, 64, 0, fake, fake, fake, fake, 0, None) == api.HG_ERR_ARG  # dh aliases dH
    assert L.hg_mean_agg_bwd(-1, 64, 0, fake, fake, fake, None, 0, None) == api.HG_ERR_ARG
    assert L.hg_home_gather(4, 64, 0, 0, fake, fake, fake, arr, arr, fake, None) == api.HG_ERR_ARG
    assert L.hg_home_gather(4, 64, 0, 1, None, fake, fake, arr, arr, fake, None) == api.HG_ERR_ARG
    # empty inputs are no-ops
    assert L.hg_mean_agg_fwd(0, 64, 0, 1, arr, arr, None, None, None) == api.HG_OK
    assert L.hg_mean_agg_bwd(0, 64, 0, None, None, None, None, 0, None) == api.HG_OK
    assert L.hg_home_gather(0, 64, 0, 1, None, None, None, arr, arr, None, None) == api.HG_OK


def test_node_keys_reject_bad_arguments(L):
    fake = C.c_void_p(0x1000)
    g = api.GraphDesc(10, 5, 2, 1, fake, fake, fake, None, None, 0, None, None, 0, 0)
    assert L.hg_node_keys(C.byref(g), 2, fake, fake, 1 << 20, None) == api.HG_ERR_ARG      # key kind
    assert L.hg_node_keys(C.byref(g), 0, None, fake, 1 << 20, None) == api.HG_ERR_ARG      # no output
    assert L.hg_node_keys(C.byref(g), 0, fake, fake, 1, None) == api.HG_ERR_CAPACITY       # workspace
    assert L.hg_node_keys(None, 0, fake, fake, 1 << 20, None) == api.HG_ERR_ARG
    big = api.GraphDesc(1 << 30, (1 << 31) - 1, 2, 1, fake, fake, fake, None, None, 0, None, None, 0, 0)
    assert L.hg_node_keys_workspace_size(C.byref(big), 0) == 0
    assert L.hg_node_keys_workspace_size(C.byref(g), 1) > L.hg_node_keys_workspace_size(C.byref(g), 0)


def test_head_rejects_bad_row_lists(L):
    fake = C.c_void_p(0x1000)
    args = lambda rows, n_list, prob: (10, 64, 64, fake, fake, None, fake, None, fake, rows, n_list, fake, prob, fake,
                                       fake, None, fake, None, fake, 1 << 30, None)
    assert L.hg_mlp_bce_fwd_bwd(*args(fake, 11, None)) == api.HG_ERR_ARG   # longer than the rows
    assert L.hg_mlp_bce_fwd_bwd(*args(fake, -1, None)) == api.HG_ERR_ARG
    assert L.hg_mlp_bce_fwd_bwd(*args(fake, 4, fake)) == api.HG_ERR_ARG    # prob needs every row


def test_hgt_descriptor_flags_and_lean_sizes(L):
    s = _sub(n_sub=1000, R=5, T=2)
    full = api.HgtDesc(64, 4, 0, 1, 1, 0)
    lean = api.HgtDesc(64, 4, 0, 1, 1, 1)
    bad = api.HgtDesc(64, 4, 0, 1, 1, 2)
    fake = C.c_void_p(0x1000)
    w = api.HgtWeights(*([fake] * 11))
    # the relation transforms (2 x rows x d floats, rows = n_sub x R in the row-indexed
    # layout) leave `saved` and go to the workspaces
    kt = 2 * 1000 * 5 * 64 * 4
    assert L.hg_hgt_saved_size(C.byref(s), C.byref(full)) - L.hg_hgt_saved_size(C.byref(s), C.byref(lean)) == kt
    assert L.hg_hgt_fwd_workspace_size(C.byref(s), C.byref(lean)) - \
        L.hg_hgt_fwd_workspace_size(C.byref(s), C.byref(full)) >= kt
    assert L.hg_hgt_bwd_workspace_size(C.byref(s), C.byref(lean)) - \
        L.hg_hgt_bwd_workspace_size(C.byref(s), C.byref(full)) >= kt
    assert L.hg_hgt_fwd(C.byref(s), C.byref(bad), fake, C.byref(w), fake, fake, fake, fake, 1 << 30,
                        None) == api.HG_ERR_ARG
