"""The C ABI without a GPU: exports, struct layout, host-side argument validation.

Every call made here returns from host validation (or the workspace size
query) before any HIP call, so it runs on a machine without a device.
"""
import ctypes as C
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gcn.h")


@pytest.fixture(scope="module")
def G():
    import paper_2512_01678_amd.gcn as G
    return G


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gcn_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(G):
    names = declared_functions()
    assert len(names) >= 17
    out = subprocess.run(["nm", "-D", "--defined-only", G.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r" T (gcn_[a-z_]+)$", out, flags=re.M))
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    for n in names:
        getattr(G.raw_lib(), n)


def test_struct_layout_matches_c(G, tmp_path):
    structs = {
        "gcn_graph": G.gcn_graph, "gcn_sparse_x": G.gcn_sparse_x, "gcn_feature_info": G.gcn_feature_info,
        "gcn_layer": G.gcn_layer, "gcn_model": G.gcn_model, "gcn_adam_tensor": G.gcn_adam_tensor,
        "gcn_profile_record": G.gcn_profile_record, "gcn_split": G.gcn_split,
    }
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "gcn.h"', "int main(void) {"]
    for sname, cls in structs.items():
        lines.append(f'printf("{sname} size %zu\\n", sizeof({sname}));')
        for fname, _ in cls._fields_:
            lines.append(f'printf("{sname} {fname} %zu\\n", offsetof({sname}, {fname}));')
    lines += ["return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
                    "-D__HIP_PLATFORM_AMD__", str(src), "-o", str(exe)], check=True)
    got = {}
    for line in subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.splitlines():
        s, f, v = line.split()
        got[(s, f)] = int(v)
    for sname, cls in structs.items():
        assert got[(sname, "size")] == C.sizeof(cls), sname
        for fname, _ in cls._fields_:
            assert got[(sname, fname)] == getattr(cls, fname).offset, (sname, fname)


def test_status_strings(G):
    L = G.raw_lib()
    assert L.gcn_status_string(0) == b"GCN_OK"
    assert L.gcn_status_string(-4) == b"GCN_E_CAPACITY"
    assert L.gcn_status_string(-99) == b"GCN_E_UNKNOWN"
    assert L.gcn_version() >= 3


def test_host_validation_rejects_bad_calls(G):
    L = G.raw_lib()
    nb = G.sz(0)
    # negative sizes
    assert L.gcn_build_csr(-1, 0, None, None, None, None, C.byref(nb), None) == G.E_INVALID
    assert L.gcn_build_csr(5, 1 << 30, None, None, None, None, C.byref(nb), None) == G.E_OVERFLOW
    # workspace size query needs no device
    assert L.gcn_build_csr(1000, 5000, None, None, None, None, C.byref(nb), None) == G.OK
    assert nb.value > 4 * (2 * 5000 + 1000)
    # ws_bytes NULL
    assert L.gcn_build_csr(10, 5, None, None, None, None, None, None) == G.E_INVALID
    # a workspace that is too small is a capacity error, before any launch
    small = G.sz(8)
    g = G.gcn_graph(10, 0, 100, 1, 1, 1, 1, 1)
    assert L.gcn_build_csr(10, 5, 1, 1, C.byref(g), 1, C.byref(small), None) == G.E_CAPACITY
    assert "needed" in L.gcn_last_error().decode()
    # feature stats: bad tau, pitch < width, bad force mode
    info = G.gcn_feature_info()
    assert L.gcn_feature_stats(1, 10, 8, 8, 4, 0, -1, None, C.byref(info), None, None, C.byref(nb), None) == G.E_INVALID
    assert L.gcn_feature_stats(1, 10, 8, 7, 4, 5, -1, None, C.byref(info), None, None, C.byref(nb), None) == G.E_INVALID
    assert L.gcn_feature_stats(1, 10, 8, 8, 4, 5, 7, None, C.byref(info), None, None, C.byref(nb), None) == G.E_INVALID
    # gemm: unknown op, pitch too small, NULL operand
    assert L.gcn_gemm(9, 4, 4, 4, 1, 4, 1, 4, 1, 4, None, 0, None, 0, None, C.byref(nb), None) == G.E_INVALID
    assert L.gcn_gemm(G.OP_NN, 4, 4, 8, 1, 4, 1, 4, 1, 4, None, 0, None, 0, None, C.byref(nb), None) == G.E_INVALID
    nb2 = G.sz(1 << 20)
    assert L.gcn_gemm(G.OP_NN, 4, 4, 4, None, 4, 1, 4, 1, 4, None, 0, None, 0, 1, C.byref(nb2), None) == G.E_INVALID
    # aggregate: NULL graph, mask epilogue without mask
    assert L.gcn_aggregate(None, 0, 4, 1, 4, None, 0, None, 0, 1, 4, None, C.byref(nb), None) == G.E_INVALID
    g2 = G.gcn_graph(10, 20, 20, 1, 1, 1, 1, 1)
    assert L.gcn_aggregate(C.byref(g2), 0, 4, 1, 4, None, G.EPI_MASK, None, 0, 1, 4, None, C.byref(nb),
                           None) == G.E_INVALID
    assert L.gcn_aggregate(C.byref(g2), 0, 4, 1, 3, None, 0, None, 0, 1, 4, None, C.byref(nb), None) == G.E_INVALID
    # the entries of A_hat are required
    noval = G.gcn_graph(10, 20, 20, 1, 1, 1, 1, None)
    assert L.gcn_aggregate(C.byref(noval), 0, 4, 1, 4, None, 0, None, 0, 1, 4, None, C.byref(nb), None) == G.E_INVALID
    assert L.gcn_build_csr(10, 5, 1, 1, C.byref(noval), 1, C.byref(G.sz(1 << 20)), None) == G.E_INVALID
    # a split plan with long rows needs its chunk sums in the workspace
    sp = G.gcn_split(3, 50, 64, 1, 1, 1, None)
    g3 = G.gcn_graph(10, 20, 20, 1, 1, 1, 1, 1, sp)
    assert L.gcn_aggregate(C.byref(g3), 0, 40, 1, 40, None, 0, None, 0, 1, 40, None, C.byref(nb), None) == G.OK
    assert nb.value == 50 * 40 * 4
    bad = G.gcn_graph(10, 20, 20, 1, 1, 1, 1, 1, G.gcn_split(3, 50, 64, 1, None, 1, None))
    assert L.gcn_aggregate(C.byref(bad), 0, 40, 1, 40, None, 0, None, 0, 1, 40, None, C.byref(nb), None) == G.E_INVALID
    # spmm: bad pitch
    assert L.gcn_spmm(10, 20, 1, 1, 1, 5, 8, 1, 7, 1, 8, None, None, C.byref(nb), None) == G.E_INVALID
    # spmm_xt: bad pitch, negative sizes; size query of the chunked form (n = 4 chunks of
    # 8192 rows, 16 entries per column and chunk): offsets (5 x 3 int64) + partials (4 x 3 x 8)
    assert L.gcn_spmm_xt(10, 3, 5, 1, 1, 1, None, 1, 7, 8, 1, 8, None, C.byref(nb), None) == G.E_INVALID
    assert L.gcn_spmm_xt(-1, 3, 5, 1, 1, 1, None, 1, 8, 8, 1, 8, None, C.byref(nb), None) == G.E_INVALID
    assert L.gcn_spmm_xt(4 * 8192, 3, 16 * 3 * 4, 1, 1, 1, None, 1, 8, 8, 1, 8, None, C.byref(nb), None) == G.OK
    assert nb.value == 256 + 512
    # adam: step 0, too many tensors
    assert L.gcn_adam(None, 0, 0, 0.01, 0.9, 0.999, 1e-8, None) == G.E_INVALID
    arr = (G.gcn_adam_tensor * 17)()
    assert L.gcn_adam(arr, 17, 1, 0.01, 0.9, 0.999, 1e-8, None) == G.E_UNSUPPORTED
    # profile read out of range
    rec = G.gcn_profile_record()
    assert L.gcn_profile_read(0, C.byref(rec)) == G.E_INVALID
    # family filter: name length bound, NULL clears
    assert L.gcn_profile_only(b"x" * 64) == G.E_INVALID
    assert L.gcn_profile_only(b"aggregate_w256") == G.OK
    assert L.gcn_profile_only(None) == G.OK


def test_layer_validation(G):
    L = G.raw_lib()
    nb = G.sz(0)
    g = G.gcn_graph(10, 20, 20, 1, 1, 1, 1, 1)
    lay = G.gcn_layer(8, 4, 8, 4, G.ACT_RELU, G.ORDER_AUTO, 1)
    # neither / both inputs
    assert L.gcn_layer_fwd(C.byref(g), C.byref(lay), None, None, 1, 1, 1, None, None, None, None, None,
                           C.byref(nb), None) == G.E_INVALID
    # pitch smaller than width
    bad = G.gcn_layer(8, 4, 7, 4, G.ACT_RELU, G.ORDER_AUTO, 1)
    assert L.gcn_layer_fwd(C.byref(g), C.byref(bad), 1, None, 1, 1, 1, None, None, None, None, None,
                           C.byref(nb), None) == G.E_INVALID
    # softmax without labels
    sm = G.gcn_layer(8, 4, 8, 4, G.ACT_SOFTMAX_CE, G.ORDER_AUTO, 1)
    assert L.gcn_layer_fwd(C.byref(g), C.byref(sm), 1, None, 1, 1, 1, None, None, None, None, None,
                           C.byref(nb), None) == G.E_INVALID
    # aggregate-first needs a saved buffer
    af = G.gcn_layer(8, 64, 8, 64, G.ACT_RELU, G.AGGREGATE_FIRST, 1)
    assert L.gcn_layer_fwd(C.byref(g), C.byref(af), 1, None, 1, 1, 1, None, None, None, None, None,
                           C.byref(nb), None) == G.E_INVALID
    # a valid transform-first layer: size query succeeds and covers the n x pitch(f_out) scratch
    assert L.gcn_layer_fwd(C.byref(g), C.byref(lay), 1, None, 1, 1, 1, None, None, None, None, None,
                           C.byref(nb), None) == G.OK
    assert nb.value >= 10 * 4 * 4
    # aggregators: unknown kind, max forced transform-first, max too wide, max on sparse X
    assert L.gcn_layer_fwd(C.byref(g), C.byref(G.gcn_layer(8, 4, 8, 4, G.ACT_RELU, G.ORDER_AUTO, 1, 9)), 1, None,
                           1, 1, 1, 1, None, None, None, None, C.byref(nb), None) == G.E_INVALID
    mx_tf = G.gcn_layer(8, 4, 8, 4, G.ACT_RELU, G.TRANSFORM_FIRST, 1, G.AGG_MAX)
    assert L.gcn_layer_fwd(C.byref(g), C.byref(mx_tf), 1, None, 1, 1, 1, 1, None, None, None, None,
                           C.byref(nb), None) == G.E_INVALID
    mx_wide = G.gcn_layer(300, 4, 300, 4, G.ACT_RELU, G.ORDER_AUTO, 1, G.AGG_MAX)
    assert L.gcn_layer_fwd(C.byref(g), C.byref(mx_wide), 1, None, 1, 1, 1, 1, None, None, None, None,
                           C.byref(nb), None) == G.E_UNSUPPORTED
    mx = G.gcn_layer(8, 4, 8, 4, G.ACT_RELU, G.ORDER_AUTO, 0, G.AGG_MAX)
    assert L.gcn_layer_order(C.byref(mx), 0) == G.AGGREGATE_FIRST
    assert L.gcn_layer_order(C.byref(mx), 1) == G.AGGREGATE_FIRST
    sxm = G.gcn_sparse_x(10, 8, 5, 1, 1, 1, 1, 1, 1)
    assert L.gcn_layer_fwd(C.byref(g), C.byref(mx), None, C.byref(sxm), 1, 1, 1, 1, None, None, None, None,
                           C.byref(nb), None) == G.E_UNSUPPORTED
    # a max loss layer is allowed (aggregate-first with the softmax epilogue)
    mx_sm = G.gcn_layer(8, 4, 8, 4, G.ACT_SOFTMAX_CE, G.ORDER_AUTO, 1, G.AGG_MAX)
    assert L.gcn_layer_fwd(C.byref(g), C.byref(mx_sm), 1, None, 1, 1, 1, 1, 1, 1, None, None,
                           C.byref(nb), None) == G.OK
    # gcn_aggregate takes the linear aggregators only; the max one has its own calls
    g2 = G.gcn_graph(10, 20, 20, 1, 1, 1, 1, 1)
    assert L.gcn_aggregate(C.byref(g2), G.AGG_MAX, 4, 1, 4, None, 0, None, 0, 1, 4, None, C.byref(nb),
                           None) == G.E_INVALID
    nb.value = 99
    assert L.gcn_aggregate_max(C.byref(g2), 4, 1, 4, 1, 4, 1, 4, None, C.byref(nb), None) == G.OK
    assert nb.value == 0
    assert L.gcn_aggregate_max(C.byref(g2), 300, 1, 300, 1, 300, 1, 300, None, C.byref(nb), None) == G.E_UNSUPPORTED
    assert L.gcn_aggregate_max_bwd(C.byref(g2), 4, 1, 4, 1, 4, None, 0, 1, 3, None, C.byref(nb),
                                   None) == G.E_INVALID
    # backward: sparse input cannot have an input gradient
    sx = G.gcn_sparse_x(10, 8, 5, 1, 1, 1, 1, 1, 1)
    assert L.gcn_layer_bwd(C.byref(g), C.byref(lay), 1, None, C.byref(sx), None, 1, 1, 1, 1, None,
                           C.byref(nb), None) == G.E_INVALID


def test_order_rule(G):
    # aggregate-first iff f_in * (1 + [l > 0]) < 2 f_out, dense input, not the loss layer
    assert G.layer_order(128, 256, 0, G.ACT_RELU) == G.AGGREGATE_FIRST     # arxiv-like layer 0
    assert G.layer_order(100, 256, 0, G.ACT_RELU) == G.AGGREGATE_FIRST     # products-like layer 0
    assert G.layer_order(256, 256, 1, G.ACT_RELU) == G.TRANSFORM_FIRST
    assert G.layer_order(602, 256, 0, G.ACT_RELU) == G.TRANSFORM_FIRST     # reddit-like layer 0
    assert G.layer_order(128, 256, 0, G.ACT_RELU, x_sparse=True) == G.TRANSFORM_FIRST
    assert G.layer_order(16, 700, 1, G.ACT_SOFTMAX_CE) == G.TRANSFORM_FIRST
    assert G.layer_order(128, 256, 0, G.ACT_RELU, order=G.TRANSFORM_FIRST) == G.TRANSFORM_FIRST


def test_epoch_rejects_hidden_layer_without_relu(G):
    """The backward of the layer above a hidden layer multiplies by 1[H > 0], ReLU's
    derivative; gcn_epoch refuses a hidden layer with another activation instead of
    producing wrong gradients.  Returns from host validation / the size query only."""
    L = G.raw_lib()
    n = 10
    g = G.gcn_graph(n, 20, 20, 1, 1, 1, 1, 1)

    def model(hidden_act):
        lays = (G.gcn_layer * 2)(G.gcn_layer(8, 4, 8, 4, hidden_act, G.TRANSFORM_FIRST, 0),
                                 G.gcn_layer(4, 3, 4, 4, G.ACT_SOFTMAX_CE, G.TRANSFORM_FIRST, 1))
        arr = lambda: (C.c_void_p * 2)(256, 512)  # stand-in device addresses, never dereferenced
        keep = {nm: arr() for nm in ("W", "b", "dW", "db", "mW", "vW", "mb", "vb", "act", "saved", "grad")}
        m = G.gcn_model(2, C.cast(lays, C.POINTER(G.gcn_layer)),
                        *[C.cast(keep[nm], C.POINTER(C.c_void_p)) for nm in
                          ("W", "b", "dW", "db", "mW", "vW", "mb", "vb", "act", "saved", "grad")],
                        0.01, 0.9, 0.999, 1e-8, 0, None)
        return m, (lays, keep)

    nb = G.sz(0)
    m, keep = model(G.ACT_NONE)
    assert L.gcn_epoch(C.byref(m), C.byref(g), 1024, None, 2048, 4096, None, C.byref(nb), None) == G.E_UNSUPPORTED
    assert "ReLU" in L.gcn_last_error().decode()
    m, keep = model(G.ACT_RELU)
    assert L.gcn_epoch(C.byref(m), C.byref(g), 1024, None, 2048, 4096, None, C.byref(nb), None) == G.OK
    assert nb.value > 0


def _epoch_ws(G, n, nnz, widths, n_chunk=0):
    """Workspace bytes gcn_epoch asks for (size query only: stand-in device addresses)."""
    L = G.raw_lib()
    nl = len(widths) - 1
    lays = (G.gcn_layer * nl)(*[
        G.gcn_layer(widths[l], widths[l + 1], G.pitch(widths[l]), G.pitch(widths[l + 1]),
                    G.ACT_SOFTMAX_CE if l == nl - 1 else G.ACT_RELU, G.ORDER_AUTO, l) for l in range(nl)])
    keep = {nm: (C.c_void_p * nl)(*[4096 * (i + 1) for i in range(nl)])
            for nm in ("W", "b", "dW", "db", "mW", "vW", "mb", "vb", "act", "saved", "grad")}
    m = G.gcn_model(nl, C.cast(lays, C.POINTER(G.gcn_layer)),
                    *[C.cast(keep[nm], C.POINTER(C.c_void_p)) for nm in
                      ("W", "b", "dW", "db", "mW", "vW", "mb", "vb", "act", "saved", "grad")],
                    0.01, 0.9, 0.999, 1e-8, 0, None)
    sp = G.gcn_split(1 if n_chunk else 0, n_chunk, max(n_chunk, 1), 256 if n_chunk else None,
                     256 if n_chunk else None, 256 if n_chunk else None, None)
    g = G.gcn_graph(n, nnz, nnz, 256, 256, 256, 256, 256, sp)
    nb = G.sz(0)
    rc = L.gcn_epoch(C.byref(m), C.byref(g), 1 << 20, None, 2 << 20, 3 << 20, None, C.byref(nb), None)
    assert rc == G.OK, L.gcn_last_error().decode()
    return nb.value


@pytest.mark.parametrize("widths", [(100, 256, 256, 47), (128, 256, 256, 40), (602, 256, 41)])
def test_epoch_memory_has_no_edge_times_width_term(G, widths):
    """Section V-F / Table III: the fused path keeps device memory at O(|V| F) with no
    per-edge message tensor.  With N and the widths fixed, the epoch workspace must not grow
    with the edge count at all (the graph itself is the caller's, 8 bytes per entry), and the
    chunk sums of split hub rows add at most 1.5 w floats per GCN_SPLIT_CHUNK entries."""
    n = 2_449_029
    base = _epoch_ws(G, n, 10 * n, widths)
    assert _epoch_ws(G, n, 100 * n, widths) == base      # 10x the entries: same workspace
    assert _epoch_ws(G, n, 1000 * n, widths) == base
    # a per-edge message tensor at the widest layer would be nnz * w * 4 bytes; the workspace
    # is a few node-sized matrices
    wmax = max(widths)
    assert base <= 4 * n * 4 * G.pitch(wmax) + (64 << 20)
    assert base < 10 * n * 4 * wmax  # far below one edge-sized message tensor at 10 entries per node
    # hub rows: chunk sums are w floats per chunk of 2048 entries
    nnz = 100 * n
    chunks = 3 * nnz // (2 * 2048) + 1
    with_split = _epoch_ws(G, n, nnz, widths, n_chunk=chunks)
    assert with_split - base <= chunks * 4 * G.pitch(wmax) + 4096
    assert (with_split - base) / nnz <= 1.5 * 4 * G.pitch(wmax) / 2048 + 1e-3


def test_epoch_memory_scales_with_nodes(G):
    """The workspace is linear in N at fixed widths (O(|V| F))."""
    w = (100, 256, 256, 47)
    a, b = _epoch_ws(G, 1_000_000, 50_000_000, w), _epoch_ws(G, 2_000_000, 50_000_000, w)
    c = _epoch_ws(G, 4_000_000, 50_000_000, w)
    assert (c - b) == pytest.approx(2 * (b - a), rel=0.02)


def test_gemm_static_checks_before_any_device_call(G):
    """gcn_gemm_static validates like gcn_gemm and rejects a product whose scratch exceeds the
    static array, both before touching a device."""
    L = G.raw_lib()
    assert L.gcn_gemm_static(9, 4, 4, 4, 1, 4, 1, 4, 1, 4, None, 0, None, 0, None) == G.E_INVALID
    assert L.gcn_gemm_static(G.OP_NN, 4, 4, 8, 1, 4, 1, 4, 1, 4, None, 0, None, 0, None) == G.E_INVALID
    # the row-panel product with a long k: its split weight planes (6 k n bytes) exceed 64 MiB
    m, n, k = 32768, 256, 50000
    nb = G.sz(0)
    assert L.gcn_gemm(G.OP_NN, m, n, k, None, k, None, n, None, n, None, 0, None, 0, None,
                      C.byref(nb), None) == G.OK
    assert nb.value > (64 << 20)
    assert L.gcn_gemm_static(G.OP_NN, m, n, k, 256, k, 256, n, 256, n, None, 0, None, 0, None) == G.E_CAPACITY
    assert "scratch" in L.gcn_last_error().decode()
