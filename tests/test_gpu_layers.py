"""GPU parity of whole layers and epochs against the fp64 oracle, through the C ABI.

Unit parity feeds the oracle the GPU's own layer inputs (so ReLU masks agree)
and compares each output element against its magnitude scale; end-to-end
parity runs the oracle from X alone and compares every tensor in the
infinity norm (max error / max value <= 1e-4).
"""
import numpy as np
import pytest
import torch

import gcn_synth as gs
from helpers import assert_mag_close, assert_norm_close, note, relu_flips

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2512_01678_amd.gcn as G
    return G


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy().astype(np.float64)


def pad(G, a):
    t = G.padded(a.shape[0], a.shape[1])
    t.copy_(dev(a.astype(np.float32)))
    return t


class Problem:
    def __init__(self, G, orc, wl, seed=0):
        self.wl = wl
        s, d = gs.make_graph(wl, seed)
        self.og = orc.build_csr(wl.n, s, d)
        self.dg = G.build_csr(wl.n, dev(s), dev(d))
        self.X = gs.make_features(wl, seed)
        self.y = gs.make_labels(wl, seed)
        self.Ws, self.bs = gs.make_weights(wl, seed)


@pytest.fixture(scope="module")
def small(G, orc):
    wl = gs.scaled(gs.WORKLOADS["arxiv_like"], 6000, 41000, name="arxiv_like_small")
    return Problem(G, orc, wl)


@pytest.fixture(scope="module")
def cora(G, orc):
    return Problem(G, orc, gs.WORKLOADS["cora_like"])


def abs_agg(orc, og, A):
    return orc.aggregate(og, np.abs(A))


# ---------------------------------------------------------------------------
# one layer forward / backward (unit parity)
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("order", ["TF", "AF"])
@pytest.mark.parametrize("fi,fo,act", [(128, 256, "relu"), (256, 40, "softmax"), (100, 256, "relu"),
                                       (41, 47, "none"), (256, 7, "softmax"), (602, 256, "relu"),
                                       (64, 300, "relu"), (33, 5, "none"), (120, 520, "relu"),
                                       (64, 128, "softmax"), (256, 200, "softmax")])
def test_layer_forward(G, orc, small, order, fi, fo, act):
    if order == "AF" and act == "softmax":
        pytest.skip("aggregate-first is never chosen for the loss layer")
    og, dg, n = small.og, small.dg, small.wl.n
    rng = np.random.default_rng(fi + fo)
    H = np.maximum(rng.standard_normal((n, fi)), 0).astype(np.float32)
    W = (rng.standard_normal((fi, fo)) / np.sqrt(fi)).astype(np.float32)
    b = rng.standard_normal(fo).astype(np.float32) * 0.1
    y = rng.integers(0, fo, n).astype(np.int32)
    code = {"relu": G.ACT_RELU, "none": G.ACT_NONE, "softmax": G.ACT_SOFTMAX_CE}[act]
    L = G.make_layer(fi, fo, G.pitch(fi), G.pitch(fo), code, 1,
                     G.TRANSFORM_FIRST if order == "TF" else G.AGGREGATE_FIRST)
    Hd = pad(G, H)
    out = G.padded(n, fo)
    saved = G.padded(n, fi) if order == "AF" else None
    loss = torch.zeros(1, device="cuda")
    logits = G.padded(n, fo) if act == "softmax" else None
    G.layer_fwd(dg, L, Hd, None, dev(W), dev(b), out, saved=saved, labels=dev(y), loss=loss, logits=logits)
    Z = orc.aggregate(og, orc.matmul(H, W), b)
    mag = orc.aggregate(og, orc.matmul(np.abs(H), np.abs(W)), np.abs(b))
    if act == "relu":
        assert_mag_close(host(out), np.maximum(Z, 0), mag, f"fwd {order} {fi}->{fo} relu")
    elif act == "none":
        assert_mag_close(host(out), Z, mag, f"fwd {order} {fi}->{fo}")
    else:
        assert_mag_close(host(logits), Z, mag, "logits")
        lo, Gr, _ = orc.softmax_ce(Z, y)
        assert host(loss)[0] == pytest.approx(lo, rel=1e-4)
        assert_norm_close(host(out), Gr, "softmax-CE gradient")
    if order == "AF":
        P, pmag = orc.aggregate(og, H, want_mag=True)
        assert_mag_close(host(saved), P, pmag, "saved A_hat H")


@pytest.mark.parametrize("fi,fo", [(128, 256), (100, 256), (41, 47), (64, 300)])
def test_aggregate_first_fused_matches_two_launches(G, small, fi, fo, monkeypatch):
    """The fused aggregate-then-transform kernel against the aggregation + GEMM pair:
    the saved aggregate is bit-identical (same accumulation code), the output agrees
    to fp32 rounding (same bf16x6 arithmetic, different grouping of k)."""
    dg, n = small.dg, small.wl.n
    rng = np.random.default_rng(fi * fo)
    H = rng.standard_normal((n, fi)).astype(np.float32)
    W = (rng.standard_normal((fi, fo)) / np.sqrt(fi)).astype(np.float32)
    b = (rng.standard_normal(fo) * 0.1).astype(np.float32)
    L = G.make_layer(fi, fo, G.pitch(fi), G.pitch(fo), G.ACT_RELU, 0, G.AGGREGATE_FIRST)
    res = {}
    for mode in ("1", "0"):
        monkeypatch.setenv("GCN_AF_FUSED", mode)
        out, saved = G.padded(n, fo), G.padded(n, fi)
        G.layer_fwd(dg, L, pad(G, H), None, dev(W), dev(b), out, saved=saved)
        res[mode] = (host(out), host(saved))
    np.testing.assert_array_equal(res["1"][1], res["0"][1])
    scale = np.abs(res["0"][0]).max()
    assert np.abs(res["1"][0] - res["0"][0]).max() <= 1e-5 * scale


@pytest.mark.parametrize("order", ["TF", "AF"])
@pytest.mark.parametrize("fi,fo,first", [(256, 40, False), (128, 256, True), (256, 256, False), (47, 41, False)])
def test_layer_backward(G, orc, small, order, fi, fo, first):
    og, dg, n = small.og, small.dg, small.wl.n
    rng = np.random.default_rng(fi * 3 + fo)
    H = np.maximum(rng.standard_normal((n, fi)), 0).astype(np.float32)
    W = (rng.standard_normal((fi, fo)) / np.sqrt(fi)).astype(np.float32)
    Gr = (rng.standard_normal((n, fo)) / n).astype(np.float32)
    L = G.make_layer(fi, fo, G.pitch(fi), G.pitch(fo), G.ACT_RELU, 0 if first else 1,
                     G.TRANSFORM_FIRST if order == "TF" else G.AGGREGATE_FIRST)
    Hd = pad(G, H)
    saved = None
    if order == "AF":
        saved = G.padded(n, fi)
        G.aggregate(dg, Hd, saved)
    dW = torch.zeros((fi, fo), device="cuda")
    db = torch.zeros(fo, device="cuda")
    Gprev = None if first else G.padded(n, fi)
    G.layer_bwd(dg, L, pad(G, Gr), Hd, None, saved, dev(W), dW, db, Gprev)
    Q = orc.aggregate(og, Gr)
    aQ = abs_agg(orc, og, Gr)
    P = orc.aggregate(og, H)
    if order == "TF":
        dW_ref, dW_mag = orc.matmul(H.T, Q), orc.matmul(np.abs(H).T, aQ)
    else:
        dW_ref, dW_mag = orc.matmul(P.T, Gr), orc.matmul(np.abs(orc.aggregate(og, np.abs(H))).T, np.abs(Gr))
    assert_mag_close(host(dW), dW_ref, dW_mag, f"dW {order}")
    assert_mag_close(host(db), Gr.astype(np.float64).sum(0), np.abs(Gr.astype(np.float64)).sum(0), "db")
    if Gprev is not None:
        ref = orc.matmul(Q, W.T) * (H > 0)
        mag = orc.matmul(aQ, np.abs(W).T)
        assert_mag_close(host(Gprev), ref, mag, f"G_prev {order}")


@pytest.mark.parametrize("xt", ["plain", "tiled"])
def test_layer_sparse_input(G, orc, cora, xt, monkeypatch):
    """xt: the CSC product for dW = X^T Q untiled, or tiled by row chunks (one chunk here)."""
    monkeypatch.setenv("GCN_XT", xt)
    og, dg, n = cora.og, cora.dg, cora.wl.n
    X, W0, b0 = cora.X, cora.Ws[0], cora.bs[0] + 0.05
    info, sx = G.feature_stats(dev(X), tau=(4, 5))
    assert info["mode"] == G.SPARSE
    L = G.make_layer(1433, 16, 1433, G.pitch(16), G.ACT_RELU, 0)
    out = G.padded(n, 16)
    G.layer_fwd(dg, L, None, sx, dev(W0), dev(b0), out)
    Z = orc.aggregate(og, orc.matmul(X, W0), b0)
    mag = orc.aggregate(og, orc.matmul(np.abs(X), np.abs(W0)), np.abs(b0))
    assert_mag_close(host(out), np.maximum(Z, 0), mag, "sparse layer-0 forward")
    Gr = (np.random.default_rng(0).standard_normal((n, 16)) / n).astype(np.float32)
    dW = torch.zeros((1433, 16), device="cuda")
    db = torch.zeros(16, device="cuda")
    G.layer_bwd(dg, L, pad(G, Gr), None, sx, None, dev(W0), dW, db, None)
    Q = orc.aggregate(og, Gr)
    assert_mag_close(host(dW), orc.matmul(X.T, Q), orc.matmul(np.abs(X).T, abs_agg(orc, og, Gr)),
                     "sparse layer-0 dW")


@pytest.mark.parametrize("w", [40, 37, 128])
def test_sparse_weight_gradient_row_chunks(G, orc, w, monkeypatch):
    """dW = X^T Q from the CSC view tiled by row chunks: three full chunks of rows and a
    ragged fourth, an empty feature column, a column with a nonzero in every row, widths
    with and without 16-byte partial rows; against the fp64 product and the untiled form.
    The graph has no edges, so Q = G."""
    n, F = 3 * 8192 + 1234, 700  # the library tiles rows in chunks of 8192
    rng = np.random.default_rng(21)
    X = np.where(rng.random((n, F)) < 0.02, rng.standard_normal((n, F)), 0.0).astype(np.float32)
    X[:, 5] = 0.0
    X[:, 9] = rng.standard_normal(n).astype(np.float32)
    dg = G.build_csr(n, dev(np.zeros(0, np.int32)), dev(np.zeros(0, np.int32)))
    info, sx = G.feature_stats(dev(X), tau=(4, 5))
    assert info["mode"] == G.SPARSE
    L = G.make_layer(F, w, F, G.pitch(w), G.ACT_RELU, 0)
    Gr = (rng.standard_normal((n, w)) / n).astype(np.float32)
    W0 = rng.standard_normal((F, w)).astype(np.float32)
    out = {}
    for xt in ("plain", "tiled"):
        monkeypatch.setenv("GCN_XT", xt)
        dW = torch.zeros((F, w), device="cuda")
        db = torch.zeros(w, device="cuda")
        G.layer_bwd(dg, L, pad(G, Gr), None, sx, None, dev(W0), dW, db, None)
        out[xt] = host(dW)
        # the same product through its own entry point
        C2 = torch.full((F, w), float("nan"), device="cuda")
        G.spmm_xt(sx, dev(Gr), C2)
        out[xt + " (gcn_spmm_xt)"] = host(C2)
        G.spmm_xt(sx, dev(Gr), C2)
        np.testing.assert_array_equal(host(C2), out[xt + " (gcn_spmm_xt)"])  # fixed order
    ref = orc.matmul(X.T, Gr)
    mag = orc.matmul(np.abs(X).T, np.abs(Gr))
    for xt, got in out.items():
        assert_mag_close(got, ref, mag, f"X^T Q ({xt})")
    assert np.all(out["tiled"][5] == 0.0)


@pytest.mark.parametrize("case", ["exact_chunks", "last_chunk_only", "one_row", "no_entries"])
def test_spmm_xt_chunk_edges(G, orc, case, monkeypatch):
    """X_csc^T Q at the edges of the row chunking, plain and tiled: a row count that is an
    exact multiple of the chunk, entries only in the last (ragged) chunk, a single row,
    and an all-zero X (nnz = 0: the result is exactly zero)."""
    rng = np.random.default_rng(23)
    n, F, w = {"exact_chunks": (2 * 8192, 300, 40), "last_chunk_only": (2 * 8192 + 100, 64, 33),
               "one_row": (1, 50, 16), "no_entries": (8192 + 1, 40, 8)}[case]
    X = np.where(rng.random((n, F)) < 0.05, rng.standard_normal((n, F)), 0.0).astype(np.float32)
    if case == "last_chunk_only":
        X[:2 * 8192] = 0.0
    if case == "one_row":
        X[0, ::10] = 1.5
    if case == "no_entries":
        X[:] = 0.0
    info, sx = G.feature_stats(dev(X), tau=(4, 5))
    assert info["mode"] == G.SPARSE and info["nnz"] == np.count_nonzero(X)
    Q = rng.standard_normal((n, w)).astype(np.float32)
    ref = orc.matmul(X.T, Q)
    mag = orc.matmul(np.abs(X).T, np.abs(Q))
    for xt in ("plain", "tiled"):
        monkeypatch.setenv("GCN_XT", xt)
        C2 = torch.full((F, w), float("nan"), device="cuda")
        G.spmm_xt(sx, pad(G, Q), C2)
        got = host(C2)
        assert_mag_close(got, ref, mag, f"X^T Q {case} ({xt})")
        assert np.all(got[np.abs(X).sum(0) == 0] == 0.0)  # empty columns give exact zeros


@pytest.mark.parametrize("w", [128, 100, 37, 16, 8])
def test_sparse_forward_product_shapes(G, orc, w):
    """The forward X_csr W of a sparse first layer (no edges, so the layer output is X W + b),
    in gcn_layer_fwd and through gcn_spmm_xw: 5000 features, empty rows, rows with every
    feature nonzero, a band of features no row touches, widths with and without 16-byte
    rows; against the fp64 product."""
    xw = "gather"
    n, F = 1000, 5000
    rng = np.random.default_rng(31 + w)
    X = np.where(rng.random((n, F)) < 0.1, rng.standard_normal((n, F)), 0.0).astype(np.float32)
    X[:, 4096 + 64:4096 + 128] = 0.0
    X[7] = 0.0
    X[500] = rng.standard_normal(F).astype(np.float32)
    X[999, :4096] = 1.0
    dg = G.build_csr(n, dev(np.zeros(0, np.int32)), dev(np.zeros(0, np.int32)))
    info, sx = G.feature_stats(dev(X), tau=(4, 5))
    assert info["mode"] == G.SPARSE
    W0 = rng.standard_normal((F, w)).astype(np.float32)
    b0 = rng.standard_normal(w).astype(np.float32)
    L = G.make_layer(F, w, F, G.pitch(w), G.ACT_NONE, 0)
    out = G.padded(n, w)
    G.layer_fwd(dg, L, None, sx, dev(W0), dev(b0), out)
    ref = orc.matmul(X, W0) + b0
    mag = orc.matmul(np.abs(X), np.abs(W0)) + np.abs(b0)
    got = host(out)
    assert_mag_close(got, ref, mag, f"X_csr W ({xw}, w = {w})")
    np.testing.assert_array_equal(got[7], b0)  # an empty row is the bias exactly
    again = G.padded(n, w)
    G.layer_fwd(dg, L, None, sx, dev(W0), dev(b0), again)
    np.testing.assert_array_equal(host(again), got)  # fixed order
    # the same product through its own entry point (no bias)
    C2 = torch.full((n, w), float("nan"), device="cuda")
    G.spmm_xw(sx, dev(W0), C2)
    assert_mag_close(host(C2), orc.matmul(X, W0), orc.matmul(np.abs(X), np.abs(W0)), f"gcn_spmm_xw ({xw}, w = {w})")
    assert np.all(host(C2)[7] == 0.0)


# ---------------------------------------------------------------------------
# whole epochs (end-to-end parity, determinism)
# ---------------------------------------------------------------------------


def snapshot(m):
    """The GPU model's parameters and Adam state, widened to fp64 on the host."""
    return {k: [host(t) for t in getattr(m, k)] for k in ("W", "b", "mW", "vW", "mb", "vb")}


AGGS = {"gcn": 0, "sum": 1, "mean": 2, "max": 4}


def gpu_relu_decisions(m, tag, orc, og, X, Ws, bs, aggs=None):
    """The ReLU factor 1[Z_l > 0] of the backward is a decision taken on the fp32
    pre-activation on the GPU and on the fp64 one in the oracle; where Z_l is within
    rounding of zero both are correct, and one flipped entry moves G, dW and db of every
    earlier layer far beyond the comparison tolerance.  The oracle takes the GPU's
    decisions (1[H_{l+1} > 0]), after checking element by element that they agree with
    its own wherever |Z_l| exceeds 1e-5 of the element's magnitude scale (sum |terms|),
    and that the flips near zero are few (counted and reported)."""
    def decide(Zs):
        on = []
        for l in range(m.L - 1):
            Z = Zs[l]
            Hin = np.asarray(X, np.float64) if l == 0 else np.maximum(Zs[l - 1], 0.0)
            Wa, ba = np.abs(np.asarray(Ws[l], np.float64)), np.abs(np.asarray(bs[l], np.float64))
            kind = aggs[l] if aggs else "gcn"
            if kind == "max":
                P, _ = orc.aggregate_max(og, Hin)
                mag = np.abs(P) @ Wa + ba
            else:
                mag = orc.aggregate(og, np.abs(Hin) @ Wa, ba, kind=kind)
            gpu_on = host(m.act[l])[:, :Z.shape[1]] > 0
            relu_flips(gpu_on, Z, mag, f"{tag} layer {l}")
            on.append(gpu_on)
        return on
    return decide


def run_epochs(G, orc, p, epochs, sparse, aggs=None, csc=True):
    """Each epoch: the oracle starts from the GPU's own pre-epoch parameters and Adam
    state, so every epoch is a well-conditioned comparison (Adam's first steps move
    each weight by about lr * sign(g), which would amplify rounding in g if the two
    trajectories were left to run apart)."""
    n = p.wl.n
    Xd = dev(p.X)
    sx = None
    if sparse:
        info, sx = G.feature_stats(Xd, tau=(4, 5), csc=csc)
        assert info["mode"] == G.SPARSE
    m = G.Model(n, p.wl.widths, p.Ws, p.bs, x_sparse=sparse, ld_x=p.wl.f,
                aggs=[AGGS[a] for a in aggs] if aggs else None)
    yd = dev(p.y)
    osx = orc.SparseX(p.X) if sparse else None
    for t in range(1, epochs + 1):
        st = snapshot(m)
        m.epoch(p.dg, X=None if sparse else Xd, x=sx, labels=yd)
        tag = f"{p.wl.name} epoch {t}"
        out = orc.epoch(p.og, p.X, p.y, st["W"], st["b"], st["mW"], st["vW"], st["mb"], st["vb"], t,
                        sparse=osx, aggs=list(aggs) if aggs else None,
                        relu_on=gpu_relu_decisions(m, tag, orc, p.og, p.X, st["W"], st["b"], aggs))
        assert host(m.loss)[0] == pytest.approx(out["loss"], rel=1e-4), tag
        for l in range(m.L):
            assert_norm_close(host(m.grad[l]), out["Gs"][l], f"{tag} G_{l}")
            assert_norm_close(host(m.dW[l]), out["dWs"][l], f"{tag} dW_{l}")
            assert_norm_close(host(m.db[l]), out["dbs"][l], f"{tag} db_{l}")
            if l < m.L - 1:
                assert_norm_close(host(m.act[l]), out["Hs"][l + 1], f"{tag} H_{l + 1}")
            # the Adam step, applied by the oracle to the GPU's own gradients
            for nm, gnm, mnm, vnm in (("W", "dW", "mW", "vW"), ("b", "db", "mb", "vb")):
                want, wm, wv = orc.adam(st[nm][l], host(getattr(m, gnm)[l]), st[mnm][l], st[vnm][l], t)
                assert_mag_close(host(getattr(m, nm)[l]), want, np.abs(st[nm][l]) + 0.01,
                                 f"{tag} Adam {nm}_{l}", rtol=1e-5)
                gg = host(getattr(m, gnm)[l])
                assert_mag_close(host(getattr(m, mnm)[l]), wm, 0.9 * np.abs(st[mnm][l]) + 0.1 * np.abs(gg),
                                 f"{tag} Adam m_{nm}_{l}", rtol=1e-5)
                assert_mag_close(host(getattr(m, vnm)[l]), wv, 0.999 * st[vnm][l] + 0.001 * gg * gg,
                                 f"{tag} Adam v_{nm}_{l}", rtol=1e-5)
    return m


def test_epochs_sparse_path_cora_like(G, orc, cora):
    m = run_epochs(G, orc, cora, 3, sparse=True)
    assert m.step == 3


def test_epochs_sparse_path_atomic_transpose(G, orc, cora):
    """Sparse path without the CSC view: X^T Q by atomic adds from X_csr (Section IV-D)."""
    m = run_epochs(G, orc, cora, 2, sparse=True, csc=False)
    assert m.step == 2


@pytest.mark.parametrize("rows", ["auto", "1"])
def test_epochs_dense_path_aggregate_first(G, orc, small, rows, monkeypatch):
    """rows=1: the row-panel products and the ReLU bitmasks below their automatic threshold."""
    if rows != "auto":
        monkeypatch.setenv("GCN_GEMM_ROWS", rows)
    m = run_epochs(G, orc, small, 2, sparse=False)
    assert m.orders()[0] == G.AGGREGATE_FIRST and m.orders()[1] == G.TRANSFORM_FIRST


# The Reddit-shaped and products-shaped models (Table II widths, the generator's degree
# distribution) on graphs small enough for whole-epoch oracle runs: reddit-like keeps
# a high mean degree (200 here, about 490 at full size) and its 602-wide input makes
# layer 0 transform-first; products-like has the aggregate-first 100-wide layer 0 and a
# 47-class loss.
SHAPED = {
    "reddit_like": (6000, 600000),
    "products_like": (20000, 500000),
}


@pytest.mark.parametrize("name", sorted(SHAPED))
@pytest.mark.parametrize("rows", ["auto", "1"])
def test_epochs_workload_shapes(G, orc, name, rows, monkeypatch):
    """rows=1: the row-panel products used at full size, forced below their automatic
    row threshold."""
    if rows != "auto":
        monkeypatch.setenv("GCN_GEMM_ROWS", rows)
    n, e = SHAPED[name]
    p = Problem(G, orc, gs.scaled(gs.WORKLOADS[name], n, e, name=f"{name}_scaled"))
    m = run_epochs(G, orc, p, 2, sparse=False)
    want = {"reddit_like": [G.TRANSFORM_FIRST, G.TRANSFORM_FIRST],
            "products_like": [G.AGGREGATE_FIRST, G.TRANSFORM_FIRST, G.TRANSFORM_FIRST]}[name]
    assert m.orders() == want


@pytest.fixture(scope="module")
def tiny(G, orc):
    wl = gs.scaled(gs.WORKLOADS["arxiv_like"], 3000, 15000, name="arxiv_like_tiny")
    wl = gs.Workload(wl.name, wl.n, wl.graph, wl.e_und, (48, 24, 16, 8), wl.features, wl.density)
    return Problem(G, orc, wl)


@pytest.fixture(scope="module")
def hubs(G, orc):
    """20,000 nodes with four rows longer than the split threshold, hidden widths 40 and 24
    (bitmask rows of a word and a half, and of a partial word)."""
    wl = gs.Workload("hub_epochs", 20000, "chung_lu", 60000, (48, 40, 24, 8), "normal", 1.0)
    p = Problem.__new__(Problem)
    p.wl = wl
    rng = np.random.default_rng(9)
    s1, d1 = gs.chung_lu(wl.n, 60000, seed=5)
    ss, dd = [s1], [d1]
    for h, k in [(3, 15000), (11, 5000), (12, 4000), (19999, 4200)]:
        ss.append(np.full(k, h, np.int32))
        dd.append(rng.choice(wl.n, k, replace=False).astype(np.int32))
    s, d = np.concatenate(ss), np.concatenate(dd)
    p.og = orc.build_csr(wl.n, s, d)
    p.dg = G.build_csr(wl.n, dev(s), dev(d))
    assert p.dg.n_long >= 3
    p.X = gs.make_features(wl, 0)
    p.y = gs.make_labels(wl, 0)
    p.Ws, p.bs = gs.make_weights(wl, 0)
    return p


def test_epochs_with_hub_rows(G, orc, hubs, monkeypatch):
    """Whole epochs on a graph with split hub rows: the ReLU bitmasks come from the row-panel
    GEMM epilogue (aggregate-first layer 0), the aggregation epilogue including its long-row
    combine (transform-first layer 1), and feed both input-gradient products (row-panel
    products forced below their automatic row threshold)."""
    monkeypatch.setenv("GCN_GEMM_ROWS", "1")
    m = run_epochs(G, orc, hubs, 2, sparse=False)
    assert m.orders() == [G.AGGREGATE_FIRST, G.TRANSFORM_FIRST, G.TRANSFORM_FIRST]


@pytest.mark.parametrize("aggs", [("sum", "mean", "gcn"), ("max", "sum", "mean"), ("mean", "max", "max")])
def test_epochs_other_aggregators(G, orc, tiny, aggs):
    """Whole epochs with sum, mean and max layers (the max loss layer goes through the
    softmax epilogue after its GEMM) against the oracle run from X alone."""
    m = run_epochs(G, orc, tiny, 2, sparse=False, aggs=aggs)
    for l, a in enumerate(aggs):
        if a == "max":
            assert m.orders()[l] == G.AGGREGATE_FIRST


@pytest.mark.parametrize("agg", ["sum", "mean", "max"])
@pytest.mark.parametrize("order", ["TF", "AF"])
def test_aggregator_layer_unit_parity(G, orc, small, agg, order):
    """One hidden layer forward and backward with the GPU's own inputs fed to the oracle."""
    if agg == "max" and order == "TF":
        pytest.skip("a max layer is always aggregate-first")
    og, dg, n = small.og, small.dg, small.wl.n
    fi, fo = 48, 64
    rng = np.random.default_rng(fi + fo + len(agg))
    H = np.maximum(rng.standard_normal((n, fi)), 0).astype(np.float32)
    W = (rng.standard_normal((fi, fo)) / np.sqrt(fi)).astype(np.float32)
    b = (rng.standard_normal(fo) * 0.1).astype(np.float32)
    code = AGGS[agg]
    L = G.make_layer(fi, fo, G.pitch(fi), G.pitch(fo), G.ACT_RELU, 1,
                     G.TRANSFORM_FIRST if order == "TF" else G.AGGREGATE_FIRST, agg=code)
    Hd = pad(G, H)
    out = G.padded(n, fo)
    saved, arg = G.saved_buffer(n, fi, G.pitch(fi), code) if order == "AF" else (None, None)
    G.layer_fwd(dg, L, Hd, None, dev(W), dev(b), out, saved=saved)
    if agg == "max":
        P, oarg = orc.aggregate_max(og, H)
        np.testing.assert_array_equal(host(saved), P)
        np.testing.assert_array_equal(arg.cpu().numpy(), oarg)
        Z, mag = orc.matmul(P, W, want_mag=True)
        Z, mag = Z + b, mag + np.abs(b)
    else:
        Z = orc.aggregate(og, orc.matmul(H, W), b, kind=agg)
        mag = orc.aggregate(og, orc.matmul(np.abs(H), np.abs(W)), np.abs(b), kind=agg)
    assert_mag_close(host(out), np.maximum(Z, 0), mag, f"{agg} {order} forward")
    Gr = (rng.standard_normal((n, fo)) / n).astype(np.float32)
    dW = torch.zeros((fi, fo), device="cuda")
    db = torch.zeros(fo, device="cuda")
    Gprev = G.padded(n, fi)
    G.layer_bwd(dg, L, pad(G, Gr), Hd, None, saved, dev(W), dW, db, Gprev)
    T, Tm = orc.matmul(Gr, W.T, want_mag=True)
    if agg == "max":
        assert_mag_close(host(dW), orc.matmul(P.T, Gr), orc.matmul(np.abs(P).T, np.abs(Gr)), "max dW")
        want = orc.aggregate_max_backward(og, T, oarg) * (H > 0)
        wmag = orc.aggregate_max_backward(og, Tm, oarg) * (H > 0)
    else:
        tk = orc.TRANSPOSE[agg]
        Q = orc.aggregate(og, Gr, kind=tk)
        Qm = orc.aggregate(og, np.abs(Gr), kind=tk)
        assert_mag_close(host(dW), orc.matmul(H.T, Q), orc.matmul(np.abs(H).T, Qm), f"{agg} dW")
        want = orc.matmul(Q, W.T) * (H > 0)
        wmag = orc.matmul(Qm, np.abs(W).T) * (H > 0)
    assert_mag_close(host(db), Gr.astype(np.float64).sum(0), np.abs(Gr).astype(np.float64).sum(0), f"{agg} db")
    assert_mag_close(host(Gprev), want, wmag, f"{agg} {order} G_prev")


def test_epochs_forced_dense_on_sparse_features(G, orc, cora):
    run_epochs(G, orc, cora, 2, sparse=False)


def test_epoch_bitwise_deterministic(G, small):
    p = small
    outs = []
    for _ in range(2):
        m = G.Model(p.wl.n, p.wl.widths, p.Ws, p.bs)
        for _ in range(3):
            m.epoch(p.dg, X=dev(p.X), labels=dev(p.y))
        torch.cuda.synchronize()
        outs.append([t.clone() for t in m.W + m.b + [m.loss]])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_epoch_column_groups_are_exact(G, small, monkeypatch):
    """The short-k input gradient (width 40 -> 256, with the bitmask and the fused bias
    gradient) split over two column groups gives bitwise the same epoch as one group."""
    monkeypatch.setenv("GCN_GEMM_ROWS", "1")
    p = small
    outs = []
    for groups in ("auto", "1"):
        monkeypatch.setenv("GCN_ROWS_GROUPS", groups)
        m = G.Model(p.wl.n, p.wl.widths, p.Ws, p.bs)
        for _ in range(2):
            m.epoch(p.dg, X=dev(p.X), labels=dev(p.y))
        torch.cuda.synchronize()
        outs.append([t.clone() for t in m.W + m.b + m.dW + m.db + [m.loss]])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


@pytest.mark.parametrize("rows", ["auto", "1"])
def test_epoch_prep_is_exact(G, small, rows, monkeypatch):
    """The epoch's weight split at its start (one launch for every row-panel product) and
    the last bias gradient taken from the loss pass are rearrangements of the same
    arithmetic: parameters, Adam moments and loss stay bitwise equal with them switched off
    (rows=1 makes the products take the row-panel kernel at this size)."""
    if rows != "auto":
        monkeypatch.setenv("GCN_GEMM_ROWS", rows)
    p = small
    outs = []
    for prep in ("1", "0"):
        monkeypatch.setenv("GCN_EPOCH_PREP", prep)
        m = G.Model(p.wl.n, p.wl.widths, p.Ws, p.bs)
        for _ in range(3):
            m.epoch(p.dg, X=dev(p.X), labels=dev(p.y))
        torch.cuda.synchronize()
        outs.append([t.clone() for t in m.W + m.b + m.mW + m.vW + m.mb + m.vb + m.dW + m.db + [m.loss]])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


# ---------------------------------------------------------------------------
# the RMAT workload's feature recipe on a small RMAT graph
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("xt", ["plain", "tiled"])
def test_epoch_rmat_4096_features_sparse(G, orc, xt, monkeypatch):
    """RMAT graph with 4096-wide nonnegative features at 10 % density (the RMAT workload's
    recipe on 2^14 nodes): sparse path chosen by the probe, one epoch against the oracle;
    xt: the untiled or the row-chunk-tiled CSC product for dW_0 (two chunks here)."""
    monkeypatch.setenv("GCN_XT", xt)
    from gcn_synth import device
    wl = gs.Workload("rmat14_p0.1", 1 << 14, "rmat", 1 << 18, (4096, 128, 32), "nonneg", 0.1, rmat_scale=14)
    s, d = gs.rmat(14, 1 << 18)
    n = wl.n
    Xd = torch.zeros((n, 4096), device="cuda")
    device.bernoulli_into(Xd, 0.1, seed=0, stream=3)
    X = gs.features_bernoulli(n, 4096, 0.1, seed=0, stream=3, binary=False)
    np.testing.assert_array_equal(host(Xd).astype(np.float32), X)
    info, sx = G.feature_stats(Xd, tau=(4, 5))
    assert info["mode"] == G.SPARSE
    p = Problem.__new__(Problem)
    p.wl, p.og, p.dg = wl, orc.build_csr(n, s, d), G.build_csr(n, dev(s), dev(d))
    p.X, p.y = X, gs.labels(n, 32)
    p.Ws, p.bs = gs.make_weights(wl)
    run_epochs(G, orc, p, 1, sparse=True)


@pytest.mark.parametrize("density", [0.5, 0.01, 0.001])
def test_epoch_rmat_4096_features_densities(G, orc, density):
    """The rest of the RMAT sweep's densities on 2^14 nodes: the probe picks the dense
    path at 50 % and the sparse one below; one epoch against the oracle."""
    from gcn_synth import device
    wl = gs.Workload(f"rmat14_p{density}", 1 << 14, "rmat", 1 << 18, (4096, 128, 32), "nonneg", density,
                     rmat_scale=14)
    s, d = gs.rmat(14, 1 << 18)
    n = wl.n
    Xd = torch.zeros((n, 4096), device="cuda")
    device.bernoulli_into(Xd, density, seed=0, stream=3)
    X = gs.features_bernoulli(n, 4096, density, seed=0, stream=3, binary=False)
    info, sx = G.feature_stats(Xd, tau=(4, 5))
    assert info["nnz"] == np.count_nonzero(X)
    sparse = density < 0.2
    assert info["mode"] == (G.SPARSE if sparse else G.DENSE)
    p = Problem.__new__(Problem)
    p.wl, p.og, p.dg = wl, orc.build_csr(n, s, d), G.build_csr(n, dev(s), dev(d))
    p.X, p.y = X, gs.labels(n, 32)
    p.Ws, p.bs = gs.make_weights(wl)
    run_epochs(G, orc, p, 1, sparse=sparse)


# ---------------------------------------------------------------------------
# degenerate cases of the method
# ---------------------------------------------------------------------------


def edge_problem(G, orc, case):
    rng = np.random.default_rng(17)
    if case == "no_edges":          # A_hat = I: the GCN is an MLP
        n, widths = 500, (8, 6, 3)
        s = d = np.zeros(0, np.int32)
    elif case == "single_node":
        n, widths = 1, (4, 3, 2)
        s = d = np.zeros(0, np.int32)
    elif case == "width1":          # a one-unit hidden layer
        n, widths = 300, (5, 1, 4)
        s, d = gs.chung_lu(n, 900, seed=4)
    else:                           # all-zero features: s = 1, sparse path with nnz(X) = 0
        n, widths = 400, (50, 7, 3)
        s, d = gs.chung_lu(n, 1500, seed=6)
    p = Problem.__new__(Problem)
    p.wl = gs.Workload(case, n, "chung_lu", s.size, widths, "normal")
    p.og, p.dg = orc.build_csr(n, s, d), G.build_csr(n, dev(s), dev(d))
    X = rng.standard_normal((n, widths[0])).astype(np.float32)
    if case == "zero_features":
        X[:] = 0.0
    p.X = X
    p.y = rng.integers(0, widths[-1], n).astype(np.int32)
    p.Ws = [(rng.standard_normal((widths[l], widths[l + 1])) * 0.6).astype(np.float32) for l in range(len(widths) - 1)]
    p.bs = [(rng.standard_normal(widths[l + 1]) * 0.2).astype(np.float32) for l in range(len(widths) - 1)]
    return p


@pytest.mark.parametrize("case", ["no_edges", "single_node", "width1", "zero_features"])
def test_epoch_degenerate_cases(G, orc, case):
    p = edge_problem(G, orc, case)
    if case == "no_edges":
        assert p.dg.nnz == p.wl.n
    run_epochs(G, orc, p, 2, sparse=(case == "zero_features"))


# ---------------------------------------------------------------------------
# one epoch captured in a HIP graph and replayed
# ---------------------------------------------------------------------------


def test_hip_graph_replay_matches_eager(G, small):
    p = small
    n = p.wl.n
    Xd, yd = dev(p.X), dev(p.y)
    eager = G.Model(n, p.wl.widths, p.Ws, p.bs, device_step=True)
    graphed = G.Model(n, p.wl.widths, p.Ws, p.bs, device_step=True)
    graphed.prepare(p.dg, X=Xd, labels=yd)
    torch.cuda.synchronize()
    cg = torch.cuda.CUDAGraph()
    with torch.cuda.graph(cg):
        graphed.epoch_captured(p.dg, X=Xd, labels=yd)
    torch.cuda.synchronize()
    for it in range(3):
        cg.replay()
        eager.epoch(p.dg, X=Xd, labels=yd)
        _ = (Xd * 2.0).sum().item()     # unrelated eager work between replays
        torch.cuda.synchronize()
        for a, b in zip(graphed.W + graphed.b + graphed.mW + graphed.vW + [graphed.loss],
                        eager.W + eager.b + eager.mW + eager.vW + [eager.loss]):
            assert torch.equal(a, b), f"replay {it}"
    assert graphed.step == eager.step == 3


def test_epoch_graph_replays_match_eager(G, small):
    """An epoch captured in a HIP graph replayed three times, with eager work between the
    replays, against an identical model stepped eagerly: equal bit for bit each time."""
    p = small
    n = p.wl.n
    Xd, yd = dev(p.X), dev(p.y)
    a = G.Model(n, p.wl.widths, p.Ws, p.bs, device_step=True)
    b = G.Model(n, p.wl.widths, p.Ws, p.bs, device_step=True)
    a.prepare(p.dg, X=Xd, labels=yd)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        a.epoch_captured(p.dg, X=Xd, labels=yd)
    torch.cuda.synchronize()
    for r in range(3):
        graph.replay()
        b.epoch(p.dg, X=Xd, labels=yd)
        torch.cuda.synchronize()
        for x, y in zip(a.W + a.b + a.dW + a.db, b.W + b.b + b.dW + b.db):
            np.testing.assert_array_equal(host(x), host(y), err_msg=f"replay {r}")
        np.testing.assert_array_equal(host(a.loss), host(b.loss))
        filler = torch.randn(4096, device="cuda")  # eager work between replays
        assert torch.isfinite(filler.sum())


def test_device_step_matches_host_step(G, small):
    p = small
    n = p.wl.n
    Xd, yd = dev(p.X), dev(p.y)
    a = G.Model(n, p.wl.widths, p.Ws, p.bs, device_step=True)
    b = G.Model(n, p.wl.widths, p.Ws, p.bs)
    for _ in range(3):
        a.epoch(p.dg, X=Xd, labels=yd)
        b.epoch(p.dg, X=Xd, labels=yd)
    torch.cuda.synchronize()
    for x, y in zip(a.W + a.b, b.W + b.b):
        np.testing.assert_allclose(host(x), host(y), rtol=1e-6, atol=1e-9)
    assert a.step == b.step == 3
