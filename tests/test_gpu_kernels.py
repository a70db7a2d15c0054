"""GPU parity of the individual steps against the fp64 oracle, through the C ABI.

Integer / index work (CSR build, degrees, dinv, nonzero counts, compressed
feature views) must match bit for bit; fp32 results must stay within 1e-4 of
the oracle relative to each element's magnitude scale (sum of |terms|).
"""
import numpy as np
import pytest
import torch

import gcn_synth as gs
from helpers import adversarial_graphs, assert_mag_close, messy

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
    return t.detach().cpu().numpy()


def pitched(a, ld):
    """Device copy of a (rows x w) with row pitch ld (extra columns filled with NaN)."""
    rows, w = a.shape
    buf = torch.full((rows, ld), float("nan"), dtype=torch.float32, device="cuda")
    buf[:, :w] = dev(a.astype(np.float32))
    return buf[:, :w]


# ---------------------------------------------------------------------------
# a1: A + I in CSR
# ---------------------------------------------------------------------------


def check_graph_equal(dg, og, n):
    assert dg.nnz == og.nnz
    np.testing.assert_array_equal(host(dg.row_ptr), og.row_ptr)
    np.testing.assert_array_equal(host(dg.col_idx)[:og.nnz], og.col_idx)
    np.testing.assert_array_equal(host(dg.deg)[:n], og.deg)
    np.testing.assert_array_equal(host(dg.dinv)[:n].view(np.int32), og.dinv.view(np.int32))
    # stored entries of A_hat: fl32(dinv[i] * dinv[j]), one IEEE rounding
    rows = np.repeat(np.arange(n), np.diff(og.row_ptr))
    want = og.dinv[rows] * og.dinv[og.col_idx]
    assert want.dtype == np.float32
    np.testing.assert_array_equal(host(dg.val)[:og.nnz].view(np.int32), want.view(np.int32))


@pytest.mark.parametrize("case", adversarial_graphs(), ids=lambda c: c[0])
def test_build_csr_bit_exact(G, orc, case):
    name, n, s, d = case
    print(f"[csr] {name} n={n} edges={s.size}", flush=True)
    check_graph_equal(G.build_csr(n, dev(s), dev(d)), orc.build_csr(n, s, d), n)


@pytest.mark.parametrize("name", ["cora_like", "arxiv_like"])
def test_build_csr_workloads(G, orc, name):
    wl = gs.WORKLOADS[name]
    s, d = gs.make_graph(wl)
    print(f"[csr] {name} n={wl.n} edges={s.size}", flush=True)
    check_graph_equal(G.build_csr(wl.n, dev(s), dev(d)), orc.build_csr(wl.n, s, d), wl.n)


def test_build_csr_rmat_small(G, orc):
    s, d = gs.rmat(14, 1 << 18)
    check_graph_equal(G.build_csr(1 << 14, dev(s), dev(d)), orc.build_csr(1 << 14, s, d), 1 << 14)


def test_build_csr_rejects_out_of_range(G):
    s = np.array([0, 1, 5], np.int32)
    d = np.array([1, 2, 0], np.int32)
    with pytest.raises(G.GcnError) as ei:
        G.build_csr(5, dev(s), dev(d))
    assert ei.value.status == G.E_RANGE
    with pytest.raises(G.GcnError):
        G.build_csr(5, dev(np.array([-1], np.int32)), dev(np.array([0], np.int32)))


# ---------------------------------------------------------------------------
# a2: density probe, decision, X_csr / X_csc
# ---------------------------------------------------------------------------


def feature_cases():
    rng = np.random.default_rng(77)
    special = rng.standard_normal((50, 70)).astype(np.float32)
    special[rng.random((50, 70)) < 0.6] = 0.0
    special[3, 4] = -0.0
    special[5, 6] = np.nan
    special[7, 8] = np.inf
    special[9, :] = 0.0
    thr = np.zeros((40, 25), np.float32)
    thr.flat[: 40 * 25 // 5] = 1.5
    rng.shuffle(thr.reshape(-1))
    return [
        ("cora_like", gs.make_features(gs.WORKLOADS["cora_like"])),
        ("nonneg10", gs.features_bernoulli(2500, 4096, 0.1, binary=False)),
        ("nonneg0.1", gs.features_bernoulli(3000, 1000, 0.001, binary=False)),
        ("special", special),
        ("zeros", np.zeros((33, 17), np.float32)),
        ("ones", np.ones((33, 17), np.float32)),
        ("identity", np.eye(64, 40, dtype=np.float32)),
        ("threshold", thr),
        ("one_col", (rng.random((1100, 1)) < 0.5).astype(np.float32)),
        ("f65", (rng.random((2100, 65)) < 0.2).astype(np.float32) * 2.0),
    ]


@pytest.mark.parametrize("case", feature_cases(), ids=lambda c: c[0])
def test_feature_stats_bit_exact(G, orc, case):
    name, X = case
    n, f = X.shape
    print(f"[features] {name} {n}x{f}", flush=True)
    nnz, rn = orc.feature_counts(X)
    mode = orc.sparse_decision(nnz, n, f)
    Xd = pitched(X, G.pitch(f) + 4)
    rnd = torch.zeros(n, dtype=torch.int64, device="cuda")
    info, sx = G.feature_stats(Xd, tau=(4, 5), materialize=True, row_nnz=rnd)
    assert info["nnz"] == nnz and info["mode"] == mode
    assert info["sparsity"] == pytest.approx(orc.sparsity(nnz, n, f), abs=1e-15)
    np.testing.assert_array_equal(host(rnd), rn)
    rp, col, val = orc.dense_to_csr(X)
    np.testing.assert_array_equal(host(sx.row_ptr), rp)
    np.testing.assert_array_equal(host(sx.col)[:nnz], col)
    np.testing.assert_array_equal(host(sx.val)[:nnz].view(np.int32), val.view(np.int32))
    cp, row, cval = orc.dense_to_csc(X)
    np.testing.assert_array_equal(host(sx.col_ptr), cp)
    np.testing.assert_array_equal(host(sx.row)[:nnz], row)
    np.testing.assert_array_equal(host(sx.cval)[:nnz].view(np.int32), cval.view(np.int32))


def test_feature_decision_tau_and_force(G, orc):
    X = np.zeros((40, 25), np.float32)
    X.flat[: 40 * 25 // 5 + 1] = 1.0
    info, _ = G.feature_stats(dev(X), tau=(4, 5), materialize=False)
    assert info["mode"] == G.DENSE
    info, _ = G.feature_stats(dev(X), tau=(3, 4), materialize=False)
    assert info["mode"] == G.SPARSE
    info, _ = G.feature_stats(dev(X), force_mode=G.SPARSE, materialize=False)
    assert info["mode"] == G.SPARSE
    # the default threshold, measured on this GPU: tau = 15/16, sparse iff nnz <= N F / 16
    assert G.TAU_MI355X == (15, 16)
    Y = np.zeros((64, 50), np.float32)
    Y.flat[: 64 * 50 // 16] = 2.0
    info, _ = G.feature_stats(dev(Y), materialize=False)
    assert info["mode"] == G.SPARSE and orc.sparse_decision(info["nnz"], 64, 50, 15, 16) == G.SPARSE
    Y.flat[64 * 50 // 16] = 2.0
    info, _ = G.feature_stats(dev(Y), materialize=False)
    assert info["mode"] == G.DENSE and orc.sparse_decision(info["nnz"], 64, 50, 15, 16) == G.DENSE


# ---------------------------------------------------------------------------
# a4 / a7: normalised aggregation (all widths, both pitches, epilogues)
# ---------------------------------------------------------------------------

WIDTHS = [1, 2, 3, 4, 5, 7, 8, 15, 16, 17, 31, 32, 33, 40, 41, 47, 63, 64, 65, 100, 127, 128, 129,
          256, 257, 602]


@pytest.fixture(scope="module")
def agg_graph(G, orc):
    rng = np.random.default_rng(5)
    s1, d1 = gs.chung_lu(3000, 20000, seed=3)
    s2 = np.zeros(5000, np.int32) + 7
    d2 = rng.integers(0, 3000, 5000).astype(np.int32)     # one hub of degree ~2600
    s = np.concatenate([s1, s2])
    d = np.concatenate([d1, d2])
    return orc.build_csr(3000, s, d), G.build_csr(3000, dev(s), dev(d))


@pytest.mark.parametrize("w", WIDTHS)
@pytest.mark.parametrize("vec", [True, False])
def test_aggregate_widths(G, orc, agg_graph, w, vec):
    og, dg = agg_graph
    rng = np.random.default_rng(w)
    n = og.n
    M = rng.standard_normal((n, w)).astype(np.float32)
    b = rng.standard_normal(w).astype(np.float32)
    ld = G.pitch(w) if vec else w
    Md = pitched(M, ld)
    Zd = pitched(np.zeros((n, w), np.float32), ld)
    mask = rng.standard_normal((n, w)).astype(np.float32)
    Z, mag = orc.aggregate(og, M, b, want_mag=True)
    for epi in (G.EPI_NONE, G.EPI_RELU, G.EPI_MASK):
        G.aggregate(dg, Md, Zd, bias=dev(b), epi=epi, mask=pitched(mask, ld) if epi == G.EPI_MASK else None)
        want = Z if epi == G.EPI_NONE else (np.maximum(Z, 0) if epi == G.EPI_RELU else Z * (mask > 0))
        assert_mag_close(host(Zd), want, mag, f"aggregate w={w} ld={ld} epi={epi}")
    # padding columns were never written
    if ld > w:
        assert torch.isnan(Zd.as_strided((n, ld), (ld, 1))[:, w:]).all()


@pytest.fixture(scope="module")
def dense_rows_graph(G, orc):
    """Mean degree about 90: slices of 16 and 32 lanes take more than 8 entries of an
    average row, so the aggregation keeps 16 neighbour loads in flight per lane."""
    s, d = gs.chung_lu(2000, 90000, seed=4)
    return orc.build_csr(2000, s, d), G.build_csr(2000, dev(s), dev(d))


@pytest.mark.parametrize("w", [33, 40, 47, 64, 65, 100, 128])
def test_aggregate_widths_long_rows(G, orc, dense_rows_graph, w):
    og, dg = dense_rows_graph
    assert og.nnz / og.n > 64
    rng = np.random.default_rng(100 + w)
    n = og.n
    M = rng.standard_normal((n, w)).astype(np.float32)
    b = rng.standard_normal(w).astype(np.float32)
    ld = G.pitch(w)
    Md = pitched(M, ld)
    Zd = pitched(np.zeros((n, w), np.float32), ld)
    mask = rng.standard_normal((n, w)).astype(np.float32)
    Z, mag = orc.aggregate(og, M, b, want_mag=True)
    for epi in (G.EPI_NONE, G.EPI_RELU, G.EPI_MASK):
        G.aggregate(dg, Md, Zd, bias=dev(b), epi=epi, mask=pitched(mask, ld) if epi == G.EPI_MASK else None)
        want = Z if epi == G.EPI_NONE else (np.maximum(Z, 0) if epi == G.EPI_RELU else Z * (mask > 0))
        assert_mag_close(host(Zd), want, mag, f"aggregate long rows w={w} epi={epi}")


def test_aggregate_no_bias_deterministic(G, orc, agg_graph):
    og, dg = agg_graph
    M = np.random.default_rng(0).standard_normal((og.n, 256)).astype(np.float32)
    Md = dev(M)
    a = torch.empty_like(Md)
    b = torch.empty_like(Md)
    G.aggregate(dg, Md, a)
    G.aggregate(dg, Md, b)
    assert torch.equal(a, b)
    Z, mag = orc.aggregate(og, M, want_mag=True)
    assert_mag_close(host(a), Z, mag, "aggregate w=256 no bias")


# ---------------------------------------------------------------------------
# a3 (sparse), a8 (sparse): X_csr W and X_csc Q
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("f,w,p", [(1433, 16, 0.013), (4096, 128, 0.01), (500, 7, 0.2), (300, 33, 0.05)])
def test_sparse_feature_products(G, orc, f, w, p):
    n = 2708
    X = gs.features_bernoulli(n, f, p, seed=1, binary=False)
    rng = np.random.default_rng(f)
    W = rng.standard_normal((f, w)).astype(np.float32)
    Q = rng.standard_normal((n, w)).astype(np.float32)
    _, sx = G.feature_stats(dev(X), materialize=True)
    out = torch.empty((n, w), dtype=torch.float32, device="cuda")
    G.spmm(sx.row_ptr, sx.col[:sx.nnz], sx.val[:sx.nnz], dev(W), out)
    rp, col, val = orc.dense_to_csr(X)
    ref, mag = orc.spmm(rp, col, val, W, want_mag=True)
    assert_mag_close(host(out), ref, mag, f"X_csr W f={f} w={w}")
    dW = torch.empty((f, w), dtype=torch.float32, device="cuda")
    G.spmm(sx.col_ptr, sx.row[:sx.nnz], sx.cval[:sx.nnz], dev(Q), dW)
    cp, row, cval = orc.dense_to_csc(X)
    ref, mag = orc.spmm(cp, row, cval, Q, want_mag=True)
    assert_mag_close(host(dW), ref, mag, f"X_csc Q f={f} w={w}")


# ---------------------------------------------------------------------------
# a3 / a5 / a8 / a9: matrix-core GEMMs
# ---------------------------------------------------------------------------

GEMM_SHAPES = [(1000, 256, 128), (1000, 40, 256), (777, 47, 256), (513, 7, 16), (300, 128, 602),
               (333, 256, 256), (65, 16, 1433), (2049, 41, 41), (1, 1, 1), (100, 300, 5)]


@pytest.mark.parametrize("op", ["NN", "NT", "TN"])
@pytest.mark.parametrize("shape", GEMM_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_gemm(G, op, shape):
    m, n, k = shape
    rng = np.random.default_rng(m * 7 + n * 3 + k)
    A = rng.standard_normal((m, k)).astype(np.float32)
    B = rng.standard_normal((k, n)).astype(np.float32)
    bias = rng.standard_normal(n).astype(np.float32)
    mask = rng.standard_normal((m, n)).astype(np.float32)
    ref = A.astype(np.float64) @ B.astype(np.float64)
    mag = np.abs(A.astype(np.float64)) @ np.abs(B.astype(np.float64))
    if op == "NN":
        Ad, Bd, code = pitched(A, G.pitch(k) + 4), pitched(B, G.pitch(n)), G.OP_NN
    elif op == "NT":
        Ad, Bd, code = pitched(A, k), pitched(np.ascontiguousarray(B.T), G.pitch(k)), G.OP_NT
    else:
        Ad, Bd, code = pitched(np.ascontiguousarray(A.T), G.pitch(m)), pitched(B, n), G.OP_TN
    C = pitched(np.zeros((m, n), np.float32), G.pitch(n) + 8)
    G.gemm(code, Ad, Bd, C, bias=dev(bias))
    assert_mag_close(host(C), ref + bias, mag + np.abs(bias), f"gemm {op} {shape}")
    if op != "TN":
        G.gemm(code, Ad, Bd, C, bias=dev(bias), epi=G.EPI_RELU)
        assert_mag_close(host(C), np.maximum(ref + bias, 0), mag + np.abs(bias), f"gemm {op} relu")
        G.gemm(code, Ad, Bd, C, epi=G.EPI_MASK, mask=dev(mask))
        assert_mag_close(host(C), ref * (mask > 0), mag, f"gemm {op} mask")


def test_gemm_huge_pitch(G):
    """Operands whose pitch is too large for 32-bit tile offsets (the fp32-mode fallback)."""
    rng = np.random.default_rng(5)
    m, n, k, ld = 3, 40, 70, (1 << 21) + 4
    A = rng.standard_normal((m, k)).astype(np.float32)
    B = rng.standard_normal((k, n)).astype(np.float32)
    Ad = pitched(A, ld)
    C = torch.empty((m, n), dtype=torch.float32, device="cuda")
    G.gemm(G.OP_NN, Ad, dev(B), C)
    ref = A.astype(np.float64) @ B.astype(np.float64)
    mag = np.abs(A.astype(np.float64)) @ np.abs(B.astype(np.float64))
    assert_mag_close(host(C), ref, mag, "gemm NN huge pitch")


@pytest.mark.parametrize("m,n,k", [(128, 256, 169343), (256, 40, 50000), (100, 256, 70001), (602, 41, 20000),
                                   (4096, 128, 4000), (16, 7, 2708)])
def test_gemm_tn_long_reduction(G, m, n, k):
    rng = np.random.default_rng(k)
    A = rng.standard_normal((k, m)).astype(np.float32)
    B = rng.standard_normal((k, n)).astype(np.float32)
    ref = A.T.astype(np.float64) @ B.astype(np.float64)
    mag = np.abs(A.T.astype(np.float64)) @ np.abs(B.astype(np.float64))
    C = torch.empty((m, n), dtype=torch.float32, device="cuda")
    G.gemm(G.OP_TN, dev(A), dev(B), C)
    C1 = host(C).copy()
    assert_mag_close(C1, ref, mag, f"gemm TN {m}x{n}x{k}")
    G.gemm(G.OP_TN, dev(A), dev(B), C)
    np.testing.assert_array_equal(host(C), C1)  # fixed-order split-k reduction


# Row-panel products (A B, A B^T with n <= 256, m >= 128, no mask): every column-tile count
# 1..8 (and so every A prefetch depth), partial and single k slabs, ragged row blocks; the
# masked product of the same operands runs on the tiled kernel.
ROWS_CASES = [(256, 1, 5), (1000, 33, 32), (4099, 64, 40), (777, 65, 256), (300, 100, 602), (2048, 130, 64),
              (513, 190, 100), (1500, 220, 17), (1025, 256, 256), (600, 256, 33)]


@pytest.mark.parametrize("op", ["NN", "NT"])
@pytest.mark.parametrize("shape", ROWS_CASES, ids=lambda s: "x".join(map(str, s)))
def test_gemm_row_panels(G, op, shape, monkeypatch):
    monkeypatch.setenv("GCN_GEMM_ROWS", "1")  # below the automatic row threshold
    m, n, k = shape
    rng = np.random.default_rng(m + 3 * n + 7 * k)
    A = (rng.standard_normal((m, k)) * np.exp(rng.standard_normal((m, 1)))).astype(np.float32)
    B = rng.standard_normal((k, n)).astype(np.float32)
    bias = rng.standard_normal(n).astype(np.float32)
    mask = rng.standard_normal((m, n)).astype(np.float32)
    ref = A.astype(np.float64) @ B.astype(np.float64)
    mag = np.abs(A.astype(np.float64)) @ np.abs(B.astype(np.float64))
    Ad = pitched(A, G.pitch(k))
    Bd = pitched(B, n) if op == "NN" else pitched(np.ascontiguousarray(B.T), k)
    code = G.OP_NN if op == "NN" else G.OP_NT
    C = pitched(np.full((m, n), np.nan, np.float32), G.pitch(n) + 4)
    G.gemm(code, Ad, Bd, C, bias=dev(bias))
    C1 = host(C).copy()
    assert_mag_close(C1, ref + bias, mag + np.abs(bias), f"rows {op} {shape}")
    G.gemm(code, Ad, Bd, C, bias=dev(bias))
    np.testing.assert_array_equal(host(C), C1)  # fixed summation order
    G.gemm(code, Ad, Bd, C, bias=dev(bias), epi=G.EPI_RELU)
    assert_mag_close(host(C), np.maximum(ref + bias, 0), mag + np.abs(bias), f"rows {op} relu")
    G.gemm(code, Ad, Bd, C, epi=G.EPI_MASK, mask=dev(mask))
    assert_mag_close(host(C), ref * (mask > 0), mag, f"rows {op} mask")


@pytest.mark.parametrize("op", ["NN", "NT"])
@pytest.mark.parametrize("shape", [(600, 256, 33), (4099, 250, 40), (300, 226, 64), (1025, 256, 256), (777, 240, 130)],
                         ids=lambda s: "x".join(map(str, s)))
def test_gemm_row_panels_column_groups(G, op, shape, monkeypatch):
    """Few row panels: the 8 column tiles go to two workgroups of 4; every output element keeps
    its summation order, so the result equals the one-group launch bit for bit."""
    monkeypatch.setenv("GCN_GEMM_ROWS", "1")
    m, n, k = shape
    rng = np.random.default_rng(m + n + k)
    A = rng.standard_normal((m, k)).astype(np.float32)
    B = rng.standard_normal((k, n)).astype(np.float32)
    bias = rng.standard_normal(n).astype(np.float32)
    Ad = pitched(A, G.pitch(k))
    Bd = pitched(B, n) if op == "NN" else pitched(np.ascontiguousarray(B.T), k)
    code = G.OP_NN if op == "NN" else G.OP_NT
    out = []
    for groups in ("auto", "1"):
        if groups == "1":
            monkeypatch.setenv("GCN_ROWS_GROUPS", "1")
        C = pitched(np.full((m, n), np.nan, np.float32), G.pitch(n))
        G.gemm(code, Ad, Bd, C, bias=dev(bias), epi=G.EPI_RELU)
        out.append(host(C).copy())
    ref = np.maximum(A.astype(np.float64) @ B.astype(np.float64) + bias, 0)
    mag = np.abs(A.astype(np.float64)) @ np.abs(B.astype(np.float64)) + np.abs(bias)
    assert_mag_close(out[0], ref, mag, f"column groups {op} {shape}")
    np.testing.assert_array_equal(out[0], out[1])


@pytest.mark.parametrize("op,n,k,epi", [("NN", 256, 256, "none"), ("NT", 256, 256, "mask"), ("NN", 40, 256, "none"),
                                        ("NT", 256, 40, "mask"), ("NN", 256, 128, "relu")])
def test_gemm_row_panels_full_size(G, op, n, k, epi):
    """The transform and input-gradient products at the arxiv-like layer sizes (169,343 rows),
    checked on sampled rows against fp64."""
    m = 169343
    rng = np.random.default_rng(n + k)
    A = dev(rng.standard_normal((m, k), dtype=np.float32))
    B = rng.standard_normal((k, n)).astype(np.float32)
    mask = dev(rng.standard_normal((m, n), dtype=np.float32)) if epi == "mask" else None
    Bd = dev(B) if op == "NN" else dev(np.ascontiguousarray(B.T))
    C = torch.empty((m, n), dtype=torch.float32, device="cuda")
    code = {"none": G.EPI_NONE, "mask": G.EPI_MASK, "relu": G.EPI_RELU}[epi]
    G.gemm(G.OP_NN if op == "NN" else G.OP_NT, A, Bd, C, epi=code, mask=mask)
    rows = np.unique(np.concatenate([rng.integers(0, m, 2000), [0, 255, 256, m - 1]]))
    As = host(A[rows]).astype(np.float64)
    ref = As @ B.astype(np.float64)
    mag = np.abs(As) @ np.abs(B.astype(np.float64))
    if epi == "mask":
        ref = ref * (host(mask[rows]) > 0)
    if epi == "relu":
        ref = np.maximum(ref, 0)
    assert_mag_close(host(C[rows]), ref, mag, f"rows {op} full size {n}x{k}")


@pytest.mark.parametrize("m,n,k", [(1, 1, 17), (33, 40, 1000), (256, 256, 5000), (100, 256, 70001),
                                   (256, 40, 50000), (200, 7, 33333), (64, 256, 123), (160, 96, 65)])
def test_gemm_tn_ragged(G, m, n, k):
    """A^T B on ragged output tiles, partial k slabs and split-k ranges (with a bias)."""
    rng = np.random.default_rng(m * 31 + n + k)
    A = (rng.standard_normal((k, m)) * np.exp(rng.standard_normal((k, 1)))).astype(np.float32)
    B = rng.standard_normal((k, n)).astype(np.float32)
    bias = rng.standard_normal(n).astype(np.float32)
    ref = A.T.astype(np.float64) @ B.astype(np.float64) + bias
    mag = np.abs(A.T.astype(np.float64)) @ np.abs(B.astype(np.float64)) + np.abs(bias)
    Ad, Bd = pitched(A, G.pitch(m) + 4), pitched(B, G.pitch(n))
    C = pitched(np.full((m, n), np.nan, np.float32), G.pitch(n))
    G.gemm(G.OP_TN, Ad, Bd, C, bias=dev(bias))
    C1 = host(C).copy()
    assert_mag_close(C1, ref, mag, f"TN ragged {m}x{n}x{k}")
    G.gemm(G.OP_TN, Ad, Bd, C, bias=dev(bias))
    np.testing.assert_array_equal(host(C), C1)  # fixed-order reduction


# ---------------------------------------------------------------------------
# bias gradient / loss mean, Adam
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("rows,w", [(169343, 256), (2708, 7), (1000, 300), (8192, 40), (8193, 40), (5, 1),
                                    (0, 3)])
@pytest.mark.parametrize("with_rv", [True, False])
def test_column_sums(G, rows, w, with_rv):
    """Column sums with and without the per-row values' mean (the loss pass's form and the
    plain bias gradient share one summation order)."""
    rng = np.random.default_rng(rows + w)
    Gm = rng.standard_normal((rows, w)).astype(np.float32)
    rv = rng.random(rows).astype(np.float32)
    out = torch.full((max(w, 1),), float("nan"), dtype=torch.float32, device="cuda")
    mean = torch.empty(1, dtype=torch.float32, device="cuda")
    use_rv = with_rv and rows > 0
    G.column_sums(pitched(Gm, G.pitch(w)), out[:w], row_vals=dev(rv) if use_rv else None,
                  mean=mean if use_rv else None)
    want = Gm.astype(np.float64).sum(0)
    mag = np.abs(Gm.astype(np.float64)).sum(0)
    assert_mag_close(host(out)[:w], want, mag, "column sums")
    if use_rv:
        assert host(mean)[0] == pytest.approx(rv.astype(np.float64).mean(), rel=1e-6)
    # fixed summation order: a second call gives the same bits
    again = torch.empty_like(out)
    G.column_sums(pitched(Gm, G.pitch(w)), again[:w], row_vals=dev(rv) if use_rv else None,
                  mean=torch.empty_like(mean) if use_rv else None)
    assert torch.equal(out[:w], again[:w])


def test_adam(G, orc):
    rng = np.random.default_rng(3)
    shapes = [(128, 256), (256,), (256, 40), (40,), (7,)]
    ps = [rng.standard_normal(s).astype(np.float32) for s in shapes]
    gs_ = [rng.standard_normal(s).astype(np.float32) for s in shapes]
    ms = [rng.standard_normal(s).astype(np.float32) * 0.1 for s in shapes]
    vs = [rng.random(s).astype(np.float32) * 0.01 for s in shapes]
    dp, dg, dm, dv = ([dev(a) for a in arrs] for arrs in (ps, gs_, ms, vs))
    G.adam(dp, dg, dm, dv, step=3)
    for i in range(len(shapes)):
        want, wm, wv = orc.adam(ps[i], gs_[i], ms[i], vs[i], 3)
        np.testing.assert_allclose(host(dm[i]), wm, rtol=2e-6, atol=1e-7)
        np.testing.assert_allclose(host(dv[i]), wv, rtol=2e-6, atol=1e-9)
        assert_mag_close(host(dp[i]), want, np.abs(ps[i]) + 0.01, f"adam tensor {i}", rtol=1e-5)


# ---------------------------------------------------------------------------
# hub rows split into chunks (rows longer than GCN_SPLIT_MIN entries)
# ---------------------------------------------------------------------------


def expected_plan(ptr, chunk, minlen):
    lens = np.diff(ptr)
    rows = np.nonzero(lens > minlen)[0]
    nch = (lens[rows] + chunk - 1) // chunk
    first = np.concatenate([[0], np.cumsum(nch)])
    owner = np.repeat(np.arange(rows.size), nch)
    return rows, first, owner


@pytest.fixture(scope="module")
def hub_graph(G, orc):
    rng = np.random.default_rng(9)
    n = 20000
    s1, d1 = gs.chung_lu(n, 60000, seed=5)
    hubs = [(3, 15000), (11, 5000), (12, 4000), (19999, 4200)]
    ss, dd = [s1], [d1]
    for h, k in hubs:
        ss.append(np.full(k, h, np.int32))
        dd.append(rng.choice(n, k, replace=False).astype(np.int32))
    s = np.concatenate(ss)
    d = np.concatenate(dd)
    og = orc.build_csr(n, s, d)
    dg = G.build_csr(n, dev(s), dev(d))
    rows, first, owner = expected_plan(og.row_ptr, G.SPLIT_CHUNK, G.SPLIT_MIN)
    assert dg.n_long == rows.size >= 3
    assert dg.c.split.n_chunk == first[-1]
    np.testing.assert_array_equal(host(dg.plan.rows)[:rows.size], rows)
    np.testing.assert_array_equal(host(dg.plan.first)[:rows.size + 1], first)
    np.testing.assert_array_equal(host(dg.plan.owner)[:first[-1]], owner)
    return og, dg


@pytest.mark.parametrize("w", [7, 40, 128, 256])
def test_aggregate_split_hubs(G, orc, hub_graph, w):
    og, dg = hub_graph
    rng = np.random.default_rng(w + 1)
    n = og.n
    M = rng.standard_normal((n, w)).astype(np.float32)
    b = rng.standard_normal(w).astype(np.float32)
    mask = rng.standard_normal((n, w)).astype(np.float32)
    ld = G.pitch(w)
    Md = pitched(M, ld)
    Zd = pitched(np.zeros((n, w), np.float32), ld)
    Z, mag = orc.aggregate(og, M, b, want_mag=True)
    for epi in (G.EPI_NONE, G.EPI_RELU, G.EPI_MASK):
        G.aggregate(dg, Md, Zd, bias=dev(b), epi=epi, mask=pitched(mask, ld) if epi == G.EPI_MASK else None)
        want = Z if epi == G.EPI_NONE else (np.maximum(Z, 0) if epi == G.EPI_RELU else Z * (mask > 0))
        assert_mag_close(host(Zd), want, mag, f"split aggregate w={w} epi={epi}")
    first = host(Zd).copy()
    G.aggregate(dg, Md, Zd, bias=dev(b), epi=G.EPI_MASK, mask=pitched(mask, ld))
    np.testing.assert_array_equal(host(Zd), first)


def test_softmax_layer_on_split_hubs(G, orc, hub_graph):
    og, dg = hub_graph
    n = og.n
    rng = np.random.default_rng(4)
    H = np.maximum(rng.standard_normal((n, 64)), 0).astype(np.float32)
    W = (rng.standard_normal((64, 41)) / 8).astype(np.float32)
    b = (rng.standard_normal(41) * 0.1).astype(np.float32)
    y = rng.integers(0, 41, n).astype(np.int32)
    L = G.make_layer(64, 41, 64, G.pitch(41), G.ACT_SOFTMAX_CE, 1)
    Hd = pitched(H, 64)
    out = pitched(np.zeros((n, 41), np.float32), G.pitch(41))
    logits = pitched(np.zeros((n, 41), np.float32), G.pitch(41))
    loss = torch.zeros(1, device="cuda")
    G.layer_fwd(dg, L, Hd, None, dev(W), dev(b), out, labels=dev(y), loss=loss, logits=logits)
    Z = orc.aggregate(og, orc.matmul(H, W), b)
    mag = orc.aggregate(og, orc.matmul(np.abs(H), np.abs(W)), np.abs(b))
    assert_mag_close(host(logits), Z, mag, "split logits")
    lo, Gr, _ = orc.softmax_ce(Z, y)
    assert host(loss)[0] == pytest.approx(lo, rel=1e-4)
    np.testing.assert_allclose(host(out), Gr, rtol=0, atol=1e-4 * np.abs(Gr).max())


def length_class(d):
    """Processing class of a row of length d (0 first): 4 classes per power of two of d."""
    d = np.asarray(d, np.int64)
    lg = np.floor(np.log2(np.maximum(d, 1))).astype(np.int64)
    key = np.where(d < 4, d, 4 * lg + ((d >> np.maximum(lg - 2, 0)) & 3))
    return np.where(d < 4, 63 - d, 63 - np.minimum(key, 63))


@pytest.mark.parametrize("case", ["hubs", "dense", "cora_like", "empty"])
def test_row_order(G, orc, hub_graph, case):
    """The row order of the aggregations: a permutation of the rows, by length class, longest
    first, ties in row order; and every aggregation result (all epilogues, split hub rows,
    the loss epilogue) is bit-identical with and without it.  The order is applied where an
    average row gathers at least 4 KB: on the dense graph (about 67 entries per row) at every
    width here, on the others at width 256."""
    if case == "hubs":
        og, dg = hub_graph
        s = d = None
    elif case == "dense":
        s, d = gs.chung_lu(6000, 200000, seed=8)
        og, dg = orc.build_csr(6000, s, d), G.build_csr(6000, dev(s), dev(d))
        assert og.nnz / og.n * 4 * 7 < 4096 < og.nnz / og.n * 4 * 40
    elif case == "cora_like":
        wl = gs.WORKLOADS["cora_like"]
        s, d = gs.make_graph(wl)
        og, dg = orc.build_csr(wl.n, s, d), G.build_csr(wl.n, dev(s), dev(d))
    else:
        s = d = np.zeros(0, np.int32)
        og, dg = orc.build_csr(300, s, d), G.build_csr(300, dev(s), dev(d))
    n = og.n
    order = host(dg.order)[:n]
    np.testing.assert_array_equal(np.sort(order), np.arange(n))
    cls = length_class(og.deg)[order]
    key = cls.astype(np.int64) * (n + 1) + order
    assert np.all(np.diff(key) > 0), "classes ascending (longest first), rows ascending within a class"
    if case == "hubs":
        e = host(dg.row_ptr)
        s_ = np.repeat(np.arange(n, dtype=np.int32), np.diff(e))
        d_ = host(dg.col_idx)[:og.nnz]
    else:
        s_, d_ = s, d
    plain = G.build_csr(n, dev(s_), dev(d_), order=False)
    assert plain.order is None and plain.nnz == dg.nnz
    rng = np.random.default_rng(n)
    for w in (7, 16, 40, 256):
        M = pitched(rng.standard_normal((n, w)).astype(np.float32), G.pitch(w))
        b = dev(rng.standard_normal(w).astype(np.float32))
        mask = pitched(rng.standard_normal((n, w)).astype(np.float32), G.pitch(w))
        for epi in (G.EPI_NONE, G.EPI_RELU, G.EPI_MASK):
            outs = []
            for g in (dg, plain):
                Z = pitched(np.zeros((n, w), np.float32), G.pitch(w))
                G.aggregate(g, M, Z, bias=b, epi=epi, mask=mask if epi == G.EPI_MASK else None)
                outs.append(host(Z))
            np.testing.assert_array_equal(outs[0], outs[1])
    # the loss epilogue (rows taken in groups of slots consecutive positions of the order)
    H = pitched(np.maximum(rng.standard_normal((n, 64)), 0).astype(np.float32), 64)
    W = dev((rng.standard_normal((64, 41)) / 8).astype(np.float32))
    bb = dev((rng.standard_normal(41) * 0.1).astype(np.float32))
    y = dev(rng.integers(0, 41, n).astype(np.int32))
    L = G.make_layer(64, 41, 64, G.pitch(41), G.ACT_SOFTMAX_CE, 1)
    res = []
    for g in (dg, plain):
        out = pitched(np.zeros((n, 41), np.float32), G.pitch(41))
        logits = pitched(np.zeros((n, 41), np.float32), G.pitch(41))
        loss = torch.zeros(1, device="cuda")
        G.layer_fwd(g, L, H, None, W, bb, out, labels=y, loss=loss, logits=logits)
        res.append((host(out), host(logits), host(loss)))
    for a, c in zip(*res):
        np.testing.assert_array_equal(a, c)


def test_tune_row_order(G, orc):
    """The tuner keeps or drops the order; either way the graph aggregates as before."""
    wl = gs.WORKLOADS["cora_like"]
    s, d = gs.make_graph(wl)
    g = G.build_csr(wl.n, dev(s), dev(d))
    rng = np.random.default_rng(3)
    M = pitched(rng.standard_normal((wl.n, 40)).astype(np.float32), G.pitch(40))
    before = pitched(np.zeros((wl.n, 40), np.float32), G.pitch(40))
    G.aggregate(g, M, before)
    kept = G.tune_row_order(g, 40)
    assert kept == (g.order is not None) and (g.c.order is not None) == kept
    after = pitched(np.zeros((wl.n, 40), np.float32), G.pitch(40))
    G.aggregate(g, M, after)
    np.testing.assert_array_equal(host(after), host(before))


@pytest.mark.parametrize("fused", ["1", "0"])
@pytest.mark.parametrize("fi,fo", [(128, 256), (48, 300)])
def test_aggregate_first_layer_on_split_hubs(G, orc, hub_graph, fi, fo, fused, monkeypatch):
    """Aggregate-then-transform layer, fused kernel and two-launch form: hub rows come from
    the chunk kernels."""
    monkeypatch.setenv("GCN_AF_FUSED", fused)
    og, dg = hub_graph
    n = og.n
    rng = np.random.default_rng(fi)
    H = rng.standard_normal((n, fi)).astype(np.float32)
    W = (rng.standard_normal((fi, fo)) / np.sqrt(fi)).astype(np.float32)
    b = (rng.standard_normal(fo) * 0.1).astype(np.float32)
    L = G.make_layer(fi, fo, G.pitch(fi), G.pitch(fo), G.ACT_RELU, 0, G.AGGREGATE_FIRST)
    out = pitched(np.zeros((n, fo), np.float32), G.pitch(fo))
    saved = pitched(np.zeros((n, fi), np.float32), G.pitch(fi))
    G.layer_fwd(dg, L, pitched(H, G.pitch(fi)), None, dev(W), dev(b), out, saved=saved)
    P, pmag = orc.aggregate(og, H, want_mag=True)
    assert_mag_close(host(saved), P, pmag, "split hubs: saved A_hat H")
    Z = orc.aggregate(og, orc.matmul(H, W), b)
    mag = orc.aggregate(og, orc.matmul(np.abs(H), np.abs(W)), np.abs(b))
    assert_mag_close(host(out), np.maximum(Z, 0), mag, f"split hubs: AF {fi}->{fo}")


# ---------------------------------------------------------------------------
# other aggregators: sum, mean and its transpose, max (forward and gradient)
# ---------------------------------------------------------------------------

AGG_CODE = {"sum": 1, "mean": 2, "mean_t": 3}


@pytest.mark.parametrize("kind", ["sum", "mean", "mean_t"])
@pytest.mark.parametrize("w", [7, 40, 256])
def test_linear_aggregators_on_split_hubs(G, orc, hub_graph, kind, w):
    og, dg = hub_graph
    rng = np.random.default_rng(w + 7)
    n = og.n
    M = rng.standard_normal((n, w)).astype(np.float32)
    b = rng.standard_normal(w).astype(np.float32)
    mask = rng.standard_normal((n, w)).astype(np.float32)
    ld = G.pitch(w)
    Md = pitched(M, ld)
    Zd = pitched(np.zeros((n, w), np.float32), ld)
    Z, mag = orc.aggregate(og, M, b, want_mag=True, kind=kind)
    for epi in (G.EPI_NONE, G.EPI_RELU, G.EPI_MASK):
        G.aggregate(dg, Md, Zd, bias=dev(b), epi=epi, mask=pitched(mask, ld) if epi == G.EPI_MASK else None,
                    agg=AGG_CODE[kind])
        want = Z if epi == G.EPI_NONE else (np.maximum(Z, 0) if epi == G.EPI_RELU else Z * (mask > 0))
        assert_mag_close(host(Zd), want, mag, f"{kind} aggregate w={w} epi={epi}")


@pytest.mark.parametrize("w,ld", [(7, 7), (7, 8), (40, 40), (128, 128), (256, 256), (41, 41)])
def test_max_aggregation_bit_exact_with_ties(G, orc, hub_graph, w, ld):
    """Max and first maximiser are exact in fp32: equal to the oracle bit for bit, also on
    rows of small integers (many ties) and on the hub rows (walked by one lane group)."""
    og, dg = hub_graph
    n = og.n
    rng = np.random.default_rng(w * 3 + ld)
    M = rng.integers(-3, 4, (n, w)).astype(np.float32)
    M[::7] = rng.standard_normal((M[::7].shape)).astype(np.float32)
    Pd = pitched(np.zeros((n, w), np.float32), ld)
    argd = torch.zeros((n, ld), dtype=torch.int32, device="cuda")[:, :w]
    G.aggregate_max(dg, pitched(M, ld), Pd, argd)
    P, arg = orc.aggregate_max(og, M)
    np.testing.assert_array_equal(host(Pd), P.astype(np.float32))
    np.testing.assert_array_equal(host(argd), arg)
    # gradient: the gather over the symmetric rows against the oracle's scatter
    dP = rng.standard_normal((n, w)).astype(np.float32)
    mask = rng.standard_normal((n, w)).astype(np.float32)
    dMd = pitched(np.zeros((n, w), np.float32), ld)
    for use_mask in (False, True):
        G.aggregate_max_bwd(dg, pitched(dP, ld), argd, dMd, mask=pitched(mask, ld) if use_mask else None)
        want = orc.aggregate_max_backward(og, dP, arg)
        mag = orc.aggregate_max_backward(og, np.abs(dP), arg)
        if use_mask:
            want, mag = want * (mask > 0), mag * (mask > 0)
        assert_mag_close(host(dMd), want, mag, f"max gradient w={w} mask={use_mask}")
    first = host(dMd).copy()
    G.aggregate_max_bwd(dg, pitched(dP, ld), argd, dMd, mask=pitched(mask, ld))
    np.testing.assert_array_equal(host(dMd), first)  # fixed order


def test_sparse_backward_atomic_transpose(G, orc):
    """X^T Q from the CSR rows with atomic adds (no CSC view): within the fp32 bar of the
    oracle; the rounding order may differ between runs, the values stay within it."""
    n, f, w = 20000, 300, 40
    X = gs.features_bernoulli(n, f, 0.05, seed=4, binary=False)
    rng = np.random.default_rng(3)
    Q = rng.standard_normal((n, w)).astype(np.float32)
    info, sx = G.feature_stats(dev(X), force_mode=G.SPARSE, csc=False)
    assert sx.col_ptr is None
    L = G.make_layer(f, w, f, G.pitch(w), G.ACT_RELU, 0)
    dW = torch.zeros((f, w), device="cuda")
    db = torch.zeros(w, device="cuda")
    g = G.build_csr(n, dev(np.zeros(0, np.int32)), dev(np.zeros(0, np.int32)))  # A + I = I: Q passes through
    G.layer_bwd(g, L, pitched(Q, G.pitch(w)), None, sx, None, dev(np.zeros((f, w), np.float32)), dW, db, None)
    rp, col, val = orc.dense_to_csr(X)
    want = orc.matmul(X.T, Q)
    mag = orc.matmul(np.abs(X).T, np.abs(Q))
    assert_mag_close(host(dW), want, mag, "atomic X^T Q")


def test_sparse_backward_long_columns(G, orc):
    """X with few, dense columns: every CSC column is long and goes through chunks
    processed chunk-index-major."""
    n, f, w = 30000, 48, 40
    X = gs.features_bernoulli(n, f, 0.4, seed=2, binary=False)
    rng = np.random.default_rng(1)
    Q = rng.standard_normal((n, w)).astype(np.float32)
    _, sx = G.feature_stats(dev(X), materialize=True)
    cp, row, cval = orc.dense_to_csc(X)
    rows, first, owner = expected_plan(cp, G.SPLIT_CHUNK, G.SPLIT_MIN)
    sp = sx.c.csc_split
    assert sp.n_long == rows.size == f and sp.n_chunk == first[-1]
    np.testing.assert_array_equal(host(sx.plan.first)[:f + 1], first)
    order = host(sx.plan.order)[:first[-1]]
    np.testing.assert_array_equal(np.sort(order), np.arange(first[-1]))
    k_of = order - first[owner[order]]
    assert (np.diff(k_of) >= 0).all()          # chunk index never decreases along the order
    dW = torch.empty((f, w), dtype=torch.float32, device="cuda")
    G.spmm(sx.col_ptr, sx.row[:sx.nnz], sx.cval[:sx.nnz], dev(Q), dW, split=sp)
    ref, mag = orc.spmm(cp, row, cval, Q, want_mag=True)
    assert_mag_close(host(dW), ref, mag, "X_csc Q with long columns")


@pytest.mark.parametrize("op", ["NN", "NT", "TN"])
@pytest.mark.parametrize("shape", [(4000, 256, 256), (3000, 40, 602), (777, 128, 4096), (50000, 64, 100)],
                         ids=lambda s: "x".join(map(str, s)))
def test_gemm_bf16x6_matches_native_fp32(G, op, shape, monkeypatch):
    """The bf16x6 split (default) and native fp32 MFMA agree to fp32 accuracy."""
    m, n, k = shape
    rng = np.random.default_rng(m + n + k)
    A = (rng.standard_normal((m, k)) * np.exp(rng.standard_normal((m, 1)))).astype(np.float32)
    B = rng.standard_normal((k, n)).astype(np.float32)
    if op == "NN":
        Ad, Bd, code = dev(A), dev(B), G.OP_NN
    elif op == "NT":
        Ad, Bd, code = dev(A), dev(np.ascontiguousarray(B.T)), G.OP_NT
    else:
        Ad, Bd, code = dev(np.ascontiguousarray(A.T)), dev(B), G.OP_TN
    mag = np.abs(A.astype(np.float64)) @ np.abs(B.astype(np.float64))
    ref = A.astype(np.float64) @ B.astype(np.float64)
    out = {}
    for mode in ("bf16x6", "fp32"):
        monkeypatch.setenv("GCN_GEMM_MODE", mode)
        C = torch.empty((m, n), dtype=torch.float32, device="cuda")
        G.gemm(code, Ad, Bd, C)
        out[mode] = host(C).astype(np.float64)
        assert_mag_close(out[mode], ref, mag, f"{mode} {op} {shape}")
    worst = assert_mag_close(out["bf16x6"], out["fp32"], mag, f"bf16x6 vs fp32 {op} {shape}", rtol=2e-6)
    print(f"bf16x6 vs fp32 {op} {shape}: max |diff| / scale = {worst:.2e}")
