"""Pins for the fp64 oracle: each oracle function checked against something other
than itself -- brute force from the definition, closed forms, invariants,
independent library routines (scipy, torch) and finite differences.

A plausible mistake anywhere in the oracle (a dropped term, a wrong sign or
index, a transposed operand, a missing dedup) fails at least one test here.
"""
import math
from decimal import Decimal, getcontext

import numpy as np
import pytest
import scipy.sparse as sp
import torch

pytestmark = []


# ---------------------------------------------------------------------------
# helpers written from the definitions, independent of the oracle
# ---------------------------------------------------------------------------


def brute_rows(n, src, dst):
    """Neighbour sets of A + I by Python sets (dedup, symmetrise, drop self, add self)."""
    rows = [set([i]) for i in range(n)]
    for u, v in zip(src, dst):
        if u != v:
            rows[u].add(v)
            rows[v].add(u)
    return [sorted(r) for r in rows]


def brute_ahat(n, src, dst):
    """Dense D^-1/2 (A + I) D^-1/2 from an adjacency matrix built entry by entry."""
    A = np.zeros((n, n))
    for u, v in zip(src, dst):
        if u != v:
            A[u, v] = 1.0
            A[v, u] = 1.0
    A += np.eye(n)
    d = A.sum(axis=1)
    Dm = np.diag(1.0 / np.sqrt(d))
    return Dm @ A @ Dm


def random_edges(rng, n, m, dup_frac=0.3, self_frac=0.1):
    src = rng.integers(0, n, m)
    dst = rng.integers(0, n, m)
    k = int(m * self_frac)
    dst[:k] = src[:k]
    j = int(m * dup_frac)
    if j and m > k + j:
        src[-j:] = src[k:k + j]
        dst[-j:] = dst[k:k + j]
    return src.astype(np.int32), dst.astype(np.int32)


def ring(n):
    s = np.arange(n, dtype=np.int32)
    return s, ((s + 1) % n).astype(np.int32)


def star(leaves):
    return np.zeros(leaves, np.int32), np.arange(1, leaves + 1, dtype=np.int32)


def complete(n):
    iu = np.triu_indices(n, 1)
    return iu[0].astype(np.int32), iu[1].astype(np.int32)


# ---------------------------------------------------------------------------
# graph construction
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("seed", range(8))
def test_csr_matches_brute_force_sets(orc, seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 40))
    m = int(rng.integers(0, 150))
    src, dst = random_edges(rng, n, m)
    g = orc.build_csr(n, src, dst)
    rows = brute_rows(n, src.tolist(), dst.tolist())
    assert g.deg.tolist() == [len(r) for r in rows]
    assert g.row_ptr.tolist() == list(np.cumsum([0] + [len(r) for r in rows]))
    assert g.col_idx.tolist() == [c for r in rows for c in r]


def test_csr_closed_forms(orc):
    g = orc.build_csr(7, *ring(7))
    assert (g.deg == 3).all()
    g = orc.build_csr(1 + 9, *star(9))
    assert g.deg[0] == 10 and (g.deg[1:] == 2).all()
    g = orc.build_csr(6, *complete(6))
    assert (g.deg == 6).all()
    assert g.col_idx.tolist() == list(range(6)) * 6
    g = orc.build_csr(5, np.zeros(0, np.int32), np.zeros(0, np.int32))
    assert (g.deg == 1).all() and g.col_idx.tolist() == [0, 1, 2, 3, 4]
    # every edge repeated in both directions, plus self pairs: same graph as the ring
    s, d = ring(7)
    s2 = np.concatenate([s, d, s, np.arange(7, dtype=np.int32)])
    d2 = np.concatenate([d, s, d, np.arange(7, dtype=np.int32)])
    g2 = orc.build_csr(7, s2, d2)
    g1 = orc.build_csr(7, s, d)
    assert (g2.row_ptr == g1.row_ptr).all() and (g2.col_idx == g1.col_idx).all()


def test_csr_rejects_out_of_range(orc):
    with pytest.raises(ValueError):
        orc.build_csr(3, np.array([0, 3], np.int32), np.array([1, 1], np.int32))
    with pytest.raises(ValueError):
        orc.build_csr(3, np.array([0, -1], np.int32), np.array([1, 1], np.int32))


def test_dinv_is_correctly_rounded(orc):
    """dinv_i is the fp32 nearest to 1/sqrt(d_i), checked with 50-digit decimals."""
    getcontext().prec = 50
    # disjoint stars with 0..K-1 leaves give hub degrees 1..K, plus a few large stars
    sizes = list(range(0, 120)) + [255, 511, 1023, 4095, 9999]
    src, dst, base = [], [], 0
    hubs = []
    for s in sizes:
        hubs.append(base)
        src += [base] * s
        dst += list(range(base + 1, base + 1 + s))
        base += s + 1
    g = orc.build_csr(base, np.array(src, np.int32), np.array(dst, np.int32))
    checked = set()
    for i in range(g.n):
        d = int(g.deg[i])
        if d in checked:
            continue
        checked.add(d)
        exact = Decimal(1) / Decimal(d).sqrt()
        got = float(g.dinv[i])
        f = np.float32(got)
        lo = np.nextafter(f, np.float32(0))
        hi = np.nextafter(f, np.float32(2))
        err = abs(Decimal(float(f)) - exact)
        assert err <= abs(Decimal(float(lo)) - exact)
        assert err <= abs(Decimal(float(hi)) - exact)
    assert len(checked) >= 120


# ---------------------------------------------------------------------------
# normalised aggregation
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("seed", range(6))
def test_aggregate_matches_dense_brute_force(orc, seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(1, 60))
    src, dst = random_edges(rng, n, int(rng.integers(0, 4 * n)))
    g = orc.build_csr(n, src, dst)
    w = int(rng.integers(1, 9))
    M = rng.standard_normal((n, w))
    b = rng.standard_normal(w)
    Z = orc.aggregate(g, M, b)
    ref = brute_ahat(n, src.tolist(), dst.tolist()) @ M + b
    np.testing.assert_allclose(Z, ref, rtol=0, atol=1e-12)


def test_aggregate_closed_form_entries(orc):
    # A_hat read off by aggregating the identity matrix
    n = 7
    g = orc.build_csr(n, *ring(n))
    A = orc.aggregate(g, np.eye(n))
    for i in range(n):
        for j in range(n):
            want = 1.0 / 3.0 if (i - j) % n in (0, 1, n - 1) else 0.0
            assert A[i, j] == pytest.approx(want, abs=1e-15)
    k = 5
    g = orc.build_csr(k, *complete(k))
    np.testing.assert_allclose(orc.aggregate(g, np.eye(k)), np.full((k, k), 1.0 / k), atol=1e-15)
    leaves = 6
    g = orc.build_csr(leaves + 1, *star(leaves))
    A = orc.aggregate(g, np.eye(leaves + 1))
    assert A[0, 0] == pytest.approx(1.0 / (leaves + 1), abs=1e-15)
    assert A[0, 3] == pytest.approx(1.0 / math.sqrt(2 * (leaves + 1)), abs=1e-15)
    assert A[3, 0] == pytest.approx(1.0 / math.sqrt(2 * (leaves + 1)), abs=1e-15)
    assert A[3, 3] == pytest.approx(0.5, abs=1e-15)
    assert A[3, 4] == 0.0
    np.testing.assert_array_equal(A, A.T)


def test_aggregate_invariants(orc):
    rng = np.random.default_rng(7)
    n = 300
    src, dst = random_edges(rng, n, 1500)
    g = orc.build_csr(n, src, dst)
    # D^-1 (A + I) is row-stochastic: A_hat sqrt(d) = sqrt(d)
    sd = np.sqrt(g.deg.astype(np.float64))[:, None]
    np.testing.assert_allclose(orc.aggregate(g, sd), sd, rtol=1e-13)
    # k-regular graph (circulant with offsets 1, 2): constant columns are preserved
    s = np.arange(50, dtype=np.int32)
    src = np.concatenate([s, s]).astype(np.int32)
    dst = np.concatenate([(s + 1) % 50, (s + 2) % 50]).astype(np.int32)
    g5 = orc.build_csr(50, src, dst)
    assert (g5.deg == 5).all()
    np.testing.assert_allclose(orc.aggregate(g5, np.full((50, 3), 2.5)), 2.5, rtol=1e-14)
    # K_n: every row is the column mean
    g6 = orc.build_csr(9, *complete(9))
    M = rng.standard_normal((9, 4))
    np.testing.assert_allclose(orc.aggregate(g6, M), np.tile(M.mean(0), (9, 1)), atol=1e-14)
    # no edges: A_hat = I, aggregation is the identity
    g0 = orc.build_csr(8, np.zeros(0, np.int32), np.zeros(0, np.int32))
    M = rng.standard_normal((8, 5))
    np.testing.assert_array_equal(orc.aggregate(g0, M), M)


def test_aggregate_rows_and_magnitude(orc):
    rng = np.random.default_rng(3)
    n = 80
    src, dst = random_edges(rng, n, 400)
    g = orc.build_csr(n, src, dst)
    M = rng.standard_normal((n, 6))
    b = rng.standard_normal(6)
    Z, mag = orc.aggregate(g, M, b, want_mag=True)
    rows = np.array([5, 0, 79, 5, 33], np.int32)
    np.testing.assert_array_equal(orc.aggregate(g, M, b, rows=rows), Z[rows])
    assert (mag >= np.abs(Z) - 1e-12).all()
    ref_mag = brute_ahat(n, src.tolist(), dst.tolist()) @ np.abs(M) + np.abs(b)
    np.testing.assert_allclose(mag, ref_mag, atol=1e-12)


# ---------------------------------------------------------------------------
# feature statistics, decision, sparse views
# ---------------------------------------------------------------------------


def test_feature_counts_and_decision(orc):
    n, f = 40, 25
    z = np.zeros((n, f), np.float32)
    nnz, rn = orc.feature_counts(z)
    assert nnz == 0 and orc.sparse_decision(nnz, n, f) == 1
    o = np.ones((n, f), np.float32)
    nnz, rn = orc.feature_counts(o)
    assert nnz == n * f and (rn == f).all() and orc.sparse_decision(nnz, n, f) == 0
    eye = np.eye(n, f, dtype=np.float32)
    assert orc.feature_counts(eye)[0] == min(n, f)
    # exact threshold: nnz = NF/5 gives s = 0.8 = tau -> sparse; one more -> dense
    x = np.zeros(n * f, np.float32)
    x[: n * f // 5] = 3.0
    assert orc.feature_counts(x.reshape(n, f))[0] == n * f // 5
    assert orc.sparse_decision(n * f // 5, n, f) == 1
    assert orc.sparse_decision(n * f // 5 + 1, n, f) == 0
    assert orc.sparse_decision(0, n, f, 1, 1) == 1 and orc.sparse_decision(1, n, f, 1, 1) == 0
    # -0.0 is a zero, NaN is a nonzero
    y = np.zeros((2, 3), np.float32)
    y[0, 0] = -0.0
    y[1, 2] = np.nan
    nnz, rn = orc.feature_counts(y)
    assert nnz == 1 and rn.tolist() == [0, 1]
    rng = np.random.default_rng(0)
    r = (rng.random((333, 77)) < 0.1).astype(np.float32) * rng.standard_normal((333, 77)).astype(np.float32)
    nnz, rn = orc.feature_counts(r)
    assert nnz == np.count_nonzero(r) and (rn == np.count_nonzero(r, axis=1)).all()
    # very large N F (64-bit products) at the threshold
    big_n, big_f = 2097152, 4096
    t = big_n * big_f // 5
    assert orc.sparse_decision(t, big_n, big_f) == 1
    assert orc.sparse_decision(t + 1, big_n, big_f) == 0


def test_sparse_views_match_scipy(orc):
    rng = np.random.default_rng(11)
    X = (rng.random((57, 91)) < 0.07).astype(np.float32) * rng.standard_normal((57, 91)).astype(np.float32)
    X[3, :] = 0
    rp, col, val = orc.dense_to_csr(X)
    ref = sp.csr_matrix(X)
    ref.sort_indices()
    assert rp.tolist() == ref.indptr.tolist()
    assert col.tolist() == ref.indices.tolist()
    np.testing.assert_array_equal(val, ref.data)
    cp, row, cval = orc.dense_to_csc(X)
    refc = sp.csc_matrix(X)
    refc.sort_indices()
    assert cp.tolist() == refc.indptr.tolist()
    assert row.tolist() == refc.indices.tolist()
    np.testing.assert_array_equal(cval, refc.data)


def test_sparse_products_match_dense(orc):
    rng = np.random.default_rng(12)
    X = (rng.random((64, 50)) < 0.1).astype(np.float32) * rng.standard_normal((64, 50)).astype(np.float32)
    W = rng.standard_normal((50, 7))
    G = rng.standard_normal((64, 7))
    rp, col, val = orc.dense_to_csr(X)
    cp, row, cval = orc.dense_to_csc(X)
    np.testing.assert_allclose(orc.spmm(rp, col, val, W), X.astype(np.float64) @ W, atol=1e-12)
    np.testing.assert_allclose(orc.spmm(cp, row, cval, G), X.astype(np.float64).T @ G, atol=1e-12)
    C, mag = orc.spmm(rp, col, val, W, want_mag=True)
    np.testing.assert_allclose(mag, np.abs(X.astype(np.float64)) @ np.abs(W), atol=1e-12)


# ---------------------------------------------------------------------------
# loss, optimizer
# ---------------------------------------------------------------------------


def test_softmax_ce_closed_form(orc):
    n, c = 10, 7
    y = np.arange(n) % c
    loss, G, li = orc.softmax_ce(np.zeros((n, c)), y)
    assert loss == pytest.approx(math.log(c), rel=1e-15)
    want = np.full((n, c), 1.0 / c)
    want[np.arange(n), y] -= 1.0
    np.testing.assert_allclose(G, want / n, atol=1e-17)


def test_softmax_ce_matches_torch(orc):
    rng = np.random.default_rng(5)
    Z = rng.standard_normal((33, 41)) * 4
    y = rng.integers(0, 41, 33)
    loss, G, _ = orc.softmax_ce(Z, y)
    zt = torch.tensor(Z, dtype=torch.float64, requires_grad=True)
    lt = torch.nn.functional.cross_entropy(zt, torch.tensor(y), reduction="mean")
    lt.backward()
    assert loss == pytest.approx(lt.item(), rel=1e-13)
    np.testing.assert_allclose(G, zt.grad.numpy(), atol=1e-15)
    np.testing.assert_allclose(G.sum(axis=1), 0.0, atol=1e-16)
    # shift invariance of the loss
    loss2, G2, _ = orc.softmax_ce(Z + 100.0, y)
    assert loss2 == pytest.approx(loss, rel=1e-12)


def test_adam_step_one_closed_form(orc):
    rng = np.random.default_rng(9)
    th = rng.standard_normal(50)
    g = rng.standard_normal(50)
    t1, m, v = orc.adam(th, g, np.zeros(50), np.zeros(50), 1)
    np.testing.assert_allclose(t1, th - 0.01 * g / (np.abs(g) + 1e-8), rtol=0, atol=1e-15)


def test_adam_matches_torch(orc):
    rng = np.random.default_rng(10)
    th0 = rng.standard_normal((6, 4))
    p = torch.nn.Parameter(torch.tensor(th0))
    opt = torch.optim.Adam([p], lr=0.01, betas=(0.9, 0.999), eps=1e-8)
    th, m, v = th0.copy(), np.zeros_like(th0), np.zeros_like(th0)
    for t in range(1, 6):
        g = rng.standard_normal((6, 4))
        p.grad = torch.tensor(g)
        opt.step()
        th, m, v = orc.adam(th, g, m, v, t)
    np.testing.assert_allclose(th, p.detach().numpy(), rtol=0, atol=1e-14)


# ---------------------------------------------------------------------------
# whole model: forward, backward, epoch
# ---------------------------------------------------------------------------


def torch_model(Ahat, X, Ws, bs, y):
    A = torch.tensor(Ahat)
    H = torch.tensor(np.asarray(X, np.float64))
    Wt = [torch.tensor(np.asarray(w, np.float64), requires_grad=True) for w in Ws]
    bt = [torch.tensor(np.asarray(b, np.float64), requires_grad=True) for b in bs]
    Zs = []
    for l in range(len(Ws)):
        Z = A @ (H @ Wt[l]) + bt[l]
        Zs.append(Z)
        H = torch.relu(Z) if l < len(Ws) - 1 else Z
    loss = torch.nn.functional.cross_entropy(Zs[-1], torch.tensor(y, dtype=torch.long))
    loss.backward()
    return loss.item(), [z.detach().numpy() for z in Zs], [w.grad.numpy() for w in Wt], \
        [b.grad.numpy() for b in bt]


def tiny_problem(seed, n=30, widths=(6, 5, 4, 3), density=1.0):
    rng = np.random.default_rng(seed)
    src, dst = random_edges(rng, n, 3 * n)
    X = rng.standard_normal((n, widths[0])).astype(np.float32)
    if density < 1.0:
        X *= (rng.random(X.shape) < density)
    Ws = [rng.standard_normal((widths[l], widths[l + 1])) * 0.7 for l in range(len(widths) - 1)]
    bs = [rng.standard_normal(widths[l + 1]) * 0.3 for l in range(len(widths) - 1)]
    y = rng.integers(0, widths[-1], n)
    return src, dst, X, Ws, bs, y


@pytest.mark.parametrize("seed", range(4))
def test_forward_backward_match_torch_autograd(orc, seed):
    src, dst, X, Ws, bs, y = tiny_problem(seed)
    n = X.shape[0]
    g = orc.build_csr(n, src, dst)
    Hs, Zs = orc.forward(g, X, Ws, bs)
    loss, G, _ = orc.softmax_ce(Zs[-1], y)
    dWs, dbs, Gs = orc.backward(g, Hs, Zs, G, Ws)
    tl, tZ, tdW, tdb = torch_model(brute_ahat(n, src.tolist(), dst.tolist()), X, Ws, bs, y)
    assert loss == pytest.approx(tl, rel=1e-12)
    for l in range(len(Ws)):
        np.testing.assert_allclose(Zs[l], tZ[l], atol=1e-12)
        np.testing.assert_allclose(dWs[l], tdW[l], atol=1e-13)
        np.testing.assert_allclose(dbs[l], tdb[l], atol=1e-13)


def test_backward_central_differences(orc):
    """Gradients against central finite differences in fp64 (inputs away from ReLU kinks)."""
    for seed in range(50):
        src, dst, X, Ws, bs, y = tiny_problem(1000 + seed, n=12, widths=(4, 5, 3))
        g = orc.build_csr(12, src, dst)
        Hs, Zs = orc.forward(g, X, Ws, bs)
        if np.abs(Zs[0]).min() > 1e-3:
            break
    else:
        pytest.fail("no kink-free sample")
    loss, G, _ = orc.softmax_ce(Zs[-1], y)
    dWs, dbs, _ = orc.backward(g, Hs, Zs, G, Ws)

    def f(Ws_, bs_):
        _, Z_ = orc.forward(g, X, Ws_, bs_)
        return orc.softmax_ce(Z_[-1], y)[0]

    h = 1e-6
    for l in range(2):
        for idx in np.ndindex(Ws[l].shape):
            Wp = [w.copy() for w in Ws]
            Wm = [w.copy() for w in Ws]
            Wp[l][idx] += h
            Wm[l][idx] -= h
            fd = (f(Wp, bs) - f(Wm, bs)) / (2 * h)
            assert fd == pytest.approx(dWs[l][idx], abs=1e-8)
        for i in range(bs[l].size):
            bp = [b.copy() for b in bs]
            bm = [b.copy() for b in bs]
            bp[l][i] += h
            bm[l][i] -= h
            fd = (f(Ws, bp) - f(Ws, bm)) / (2 * h)
            assert fd == pytest.approx(dbs[l][i], abs=1e-8)


def test_sparse_path_equals_dense_path(orc):
    src, dst, X, Ws, bs, y = tiny_problem(21, n=40, widths=(30, 8, 4), density=0.1)
    g = orc.build_csr(40, src, dst)
    sx = orc.SparseX(X)
    Hd, Zd = orc.forward(g, X, Ws, bs)
    Hsp, Zsp = orc.forward(g, X, Ws, bs, sparse=sx)
    for a, b in zip(Zd, Zsp):
        np.testing.assert_allclose(a, b, atol=1e-13)
    loss, G, _ = orc.softmax_ce(Zd[-1], y)
    dWd, dbd, _ = orc.backward(g, Hd, Zd, G, Ws)
    dWs, dbs, _ = orc.backward(g, Hsp, Zsp, G, Ws, sparse=sx)
    for a, b in zip(dWd, dWs):
        np.testing.assert_allclose(a, b, atol=1e-14)


@pytest.mark.parametrize("sparse", [False, True])
@pytest.mark.parametrize("widths", [(30, 8, 4), (20, 7, 6, 3)])
def test_row_block_epoch_equals_epoch(orc, sparse, widths):
    """The row-block epoch (for features too large to hold) against the whole-matrix epoch:
    same loss, gradients and Adam step, with blocks that do not divide n."""
    n = 40
    src, dst, X, Ws, bs, y = tiny_problem(23, n=n, widths=widths, density=0.1)
    g = orc.build_csr(n, src, dst)
    z = [np.zeros_like(w) for w in Ws]
    zb = [np.zeros_like(b) for b in bs]
    want = orc.epoch(g, X, y, Ws, bs, z, z, zb, zb, 1, sparse=orc.SparseX(X) if sparse else None)
    got = orc.epoch_row_blocks(g, lambda r0, r1: X[r0:r1], X.shape[1], y, Ws, bs, z, z, zb, zb, 1,
                               sparse=sparse, block_rows=7)
    assert got["loss"] == pytest.approx(want["loss"], rel=1e-14)
    for k in ("dWs", "dbs", "Ws", "bs"):
        for a, b in zip(got[k], want[k]):
            np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-15)


def test_epochs_match_torch_training(orc):
    """Three oracle epochs against torch autograd + torch.optim.Adam on a dense A_hat."""
    src, dst, X, Ws, bs, y = tiny_problem(31, n=25, widths=(5, 6, 3))
    n = 25
    g = orc.build_csr(n, src, dst)
    A = torch.tensor(brute_ahat(n, src.tolist(), dst.tolist()))
    Wt = [torch.nn.Parameter(torch.tensor(w)) for w in Ws]
    bt = [torch.nn.Parameter(torch.tensor(b)) for b in bs]
    opt = torch.optim.Adam(Wt + bt, lr=0.01, betas=(0.9, 0.999), eps=1e-8)
    st = dict(Ws=[w.copy() for w in Ws], bs=[b.copy() for b in bs],
              mW=[np.zeros_like(w) for w in Ws], vW=[np.zeros_like(w) for w in Ws],
              mb=[np.zeros_like(b) for b in bs], vb=[np.zeros_like(b) for b in bs])
    for t in range(1, 4):
        out = orc.epoch(g, X, y, st["Ws"], st["bs"], st["mW"], st["vW"], st["mb"], st["vb"], t)
        opt.zero_grad()
        H = torch.tensor(X.astype(np.float64))
        for l in range(2):
            Z = A @ (H @ Wt[l]) + bt[l]
            H = torch.relu(Z) if l == 0 else Z
        loss = torch.nn.functional.cross_entropy(H, torch.tensor(y))
        loss.backward()
        opt.step()
        assert out["loss"] == pytest.approx(loss.item(), rel=1e-12)
        st = {k: out[k] for k in ("Ws", "bs", "mW", "vW", "mb", "vb")}
    for l in range(2):
        np.testing.assert_allclose(st["Ws"][l], Wt[l].detach().numpy(), atol=1e-12)
        np.testing.assert_allclose(st["bs"][l], bt[l].detach().numpy(), atol=1e-12)


def test_backward_relu_decisions_hook(orc):
    """The optional ReLU decisions of the backward: the oracle's own decisions reproduce
    the default exactly, and flipping one decision changes only that entry of G (the
    flipped factor times (Q W^T) there) before it propagates."""
    src, dst, X, Ws, bs, y = tiny_problem(33, n=25, widths=(5, 6, 3))
    g = orc.build_csr(25, src, dst)
    Hs, Zs = orc.forward(g, X, Ws, bs)
    _, G, _ = orc.softmax_ce(Zs[-1], y)
    ref = orc.backward(g, Hs, Zs, G, Ws)
    same = orc.backward(g, Hs, Zs, G, Ws, relu_on=[Zs[0] > 0])
    for a, b in zip(ref[0] + ref[1] + ref[2], same[0] + same[1] + same[2]):
        np.testing.assert_array_equal(a, b)
    on = Zs[0] > 0
    i, j = np.argwhere(on)[0]
    on[i, j] = False
    flip = orc.backward(g, Hs, Zs, G, Ws, relu_on=[on])
    diff = flip[2][0] != ref[2][0]
    assert diff.sum() == 1 and diff[i, j] and flip[2][0][i, j] == 0.0
    np.testing.assert_array_equal(flip[2][1], ref[2][1])  # the last layer's G is upstream


# ---------------------------------------------------------------------------
# other aggregators: sum (A + I), mean (D^-1 (A + I)) and its transpose, max
# ---------------------------------------------------------------------------


def brute_operator(n, src, dst, kind):
    """Dense aggregation operator from an adjacency matrix built entry by entry."""
    A = np.zeros((n, n))
    for u, v in zip(src, dst):
        if u != v:
            A[u, v] = 1.0
            A[v, u] = 1.0
    A += np.eye(n)
    d = A.sum(axis=1)
    return {"sum": A, "mean": A / d[:, None], "mean_t": A / d[None, :]}[kind]


@pytest.mark.parametrize("kind", ["sum", "mean", "mean_t"])
@pytest.mark.parametrize("seed", range(3))
def test_linear_aggregators_match_dense_brute_force(orc, kind, seed):
    rng = np.random.default_rng(100 + seed)
    n = 40
    src, dst = random_edges(rng, n, 90)
    g = orc.build_csr(n, src, dst)
    M = rng.standard_normal((n, 5))
    b = rng.standard_normal(5)
    S = brute_operator(n, src.tolist(), dst.tolist(), kind)
    Z, mag = orc.aggregate(g, M, b, want_mag=True, kind=kind)
    np.testing.assert_allclose(Z, S @ M + b, atol=1e-12)
    np.testing.assert_allclose(mag, np.abs(S) @ np.abs(M) + np.abs(b), atol=1e-12)
    np.testing.assert_allclose(orc.dense_operator(g, kind), S, atol=1e-15)


def test_linear_aggregator_closed_forms(orc):
    n = 9
    s, d = star(n - 1)
    g = orc.build_csr(n, s, d)
    ones = np.ones((n, 1))
    # sum of ones is the degree: hub n, leaves 2
    np.testing.assert_array_equal(orc.aggregate(g, ones, kind="sum")[:, 0], [n] + [2] * (n - 1))
    # the mean keeps constant columns; the transpose of the mean sums 1/d over a row
    np.testing.assert_allclose(orc.aggregate(g, 3.5 * ones, kind="mean"), 3.5 * ones, rtol=1e-15)
    np.testing.assert_allclose(orc.aggregate(g, ones, kind="mean_t")[0, 0], 1 / n + (n - 1) / 2, rtol=1e-15)
    # complete graph: the mean is the column mean
    s, d = complete(6)
    g = orc.build_csr(6, s, d)
    M = np.arange(18.0).reshape(6, 3)
    np.testing.assert_allclose(orc.aggregate(g, M, kind="mean"), np.tile(M.mean(0), (6, 1)), rtol=1e-15)


def brute_max(n, rows, M):
    P = np.zeros_like(M)
    arg = np.zeros(M.shape, np.int32)
    for u in range(n):
        for c in range(M.shape[1]):
            vals = [M[v, c] for v in rows[u]]
            best = max(vals)
            P[u, c] = best
            arg[u, c] = rows[u][vals.index(best)]  # first maximal, columns ascending
    return P, arg


@pytest.mark.parametrize("seed", range(4))
def test_max_aggregation_brute_force_with_ties(orc, seed):
    rng = np.random.default_rng(200 + seed)
    n = 35
    src, dst = random_edges(rng, n, 80)
    g = orc.build_csr(n, src, dst)
    rows = brute_rows(n, src.tolist(), dst.tolist())
    M = rng.integers(-2, 3, (n, 6)).astype(np.float64)  # small integers: many ties
    P, arg = orc.aggregate_max(g, M)
    Pb, argb = brute_max(n, rows, M)
    np.testing.assert_array_equal(P, Pb)
    np.testing.assert_array_equal(arg, argb)
    assert (P >= M).all()  # the row includes the node itself
    # gradient: each output passes its gradient to the one input it copied
    dP = rng.standard_normal((n, 6))
    dM = orc.aggregate_max_backward(g, dP, arg)
    want = np.zeros_like(dM)
    for u in range(n):
        for v in rows[u]:  # gather form over the symmetric rows
            want[u] += dP[v] * (arg[v] == u)
    np.testing.assert_allclose(dM, want, atol=1e-14)
    np.testing.assert_allclose(dM.sum(0), dP.sum(0), atol=1e-12)


def torch_model_aggs(n, src, dst, X, Ws, bs, y, aggs):
    """Reference model in torch autograd: dense operators for the linear aggregators, a
    padded neighbour gather with max over the neighbourhood for the max one."""
    rows = brute_rows(n, src, dst)
    dmax = max(len(r) for r in rows)
    nb = torch.tensor([r + [r[0]] * (dmax - len(r)) for r in rows])  # pad with a repeat
    H = torch.tensor(np.asarray(X, np.float64))
    Wt = [torch.tensor(np.asarray(w, np.float64), requires_grad=True) for w in Ws]
    bt = [torch.tensor(np.asarray(b, np.float64), requires_grad=True) for b in bs]
    Zs = []
    for l, a in enumerate(aggs):
        if a == "max":
            P = H[nb].max(dim=1).values  # (n, dmax, w) -> (n, w)
            Z = P @ Wt[l] + bt[l]
        else:
            S = torch.tensor(brute_ahat(n, src, dst) if a == "gcn" else brute_operator(n, src, dst, a))
            Z = S @ (H @ Wt[l]) + bt[l]
        Zs.append(Z)
        H = torch.relu(Z) if l < len(Ws) - 1 else Z
    loss = torch.nn.functional.cross_entropy(Zs[-1], torch.tensor(y, dtype=torch.long))
    loss.backward()
    return loss.item(), [z.detach().numpy() for z in Zs], [w.grad.numpy() for w in Wt], \
        [b.grad.numpy() for b in bt]


@pytest.mark.parametrize("aggs", [("max", "sum", "mean"), ("sum", "max", "gcn"), ("mean", "mean", "max")])
def test_aggregator_models_match_torch_autograd(orc, aggs):
    src, dst, X, Ws, bs, y = tiny_problem(7, n=30, widths=(6, 5, 4, 3))
    n = X.shape[0]
    g = orc.build_csr(n, src, dst)
    Hs, Zs, aux = orc.forward_aux(g, X, Ws, bs, aggs=list(aggs))
    loss, G, _ = orc.softmax_ce(Zs[-1], y)
    dWs, dbs, _ = orc.backward(g, Hs, Zs, G, Ws, aggs=list(aggs), aux=aux)
    tl, tZ, tdW, tdb = torch_model_aggs(n, src.tolist(), dst.tolist(), X, Ws, bs, y, aggs)
    assert loss == pytest.approx(tl, rel=1e-12)
    for l in range(len(Ws)):
        np.testing.assert_allclose(Zs[l], tZ[l], atol=1e-12)
        np.testing.assert_allclose(dWs[l], tdW[l], atol=1e-12)
        np.testing.assert_allclose(dbs[l], tdb[l], atol=1e-13)


def test_max_model_central_differences(orc):
    """Max-aggregator model against central differences (inputs away from kinks and ties)."""
    for seed in range(200):
        src, dst, X, Ws, bs, y = tiny_problem(3000 + seed, n=12, widths=(4, 5, 3))
        g = orc.build_csr(12, src, dst)
        aggs = ["max", "max"]
        Hs, Zs, aux = orc.forward_aux(g, X, Ws, bs, aggs=aggs)
        # distinct values near every max: second-best at least 1e-3 below the best
        ok = np.abs(Zs[0]).min() > 1e-3
        for l in range(2):
            M = Hs[l]
            for u in range(12):
                row = g.col_idx[g.row_ptr[u]:g.row_ptr[u + 1]]
                srt = np.sort(M[row], axis=0)
                if row.size > 1 and (srt[-1] - srt[-2]).min() < 1e-3:
                    ok = False
        if ok:
            break
    else:
        pytest.fail("no kink-free sample")
    loss, G, _ = orc.softmax_ce(Zs[-1], y)
    dWs, dbs, _ = orc.backward(g, Hs, Zs, G, Ws, aggs=aggs, aux=aux)

    def f(Ws_, bs_):
        _, Z_ = orc.forward(g, X, Ws_, bs_, aggs=aggs)
        return orc.softmax_ce(Z_[-1], y)[0]

    h = 1e-6
    for l in range(2):
        for idx in np.ndindex(Ws[l].shape):
            Wp = [w.copy() for w in Ws]
            Wm = [w.copy() for w in Ws]
            Wp[l][idx] += h
            Wm[l][idx] -= h
            assert (f(Wp, bs) - f(Wm, bs)) / (2 * h) == pytest.approx(dWs[l][idx], abs=1e-8)
