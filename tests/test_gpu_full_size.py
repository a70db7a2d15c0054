"""Parity at the full size of every workload, in the benchmark's launch configuration.

One training epoch (Algorithm 1 forward and backward, the softmax cross-entropy, Adam)
of each full-size workload runs on the GPU as bench.py runs it: X at the bench's pitch,
the density probe choosing the path (with the paper's tau = 4/5, so that the RMAT
features at 10 % density take the sparse path too), the CSC view for a sparse first
layer, the row order of the aggregations kept or dropped by the same timing, every
product at its automatic kernel choice.  Then the fp64 oracle
checks, from the GPU's own layer inputs (unit parity, each element against its
magnitude scale sum |terms|):
  * every hidden layer's output H_{l+1} (and the saved aggregate of an aggregate-first
    layer) on about 400 random rows plus every hub row longer than GCN_SPLIT_MIN (the
    rows the library cuts into chunks) and the 20 longest rows, with the ReLU decisions
    that differ counted and bounded;
  * the loss and G = dLoss/dZ of the last layer on all rows;
  * every layer's backward from the GPU's own G_l: the full weight gradient dW_l (on the
    RMAT workloads 128 sampled rows of dW_0 = X^T Q_0, each a sum over all 2^21 nodes),
    the full bias gradient, and G_{l-1} on the sampled rows;
  * the Adam step of every parameter.
The arxiv-shaped workload is checked on every row, also with the sum, mean and max
aggregators on every layer (there the loss layer's gradient is held to what its logits'
rounding allows per row: dG/dz moves G by at most 2/N of a logit's error, and the sum
aggregator's logits reach thousands).  These sizes reach what the small
tests cannot: operands above 2 GiB (H of the products-shaped graph is 2.5 GB, the RMAT
features 34 GB), split-k weight gradients over 2.45 M rows, the row-panel products
with 19,133 row panels, hub splitting on the RMAT graph and the row-chunk-tiled
X^T Q over 256 chunks.
"""
import numpy as np
import pytest
import torch

import gcn_synth as gs
from helpers import assert_mag_close, assert_norm_close, note, relu_flips

pytestmark = pytest.mark.gpu

SPLIT_MIN = 4096  # GCN_SPLIT_MIN of include/gcn.h


@pytest.fixture(scope="module")
def G():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2512_01678_amd.gcn as G
    return G


def host(t, w=None):
    torch.cuda.synchronize()
    a = t.detach().cpu().numpy()
    if w is not None:
        a = a[:, :w]
    return a.astype(np.float64)


def sample_rows(og, count, seed=0):
    rng = np.random.default_rng(seed)
    n = og.n
    hubs = np.nonzero(og.deg > SPLIT_MIN)[0]
    top = np.argsort(og.deg, kind="stable")[-20:]
    return np.unique(np.concatenate([rng.integers(0, n, count), hubs, top])).astype(np.int32), hubs.size


def neighbours(og, rows):
    parts = [og.col_idx[og.row_ptr[r]:og.row_ptr[r + 1]] for r in rows]
    return np.unique(np.concatenate(parts)).astype(np.int64)


class Run:
    """One workload set up and trained for one epoch as bench.py does it."""

    def __init__(self, G, orc, wl, graph=None, agg=None, csc=True):
        self.wl = wl
        self.agg = agg  # None: the normalised GCN operator; else "sum", "mean" or "max" on every layer
        n = wl.n
        note(f"{wl.name}: drawing inputs")
        if graph is None:
            s, d = gs.make_graph(wl)
            note(f"{wl.name}: {s.size} edges drawn; oracle CSR")
            self.og = orc.build_csr(n, s, d)
            self.dg = G.build_csr(n, torch.from_numpy(s).cuda(), torch.from_numpy(d).cuda())
            del s, d
            # the row order, kept or dropped by the same setup-time timing as the bench's
            kept = G.tune_row_order(self.dg, max(wl.widths[1:-1]) if len(wl.widths) > 2 else wl.widths[-1])
            note(f"{wl.name}: row order {'kept' if kept else 'dropped'}")
        else:
            self.og, self.dg = graph
        assert self.dg.nnz == self.og.nnz
        self.on_device = n * wl.f > (1 << 28)
        self.X = None if self.on_device else gs.make_features(wl)
        self.y = gs.make_labels(wl)
        self.Ws, self.bs = gs.make_weights(wl)
        ld_x = G.pitch(wl.f)
        self.Xd = torch.zeros((n, ld_x), dtype=torch.float32, device="cuda")
        self.Xv = self.Xd[:, :wl.f]
        if self.on_device:
            from gcn_synth import device
            device.bernoulli_into(self.Xv, wl.density, seed=0, stream=3, binary=(wl.features == "binary"))
        else:
            self.Xv.copy_(torch.from_numpy(self.X).cuda())
        torch.cuda.synchronize()
        info, self.sx = G.feature_stats(self.Xv, tau=(4, 5), force_mode=-1, csc=csc)
        self.sparse = info["mode"] == G.SPARSE
        note(f"{wl.name}: nnz(A+I) {self.og.nnz}, probe s = {info['sparsity']:.4f} -> "
             f"{'sparse' if self.sparse else 'dense'}; one GPU epoch")
        aggs = None if agg is None else [{"sum": G.AGG_SUM, "mean": G.AGG_MEAN, "max": G.AGG_MAX}[agg]] * (len(wl.widths) - 1)
        self.m = G.Model(n, wl.widths, self.Ws, self.bs, x_sparse=self.sparse, ld_x=ld_x, aggs=aggs)
        self.m.epoch(self.dg, X=None if self.sparse else self.Xv, x=self.sx,
                     labels=torch.from_numpy(self.y).cuda())
        torch.cuda.synchronize()

    def x_rows(self, rows):
        """Rows of X in fp64 on the host (drawn on the device for the RMAT features, by the
        same counter stream as the host generator)."""
        if self.X is not None:
            return self.X[rows].astype(np.float64)
        out = np.empty((rows.size, self.wl.f), np.float64)
        idx = torch.from_numpy(np.asarray(rows, np.int64))
        for r0 in range(0, rows.size, 32768):
            sel = idx[r0:r0 + 32768].cuda()
            out[r0:r0 + sel.numel()] = self.Xv.index_select(0, sel).cpu().numpy()
        return out


def check_run(G, orc, run, rows, what, x_cols=None):
    """The oracle checks described in the module docstring; rows=None: every row."""
    wl, og, m = run.wl, run.og, run.m
    n, L = wl.n, m.L
    all_rows = rows is None
    if all_rows:
        rows = np.arange(n, dtype=np.int32)
    need = np.arange(n) if all_rows else neighbours(og, rows)
    Ws = [w.astype(np.float64) for w in run.Ws]
    bs = [b.astype(np.float64) for b in run.bs]
    Hs = [None] + [host(a, wl.widths[l + 1]) for l, a in enumerate(m.act)]
    flips = 0
    # forward of every hidden layer on the sampled rows, from the GPU's own layer input
    for l in range(L - 1):
        note(f"{what}: forward layer {l} on {rows.size} rows ({need.size} neighbour rows)")
        M = np.zeros((n, wl.widths[l + 1]))
        Ma = np.zeros_like(M)
        for b0 in range(0, need.size, 65536):  # row blocks bound the host memory of wide X
            blk = need[b0:b0 + 65536]
            Hin = run.x_rows(blk) if l == 0 else Hs[l][blk]
            M[blk] = Hin @ Ws[l]
            Ma[blk] = np.abs(Hin) @ np.abs(Ws[l])
        del Hin
        Z = orc.aggregate(og, M, bs[l], rows=rows)
        mag = orc.aggregate(og, Ma, np.abs(bs[l]), rows=rows)
        got = Hs[l + 1][rows]
        flips += relu_flips(got > 0, Z, mag, f"{what} H_{l + 1}")
        assert_mag_close(got, np.maximum(Z, 0), mag, f"{what} H_{l + 1}")
        if m.saved[l] is not None:
            Xn = np.zeros((n, wl.widths[l]))
            Xn[need] = run.x_rows(need) if l == 0 else Hs[l][need]
            P, pmag = orc.aggregate(og, Xn, rows=rows, want_mag=True)
            assert_mag_close(host(m.saved[l], wl.widths[l])[rows], P, pmag, f"{what} saved aggregate {l}")
        del M, Ma
    # loss layer on every row
    note(f"{what}: loss layer")
    Zl = orc.aggregate(og, Hs[L - 1] @ Ws[L - 1], bs[L - 1])
    lo, Gl, _ = orc.softmax_ce(Zl, run.y)
    assert float(m.loss.cpu()[0]) == pytest.approx(lo, rel=1e-4), f"{what} loss"
    assert_norm_close(host(m.grad[L - 1], wl.widths[L]), Gl, f"{what} G_{L - 1}")
    del Zl, Gl
    # backward of every layer from the GPU's own G_l
    for l in range(L - 1, -1, -1):
        note(f"{what}: backward layer {l}")
        Gg = host(m.grad[l], wl.widths[l + 1])
        Q, aQ = orc.aggregate(og, Gg, want_mag=True)
        assert_mag_close(host(m.db[l][None, :])[0], Gg.sum(axis=0), np.abs(Gg).sum(axis=0), f"{what} db_{l}")
        if l == 0 and x_cols is not None:
            # sampled rows k of dW_0 = X^T Q_0: column k of X over all nodes (X >= 0 here)
            Xc = run.Xv[:, torch.from_numpy(x_cols).cuda()].cpu().numpy().astype(np.float64)
            assert (Xc >= 0).all()
            assert_mag_close(host(m.dW[0])[x_cols], Xc.T @ Q, Xc.T @ aQ, f"{what} dW_0 rows")
            del Xc
        else:
            Hin = run.x_rows(np.arange(n)) if l == 0 else Hs[l]
            assert_mag_close(host(m.dW[l]), Hin.T @ Q, np.abs(Hin).T @ aQ, f"{what} dW_{l}")
            del Hin
        if l > 0:
            ref = (Q[rows] @ Ws[l].T) * (Hs[l][rows] > 0)
            mag = aQ[rows] @ np.abs(Ws[l]).T
            assert_mag_close(host(m.grad[l - 1], wl.widths[l])[rows], ref, mag, f"{what} G_{l - 1}")
        del Gg, Q, aQ
    # Adam step 1 from the initial parameters with the GPU's own gradients
    for l in range(L):
        for nm, gnm, p0 in (("W", "dW", Ws[l]), ("b", "db", bs[l])):
            g = host(getattr(m, gnm)[l][None] if nm == "b" else getattr(m, gnm)[l])
            g = g[0] if nm == "b" else g
            want, _, _ = orc.adam(p0, g, np.zeros_like(p0), np.zeros_like(p0), 1)
            got = host(getattr(m, nm)[l][None] if nm == "b" else getattr(m, nm)[l])
            got = got[0] if nm == "b" else got
            assert_mag_close(got, want, np.abs(p0) + 0.01, f"{what} Adam {nm}_{l}", rtol=1e-5)
    note(f"{what}: passed ({flips} ReLU flips near zero in total)")


def test_full_size_arxiv_like_every_row(G, orc):
    run = Run(G, orc, gs.WORKLOADS["arxiv_like"])
    assert run.m.orders() == [G.AGGREGATE_FIRST, G.TRANSFORM_FIRST, G.TRANSFORM_FIRST]
    check_run(G, orc, run, None, "arxiv_like")


@pytest.mark.parametrize("name", ["reddit_like", "products_like"])
def test_full_size_sampled_rows(G, orc, name):
    run = Run(G, orc, gs.WORKLOADS[name])
    rows, n_hubs = sample_rows(run.og, 400)
    note(f"{name}: {rows.size} sampled rows, {n_hubs} hub rows above {SPLIT_MIN} entries")
    want = {"reddit_like": [G.TRANSFORM_FIRST, G.TRANSFORM_FIRST],
            "products_like": [G.AGGREGATE_FIRST, G.TRANSFORM_FIRST, G.TRANSFORM_FIRST]}[name]
    assert run.m.orders() == want
    check_run(G, orc, run, rows, name)


@pytest.fixture(scope="module")
def rmat_graph(G, orc):
    wl = gs.WORKLOADS["rmat21_p0.5"]
    note("rmat21: drawing 2^25 samples")
    s, d = gs.make_graph(wl)
    og = orc.build_csr(wl.n, s, d)
    dg = G.build_csr(wl.n, torch.from_numpy(s).cuda(), torch.from_numpy(d).cuda())
    kept = G.tune_row_order(dg, max(wl.widths[1:-1]))
    note(f"rmat21: row order {'kept' if kept else 'dropped'}")
    return og, dg


@pytest.mark.parametrize("density", [0.5, 0.1, 0.01, 0.001])
def test_full_size_rmat(G, orc, rmat_graph, density):
    wl = gs.WORKLOADS[f"rmat21_p{density:g}"]
    run = Run(G, orc, wl, graph=rmat_graph)
    assert run.sparse == (density < 0.2)
    # the device-drawn features equal the host generator's on sampled rows
    rng = np.random.default_rng(1)
    for r in rng.integers(0, wl.n, 4):
        want = gs.features_bernoulli(wl.n, wl.f, density, seed=0, stream=3, row0=int(r), rows=1, binary=False)
        np.testing.assert_array_equal(run.Xv[int(r)].cpu().numpy(), want[0])
    rows, n_hubs = sample_rows(run.og, 400)
    note(f"{wl.name}: {rows.size} sampled rows, {n_hubs} hub rows above {SPLIT_MIN} entries")
    x_cols = np.unique(np.concatenate([rng.integers(0, wl.f, 120), [0, 1, wl.f - 2, wl.f - 1]])).astype(np.int64)
    check_run(G, orc, run, rows, wl.name, x_cols=x_cols)
    del run
    torch.cuda.empty_cache()


def test_full_size_rmat_atomic_transpose(G, orc, rmat_graph):
    """The sparse path without the CSC view (`bench.py --csc off`): dW_0 = X^T Q_0 by atomic
    adds from X_csr rows, at the 1 % RMAT workload's full size; its rounding order varies
    from run to run, the result stays within the magnitude bar."""
    wl = gs.WORKLOADS["rmat21_p0.01"]
    run = Run(G, orc, wl, graph=rmat_graph, csc=False)
    assert run.sparse and run.sx.col_ptr is None
    rng = np.random.default_rng(2)
    rows, n_hubs = sample_rows(run.og, 400)
    x_cols = np.unique(np.concatenate([rng.integers(0, wl.f, 120), [0, wl.f - 1]])).astype(np.int64)
    check_run(G, orc, run, rows, wl.name + " (atomic X^T Q)", x_cols=x_cols)
    del run
    torch.cuda.empty_cache()


def check_run_agg(G, orc, run, what):
    """check_run's unit parity on every row for a model whose layers all use run.agg (sum,
    mean or max): each layer from the GPU's own input, the loss layer's gradient per row
    within what its logits' rounding allows, every backward from the GPU's own G_l."""
    wl, og, m, agg = run.wl, run.og, run.m, run.agg
    n, L = wl.n, m.L
    Ws = [w.astype(np.float64) for w in run.Ws]
    bs = [b.astype(np.float64) for b in run.bs]
    Hs = [run.x_rows(np.arange(n))] + [host(a, wl.widths[l + 1]) for l, a in enumerate(m.act)]
    Ps = [None] * L  # max: the oracle's aggregate of each layer input (exact, as the GPU's)
    args = [None] * L
    flips = 0

    def layer(l):
        """Z_l and its magnitude scale from the GPU's own H_l."""
        if agg == "max":
            P, arg = orc.aggregate_max(og, Hs[l])
            got_p = host(m.saved[l], wl.widths[l])
            np.testing.assert_array_equal(got_p, P, err_msg=f"{what} max aggregate {l}")
            ld = m.saved[l].stride(0)
            # the maximisers follow the n rows of the saved aggregate in the same buffer
            full = torch.as_strided(m.saved[l], (2 * n, ld), (ld, 1))
            got_arg = full[n:].view(torch.int32)[:, :wl.widths[l]]
            np.testing.assert_array_equal(host(got_arg), arg, err_msg=f"{what} argmax {l}")
            Ps[l], args[l] = P, arg
            return P @ Ws[l] + bs[l], np.abs(P) @ np.abs(Ws[l]) + np.abs(bs[l])
        Z = orc.aggregate(og, Hs[l] @ Ws[l], bs[l], kind=agg)
        mag = orc.aggregate(og, np.abs(Hs[l]) @ np.abs(Ws[l]), np.abs(bs[l]), kind=agg)
        if m.saved[l] is not None:
            P, pmag = orc.aggregate(og, Hs[l], kind=agg, want_mag=True)
            assert_mag_close(host(m.saved[l], wl.widths[l]), P, pmag, f"{what} saved aggregate {l}")
        return Z, mag

    for l in range(L - 1):
        note(f"{what}: forward layer {l}")
        Z, mag = layer(l)
        got = Hs[l + 1]
        flips += relu_flips(got > 0, Z, mag, f"{what} H_{l + 1}")
        assert_mag_close(got, np.maximum(Z, 0), mag, f"{what} H_{l + 1}")
    note(f"{what}: loss layer")
    Zl, zmag = layer(L - 1)
    lo, Gl, _ = orc.softmax_ce(Zl, run.y)
    assert float(m.loss.cpu()[0]) == pytest.approx(lo, rel=1e-4), f"{what} loss"
    # dG/dz has row sums of absolute values <= 2 / N, so a logit error within 1e-4 of its
    # scale moves G by at most 2e-4 / N times the row's largest logit scale
    gg = host(m.grad[L - 1], wl.widths[L])
    bound = 2e-4 * zmag.max(axis=1, keepdims=True) / n + 1e-7 / n
    worst = float((np.abs(gg - Gl) / bound).max())
    assert worst <= 1.0, f"{what} G_{L - 1}: error {worst:.3f} of its per-row bound"
    del Zl, Gl
    for l in range(L - 1, -1, -1):
        note(f"{what}: backward layer {l}")
        Gg = host(m.grad[l], wl.widths[l + 1])
        assert_mag_close(host(m.db[l][None, :])[0], Gg.sum(axis=0), np.abs(Gg).sum(axis=0), f"{what} db_{l}")
        if agg == "max":
            P = Ps[l]
            assert_mag_close(host(m.dW[l]), P.T @ Gg, np.abs(P).T @ np.abs(Gg), f"{what} dW_{l}")
            if l > 0:
                dP = Gg @ Ws[l].T
                dPm = np.abs(Gg) @ np.abs(Ws[l]).T
                ref = orc.aggregate_max_backward(og, dP, args[l]) * (Hs[l] > 0)
                mag = orc.aggregate_max_backward(og, dPm, args[l])
                assert_mag_close(host(m.grad[l - 1], wl.widths[l]), ref, mag, f"{what} G_{l - 1}")
        else:
            Q, aQ = orc.aggregate(og, Gg, kind="mean_t" if agg == "mean" else agg, want_mag=True)
            assert_mag_close(host(m.dW[l]), Hs[l].T @ Q, np.abs(Hs[l]).T @ aQ, f"{what} dW_{l}")
            if l > 0:
                ref = (Q @ Ws[l].T) * (Hs[l] > 0)
                assert_mag_close(host(m.grad[l - 1], wl.widths[l]), ref, aQ @ np.abs(Ws[l]).T, f"{what} G_{l - 1}")
    for l in range(L):
        for nm, gnm, p0 in (("W", "dW", Ws[l]), ("b", "db", bs[l])):
            g = host(getattr(m, gnm)[l][None] if nm == "b" else getattr(m, gnm)[l])
            g = g[0] if nm == "b" else g
            want, _, _ = orc.adam(p0, g, np.zeros_like(p0), np.zeros_like(p0), 1)
            got = host(getattr(m, nm)[l][None] if nm == "b" else getattr(m, nm)[l])
            got = got[0] if nm == "b" else got
            assert_mag_close(got, want, np.abs(p0) + 0.01, f"{what} Adam {nm}_{l}", rtol=1e-5)
    note(f"{what}: passed ({flips} ReLU flips near zero in total)")


@pytest.mark.parametrize("agg", ["sum", "mean", "max"])
def test_full_size_arxiv_like_aggregators(G, orc, agg):
    """The full arxiv-shaped workload with every layer on the sum, mean or max aggregator
    (`bench.py --workload arxiv_like --agg ...`), checked on every row."""
    run = Run(G, orc, gs.WORKLOADS["arxiv_like"], agg=agg)
    if agg == "max":
        assert run.m.orders() == [G.AGGREGATE_FIRST] * 3
    check_run_agg(G, orc, run, f"arxiv_like {agg}")
