"""fp64 CPU oracle for the GCN training path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` import this module.  It shares no code with the HIP library
(``paper_2512_01678_amd``) and never imports it.

It computes, slowly and plainly, what one epoch of full-batch GCN training
computes (paper: "Morphling: Fast, Fused, and Flexible GNN Training at
Scale", arXiv 2512.01678):

* the graph operator A_hat = D^-1/2 (A + I) D^-1/2 in CSR form (Section III-A,
  GCN "normalized mean aggregation"), and the other aggregators Section III-A and
  Listing 1 name: sum (A + I), mean (D^-1 (A + I)) and max (with its argmax),
* the density probe and the dense/sparse decision s >= tau (Section IV-B,
  Algorithm 1, Initialize), with DenseToCSR / DenseToCSC,
* the forward pass Z_l = A_hat (H_l W_l) + b_l, H_{l+1} = ReLU(Z_l) (the
  layer update of Section III-A; sparse X W on the sparse path, Algorithm 1,
  Forward),
* softmax cross-entropy over all nodes (the paper names no loss; this is the
  reading used throughout),
* the backward pass: Q_l = A_hat G_l (A_hat is symmetric), dW_l = H_l^T Q_l,
  db_l = sum_i G_l[i], G_{l-1} = (Q_l W_l^T) * 1[Z_{l-1} > 0] (Algorithm 1,
  Backward, with X^T G from the CSC view on the sparse path),
* Adam with bias correction (Listing 1: optimizer("adam", 0.01, 0.9, 0.999)).

Arithmetic is fp64; fp32 inputs are widened exactly.  The graph-shaped loops
live in ``gcn_oracle.c`` (plain C, compiled here with gcc, no fast-math); the
dense products use numpy's fp64 matmul as a library primitive.

Every function here is pinned by ``tests/test_oracle_pins.py`` against
something other than itself (brute force, closed forms, invariants,
independent library routines, finite differences).
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "gcn_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile gcn_oracle.c into liboracle.so (gcc -O2 -fopenmp, IEEE fp64)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-fno-fast-math", "-ffp-contract=off", SRC, "-o", tmp, "-lm"])
        os.replace(tmp, LIB)
    return LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = C.CDLL(LIB)
        P = C.c_void_p
        i32, i64 = C.c_int32, C.c_int64
        L.orc_build_csr.restype = i64
        L.orc_build_csr.argtypes = [i32, i64, P, P, i64, P, P, P, P]
        L.orc_feature_counts.restype = i64
        L.orc_feature_counts.argtypes = [P, i32, i32, i64, P]
        L.orc_sparse_decision.restype = i32
        L.orc_sparse_decision.argtypes = [i64, i64, i64, i32, i32]
        L.orc_dense_to_csr.restype = None
        L.orc_dense_to_csr.argtypes = [P, i32, i32, i64, P, P, P]
        L.orc_dense_to_csc.restype = None
        L.orc_dense_to_csc.argtypes = [P, i32, i32, i64, P, P, P]
        L.orc_aggregate.restype = None
        L.orc_aggregate.argtypes = [i32, P, P, P, P, i64, i32, P, P, i64, P, P, i64, i32]
        L.orc_aggregate_max.restype = None
        L.orc_aggregate_max.argtypes = [i32, P, P, P, i64, i32, P, P]
        L.orc_aggregate_max_backward.restype = None
        L.orc_aggregate_max_backward.argtypes = [i32, P, i32, P, P, i64]
        L.orc_spmm.restype = None
        L.orc_spmm.argtypes = [i64, P, P, P, P, i64, i32, P, i64, P]
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


# ---------------------------------------------------------------------------
# graph and feature statistics
# ---------------------------------------------------------------------------


class Graph:
    """CSR of A + I with degrees (see ``build_csr``)."""

    def __init__(self, n, row_ptr, col_idx, deg, dinv):
        self.n = n
        self.row_ptr = row_ptr
        self.col_idx = col_idx
        self.deg = deg
        self.dinv = dinv

    @property
    def nnz(self):
        return int(self.row_ptr[-1])


def build_csr(n: int, src: np.ndarray, dst: np.ndarray) -> Graph:
    """Neighbour sets of A + I as sorted CSR rows (Section III-A / GCN normalisation).

    Raises ValueError for an id outside [0, n).
    """
    src = np.ascontiguousarray(src, np.int32)
    dst = np.ascontiguousarray(dst, np.int32)
    cap = 2 * src.size + n
    row_ptr = np.zeros(n + 1, np.int64)
    col_idx = np.zeros(max(cap, 1), np.int32)
    deg = np.zeros(n, np.int32)
    dinv = np.zeros(n, np.float32)
    nnz = lib().orc_build_csr(n, src.size, _p(src), _p(dst), cap, _p(row_ptr), _p(col_idx),
                              _p(deg), _p(dinv))
    if nnz < 0:
        raise ValueError(f"orc_build_csr failed with code {nnz}")
    return Graph(n, row_ptr, col_idx[:nnz].copy(), deg, dinv)


def feature_counts(X: np.ndarray):
    """(nnz(X), per-row nnz) with x != 0.0f as the nonzero test (Section IV-B)."""
    X = np.ascontiguousarray(X, np.float32)
    n, f = X.shape
    rn = np.zeros(n, np.int64)
    nnz = lib().orc_feature_counts(_p(X), n, f, f, _p(rn))
    return int(nnz), rn


def sparse_decision(nnz: int, n: int, f: int, tau_num: int = 4, tau_den: int = 5) -> int:
    """1 (sparse path) iff s = 1 - nnz/(N F) >= tau_num/tau_den (Algorithm 1)."""
    return int(lib().orc_sparse_decision(nnz, n, f, tau_num, tau_den))


def sparsity(nnz: int, n: int, f: int) -> float:
    """s = 1 - nnz(X)/(N F) (Section IV-B), for display."""
    return 1.0 - nnz / float(n * f)


def dense_to_csr(X: np.ndarray):
    """DenseToCSR (Algorithm 1): (row_ptr int64, col int32, val fp32)."""
    X = np.ascontiguousarray(X, np.float32)
    n, f = X.shape
    nnz, _ = feature_counts(X)
    rp = np.zeros(n + 1, np.int64)
    col = np.zeros(max(nnz, 1), np.int32)
    val = np.zeros(max(nnz, 1), np.float32)
    lib().orc_dense_to_csr(_p(X), n, f, f, _p(rp), _p(col), _p(val))
    return rp, col[:nnz].copy(), val[:nnz].copy()


def dense_to_csc(X: np.ndarray):
    """DenseToCSC (Algorithm 1): (col_ptr int64, row int32, val fp32)."""
    X = np.ascontiguousarray(X, np.float32)
    n, f = X.shape
    nnz, _ = feature_counts(X)
    cp = np.zeros(f + 1, np.int64)
    row = np.zeros(max(nnz, 1), np.int32)
    val = np.zeros(max(nnz, 1), np.float32)
    lib().orc_dense_to_csc(_p(X), n, f, f, _p(cp), _p(row), _p(val))
    return cp, row[:nnz].copy(), val[:nnz].copy()


# ---------------------------------------------------------------------------
# per-step products
# ---------------------------------------------------------------------------


# linear aggregators (the AGGREGATE step of Section III-A): operator over the rows of A + I
KINDS = {"gcn": 0, "sum": 1, "mean": 2, "mean_t": 3}
# the operator that carries gradients back through each one (A_hat and A + I are symmetric)
TRANSPOSE = {"gcn": "gcn", "sum": "sum", "mean": "mean_t", "mean_t": "mean"}


def aggregate(g: Graph, M: np.ndarray, bias=None, rows=None, want_mag: bool = False, kind: str = "gcn"):
    """Z = S M + 1 b^T on all rows, or on the listed rows (Section III-A, Algorithm 3).

    S = A_hat = D^-1/2 (A+I) D^-1/2 ("gcn"), A + I ("sum"), D^-1 (A+I) ("mean") or
    (A+I) D^-1 ("mean_t", the transpose of the mean).  Returns Z (and the magnitude
    scale sum |S||M| + |b| when want_mag).
    """
    M = np.ascontiguousarray(M, np.float64)
    w = M.shape[1]
    b = None if bias is None else np.ascontiguousarray(bias, np.float64)
    r = None if rows is None else np.ascontiguousarray(rows, np.int32)
    cnt = g.n if r is None else r.size
    Z = np.zeros((cnt, w), np.float64)
    mag = np.zeros((cnt, w), np.float64) if want_mag else None
    if w > 0 and cnt > 0:
        lib().orc_aggregate(g.n, _p(g.row_ptr), _p(g.col_idx), _p(g.deg), _p(M), w, w, _p(b),
                            _p(Z), w, _p(mag), _p(r), cnt, KINDS[kind])
    return (Z, mag) if want_mag else Z


def aggregate_max(g: Graph, M: np.ndarray):
    """Max aggregation over the rows of A + I (the "Max" aggregator of Listing 1).

    Returns (P, argmax): P[u,c] = max_v M[v,c] over u's row, argmax the first such v.
    """
    M = np.ascontiguousarray(M, np.float64)
    w = M.shape[1]
    P = np.zeros((g.n, w), np.float64)
    arg = np.zeros((g.n, w), np.int32)
    if w > 0 and g.n > 0:
        lib().orc_aggregate_max(g.n, _p(g.row_ptr), _p(g.col_idx), _p(M), w, w, _p(P), _p(arg))
    return P, arg


def aggregate_max_backward(g: Graph, dP: np.ndarray, argmax: np.ndarray):
    """Gradient of the max aggregation: dM[argmax[u,c], c] += dP[u,c]."""
    dP = np.ascontiguousarray(dP, np.float64)
    arg = np.ascontiguousarray(argmax, np.int32)
    w = dP.shape[1]
    dM = np.zeros((g.n, w), np.float64)
    if w > 0 and g.n > 0:
        lib().orc_aggregate_max_backward(g.n, _p(dP), w, _p(arg), _p(dM), w)
    return dM


def spmm(ptr, idx, val, B, want_mag: bool = False):
    """C[i] = sum_e val[e] B[idx[e]] over compressed row i (sparse X W or X^T G)."""
    B = np.ascontiguousarray(B, np.float64)
    w = B.shape[1]
    ptr = np.ascontiguousarray(ptr, np.int64)
    idx = np.ascontiguousarray(idx, np.int32)
    v = np.ascontiguousarray(val, np.float64)
    nrows = ptr.size - 1
    Cm = np.zeros((nrows, w), np.float64)
    mag = np.zeros((nrows, w), np.float64) if want_mag else None
    if w > 0 and nrows > 0:
        lib().orc_spmm(nrows, _p(ptr), _p(idx), _p(v), _p(B), w, w, _p(Cm), w, _p(mag))
    return (Cm, mag) if want_mag else Cm


def matmul(A, B, want_mag: bool = False):
    """Dense fp64 product A B (the vendor-BLAS step of Algorithm 1), with |A||B| scale."""
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    out = A @ B
    return (out, np.abs(A) @ np.abs(B)) if want_mag else out


def softmax_ce(Z: np.ndarray, y: np.ndarray):
    """Mean softmax cross-entropy over all N rows and its gradient w.r.t. the logits.

    l_i = log sum_c exp(z_ic - max_i) + max_i - z_{i,y_i};  loss = (1/N) sum_i l_i;
    G = (softmax(Z) - onehot(y)) / N.  Returns (loss, G, per-row l).
    """
    Z = np.asarray(Z, np.float64)
    n = Z.shape[0]
    mx = Z.max(axis=1, keepdims=True)
    ex = np.exp(Z - mx)
    se = ex.sum(axis=1, keepdims=True)
    rows = np.arange(n)
    li = np.log(se[:, 0]) + mx[:, 0] - Z[rows, y]
    G = ex / se
    G[rows, y] -= 1.0
    G /= n
    return float(li.sum() / n), G, li


def adam(theta, g, m, v, t: int, lr=0.01, b1=0.9, b2=0.999, eps=1e-8):
    """One Adam step with bias correction (Listing 1 optimizer("adam", 0.01, 0.9, 0.999)).

    m <- b1 m + (1-b1) g;  v <- b2 v + (1-b2) g^2;
    theta <- theta - lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps).  Returns new arrays.
    """
    theta = np.asarray(theta, np.float64)
    g = np.asarray(g, np.float64)
    m = b1 * np.asarray(m, np.float64) + (1.0 - b1) * g
    v = b2 * np.asarray(v, np.float64) + (1.0 - b2) * g * g
    mhat = m / (1.0 - b1 ** t)
    vhat = v / (1.0 - b2 ** t)
    return theta - lr * mhat / (np.sqrt(vhat) + eps), m, v


# ---------------------------------------------------------------------------
# whole layers and one epoch
# ---------------------------------------------------------------------------


class SparseX:
    """X in both compressed forms (Algorithm 1: X_csr for Forward, X_csc for Backward)."""

    def __init__(self, X):
        self.n, self.f = X.shape
        self.csr = dense_to_csr(X)
        self.csc = dense_to_csc(X)


def forward(g: Graph, X, Ws, bs, sparse: SparseX | None = None, aggs=None):
    """Z_l = AGG_l(H_l W_l) + b_l;  H_{l+1} = ReLU(Z_l) for l < L-1;  H_0 = X.

    AGG_l is A_hat (default) or the aggregator aggs[l] ("gcn", "sum", "mean", "max");
    a linear aggregator commutes with W, the max one is applied first:
    Z_l = max-aggregate(H_l) W_l + b_l.  With ``sparse`` the first transform of a
    linear layer is X_csr W_0 (Algorithm 1, Forward).
    Returns (Hs, Zs): Hs[l] is the input of layer l, Zs[l] its pre-activation.
    """
    Hs, Zs, _ = forward_aux(g, X, Ws, bs, sparse, aggs)
    return Hs, Zs


def forward_aux(g: Graph, X, Ws, bs, sparse: SparseX | None = None, aggs=None):
    """``forward`` plus, for max layers, the saved (P, argmax) in aux[l]."""
    L = len(Ws)
    aggs = aggs or ["gcn"] * L
    Hs = [np.asarray(X, np.float64)]
    Zs, aux = [], [None] * L
    for l in range(L):
        if aggs[l] == "max":
            P, arg = aggregate_max(g, Hs[l])
            aux[l] = (P, arg)
            Z = matmul(P, Ws[l]) + np.asarray(bs[l], np.float64)
        else:
            if l == 0 and sparse is not None:
                rp, col, val = sparse.csr
                Mt = spmm(rp, col, val, Ws[0])
            else:
                Mt = matmul(Hs[l], Ws[l])
            Z = aggregate(g, Mt, bs[l], kind=aggs[l])
        Zs.append(Z)
        if l < L - 1:
            Hs.append(np.maximum(Z, 0.0))
    return Hs, Zs, aux


def backward(g: Graph, Hs, Zs, G_last, Ws, sparse: SparseX | None = None, aggs=None, aux=None,
             relu_on=None):
    """Gradients of the mean loss for every layer (Algorithm 1, Backward).

    Linear layers: Q_l = S_l^T G_l (A_hat and A + I are symmetric, the mean's transpose
    is (A+I) D^-1);  dW_l = H_l^T Q_l (X_csc Q_0 on the sparse path);
    G_{l-1} = (Q_l W_l^T) * 1[Z_{l-1} > 0].
    Max layers: dW_l = P_l^T G_l;  G_{l-1} = maxgrad(G_l W_l^T) * 1[Z_{l-1} > 0].
    db_l = sum_i G_l[i,:].  Returns (dWs, dbs, Gs) with Gs[l] = dLoss/dZ_l.

    relu_on: optional list; relu_on[l] (boolean, the shape of Z_l) replaces 1[Z_l > 0],
    so that a comparison can take the ReLU decisions where another implementation took
    them (a decision on a pre-activation within rounding of zero is precision-dependent).
    """
    L = len(Ws)
    aggs = aggs or ["gcn"] * L
    on = [relu_on[l] if relu_on is not None and relu_on[l] is not None else (Zs[l] > 0.0)
          for l in range(L - 1)]
    dWs, dbs, Gs = [None] * L, [None] * L, [None] * L
    G = np.asarray(G_last, np.float64)
    for l in range(L - 1, -1, -1):
        Gs[l] = G
        dbs[l] = G.sum(axis=0)
        Wt = np.asarray(Ws[l], np.float64).T
        if aggs[l] == "max":
            P, arg = aux[l]
            dWs[l] = matmul(P.T, G)
            if l > 0:
                G = aggregate_max_backward(g, matmul(G, Wt), arg) * on[l - 1]
            continue
        Q = aggregate(g, G, kind=TRANSPOSE[aggs[l]])
        if l == 0 and sparse is not None:
            cp, row, val = sparse.csc
            dWs[l] = spmm(cp, row, val, Q)
        else:
            dWs[l] = matmul(Hs[l].T, Q)
        if l > 0:
            G = matmul(Q, Wt) * on[l - 1]
    return dWs, dbs, Gs


def epoch(g: Graph, X, y, Ws, bs, mW, vW, mb, vb, t: int, sparse: SparseX | None = None,
          lr=0.01, b1=0.9, b2=0.999, eps=1e-8, aggs=None, relu_on=None):
    """One training epoch: forward, softmax-CE loss, backward, Adam step t (t >= 1).

    aggs: per-layer aggregator ("gcn" default, "sum", "mean", "max").  relu_on: optional
    callable (Zs -> list of boolean masks) giving the backward's ReLU decisions (see
    backward).  Returns a dict with loss, activations, gradients and updated
    parameters/state.
    """
    Hs, Zs, aux = forward_aux(g, X, Ws, bs, sparse, aggs)
    loss, G, _ = softmax_ce(Zs[-1], y)
    dWs, dbs, Gs = backward(g, Hs, Zs, G, Ws, sparse, aggs, aux,
                            relu_on=relu_on(Zs) if relu_on is not None else None)
    nW, nmW, nvW, nb, nmb, nvb = [], [], [], [], [], []
    for l in range(len(Ws)):
        a, m_, v_ = adam(Ws[l], dWs[l], mW[l], vW[l], t, lr, b1, b2, eps)
        nW.append(a), nmW.append(m_), nvW.append(v_)
        a, m_, v_ = adam(bs[l], dbs[l], mb[l], vb[l], t, lr, b1, b2, eps)
        nb.append(a), nmb.append(m_), nvb.append(v_)
    return dict(loss=loss, Hs=Hs, Zs=Zs, G=G, Gs=Gs, dWs=dWs, dbs=dbs, Ws=nW, bs=nb, mW=nmW,
                vW=nvW, mb=nmb, vb=nvb, aux=aux)


def epoch_row_blocks(g: Graph, x_rows, f: int, y, Ws, bs, mW, vW, mb, vb, t: int, sparse: bool = False,
                     block_rows: int = 65536, lr=0.01, b1=0.9, b2=0.999, eps=1e-8):
    """``epoch`` for input features too large to hold whole (GCN aggregator, ReLU hidden layers).

    x_rows(r0, r1) returns rows r0 .. r1-1 of X (fp32).  The two products that read X,
    X W_0 in the forward pass and dW_0 = X^T Q_0 in the backward pass, run over row blocks
    (dW_0 as the sum of the blocks' X_b^T Q_0[b], in block order); with ``sparse`` each block
    goes through DenseToCSR / DenseToCSC and the sparse products of Algorithm 1.  Every
    other step is the one ``epoch`` takes.  Returns loss, gradients and updated parameters.
    """
    n = g.n
    L = len(Ws)
    Wd = [np.asarray(w, np.float64) for w in Ws]
    blocks = [(r0, min(n, r0 + block_rows)) for r0 in range(0, n, block_rows)]
    M0 = np.zeros((n, Wd[0].shape[1]))
    for r0, r1 in blocks:
        Xb = np.asarray(x_rows(r0, r1), np.float32)
        if sparse:
            rp, col, val = dense_to_csr(Xb)
            M0[r0:r1] = spmm(rp, col, val, Wd[0])
        else:
            M0[r0:r1] = matmul(Xb, Wd[0])
    Zs = [aggregate(g, M0, bs[0])]
    Hs = [None]
    for l in range(1, L):
        Hs.append(np.maximum(Zs[-1], 0.0))
        Zs.append(aggregate(g, matmul(Hs[l], Wd[l]), bs[l]))
    loss, G, _ = softmax_ce(Zs[-1], y)
    dWs, dbs = [None] * L, [None] * L
    for l in range(L - 1, -1, -1):
        dbs[l] = G.sum(axis=0)
        Q = aggregate(g, G)
        if l > 0:
            dWs[l] = matmul(Hs[l].T, Q)
            G = matmul(Q, Wd[l].T) * (Zs[l - 1] > 0.0)
            continue
        dW0 = np.zeros_like(Wd[0])
        for r0, r1 in blocks:
            Xb = np.asarray(x_rows(r0, r1), np.float32)
            if sparse:
                cp, row, val = dense_to_csc(Xb)
                dW0 += spmm(cp, row, val, Q[r0:r1])
            else:
                dW0 += matmul(Xb.T, Q[r0:r1])
        dWs[0] = dW0
    out = dict(loss=loss, dWs=dWs, dbs=dbs, Ws=[], bs=[], mW=[], vW=[], mb=[], vb=[])
    for l in range(L):
        a, m_, v_ = adam(Ws[l], dWs[l], mW[l], vW[l], t, lr, b1, b2, eps)
        out["Ws"].append(a), out["mW"].append(m_), out["vW"].append(v_)
        a, m_, v_ = adam(bs[l], dbs[l], mb[l], vb[l], t, lr, b1, b2, eps)
        out["bs"].append(a), out["mb"].append(m_), out["vb"].append(v_)
    return out


def dense_operator(g: Graph, kind: str = "gcn") -> np.ndarray:
    """The aggregation operator (A_hat by default) as a dense fp64 matrix (small graphs only)."""
    A = np.zeros((g.n, g.n), np.float64)
    for u in range(g.n):
        for e in range(g.row_ptr[u], g.row_ptr[u + 1]):
            v = g.col_idx[e]
            du, dv = float(g.deg[u]), float(g.deg[v])
            A[u, v] = {"gcn": 1.0 / np.sqrt(du * dv), "sum": 1.0, "mean": 1.0 / du, "mean_t": 1.0 / dv}[kind]
    return A
