"""gcn_gemm_static, the entry point that allocates nothing, against gcn_gemm (through the C ABI).

Two calls in a row on one device, the second with a smaller product, each checked
bitwise against gcn_gemm with a caller workspace (the same kernels and launch plan) and
against the fp64 product within the 1e-4 bar.  Covers the split-k A^T B (partials in the
static scratch) and the row-panel A B (split weight planes in the static scratch).
"""
import ctypes as C

import numpy as np
import pytest
import torch

from helpers import assert_mag_close

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2512_01678_amd.gcn as G
    return G


def operands(op, m, n, k, seed, G):
    rng = np.random.default_rng(seed)
    a_shape = (k, m) if op == G.OP_TN else (m, k)
    b_shape = (n, k) if op == G.OP_NT else (k, n)
    A = rng.standard_normal(a_shape).astype(np.float32)
    B = rng.standard_normal(b_shape).astype(np.float32)
    bias = rng.standard_normal(n).astype(np.float32)
    return A, B, bias


def reference(op, A, B, bias):
    A64, B64 = A.astype(np.float64), B.astype(np.float64)
    if op == 2:  # TN
        return A64.T @ B64 + bias, np.abs(A64).T @ np.abs(B64) + np.abs(bias)
    if op == 1:  # NT
        return A64 @ B64.T + bias, np.abs(A64) @ np.abs(B64).T + np.abs(bias)
    return A64 @ B64 + bias, np.abs(A64) @ np.abs(B64) + np.abs(bias)


@pytest.mark.parametrize("shapes", [
    # split-k A^T B: 256 x 256 over 169,343 rows needs the whole 64 MiB, then a smaller one
    [("TN", 256, 256, 169343), ("TN", 100, 64, 40000)],
    # row-panel A B (the layer transform), then a smaller row-panel product
    [("NN", 100000, 256, 128), ("NN", 40000, 40, 256)],
    # a mixed pair: the row-panel scratch, then split-k partials over the same array
    [("NN", 60000, 128, 64), ("TN", 64, 47, 50000)],
])
def test_gemm_static_matches_gemm(G, shapes):
    L = G.raw_lib()
    for i, (opname, m, n, k) in enumerate(shapes):
        op = {"NN": G.OP_NN, "NT": G.OP_NT, "TN": G.OP_TN}[opname]
        A, B, bias = operands(op, m, n, k, 100 + i, G)
        Ad, Bd, bd = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda(), torch.from_numpy(bias).cuda()
        want = torch.full((m, n), float("nan"), device="cuda")
        got = torch.full((m, n), float("nan"), device="cuda")
        G.gemm(op, Ad, Bd, want, bias=bd)
        st = torch.cuda.current_stream().cuda_stream
        rc = L.gcn_gemm_static(op, m, n, k, Ad.data_ptr(), Ad.stride(0), Bd.data_ptr(), Bd.stride(0),
                               got.data_ptr(), got.stride(0), bd.data_ptr(), G.EPI_NONE, None, 0, C.c_void_p(st))
        assert rc == G.OK, L.gcn_last_error().decode()
        torch.cuda.synchronize()
        assert torch.equal(got, want), f"call {i} {opname} {m}x{n}x{k}: differs from gcn_gemm"
        ref, mag = reference(op, A, B, bias)
        assert_mag_close(got.cpu().numpy(), ref, mag, f"call {i} {opname} {m}x{n}x{k}")


def test_gemm_static_rejects_products_beyond_its_scratch(G):
    """A row-panel product with a long k, whose split weight planes (6 k n bytes) exceed the
    static array: GCN_E_CAPACITY, nothing launched, the output untouched."""
    L = G.raw_lib()
    m, n, k = 32768, 256, 50000
    Ad = torch.zeros((m, k), device="cuda")
    Bd = torch.zeros((k, n), device="cuda")
    out = torch.full((m, n), 7.0, device="cuda")
    nb = G.sz(0)
    assert L.gcn_gemm(G.OP_NN, m, n, k, None, k, None, n, None, n, None, 0, None, 0, None, C.byref(nb), None) == G.OK
    assert nb.value > (64 << 20)
    rc = L.gcn_gemm_static(G.OP_NN, m, n, k, Ad.data_ptr(), k, Bd.data_ptr(), n, out.data_ptr(), n, None,
                           G.EPI_NONE, None, 0, None)
    assert rc == G.E_CAPACITY
    torch.cuda.synchronize()
    assert (out == 7.0).all()
