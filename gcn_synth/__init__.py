"""Seeded synthetic inputs for the GCN training path.

This module only draws inputs: graphs, feature matrices, labels and initial
weights.  It holds none of the method's arithmetic (no normalisation, no
aggregation, no transform, no loss), so both the fp64 oracle and the HIP
library can consume what it produces without sharing code with each other.

Random numbers come from one counter-based generator: SplitMix64 (Steele,
Lea and Flood, "Fast splittable pseudorandom number generators", OOPSLA
2014).  A (seed, stream) pair names one SplitMix64 sequence; its i-th output
is the published finaliser applied to ``state + (i + 1) * GAMMA`` and can be
computed for any i without the ones before it, so a row range of a large
matrix can be regenerated on demand.

Workload shapes follow the datasets of the paper's evaluation (Table II:
ogbn-arxiv, Reddit, ogbn-products) plus a Cora-sized graph and a Graph500-style
RMAT graph; the datasets themselves are not used.
"""
from __future__ import annotations

import ctypes
import hashlib
import math
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_U64 = np.uint64
GAMMA = 0x9E3779B97F4A7C15
_M1 = 0xBF58476D1CE4E5B9
_M2 = 0x94D049BB133111EB
_MASK64 = (1 << 64) - 1

# ---------------------------------------------------------------------------
# counter-based generator
# ---------------------------------------------------------------------------


def _mix64_int(z: int) -> int:
    z &= _MASK64
    z = ((z ^ (z >> 30)) * _M1) & _MASK64
    z = ((z ^ (z >> 27)) * _M2) & _MASK64
    return z ^ (z >> 31)


def stream_state(seed: int, stream: int) -> int:
    """Starting state of the SplitMix64 sequence named by (seed, stream)."""
    return _mix64_int((seed * GAMMA + stream * 0xD1B54A32D192ED03 + 0x632BE59BD9B4E019) & _MASK64)


def _mix64_inplace(z: np.ndarray, t: np.ndarray) -> np.ndarray:
    """SplitMix64 finaliser applied in place to z (t is scratch of the same shape)."""
    np.right_shift(z, _U64(30), out=t)
    np.bitwise_xor(z, t, out=z)
    np.multiply(z, _U64(_M1), out=z)
    np.right_shift(z, _U64(27), out=t)
    np.bitwise_xor(z, t, out=z)
    np.multiply(z, _U64(_M2), out=z)
    np.right_shift(z, _U64(31), out=t)
    np.bitwise_xor(z, t, out=z)
    return z


_CHUNK = 1 << 20
_IOTA = np.arange(_CHUNK, dtype=np.uint64)


def draws(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """Outputs start .. start+count-1 of the (seed, stream) sequence, uint64."""
    out = np.empty(count, np.uint64)
    t = np.empty(min(count, _CHUNK), np.uint64)
    state = _U64(stream_state(seed, stream))
    for c0 in range(0, count, _CHUNK):
        k = min(_CHUNK, count - c0)
        z = out[c0:c0 + k]
        # z = state + (start + c0 + 1 + i) * GAMMA, in place (uint64 wraps)
        np.add(_IOTA[:k], _U64(start + c0 + 1), out=z)
        np.multiply(z, _U64(GAMMA), out=z)
        np.add(z, state, out=z)
        _mix64_inplace(z, t[:k])
    return out


def u01_f64(h: np.ndarray) -> np.ndarray:
    """Uniform in [0, 1) from the top 53 bits."""
    return (h >> _U64(11)).astype(np.float64) * (1.0 / 9007199254740992.0)


def u01_f64_open0(h: np.ndarray) -> np.ndarray:
    """Uniform in (0, 1] from the top 53 bits."""
    return ((h >> _U64(11)).astype(np.float64) + 1.0) * (1.0 / 9007199254740992.0)


# ---------------------------------------------------------------------------
# graphs
# ---------------------------------------------------------------------------


def _chung_lu_offset(n: int, mean_deg: float, dmax: float, alpha: float) -> float:
    """i0 such that the expected degree of node 0 is dmax for weights (i+i0)^-alpha."""
    i = np.arange(n, dtype=np.float64)

    def top(i0):
        w = (i + i0) ** (-alpha)
        return n * mean_deg * w[0] / w.sum()

    lo, hi = 1e-9, 1e12
    for _ in range(200):
        mid = math.sqrt(lo * hi)
        if top(mid) > dmax:
            lo = mid
        else:
            hi = mid
    return math.sqrt(lo * hi)


def permutation(n: int, seed: int, stream: int) -> np.ndarray:
    """A seeded random permutation of 0..n-1 (argsort of uniform keys)."""
    keys = draws(seed, stream, 0, n)
    return np.argsort(keys, kind="stable").astype(np.int32)


_HOST_LIB = None
_HOST_SRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "host_gen.c")
_HOST_SO = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsynth_host.so")


def build_host(force: bool = True) -> str:
    """Compile host_gen.c (the C edge sampler) into libsynth_host.so."""
    if force or not os.path.exists(_HOST_SO):
        tmp = _HOST_SO + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", _HOST_SRC, "-o", tmp])
        os.replace(tmp, _HOST_SO)
    return _HOST_SO


def host_lib():
    """The C edge sampler, or None when it is not built (the numpy loop then runs)."""
    global _HOST_LIB
    if _HOST_LIB is None and os.path.exists(_HOST_SO):
        L = ctypes.CDLL(_HOST_SO)
        L.synth_chung_lu_keys.restype = ctypes.c_int
        L.synth_chung_lu_keys.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_uint64,
                                          ctypes.c_void_p]
        _HOST_LIB = L
    return _HOST_LIB


def chung_lu(n: int, e_und: int, seed: int = 0, stream: int = 1, alpha: float = 2.0 / 3.0,
             dmax: float | None = None, permute: bool = True, use_c: bool = True):
    """Chung-Lu power-law graph with exactly ``e_und`` distinct undirected edges.

    Node i gets weight (i + i0)^-alpha (degree exponent 1 + 1/alpha); i0 puts the
    expected maximum degree at ``dmax`` (default min(n/8, 100 * mean)).  Both
    endpoints are drawn proportional to weight; self pairs are discarded and each
    pair is kept once, in (min, max) form, in sampling order, until exactly
    ``e_und`` remain.  Node ids are then randomly permuted.  Returns (src, dst)
    int32 arrays, one entry per undirected edge.  ``use_c``: draw the pairs with the C
    sampler when it is built (the same pairs as the numpy loop, much faster).
    """
    if e_und == 0:
        z = np.zeros(0, np.int32)
        return z, z.copy()
    mean = 2.0 * e_und / n
    if dmax is None:
        dmax = min(n / 8.0, 100.0 * mean)
    i0 = _chung_lu_offset(n, mean, dmax, alpha)
    w = (np.arange(n, dtype=np.float64) + i0) ** (-alpha)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    have = np.zeros(0, np.int64)
    off = 0
    hl = host_lib() if use_c else None
    if hl is not None:  # the same sampling rule in C (host_gen.c)
        keys = np.empty(e_und, np.int64)
        cdf = np.ascontiguousarray(cdf)
        rc = hl.synth_chung_lu_keys(n, e_und, cdf.ctypes.data, stream_state(seed, stream), keys.ctypes.data)
        if rc != 0:
            raise MemoryError("synth_chung_lu_keys: out of host memory")
        have = np.sort(keys)
    while have.size < e_und:
        need = e_und - have.size
        b = int(need * 1.15) + 1024
        h = draws(seed, stream, off, 2 * b)
        off += 2 * b
        u = np.minimum(np.searchsorted(cdf, u01_f64(h[:b]), side="right"), n - 1)
        v = np.minimum(np.searchsorted(cdf, u01_f64(h[b:]), side="right"), n - 1)
        keep = u != v
        lo = np.minimum(u, v)[keep].astype(np.int64)
        hi = np.maximum(u, v)[keep].astype(np.int64)
        keys = lo * n + hi
        uk, first = np.unique(keys, return_index=True)
        if have.size:
            pos = np.searchsorted(have, uk)
            pos_c = np.minimum(pos, have.size - 1)
            fresh = have[pos_c] != uk
            uk, first = uk[fresh], first[fresh]
        take = uk[np.argsort(first, kind="stable")][:need]
        have = np.union1d(have, take)
    src = (have // n).astype(np.int32)
    dst = (have % n).astype(np.int32)
    if permute:
        p = permutation(n, seed, stream + 1000)
        src, dst = p[src], p[dst]
    return src, dst


def rmat(scale: int, n_samples: int, a=0.57, b=0.19, c=0.19, seed: int = 0, stream: int = 1,
         permute: bool = True):
    """Graph500-style RMAT samples: 2^scale nodes, ``n_samples`` raw edges.

    At each of ``scale`` levels a uniform draw picks the quadrant (a, b, c,
    d = 1-a-b-c).  Raw samples keep their duplicates and self pairs.  Node ids
    are randomly permuted.  Returns (src, dst) int32.
    """
    n = 1 << scale
    src = np.zeros(n_samples, np.int64)
    dst = np.zeros(n_samples, np.int64)
    ab, abc = a + b, a + b + c
    chunk = 1 << 22
    for s0 in range(0, n_samples, chunk):
        cnt = min(chunk, n_samples - s0)
        su = np.zeros(cnt, np.int64)
        sv = np.zeros(cnt, np.int64)
        for lvl in range(scale):
            r = u01_f64(draws(seed, stream + lvl, s0, cnt))
            bit_u = r >= ab                      # quadrants c, d
            bit_v = ((r >= a) & (r < ab)) | (r >= abc)  # quadrants b, d
            su |= bit_u.astype(np.int64) << lvl
            sv |= bit_v.astype(np.int64) << lvl
        src[s0:s0 + cnt] = su
        dst[s0:s0 + cnt] = sv
    src = src.astype(np.int32)
    dst = dst.astype(np.int32)
    if permute:
        p = permutation(n, seed, stream + 1000)
        src, dst = p[src], p[dst]
    return src, dst


# ---------------------------------------------------------------------------
# features, labels, weights
# ---------------------------------------------------------------------------


def features_normal(n: int, f: int, seed: int = 0, stream: int = 3, row0: int = 0,
                    rows: int | None = None) -> np.ndarray:
    """Rows row0.. of an n x f matrix of N(0,1) values (Box-Muller in fp64, cast to fp32)."""
    rows = n - row0 if rows is None else rows
    out = np.empty((rows, f), np.float32)
    step = max(1, (1 << 22) // max(f, 1))
    for r in range(0, rows, step):
        k = min(step, rows - r)
        e0 = (row0 + r) * f
        h = draws(seed, stream, 2 * e0, 2 * k * f)
        u1 = u01_f64_open0(h[0::2])
        u2 = u01_f64(h[1::2])
        z = np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * np.pi * u2)
        out[r:r + k] = z.reshape(k, f).astype(np.float32)
    return out


def features_bernoulli(n: int, f: int, p: float, seed: int = 0, stream: int = 3, row0: int = 0,
                       rows: int | None = None, binary: bool = True) -> np.ndarray:
    """Rows row0.. of an n x f matrix with each entry nonzero with probability p.

    One 64-bit draw per entry: its top 32 bits decide presence (u32 < p * 2^32);
    a present entry is 1.0 when ``binary``, else (k + 1) * 2^-24 with k the low 24
    bits, a value in (0, 1].
    """
    rows = n - row0 if rows is None else rows
    out = np.zeros((rows, f), np.float32)
    thr = _U64(min(int(round(p * 4294967296.0)), 4294967296))
    step = max(1, (1 << 22) // max(f, 1))
    for r in range(0, rows, step):
        k = min(step, rows - r)
        h = draws(seed, stream, (row0 + r) * f, k * f)
        present = (h >> _U64(32)) < thr
        if binary:
            vals = present.astype(np.float32)
        else:
            mant = (h & _U64(0xFFFFFF)).astype(np.float64) + 1.0
            vals = np.where(present, mant * (1.0 / 16777216.0), 0.0).astype(np.float32)
        out[r:r + k] = vals.reshape(k, f)
    return out


def labels(n: int, classes: int, seed: int = 0, stream: int = 4) -> np.ndarray:
    """Uniform class labels in [0, classes), int32."""
    h = draws(seed, stream, 0, n)
    return (((h >> _U64(32)) * _U64(classes)) >> _U64(32)).astype(np.int32)


def glorot(fan_in: int, fan_out: int, seed: int = 0, stream: int = 10) -> np.ndarray:
    """Glorot/Xavier-uniform fan_in x fan_out fp32 matrix, bound sqrt(6/(fan_in+fan_out))."""
    a = math.sqrt(6.0 / (fan_in + fan_out))
    u = u01_f64(draws(seed, stream, 0, fan_in * fan_out))
    return (a * (2.0 * u - 1.0)).astype(np.float32).reshape(fan_in, fan_out)


# ---------------------------------------------------------------------------
# workloads shaped like the paper's evaluation graphs
# ---------------------------------------------------------------------------


@dataclass(frozen=True)
class Workload:
    name: str
    n: int
    graph: str            # "chung_lu" or "rmat"
    e_und: int            # undirected edges (chung_lu) or raw samples (rmat)
    widths: tuple         # (F, hidden..., classes)
    features: str         # "normal", "binary", "nonneg"
    density: float = 1.0
    rmat_scale: int = 0
    note: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def f(self) -> int:
        return self.widths[0]

    @property
    def classes(self) -> int:
        return self.widths[-1]

    @property
    def n_layers(self) -> int:
        return len(self.widths) - 1


WORKLOADS = {
    # Cora-sized citation graph: 2-layer GCN, binary bag-of-words features at 1.3 %
    "cora_like": Workload("cora_like", 2708, "chung_lu", 5278, (1433, 16, 7), "binary", 0.013,
                          note="2,708 nodes, 5,278 undirected edges, 1433-d binary X"),
    # ogbn-arxiv shape (Table II): 3-layer GCN, dense 128-d features, 40 classes
    "arxiv_like": Workload("arxiv_like", 169343, "chung_lu", 1166243, (128, 256, 256, 40), "normal",
                           note="169,343 nodes, 1,166,243 undirected edges, 128-d N(0,1) X"),
    # Reddit shape (Table II): 2-layer GCN, 602-d dense features, heavy-tailed degree (mean ~490)
    "reddit_like": Workload("reddit_like", 232965, "chung_lu", 57307946, (602, 256, 41), "normal",
                            note="232,965 nodes, 57.3M undirected edges, 602-d N(0,1) X"),
    # ogbn-products shape (Table II): 3-layer GCN, 100-d dense features, 47 classes
    "products_like": Workload("products_like", 2449029, "chung_lu", 61859140, (100, 256, 256, 47),
                              "normal", note="2,449,029 nodes, 61,859,140 undirected edges, 100-d X"),
}
for _p in (0.5, 0.1, 0.01, 0.001):
    _nm = f"rmat21_p{_p:g}"
    WORKLOADS[_nm] = Workload(_nm, 1 << 21, "rmat", 1 << 25, (4096, 128, 32), "nonneg", _p,
                              rmat_scale=21,
                              note=f"RMAT SCALE 21, 2^25 samples, 4096-d nonneg X at {_p:g} density")


def make_graph(wl: Workload, seed: int = 0):
    if wl.graph == "chung_lu":
        return chung_lu(wl.n, wl.e_und, seed=seed, stream=1)
    return rmat(wl.rmat_scale, wl.e_und, seed=seed, stream=1)


def make_features(wl: Workload, seed: int = 0, row0: int = 0, rows: int | None = None):
    if wl.features == "normal":
        return features_normal(wl.n, wl.f, seed=seed, stream=3, row0=row0, rows=rows)
    return features_bernoulli(wl.n, wl.f, wl.density, seed=seed, stream=3, row0=row0, rows=rows,
                              binary=(wl.features == "binary"))


def make_labels(wl: Workload, seed: int = 0):
    return labels(wl.n, wl.classes, seed=seed, stream=4)


def make_weights(wl: Workload, seed: int = 0):
    """Glorot weights and zero biases for every layer (fp32)."""
    ws, bs = [], []
    for l in range(wl.n_layers):
        ws.append(glorot(wl.widths[l], wl.widths[l + 1], seed=seed, stream=10 + l))
        bs.append(np.zeros(wl.widths[l + 1], np.float32))
    return ws, bs


def scaled(wl: Workload, n: int, e_und: int, name: str | None = None) -> Workload:
    """The same layer widths and feature recipe on a smaller graph."""
    return Workload(name or f"{wl.name}_n{n}", n, "chung_lu", e_und, wl.widths, wl.features,
                    wl.density, note=f"{wl.name} widths on {n} nodes")


def digest(*arrays) -> str:
    """sha256 over the raw bytes of the given arrays (golden-hash helper)."""
    hsh = hashlib.sha256()
    for a in arrays:
        a = np.ascontiguousarray(a)
        hsh.update(str(a.dtype).encode())
        hsh.update(str(a.shape).encode())
        hsh.update(a.tobytes())
    return hsh.hexdigest()
