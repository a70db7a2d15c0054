"""Dense/sparse crossover of the input-feature products on this GPU (the paper's
calibration of gamma and tau, Section IV-B "Sparsity Decision Model").

For each feature width F and density p, X (N x F, nonnegative values on a random
support of density p, as in the RMAT workload) is drawn on the device and both
products of layer 0 are timed both ways:

  forward   X W    (F x F1):  dense MFMA GEMM      vs  X_csr SpMM
  backward  X^T Q  (N x F1):  dense MFMA GEMM (TN) vs  X_csc SpMM (gcn_spmm_xt)

Efficiencies count useful work only: eta_dense = 2 N F F1 / t_dense and
eta_sparse = 2 nnz F1 / t_sparse, so gamma = eta_sparse / eta_dense and the sparse
product is the faster one iff density < gamma, i.e. iff s = 1 - density > 1 - gamma.
The crossover density is interpolated linearly in log(density) between the measured
points; tau = 1 - crossover.

    python calibrate.py [--rows N] [--features 1024,4096] [--densities ...] [--out f.json]
"""
import argparse
import json
import math
import sys
import time


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--rows", type=int, default=1 << 21)
    ap.add_argument("--features", default="1024,4096")
    ap.add_argument("--hidden", type=int, default=128)
    ap.add_argument("--densities", default="0.5,0.3,0.2,0.1,0.05,0.01,0.001")
    ap.add_argument("--reps", type=int, default=5)
    ap.add_argument("--out", default=None)
    return ap.parse_args()


def timed(fn, reps):
    import torch
    fn()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    for _ in range(reps):
        fn()
    ev[1].record()
    torch.cuda.synchronize()
    return ev[0].elapsed_time(ev[1]) / reps


def crossover(points):
    """Density where t_sparse = t_dense, interpolated in log(density); None if no sign change."""
    pts = sorted(points)
    for (p0, r0), (p1, r1) in zip(pts, pts[1:]):  # r = t_sparse / t_dense
        if (r0 - 1) * (r1 - 1) <= 0 and r0 != r1:
            a = (1 - r0) / (r1 - r0)
            return math.exp(math.log(p0) + a * (math.log(p1) - math.log(p0)))
    return None


def main():
    args = parse()
    import torch
    import paper_2512_01678_amd.gcn as G
    from gcn_synth import device as gdev

    n, f1 = args.rows, args.hidden
    rows = []
    for F in (int(v) for v in args.features.split(",")):
        X = torch.zeros((n, G.pitch(F)), dtype=torch.float32, device="cuda")[:, :F]
        W = torch.randn(F, f1, device="cuda") / math.sqrt(F)
        Q = torch.randn(n, f1, device="cuda")
        out = torch.empty(n, f1, device="cuda")
        dW = torch.empty(F, f1, device="cuda")
        ws = G._Workspace()
        for p in (float(v) for v in args.densities.split(",")):
            t0 = time.perf_counter()
            gdev.bernoulli_into(X, p, seed=0, stream=3, binary=False)
            info, sx = G.feature_stats(X, force_mode=G.SPARSE)
            nnz = sx.nnz
            dense_f = timed(lambda: G.gemm(G.OP_NN, X, W, out, ws=ws), args.reps)
            dense_b = timed(lambda: G.gemm(G.OP_TN, X, Q, dW, ws=ws), args.reps)
            # both sparse products in the form layer 0 takes them
            sparse_f = timed(lambda: G.spmm_xw(sx, W, out), args.reps)
            sparse_b = timed(lambda: G.spmm_xt(sx, Q, dW), args.reps)
            dflop, sflop = 2.0 * n * F * f1, 2.0 * nnz * f1
            r = {"F": F, "density": nnz / (n * F), "nnz": nnz,
                 "dense_fwd_ms": round(dense_f, 3), "sparse_fwd_ms": round(sparse_f, 3),
                 "dense_bwd_ms": round(dense_b, 3), "sparse_bwd_ms": round(sparse_b, 3),
                 "gamma_fwd": round((sflop / sparse_f) / (dflop / dense_f), 4),
                 "gamma_bwd": round((sflop / sparse_b) / (dflop / dense_b), 4)}
            rows.append(r)
            print(f"[calibrate] F={F} p={p}: dense {dense_f:.2f}/{dense_b:.2f} ms, sparse {sparse_f:.2f}/"
                  f"{sparse_b:.2f} ms (fwd/bwd), gamma {r['gamma_fwd']}/{r['gamma_bwd']} "
                  f"({time.perf_counter() - t0:.1f} s)", file=sys.stderr, flush=True)
            del sx
            torch.cuda.empty_cache()
        del X, Q, out
        torch.cuda.empty_cache()

    summary = {}
    for F in sorted({r["F"] for r in rows}):
        sel = [r for r in rows if r["F"] == F]
        cf = crossover([(r["density"], r["sparse_fwd_ms"] / r["dense_fwd_ms"]) for r in sel])
        cb = crossover([(r["density"], r["sparse_bwd_ms"] / r["dense_bwd_ms"]) for r in sel])
        cp = crossover([(r["density"], (r["sparse_fwd_ms"] + r["sparse_bwd_ms"]) /
                         (r["dense_fwd_ms"] + r["dense_bwd_ms"])) for r in sel])
        summary[str(F)] = {"crossover_fwd": cf, "crossover_bwd": cb, "crossover_pair": cp,
                           "tau_pair": None if cp is None else round(1 - cp, 4)}
    result = {"rows": n, "hidden": f1, "points": rows, "summary": summary}
    text = json.dumps(result, indent=1)
    if args.out:
        open(args.out, "w").write(text + "\n")
    print(text)


if __name__ == "__main__":
    main()
