"""Benchmark: full-batch GCN training epochs per second on one MI355X.

One step = one training epoch of the whole hot path (forward through every
layer with the fused aggregation, softmax cross-entropy, backward, Adam) on a
seeded synthetic graph resident in HBM.  Graph generation, upload, the CSR
build and the density probe run once before timing (the paper also excludes
one-time setup from its per-epoch times).

Prints ONE JSON line.  Extra objects:
  roofline      the dominant kernel family's algorithmic bytes (or flops) per
                launch over its average launch time, from HIP events recorded
                around that family's launches inside the timed region (an
                untimed pass before it brackets every launch for the
                per-kernel table and picks the family);
  cpu_baseline  the fp64 oracle's epoch time on this host's cores (bounded sample).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GCN train epochs/sec (fwd+bwd) on 1 MI355X; SpMM achieved HBM GB/s"
HBM_PEAK_GBS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="products_like",
                    help="products_like (the default: the largest single-GPU workload, 2,449,029 nodes), "
                         "arxiv_like, reddit_like, cora_like, rmat21_p{0.5,0.1,0.01,0.001}")
    ap.add_argument("--tau", default="15/16",
                    help="sparse-path threshold tau as num/den (15/16: measured on MI355X; the paper's is 4/5)")
    ap.add_argument("--force-mode", default="auto", choices=["auto", "dense", "sparse"])
    ap.add_argument("--row-order", default="auto", choices=["auto", "on", "off"],
                    help="aggregations take the graph rows longest first (on) or in row order (off); "
                         "auto: whichever times faster for the widest hidden layer (untimed setup)")
    ap.add_argument("--csc", default="on", choices=["on", "off"],
                    help="off: no X_csc view; the sparse backward X^T Q uses atomic adds from X_csr")
    ap.add_argument("--agg", default="gcn", choices=["gcn", "sum", "mean", "max"],
                    help="aggregator of every layer (Section III-A); gcn is the normalised A_hat")
    ap.add_argument("--cpu-baseline", default="auto", choices=["auto", "off"])
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="CPU work budget for the oracle leg")
    ap.add_argument("--no-profile", action="store_true", help="no launch events at all (pure epoch timing)")
    ap.add_argument("--graph", action="store_true",
                    help="capture one epoch in a HIP graph and time K replays (per-launch events off)")
    ap.add_argument("--copy-gib", type=float, default=0.0,
                    help="instead of training, time a plain device copy of this many GiB "
                         "(calibrates HBM counters against a kernel of known traffic)")
    return ap.parse_args()


def alg_bytes_aggregate(nnz: int, rows: int, w: int) -> int:
    """Algorithmic bytes of one normalised aggregation at width w: neighbour-row gathers
    4 nnz w, column indices and entry values 8 nnz, row offsets 8 (rows + 1), output 4 rows w."""
    return 4 * nnz * w + 8 * nnz + 8 * (rows + 1) + 4 * rows * w


def compulsory_bytes_aggregate(nnz: int, rows: int, w: int) -> int:
    """Bytes any aggregation at width w must move at least once: the column indices 4 nnz,
    row offsets and dinv 12 N, every input row once and the output, 8 N w."""
    return 4 * nnz + 12 * rows + 8 * rows * w


def sha_of(path):
    return hashlib.sha256(open(path, "rb").read()).hexdigest()


def traffic_for(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if the kernel's
    source files are unchanged since the counters were taken; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        table = json.load(open(path))
    except (OSError, ValueError):
        return None
    rec = table.get(f"{kernel}@{workload}")
    if not isinstance(rec, dict) or not isinstance(rec.get("sources"), dict) or not rec["sources"]:
        return None
    for rel, sha in rec["sources"].items():
        src = os.path.join(ROOT, rel)
        if not os.path.exists(src) or sha_of(src) != sha:
            return None
    return rec.get("bytes_per_launch")


def copy_calibration(gib: float):
    import torch
    n = int(gib * (1 << 30)) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    reps = 10
    for _ in range(reps):
        b.copy_(a)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / reps
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "ms": ms,
                      "GBps": 2 * n * 4 / ms / 1e6}))


def cpu_baseline(wl, s, d, X, y, Ws, bs, sparse: bool, budget_s: float):
    """The oracle as it stands, timed on this host: full epochs of the same workload,
    repeated until about budget_s seconds of work (at least one)."""
    from oracle import oracle as orc
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    og = orc.build_csr(wl.n, s, d)
    osx = orc.SparseX(X) if sparse else None
    Wd = [w.astype(np.float64) for w in Ws]
    bd = [b.astype(np.float64) for b in bs]
    z = [np.zeros(w.shape) for w in Ws]
    zb = [np.zeros(b.shape) for b in bs]
    times = []
    t_all = time.perf_counter()
    while True:
        t0 = time.perf_counter()
        orc.epoch(og, X, y, Wd, bd, z, z, zb, zb, 1, sparse=osx)
        times.append(time.perf_counter() - t0)
        if time.perf_counter() - t_all >= budget_s or len(times) >= 50:
            break
    sec = float(np.median(times))
    return {"value": 1.0 / sec, "unit": "epochs/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(times)} full fp64 oracle epoch(s) of {wl.name} (forward, loss, backward, "
                      f"Adam), median {sec:.3f} s/epoch; graph loops in plain C with OpenMP over rows, "
                      f"dense products through numpy's fp64 matmul (multi-threaded BLAS)"}


def cpu_baseline_device_x(wl, s, d, y, Ws, bs, sparse: bool, budget_s: float):
    """The oracle's epoch for features drawn on the device (too large to draw on the host in
    reasonable time): X is drawn again block by block from the same counter stream into host
    memory before timing, and the oracle's row-block epoch (the products that read X taken
    over row blocks, every other step as in its plain epoch) is timed."""
    import torch
    from gcn_synth import device as gdev
    from oracle import oracle as orc
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    og = orc.build_csr(wl.n, s, d)
    X = np.empty((wl.n, wl.f), np.float32)
    rows = 65536
    buf = torch.empty((rows, wl.f), dtype=torch.float32, device="cuda")
    for r0 in range(0, wl.n, rows):
        r1 = min(wl.n, r0 + rows)
        gdev.bernoulli_into(buf[:r1 - r0], wl.density, seed=0, stream=3, row0=r0, binary=(wl.features == "binary"))
        X[r0:r1] = buf[:r1 - r0].cpu().numpy()
    del buf
    z = [np.zeros(w.shape) for w in Ws]
    zb = [np.zeros(b.shape) for b in bs]
    times = []
    t_all = time.perf_counter()
    while True:
        t0 = time.perf_counter()
        orc.epoch_row_blocks(og, lambda r0, r1: X[r0:r1], wl.f, y, Ws, bs, z, z, zb, zb, 1, sparse=sparse,
                             block_rows=rows)
        times.append(time.perf_counter() - t0)
        if time.perf_counter() - t_all >= budget_s or len(times) >= 50:
            break
    sec = float(np.median(times))
    return {"value": 1.0 / sec, "unit": "epochs/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(times)} full fp64 oracle epoch(s) of {wl.name} (forward, loss, backward, Adam), "
                      f"median {sec:.3f} s/epoch; the {wl.n:,} x {wl.f} features redrawn in {rows}-row blocks "
                      f"from the counter stream before timing, the two products that read them taken over those "
                      f"blocks ({'DenseToCSR / DenseToCSC and sparse products per block' if sparse else 'dense'}); "
                      f"graph loops in plain C with OpenMP over rows, dense products through numpy's fp64 "
                      f"matmul (multi-threaded BLAS)"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the multi-GPU form "
              "(one process per GPU over a row partition of A_hat, halo rows exchanged over RCCL) "
              "is not built", file=sys.stderr)
        sys.exit(2)
    import torch
    if args.copy_gib > 0:
        copy_calibration(args.copy_gib)
        return

    import gcn_synth as gs
    import paper_2512_01678_amd.gcn as G

    wl = gs.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    # matrices too large to draw on the host (the RMAT workloads' 2^21 x 4096 X) are
    # drawn on the device from the same counter stream
    on_device = wl.n * wl.f > (1 << 28)
    t0 = time.perf_counter()
    s, d = gs.make_graph(wl)
    X = None if on_device else gs.make_features(wl)
    y = gs.make_labels(wl)
    Ws, bs = gs.make_weights(wl)
    ld_x = G.pitch(wl.f)
    Xd = torch.zeros((wl.n, ld_x), dtype=torch.float32, device=dev)
    Xv = Xd[:, :wl.f]
    if on_device:
        from gcn_synth import device as gdev
        gdev.bernoulli_into(Xv, wl.density, seed=0, stream=3, binary=(wl.features == "binary"))
    else:
        Xv.copy_(torch.from_numpy(X).to(dev))
    torch.cuda.synchronize()
    t_gen = time.perf_counter() - t0
    print(f"[bench] {wl.name}: inputs generated in {t_gen:.1f} s", file=sys.stderr, flush=True)
    sd, dd = torch.from_numpy(s).to(dev), torch.from_numpy(d).to(dev)
    yd = torch.from_numpy(y).to(dev)
    torch.cuda.synchronize()

    t0 = time.perf_counter()
    g = G.build_csr(wl.n, sd, dd, order=args.row_order != "off")
    if args.row_order == "auto":
        G.tune_row_order(g, max(wl.widths[1:-1]) if len(wl.widths) > 2 else wl.widths[-1])
    t_csr = time.perf_counter() - t0
    tau = tuple(int(v) for v in args.tau.split("/"))
    force = {"auto": -1, "dense": G.DENSE, "sparse": G.SPARSE}[args.force_mode]
    t0 = time.perf_counter()
    info, sx = G.feature_stats(Xv, tau=tau, force_mode=force, csc=args.csc == "on")
    t_probe = time.perf_counter() - t0
    sparse = info["mode"] == G.SPARSE
    print(f"[bench] nnz(A+I)={g.nnz} csr {t_csr * 1e3:.1f} ms; probe s={info['sparsity']:.4f} -> "
          f"{'sparse' if sparse else 'dense'} ({t_probe * 1e3:.1f} ms)", file=sys.stderr, flush=True)
    del sd, dd

    if sparse:
        del Xv, Xd  # the sparse path reads only X_csr / X_csc
        torch.cuda.empty_cache()
    setup_peak = torch.cuda.max_memory_allocated(dev)
    torch.cuda.reset_peak_memory_stats(dev)
    agg = {"gcn": G.AGG_NORM, "sum": G.AGG_SUM, "mean": G.AGG_MEAN, "max": G.AGG_MAX}[args.agg]
    if agg == G.AGG_MAX and sparse:
        sys.exit("bench.py: the max aggregator needs dense input features (use --force-mode dense)")
    m = G.Model(wl.n, wl.widths, Ws, bs, device=dev, x_sparse=sparse, ld_x=ld_x, device_step=args.graph,
                aggs=[agg] * (len(wl.widths) - 1))
    Xin = None if sparse else Xv
    for _ in range(args.warmup):
        m.epoch(g, X=Xin, x=sx, labels=yd)
    torch.cuda.synchronize()
    print(f"[bench] {args.warmup} warm-up epochs done", file=sys.stderr, flush=True)

    profile = not (args.no_profile or args.graph)
    cg = None
    if args.graph:
        m.prepare(g, X=Xin, x=sx, labels=yd)
        torch.cuda.synchronize()
        cg = torch.cuda.CUDAGraph()
        with torch.cuda.graph(cg):
            m.epoch_captured(g, X=Xin, x=sx, labels=yd)
        torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    launches_per_epoch = 64

    def run(steps):
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        t = time.perf_counter()
        for _ in range(steps):
            if cg is not None:
                cg.replay()
            else:
                m.epoch(g, X=Xin, x=sx, labels=yd)
        ev1.record(stream)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1), time.perf_counter() - t

    def families(records):
        fam = {}
        for r in records:
            f = fam.setdefault(r["name"], dict(ms=0.0, count=0, width=r["width"], rows=r["rows"], nnz=r["nnz"]))
            f["ms"] += r["ms"]
            f["count"] += 1
        return fam

    # Untimed pass with an event pair around every launch: the per-kernel table and the
    # dominant aggregation family.  Each pair adds a few microseconds of queue time, so the
    # timed pass below brackets only that family's launches.
    fam, dominant, prof_steps, ms_prof = {}, None, 0, 0.0
    if profile:
        prof_steps = max(2, min(args.steps, 10))
        G.profile_only(None)
        G.profile_enable(launches_per_epoch * prof_steps)
        ms_prof, _ = run(prof_steps)
        fam = families(G.profile_records())
        G.profile_enable(0)
        aggs = {k: v for k, v in fam.items() if k.startswith("aggregate_w")}
        if aggs:
            dominant = max(aggs.items(), key=lambda kv: kv[1]["ms"])[0]
            G.profile_only(dominant)
            G.profile_enable(launches_per_epoch * args.steps)

    ms_total, t_wall = run(args.steps)
    ms_per_step = ms_total / args.steps
    timed_dom = None
    if dominant is not None:
        timed_dom = families(G.profile_records()).get(dominant)
        G.profile_enable(0)
        G.profile_only(None)
    loss = float(m.loss.cpu()[0])
    print(f"[bench] {args.steps} epochs: {ms_per_step:.3f} ms/epoch (wall {t_wall * 1e3 / args.steps:.3f}), "
          f"loss {loss:.5f}, Adam steps {m.step}", file=sys.stderr, flush=True)

    kernels = {}
    for name, f in sorted(fam.items(), key=lambda kv: -kv[1]["ms"]):
        avg = f["ms"] / f["count"]
        k = {"avg_ms": round(avg, 5), "launches_per_epoch": f["count"] // prof_steps,
             "share": round(f["ms"] / ms_prof, 4)}
        if name.startswith("aggregate_w"):
            by = alg_bytes_aggregate(g.nnz, f["rows"], f["width"])
            k["alg_GBps"] = round(by / (avg * 1e-3) / 1e9, 1)
            k["compulsory_frac"] = round(compulsory_bytes_aggregate(g.nnz, f["rows"], f["width"]) /
                                         (avg * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
        elif name.startswith("aggmax_bwd_w"):  # gathers dP and maximisers, mask and output rows
            w = f["width"]
            by = 8 * g.nnz * w + 4 * g.nnz + 8 * (f["rows"] + 1) + 8 * f["rows"] * w
            k["alg_GBps"] = round(by / (avg * 1e-3) / 1e9, 1)
        elif name.startswith("aggmax_w"):  # gathers, indices, offsets, maxima and maximisers out
            w = f["width"]
            by = 4 * g.nnz * w + 4 * g.nnz + 8 * (f["rows"] + 1) + 8 * f["rows"] * w
            k["alg_GBps"] = round(by / (avg * 1e-3) / 1e9, 1)
        elif name.startswith("agg_gemm_"):
            fi, fo = (int(v) for v in name.split("_")[2].split("x"))
            by = alg_bytes_aggregate(g.nnz, f["rows"], fi) + 4 * f["rows"] * fo
            k["alg_GBps"] = round(by / (avg * 1e-3) / 1e9, 1)
            k["TFLOPs"] = round(2 * f["rows"] * fi * fo / (avg * 1e-3) / 1e12, 2)
        elif name.startswith("gemm_"):
            mm, nn, kk = (int(v) for v in name.split("_")[2].split("x"))
            k["TFLOPs"] = round(2 * mm * nn * kk / (avg * 1e-3) / 1e12, 2)
        kernels[name] = k

    roofline = None
    if timed_dom is not None and timed_dom["count"]:
        # dominant kernel family (largest total time in the profiled pass), its launches
        # timed inside the timed region
        f = timed_dom
        avg_s = f["ms"] / f["count"] * 1e-3
        by = alg_bytes_aggregate(g.nnz, f["rows"], f["width"])
        bmin = compulsory_bytes_aggregate(g.nnz, f["rows"], f["width"])
        traffic = traffic_for(dominant, wl.name)
        # The algorithmic bytes count every neighbour-row gather as an HBM read.  Where the
        # gathered rows are so concentrated on hub nodes that caches serve them (the RMAT
        # graph), that rate exceeds the HBM peak and is no bound; the roofline is then taken
        # on the bytes the HBM counters saw, or, without counters, on the compulsory bytes.
        basis, used = "algorithmic", by
        if by / avg_s / 1e9 > HBM_PEAK_GBS:
            basis, used = ("hbm_counters", traffic) if traffic else ("compulsory", bmin)
        achieved = used / avg_s / 1e9
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                    "kernel": dominant, "basis": basis, "alg_bytes_per_launch": by,
                    "alg_GBps": round(by / avg_s / 1e9, 1),
                    "compulsory_bytes_per_launch": bmin,
                    "compulsory_frac": round(bmin / avg_s / 1e9 / HBM_PEAK_GBS, 4),
                    "traffic_frac": None if not traffic else round(traffic / avg_s / 1e9 / HBM_PEAK_GBS, 4),
                    "avg_launch_ms": round(avg_s * 1e3, 5), "launches_timed": f["count"]}

    # every aggregation launch of the profiled pass: bytes-weighted achieved rate of the graph SpMM
    spmm = None
    agg_fams = [(f, alg_bytes_aggregate(g.nnz, f["rows"], f["width"])) for k, f in fam.items()
                if k.startswith("aggregate_w")]
    if agg_fams:
        tot_b = sum(by * f["count"] for f, by in agg_fams)
        tot_min = sum(compulsory_bytes_aggregate(g.nnz, f["rows"], f["width"]) * f["count"] for f, _ in agg_fams)
        tot_s = sum(f["ms"] for f, _ in agg_fams) * 1e-3
        spmm = {"weighted_GBps": round(tot_b / tot_s / 1e9, 1),
                "frac": round(tot_b / tot_s / 1e9 / HBM_PEAK_GBS, 4),
                "compulsory_frac": round(tot_min / tot_s / 1e9 / HBM_PEAK_GBS, 4),
                "launches_per_epoch": sum(f["count"] for f, _ in agg_fams) // prof_steps}

    # device memory during training (allocator high-water mark from the model's creation
    # on) against the O(N F) model: nothing may scale with nnz times a feature width
    # offsets, indices + values, deg + dinv, and the row order when kept
    graph_bytes = 8 * (wl.n + 1) + 8 * g.col_idx.numel() + 8 * wl.n + (4 * wl.n if g.order is not None else 0)
    x_bytes = 0 if sparse else 4 * wl.n * ld_x
    if sparse:  # X_csr (and X_csc): offsets, indices, values
        x_bytes = 8 * (wl.n + 1) + 8 * sx.col.numel()
        if sx.col_ptr is not None:
            x_bytes += 8 * (wl.f + 1) + 8 * sx.col.numel()
    train_peak = torch.cuda.max_memory_allocated(dev)
    memory = {"train_peak_bytes": train_peak, "setup_peak_bytes": setup_peak, "graph_bytes": graph_bytes,
              "x_bytes": x_bytes,
              "other_floats_per_node": round((train_peak - graph_bytes - x_bytes) / (4 * wl.n), 1),
              "layer_output_floats_per_node": sum(G.pitch(w) for w in wl.widths[1:])}

    cpu = None
    if args.cpu_baseline == "auto" and X is None and args.agg == "gcn":
        print("[bench] timing the fp64 oracle on the host (features redrawn in row blocks)", file=sys.stderr,
              flush=True)
        cpu = cpu_baseline_device_x(wl, s, d, y, Ws, bs, sparse, args.cpu_seconds)
    elif args.cpu_baseline == "auto" and args.agg != "gcn":
        print("[bench] cpu_baseline is timed for the gcn aggregator only", file=sys.stderr, flush=True)
    elif args.cpu_baseline == "auto":
        print("[bench] timing the fp64 oracle on the host", file=sys.stderr, flush=True)
        cpu = cpu_baseline(wl, s, d, X, y, Ws, bs, sparse, args.cpu_seconds)

    out = {
        "metric": METRIC, "value": round(1000.0 / ms_per_step, 3), "unit": "epochs/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "nodes": wl.n, "nnz_A_plus_I": g.nnz, "widths": list(wl.widths),
                   "feature_path": "sparse" if sparse else "dense", "sparsity": round(info["sparsity"], 6),
                   "orders": ["AF" if o == G.AGGREGATE_FIRST else "TF" for o in m.orders()],
                   "aggregator": args.agg, "row_order": g.order is not None, "x_csc": sparse and args.csc == "on",
                   "timed_events": dominant, "hip_graph": bool(args.graph),
                   "af_layer": None if G.AGGREGATE_FIRST not in m.orders() else
                   "fused kernel" if os.environ.get("GCN_AF_FUSED") == "1" else "aggregation + GEMM",
                   "gemm_mode": "fp32 MFMA" if os.environ.get("GCN_GEMM_MODE") == "fp32"
                   else "fp32 via exact 3-way bf16 split, 6 bf16 MFMA products"},
        "roofline": roofline, "cpu_baseline": cpu, "spmm": spmm, "memory": memory, "kernels": kernels,
        "setup_ms": {"csr_build": round(t_csr * 1e3, 2), "density_probe": round(t_probe * 1e3, 2)},
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
