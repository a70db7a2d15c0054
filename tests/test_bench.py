"""Host-side logic of bench.py: the HBM-traffic lookup and the single-GPU guard (no GPU)."""
import hashlib
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.fixture
def fake_root(tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    src = tmp_path / "k.hip"
    src.write_text("kernel source\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    return tmp_path, hashlib.sha256(src.read_bytes()).hexdigest()


def write_table(root, table):
    (root / "profiles" / "traffic.json").write_text(json.dumps(table) if not isinstance(table, str) else table)


def test_traffic_lookup(fake_root):
    root, sha = fake_root
    assert bench.traffic_for("aggregate_w256", "wl") is None  # no table
    write_table(root, "{not json")
    assert bench.traffic_for("aggregate_w256", "wl") is None
    write_table(root, {"aggregate_w256@wl": {"bytes_per_launch": 7}})  # no source hashes
    assert bench.traffic_for("aggregate_w256", "wl") is None
    write_table(root, {"aggregate_w256@wl": {"bytes_per_launch": 7, "sources": {"k.hip": "0" * 64}}})
    assert bench.traffic_for("aggregate_w256", "wl") is None  # kernel changed since the counters
    write_table(root, {"aggregate_w256@wl": {"bytes_per_launch": 7, "sources": {"k.hip": sha}}})
    assert bench.traffic_for("aggregate_w256", "wl") == 7
    assert bench.traffic_for("aggregate_w128", "wl") is None
    write_table(root, {"aggregate_w256@wl": {"bytes_per_launch": 7, "sources": {"gone.hip": sha}}})
    assert bench.traffic_for("aggregate_w256", "wl") is None


def test_committed_traffic_record_is_well_formed():
    table = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    for key, rec in table.items():
        kernel, workload = key.split("@")
        assert rec["bytes_per_launch"] > 0 and rec["sources"]
        for rel in rec["sources"]:
            assert os.path.exists(os.path.join(ROOT, rel)), rel
        assert os.path.exists(os.path.join(ROOT, rec["summary"]))


def test_algorithmic_bytes():
    # gathers 4 nnz w + indices and values 8 nnz + offsets 8 (N + 1) + output 4 N w
    assert bench.alg_bytes_aggregate(10, 3, 2) == 4 * 10 * 2 + 8 * 10 + 8 * 4 + 4 * 3 * 2


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, env={**os.environ, "HIP_VISIBLE_DEVICES": ""})
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_calibration_crossover_interpolation():
    import calibrate
    # ratio t_sparse / t_dense crosses 1 between densities 0.01 and 0.1, at the geometric mean
    # when the two ratios are symmetric about 1
    c = calibrate.crossover([(0.1, 1.5), (0.01, 0.5), (0.5, 4.0)])
    assert c == pytest.approx((0.01 * 0.1) ** 0.5, rel=1e-12)
    assert calibrate.crossover([(0.1, 0.5), (0.5, 0.9)]) is None  # sparse faster everywhere


def test_compulsory_bytes_are_below_algorithmic():
    # indices 4 nnz, offsets and dinv 12 N, each input row once and the output 8 N w
    assert bench.compulsory_bytes_aggregate(10, 3, 2) == 4 * 10 + 12 * 3 + 8 * 3 * 2
    for nnz, n, w in [(2_501_829, 169_343, 256), (126_167_309, 2_449_029, 47), (5, 5, 1)]:
        assert bench.compulsory_bytes_aggregate(nnz, n, w) <= bench.alg_bytes_aggregate(nnz, n, w)


def test_default_workload_is_the_largest_single_gpu_config():
    import gcn_synth as gs
    args = sys.argv
    try:
        sys.argv = ["bench.py"]
        wl = gs.WORKLOADS[bench.parse().workload]
    finally:
        sys.argv = args
    assert wl.n == max(w.n for w in gs.WORKLOADS.values())
    assert wl.name == "products_like"
