"""Writes synth_hashes.json: sha256 digests of small seeded inputs.

Calls only the input generators (gcn_synth); the digests pin the generators'
determinism, so the oracle and the HIP path are always fed the same arrays.
Run from the repository root: python tests/golden/make_synth_hashes.py
"""
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
import gcn_synth as gs  # noqa: E402


def cases():
    wl = gs.WORKLOADS["cora_like"]
    s, d = gs.make_graph(wl)
    ws, bs = gs.make_weights(wl)
    yield "cora_like_graph", gs.digest(s, d)
    yield "cora_like_features", gs.digest(gs.make_features(wl))
    yield "cora_like_labels", gs.digest(gs.make_labels(wl))
    yield "cora_like_weights", gs.digest(*ws, *bs)
    small = gs.scaled(gs.WORKLOADS["arxiv_like"], 5000, 34000)
    yield "arxiv_like_n5000_graph", gs.digest(*gs.make_graph(small))
    yield "arxiv_like_n5000_features", gs.digest(gs.make_features(small))
    yield "rmat10_graph", gs.digest(*gs.rmat(10, 1 << 14))
    yield "nonneg_p0.1_rows", gs.digest(gs.features_bernoulli(300, 4096, 0.1, binary=False))


if __name__ == "__main__":
    out = dict(cases())
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "synth_hashes.json")
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1, sort_keys=True)
    print(f"wrote {len(out)} digests to {path}")
