"""Shared test helpers: tolerances and small graph builders (no method arithmetic)."""
import numpy as np

# fp32 results against the fp64 oracle: max relative error 1e-4, measured per element
# against the element's magnitude scale sum |terms| (which is >= |value|).
RTOL = 1e-4


def assert_mag_close(got, want, mag, what="", rtol=RTOL):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    mag = np.asarray(mag, np.float64)
    assert got.shape == want.shape, f"{what}: shape {got.shape} vs {want.shape}"
    err = np.abs(got - want)
    zero = mag == 0
    assert not (zero & (got != 0)).any(), f"{what}: nonzero where every term is zero"
    ratio = np.where(zero, 0.0, err / np.where(zero, 1.0, mag))
    worst = float(ratio.max()) if ratio.size else 0.0
    assert worst <= rtol, f"{what}: max |gpu - oracle| / scale = {worst:.3e} > {rtol}"
    return worst


def assert_norm_close(got, want, what="", rtol=RTOL):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    den = np.abs(want).max() if want.size else 0.0
    err = np.abs(got - want).max() if want.size else 0.0
    rel = err / den if den > 0 else err
    assert rel <= rtol, f"{what}: ||gpu - oracle||_inf / ||oracle||_inf = {rel:.3e} > {rtol}"
    return rel


def ring(n):
    s = np.arange(n, dtype=np.int32)
    return s, ((s + 1) % n).astype(np.int32)


def star(leaves, hub=0):
    others = np.array([i for i in range(leaves + 1) if i != hub], np.int32)
    return np.full(leaves, hub, np.int32), others


def complete(n):
    iu = np.triu_indices(n, 1)
    return iu[0].astype(np.int32), iu[1].astype(np.int32)


def messy(rng, n, m, self_frac=0.1, dup_frac=0.3):
    src = rng.integers(0, n, m)
    dst = rng.integers(0, n, m)
    k = int(m * self_frac)
    dst[:k] = src[:k]
    j = int(m * dup_frac)
    if j and m > k + j:
        src[-j:] = dst[k:k + j]
        dst[-j:] = src[k:k + j]
    return src.astype(np.int32), dst.astype(np.int32)


def adversarial_graphs():
    """(name, n, src, dst) covering every row-length class of the device CSR build."""
    rng = np.random.default_rng(1234)
    out = [("empty", 5, np.zeros(0, np.int32), np.zeros(0, np.int32)),
           ("single", 1, np.zeros(0, np.int32), np.zeros(0, np.int32)),
           ("self_only", 4, np.arange(4, dtype=np.int32), np.arange(4, dtype=np.int32)),
           ("ring", 97, *ring(97)),
           ("star63", 64, *star(63)),
           ("star64", 65, *star(64, hub=17)),
           ("star300", 301, *star(300, hub=300)),
           ("star4095", 4096, *star(4095)),
           ("star9000", 9001, *star(9000, hub=4500)),
           ("k40", 40, *complete(40)),
           ("messy", 500, *messy(rng, 500, 6000)),
           ]
    # disconnected: two rings and isolated nodes
    s1, d1 = ring(10)
    s2, d2 = ring(7)
    out.append(("disconnected", 30, np.concatenate([s1, s2 + 12]), np.concatenate([d1, d2 + 12])))
    # a hub whose raw row has heavy duplication (many repeated pairs in both directions)
    hs = np.concatenate([np.zeros(20000, np.int32), rng.integers(1, 700, 20000).astype(np.int32)])
    hd = np.concatenate([rng.integers(1, 700, 20000).astype(np.int32), np.zeros(20000, np.int32)])
    out.append(("dup_hub", 700, hs, hd))
    return out


def note(msg):
    """A progress line for long GPU tests: to stderr and appended to gpurun_out/test_progress.log
    (a long test then shows activity while it runs)."""
    import os
    import sys
    import time
    line = f"[{time.strftime('%H:%M:%S')}] {msg}"
    print(line, file=sys.stderr, flush=True)
    root = os.environ.get("GRAFT_REPO_ROOT") or os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    try:
        os.makedirs(os.path.join(root, "gpurun_out"), exist_ok=True)
        with open(os.path.join(root, "gpurun_out", "test_progress.log"), "a") as f:
            f.write(line + "\n")
    except OSError:
        pass


def relu_flips(gpu_on, Z, mag, what, band=1e-5):
    """ReLU decisions: the GPU's 1[H > 0] (taken on its fp32 pre-activation) against the
    oracle's 1[Z > 0] (fp64).  Where Z is within rounding of zero both are correct; a
    differing decision is accepted only where |Z| <= band * (the element's magnitude scale
    sum |terms|), and the number of accepted flips must stay small.  Returns the count."""
    gpu_on = np.asarray(gpu_on, bool)
    Z = np.asarray(Z, np.float64)
    mag = np.asarray(mag, np.float64)
    differ = gpu_on != (Z > 0)
    far = differ & (np.abs(Z) > band * mag)
    assert not far.any(), (f"{what}: {int(far.sum())} ReLU decisions differ away from zero "
                           f"(worst |Z|/scale {float((np.abs(Z) / np.maximum(mag, 1e-300))[far].max()):.3e})")
    flips = int(differ.sum())
    limit = 5 + int(1e-5 * Z.size)
    assert flips <= limit, f"{what}: {flips} ReLU flips near zero (limit {limit})"
    note(f"{what}: {flips} ReLU flips within {band:g} x scale of zero, of {Z.size} entries")
    return flips
