"""Write the stored oracle values the full-size parity tests compare with.

    python tests/golden/make_golden.py mlp1000_n20 mlp2000_n40 wide_bf16

For each named workload this runs the CPU oracle (and nothing else) over the
workload's rounds on its seeded synthetic data and commit orders, and stores
in tests/golden/<name>.npz, after round 1 and after the last round:
  - the oracle's max-abs value of every parameter tensor of the central
    variable (the denominator of the normwise parity metric),
  - the central variable at seeded sample positions of every tensor,
  - the per-worker loss of that round;
and the SHA-256 digest of the data, so a test can tell when its regenerated
inputs differ from the ones the values were computed on.
"""
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402
from oracle import AGNOracle  # noqa: E402

SAMPLES_PER_TENSOR = 1024


def tensor_slices(dims):
    out, o = [], 0
    for l in range(len(dims) - 1):
        w = dims[l] * dims[l + 1]
        out.append((o, o + w))
        o += w
        out.append((o, o + dims[l + 1]))
        o += dims[l + 1]
    return out


def sample_positions(dims, seed):
    rng = np.random.default_rng([seed, 7])
    pos = []
    for a, b in tensor_slices(dims):
        n = b - a
        k = min(n, SAMPLES_PER_TENSOR)
        pos.append(a + np.sort(rng.choice(n, size=k, replace=False)))
    return pos


def snapshot(o, dims, pos, tag, out):
    c = o.central_flat()
    out[f"{tag}_maxabs"] = np.array([np.max(np.abs(c[a:b])) for a, b in tensor_slices(dims)], np.float64)
    out[f"{tag}_values"] = np.concatenate([c[p] for p in pos]).astype(np.float32)
    out[f"{tag}_loss"] = o.last_loss.astype(np.float32)


def make(name):
    wl = W.workload(name)
    t0 = time.time()
    X, y = W.make_data(wl)
    orders = W.commit_orders(wl)
    pos = sample_positions(wl.dims, wl.seed)
    o = AGNOracle(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, bf16=wl.dtype == "bf16")
    out = {"digest": np.array(W.data_digest(X, y)), "positions": np.concatenate(pos).astype(np.int64),
           "rounds": np.array(wl.rounds)}
    for r, order in enumerate(orders, start=1):
        o.round(X, y, order)
        print(f"{name}: round {r}/{wl.rounds} done at {time.time() - t0:.0f} s", flush=True)
        if r == 1:
            snapshot(o, wl.dims, pos, "r1", out)
    snapshot(o, wl.dims, pos, "last", out)
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), f"{name}.npz")
    np.savez_compressed(path, **out)
    print(f"wrote {path} ({os.path.getsize(path)} bytes) in {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    for n in sys.argv[1:]:
        make(n)
