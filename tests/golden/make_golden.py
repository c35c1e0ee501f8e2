"""Write the stored oracle values the full-size parity tests compare with.

    python tests/golden/make_golden.py mlp2000_n40 wide_bf16

For each named workload this runs the CPU oracle (and nothing else) over the
workload's rounds on its seeded synthetic data and commit orders, and stores
in tests/golden/<name>.npz, after round 1 and after the last round:
  - the oracle's max-abs value of every parameter tensor of the central
    variable (the denominator of the per-tensor max-norm parity metric),
  - the central variable at the stored positions: every bias element, and
    in every weight tensor SAMPLES_PER_TILE seeded positions inside every
    64 x 64 block of the [d_out][d_in] matrix (the output tile of the
    float32 weight-gradient products; the bf16 products use 128 x 128 tiles,
    each of which holds four such blocks), so a wrong tile, edge or worker
    cannot hide between the samples,
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

BLOCK = 64
SAMPLES_PER_TILE = 8


def tensor_slices(dims):
    """(start, stop, rows, cols) of every tensor in the packed layout."""
    out, o = [], 0
    for l in range(len(dims) - 1):
        w = dims[l] * dims[l + 1]
        out.append((o, o + w, dims[l + 1], dims[l]))
        o += w
        out.append((o, o + dims[l + 1], 1, dims[l + 1]))
        o += dims[l + 1]
    return out


def sample_positions(dims, seed):
    """Every bias element; per weight tensor SAMPLES_PER_TILE distinct
    positions inside every BLOCK x BLOCK block (all of a smaller ragged
    block), plus the last row and column of the matrix at seeded places."""
    rng = np.random.default_rng([seed, 7])
    pos = []
    for a, b, rows, cols in tensor_slices(dims):
        if rows == 1:
            pos.append(np.arange(a, b, dtype=np.int64))
            continue
        sel = []
        for r0 in range(0, rows, BLOCK):
            for c0 in range(0, cols, BLOCK):
                h, w = min(BLOCK, rows - r0), min(BLOCK, cols - c0)
                k = min(h * w, SAMPLES_PER_TILE)
                flat = rng.choice(h * w, size=k, replace=False)
                sel.append((r0 + flat // w) * cols + (c0 + flat % w))
        sel.append((rows - 1) * cols + rng.choice(cols, size=min(cols, 64), replace=False))
        sel.append(rng.choice(rows, size=min(rows, 64), replace=False) * cols + (cols - 1))
        pos.append(a + np.unique(np.concatenate(sel)).astype(np.int64))
    return pos


def snapshot(o, dims, pos, tag, out):
    c = o.central_flat()
    out[f"{tag}_maxabs"] = np.array([np.max(np.abs(c[a:b])) for a, b, _, _ in tensor_slices(dims)], np.float64)
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
           "rounds": np.array(wl.rounds), "block": np.array(BLOCK)}
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
