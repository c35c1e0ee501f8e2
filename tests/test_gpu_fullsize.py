"""GPU path against the oracle at the five workloads' full sizes, through the
same library calls and launch configuration bench.py times (captured round
graph replays).

Metrics (see helpers.parity_report).  The gate is the whole central
variable's normwise relative error: <= 1e-4 after round 1 and <= 1e-3 after
the last round for float32, <= 2e-2 for bf16.  Every weight tensor must meet
the same bound by itself (max-norm).  Bias tensors start at zero, so after
a round they hold only the sum of the workers' deltas; a ReLU derivative
flipped by a rounding-level difference (the derivative is a step at zero)
changes one worker's delta locally, and the oracle run against itself with
a 1e-7 relative perturbation of its start already differs by 6.4e-4 in a
bias tensor after one round of the n=8 workload.  Biases are therefore held
to 10x the bound in the Frobenius norm.

* 784-1000-1000-10, n=8, lambda=15, 10 rounds: the live oracle runs all ten
  rounds; also the losses and every worker's pulled copy.
* The three larger workloads: stored oracle values (tests/golden/*.npz,
  written by tests/golden/make_golden.py, which calls only the oracle) at
  seeded sample positions of every parameter tensor after round 1 and after
  the last round, with the oracle's per-tensor max-abs as the max-norm
  denominators.
* Round 1 for sampled workers of the two largest workloads, live: every
  worker starts round 1 from the initial central variable, so the oracle
  computes one worker with 1/n of a round's work.  The committed delta is
  compared with the oracle's displacement (theta_lambda - theta_0) / lambda.
"""
import os

import numpy as np
import pytest

import workloads as W
from oracle import AGNOracle, flat_params
from tests.helpers import parity_report, rel_err, rel_fro, tensor_slices, to_device, require_gpu

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TOL = {"fp32": (1e-4, 1e-3), "bf16": (2e-2, 2e-2)}
BIAS_FACTOR = 10.0
# One worker's delta, Frobenius norm.  Nothing dilutes a flipped ReLU
# derivative here (fp32), and in bf16 mode every product operand is rounded
# to 8 bits, so a rounding-level difference in a float32 sum moves some
# operands by one bf16 step and the change cascades through the layers: the
# oracle run against itself with its start perturbed by 1e-7 already
# differs by 1.6e-2 (one step) and 3.3e-2 (three steps) at the 3072-2048x3-100
# shape (pinned on the CPU in test_oracle_sensitivity.py).
DELTA_FRO = {"fp32": 1e-2, "bf16": 1e-1}

_DATA = {}


def data_for(wl):
    key = (wl.data_seed or wl.seed, wl.N, wl.dims[0], wl.data, wl.dtype, wl.dims[-1])
    if key not in _DATA:
        _DATA.clear()
        X, y = W.make_data(wl)
        _DATA[key] = (X, y, to_device(X, y))
    return _DATA[key]


def _agn():
    require_gpu()
    import paper_1710_02368_amd as agn
    return agn


def check(rep, tol, label):
    print(f"{label}: vec {rep['vec']:.2e}  W(max) {rep['W']:.2e}  b(fro) {rep['b']:.2e}", flush=True)
    assert rep["vec"] <= tol, (label, rep)
    assert rep["W"] <= tol, (label, rep)
    assert rep["b"] <= BIAS_FACTOR * tol, (label, rep)


def sampled_report(got_flat, positions, ref_values, ref_maxabs, dims):
    got = got_flat[positions].astype(np.float64)
    ref = ref_values.astype(np.float64)
    vec = np.max(np.abs(got - ref)) / np.max(ref_maxabs)
    w = b = 0.0
    for t, (name, a, c) in enumerate(tensor_slices(dims)):
        sel = (positions >= a) & (positions < c)
        d = got[sel] - ref[sel]
        if name[0] == "W":
            w = max(w, np.max(np.abs(d)) / ref_maxabs[t])
        else:
            b = max(b, np.linalg.norm(d) / max(np.linalg.norm(ref[sel]), 1e-300))
    return {"vec": vec, "W": w, "b": b}


def test_mlp1000_n8_ten_rounds_live_oracle():
    agn = _agn()
    wl = W.workload("mlp1000_n8")
    X, y, (xd, yd) = data_for(wl)
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed)
    o = AGNOracle(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed)
    tol1, tolR = TOL["fp32"]
    for r, order in enumerate(W.commit_orders(wl), start=1):
        g.round(xd, yd, order)
        o.round(X, y, order)
        tol = tol1 if r == 1 else tolR
        check(parity_report(g.central().cpu().numpy(), o.central_flat(), wl.dims), tol,
              f"mlp1000_n8 round {r} central")
        np.testing.assert_allclose(g.loss().cpu().numpy(), o.last_loss, rtol=1e-4)
    for k in range(wl.n):
        check(parity_report(g.worker_params(k).cpu().numpy(), o.worker_flat(k), wl.dims), tolR,
              f"mlp1000_n8 worker {k} pulled copy")
    g.close()


@pytest.mark.parametrize("name", ["mlp1000_n20", "mlp2000_n40", "wide_bf16"])
def test_full_rounds_against_stored_oracle_values(name):
    agn = _agn()
    path = os.path.join(GOLDEN, f"{name}.npz")
    assert os.path.exists(path), f"{path} missing: run tests/golden/make_golden.py {name}"
    gold = np.load(path, allow_pickle=False)
    wl = W.workload(name)
    X, y, (xd, yd) = data_for(wl)
    assert str(gold["digest"]) == W.data_digest(X, y), "regenerated inputs differ from the stored ones"
    pos = gold["positions"]
    tol1, tolR = TOL[wl.dtype]
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, dtype=wl.dtype)
    for r, order in enumerate(W.commit_orders(wl), start=1):
        g.round(xd, yd, order)
        if r == 1 or r == wl.rounds:
            tag, tol = ("r1", tol1) if r == 1 else ("last", tolR)
            c = g.central().cpu().numpy()
            check(sampled_report(c, pos, gold[f"{tag}_values"], gold[f"{tag}_maxabs"], wl.dims), tol,
                  f"{name} round {r} central (sampled)")
            np.testing.assert_allclose(g.loss().cpu().numpy(), gold[f"{tag}_loss"],
                                       rtol=1e-3 if wl.dtype == "fp32" else 2e-2)
    g.close()


@pytest.mark.parametrize("name", ["mlp2000_n40", "wide_bf16"])
def test_round1_sampled_workers_live(name):
    agn = _agn()
    wl = W.workload(name)
    X, y, (xd, yd) = data_for(wl)
    order = W.commit_orders(wl)[0]
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, dtype=wl.dtype)
    g.round(xd, yd, order)
    # the last committer pulls the final central variable
    assert np.array_equal(g.worker_params(int(order[-1])).cpu().numpy(), g.central().cpu().numpy())
    workers = [int(order[0]), wl.n - 1]
    got = {k: g.delta(k).cpu().numpy() for k in workers}
    loss = g.loss().cpu().numpy()
    g.close()
    o = AGNOracle(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, bf16=wl.dtype == "bf16")
    Xo = X if X.dtype != np.uint16 else W.f32_from_bf16_bits(X)
    start = o.worker_flat(0).astype(np.float64)
    for k in workers:
        _, lk, theta_fin = o._worker_round(k, Xo, y, wl.N // wl.n)
        disp = (flat_params(theta_fin).astype(np.float64) - start) / wl.lam
        fro, fw = rel_fro(got[k], disp, wl.dims)
        inf, iw = rel_err(got[k], disp, wl.dims)
        print(f"{name} round 1 worker {k}: delta vs displacement/lambda: fro {fro:.2e} ({fw}), "
              f"max {inf:.2e} ({iw})", flush=True)
        # a worker's delta has no large initial part to dilute a flipped ReLU
        # derivative, so only its Frobenius norm is gated
        assert fro <= DELTA_FRO[wl.dtype], (k, fw, fro)
        assert abs(loss[k] - lk) <= 1e-3 * abs(lk) + 1e-6
