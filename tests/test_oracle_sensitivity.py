"""How far two correct implementations of the AGN round can drift apart.

The oracle is run against itself with its starting parameters perturbed by
a rounding-level 1e-7 (relative); the spread that results is a floor no
implementation with a different float32 summation order can beat.  These
measurements justify the full-size parity metrics and tolerances:

* float32: ReLU' is a step at zero, so a pre-activation within rounding
  distance of zero can flip its derivative; the flip changes one sample's
  contribution to one worker's gradient locally.  In the max-norm this can
  exceed 1e-4 for a single worker's delta after one step.
* bf16: every product operand is rounded to 8 significant bits; a
  rounding-level change moves some operands by one bf16 step and the change
  cascades through the layers, so single-step deltas differ by percent.
"""
import numpy as np
import pytest

import workloads as W
from oracle import AGNOracle, flat_params
from tests.helpers import rel_fro, tensor_slices


def spread(dims, m, lam, eta, dtype, pert=1e-7, seed=20171005):
    wl = W.small_workload("s", dims, 2, lam, m, eta, 1, N=2 * m * 10, data="gauss_linear",
                          order="sequential", dtype=dtype, seed=seed)
    X, y = W.make_data(wl)
    Xo = X if X.dtype != np.uint16 else W.f32_from_bf16_bits(X)
    out = []
    for p in (0.0, pert):
        o = AGNOracle(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, bf16=dtype == "bf16")
        rng = np.random.default_rng(3)
        o.workers[0] = [(Wt * (1 + p * rng.standard_normal(Wt.shape)).astype(np.float32), b)
                        for Wt, b in o.workers[0]]
        a, _, _ = o._worker_round(0, Xo, y, wl.N // wl.n)
        out.append(flat_params(a))
    return out


@pytest.mark.slow
def test_bf16_single_step_spread_is_percent_level():
    a, b = spread((3072, 2048, 2048, 2048, 100), 256, 1, 0.005, "bf16")
    err, where = rel_fro(b, a, (3072, 2048, 2048, 2048, 100))
    assert err > 5e-3, (err, where)


def test_fp32_single_step_spread_is_rounding_level():
    dims = (512, 256, 256, 100)
    a, b = spread(dims, 128, 1, 0.005, "fp32")
    err, where = rel_fro(b, a, dims)
    assert err < 1e-5, (err, where)


def test_bf16_spread_exceeds_fp32_at_the_same_shape():
    dims = (512, 256, 256, 100)
    a32, b32 = spread(dims, 128, 1, 0.005, "fp32")
    a16, b16 = spread(dims, 128, 1, 0.005, "bf16")
    assert rel_fro(b16, a16, dims)[0] > 10 * rel_fro(b32, a32, dims)[0]
