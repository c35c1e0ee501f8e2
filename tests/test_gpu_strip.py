"""The strip schedule of a float32 hidden layer's backward launch (input
gradient and weight gradient + update sharing each weight block in LDS)
against the oracle.  The library takes that schedule when workers x column
strips of 64 reach 1024 (one workgroup per compute unit at a time), so these
shapes use many workers: 64 x 16 and 128 x 8 strips.

Shapes: strips and row blocks with ragged ends (996 and 1004 are not
multiples of 64), a row stride padded past the width (996 -> 1000), a
mini-batch below the 128 rows the schedule holds (m = 100), several local
steps (the round's last step stores the normalized displacement), two
rounds.  Gates as in the full-size tests (test_gpu_fullsize.py): round 1
against the live oracle on the whole central variable, every delta and every
pulled copy, and the commit bit for bit; round 2 on the central variable and
the pulled copies.
"""
import numpy as np
import pytest

import workloads as W
from oracle import AGNOracle
from tests.helpers import to_device, require_gpu
from tests.test_gpu_fullsize import BIAS_FACTOR, TOL, check_params, round1_against_live_oracle

pytestmark = pytest.mark.gpu

STRIP_CASES = [
    # name, dims, n, lam, m, eta, rounds, N, data
    ("strip_ragged", (96, 996, 1004, 12), 64, 2, 100, 0.02, 2, 64 * 300, "sparse_teacher2"),
    ("strip_two_hidden", (64, 512, 768, 512, 10), 128, 3, 128, 0.02, 2, 128 * 256, "sparse_teacher2"),
]


def strip_groups(dims, n, layer):
    return n * -(-dims[layer] // 64)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("case", STRIP_CASES, ids=[c[0] for c in STRIP_CASES])
def test_strip_schedule(case):
    require_gpu()
    import paper_1710_02368_amd as agn
    name, dims, n, lam, m, eta, R, N, data = case
    # every hidden layer l >= 1 below the output layer runs the strip schedule
    assert all(strip_groups(dims, n, l) >= 1024 for l in range(1, len(dims) - 2))
    wl = W.small_workload(name, dims, n, lam, m, eta, R, N, data=data, order="permutation")
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed)
    o = AGNOracle(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed)
    orders = W.commit_orders(wl)
    round1_against_live_oracle(g, o, wl, X, y, xd, yd, orders[0])
    tol = TOL["fp32"][1]
    for r, order in enumerate(orders[1:], start=2):
        g.round(xd, yd, order)
        o.round(X, y, order)
        check_params(g.central().cpu().numpy(), o.central_flat(), wl.dims, tol, BIAS_FACTOR["fp32"] * tol,
                     f"{name} round {r} central")
        np.testing.assert_allclose(g.loss().cpu().numpy(), o.last_loss, rtol=1e-4)
        for k in range(wl.n):
            check_params(g.worker_params(k).cpu().numpy(), o.worker_flat(k), wl.dims, tol,
                         BIAS_FACTOR["fp32"] * tol, f"{name} round {r} pulled copy {k}")
    g.close()
