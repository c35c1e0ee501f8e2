"""The strip schedules against the oracle: the backward launch of a float32
hidden layer (input gradient and weight gradient + update sharing each
weight block in LDS) and the first layer's weight gradient + update as
64-row strips of W_0 (gathered data rows streamed past a dZ_1 strip held in
LDS).  The library takes them when workers x strips of 64
reach 1024 (one workgroup per compute unit at a time), so these shapes use
many workers: 64 x 16 and 128 x 8 strips.

Shapes: strips and row blocks with ragged ends (996 and 1004 are not
multiples of 64; 968 leaves 8 rows in the last block, so most of its MFMA
groups are skipped), a row stride padded past the width (996 -> 1000), a
mini-batch below the 128 rows the schedule holds (m = 100), several local
steps (the round's last step stores the normalized displacement), two
rounds, Adam as the local rule (also on the first layer's strips, over
several column blocks of W_0 with a ragged last one).  Gates as in the full-size tests
(test_gpu_fullsize.py): round 1 against the live oracle on the whole central
variable, every delta and every pulled copy, and the commit bit for bit;
round 2 on the central variable and the pulled copies.  Adam: see
check_adam_round1 (test_gpu_fullsize.py).
"""
import numpy as np
import pytest

import workloads as W
from oracle import AGNOracle
from tests.helpers import to_device, require_gpu
from tests.test_gpu_fullsize import (BIAS_FACTOR, TOL, check_adam_round1, check_commit_prefix_sums, check_params,
                                     round1_against_live_oracle)

pytestmark = pytest.mark.gpu

ADAM = (0.9, 0.999, 1e-8)

STRIP_CASES = [
    # name, dims, n, lam, m, eta, rounds, N, data[, adam]
    ("strip_ragged", (96, 996, 1004, 12), 64, 2, 100, 0.02, 2, 64 * 300, "sparse_teacher2"),
    ("strip_short_tail", (96, 1000, 968, 12), 64, 2, 128, 0.02, 2, 64 * 300, "sparse_teacher2"),
    ("strip_two_hidden", (64, 512, 768, 512, 10), 128, 3, 128, 0.02, 2, 128 * 256, "sparse_teacher2"),
    ("strip_adam", (64, 516, 512, 10), 128, 3, 120, 0.002, 2, 128 * 256, "sparse_teacher2", ADAM),
    ("strip_adam_first_layer", (200, 516, 10), 128, 3, 120, 0.002, 2, 128 * 256, "sparse_teacher2", ADAM),
]


def strip_groups(dims, n, layer):
    return n * -(-dims[layer] // 64)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("case", STRIP_CASES, ids=[c[0] for c in STRIP_CASES])
def test_strip_schedule(case):
    require_gpu()
    import paper_1710_02368_amd as agn
    name, dims, n, lam, m, eta, R, N, data = case[:9]
    adam = case[9] if len(case) > 9 else None
    # every hidden layer l >= 1 below the output layer runs the strip schedule
    assert all(strip_groups(dims, n, l) >= 1024 for l in range(1, len(dims) - 2))
    wl = W.small_workload(name, dims, n, lam, m, eta, R, N, data=data, order="permutation")
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, adam=adam)
    o = AGNOracle(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, adam=adam)
    orders = W.commit_orders(wl)
    if adam is not None:
        check_adam_round1(g, o, wl, X, y, xd, yd, orders[0], adam)
        for r, order in enumerate(orders[1:], start=2):
            start = g.central().cpu().numpy()
            g.round(xd, yd, order)
            gdel = [g.delta(k).cpu().numpy() for k in range(wl.n)]
            check_commit_prefix_sums(start, gdel, [g.worker_params(k).cpu().numpy() for k in range(wl.n)],
                                     g.central().cpu().numpy(), order, f"{name} round {r}")
        g.close()
        return
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
