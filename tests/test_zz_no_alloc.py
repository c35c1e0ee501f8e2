"""agn_evaluate_noalloc (the allocation-free evaluation) against
agn_evaluate, through the C ABI, on two calls in a row (the second with
fewer rows), and its rejection of models whose buffers exceed its scratch
array.

The bar: predictions and the correct count equal (integer results), the
per-row losses equal bit for bit (the same kernels on the same rows; the
rows of a forward pass are independent), the float64 mean loss equal to
1e-12 relative (its partial sums may group differently when the variant
takes fewer rows per forward pass).
"""
import numpy as np
import pytest

import workloads as W
from tests.helpers import to_device, require_gpu

pytestmark = pytest.mark.gpu


def _agn():
    require_gpu()
    import paper_1710_02368_amd as agn
    return agn


CASES = [
    # name, dims, n, m, rows of the two calls, data, dtype
    ("fused_head", (200, 130, 70, 10), 3, 40, (9000, 777), "gauss_linear", "fp32"),
    # 4000-wide hidden layer: 32 KB of activations per row, so the scratch
    # array holds a few hundred rows and the 3000 rows take several passes
    ("wide_hidden", (64, 4000, 10), 2, 16, (3000, 513), "gauss_linear", "fp32"),
    ("many_classes", (60, 50, 40), 3, 24, (9000, 100), "gauss_linear", "fp32"),
    ("single_layer", (33, 7), 2, 16, (8193, 5), "gauss_linear", "fp32"),
    ("bf16", (256, 300, 300, 100), 4, 70, (5000, 1000), "gauss_linear", "bf16"),
]


def evaluate_both(agn, g, xd, yd, rows, dtype):
    import torch
    x, y = xd[:rows], yd[:rows]
    xdt = agn.AGN_BF16 if dtype == "bf16" else agn.AGN_FP32
    out = {}
    for name, fn in (("noalloc", agn.agn_evaluate_noalloc), ("evaluate", agn.agn_evaluate)):
        rl = torch.full((rows,), float("nan"), dtype=torch.float32, device="cuda")
        rp = torch.full((rows,), -1, dtype=torch.int32, device="cuda")
        res = fn(g.ctx, x, y, rows, xdt, rl, rp)
        out[name] = (res, rl.cpu().numpy(), rp.cpu().numpy())
    return out


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_evaluate(case):
    agn = _agn()
    name, dims, n, m, rows, data, dtype = case
    N = max(rows)
    wl = W.small_workload(name, dims, n, 2, m, 0.05, 1, N, data=data, dtype=dtype)
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, dtype=dtype)
    # the first call on a fresh context, before any agn_evaluate (so before
    # the allocating path's workspace exists), at the initial model
    first = evaluate_both(agn, g, xd, yd, rows[0], dtype)
    g.round(xd, yd, W.commit_orders(wl)[0])
    calls = [first] + [evaluate_both(agn, g, xd, yd, r, dtype) for r in rows]
    for i, res in enumerate(calls):
        (ra, la, pa), (rb, lb, pb) = res["noalloc"], res["evaluate"]
        assert not np.isnan(la).any()
        np.testing.assert_array_equal(pa, pb, err_msg=f"{name} call {i}: predictions")
        np.testing.assert_array_equal(la.view(np.int32), lb.view(np.int32), err_msg=f"{name} call {i}: losses")
        assert ra[2] == rb[2] and ra[1] == rb[1], (name, i, ra, rb)
        assert ra[0] == pytest.approx(rb[0], rel=1e-12), (name, i, ra, rb)
    g.close()


def test_noalloc_rejects_models_beyond_its_scratch():
    agn = _agn()
    # a 40,000-wide hidden layer: 64 rows of float32 activations, twice,
    # take 20 MB, more than the 16 MiB array
    wl = W.small_workload("too_wide", (16, 40000, 10), 2, 1, 8, 0.05, 1, 64)
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed)
    with pytest.raises(agn.AGNError) as e:
        agn.agn_evaluate_noalloc(g.ctx, xd, yd, 64)
    assert e.value.code == agn.AGN_EINVAL and "scratch" in str(e.value)
    # the context is not poisoned: the allocating path still works
    res = g.evaluate(xd, yd)
    assert 0 <= res[2] <= 64
    g.close()
