"""GPU path (libagn on gfx950) against the CPU oracle, element by element,
on the same seeded inputs and commit orders.

Tolerances (normwise per parameter tensor, maximum over tensors): float32
<= 1e-4 after one round and <= 1e-3 after several; bf16 <= 2e-2.  The
per-worker normalized deltas are compared in round 1, where both sides
start from the same central variable; in later rounds a rounding-level
difference in a worker's start can flip a ReLU derivative (a step function)
and change that worker's delta by far more than the central variable, so
later rounds compare the central variable, the pulled copies and the loss.  Integer
work (batch indices) is bit-exact.  Shapes are chosen to span several
64x64 tiles with ragged tails, unaligned input widths (scalar load path),
mini-batches that straddle the end of a shard, shards with an unused
remainder, a single layer, one worker, lambda = 1 and m = 1.
"""
import numpy as np
import pytest

import workloads as W
from oracle import AGNOracle, he_normal_init, flat_params, batch_indices
from tests.helpers import rel_err, tensor_slices, to_device, require_gpu

pytestmark = pytest.mark.gpu

ADAM = (0.9, 0.999, 1e-8)
FP32_TOL_1 = 1e-4
FP32_TOL_N = 1e-3
BF16_TOL = 2e-2


def _agn():
    require_gpu()
    import paper_1710_02368_amd as agn
    return agn


SMALL = [
    # name, dims, n, lam, m, eta, rounds, N, data, order, dtype
    ("ragged_deep", (200, 130, 70, 10), 3, 3, 40, 0.05, 3, 650, "gauss_linear", "permutation", "fp32"),
    ("unaligned_d0", (37, 29, 5), 4, 2, 9, 0.1, 4, 101, "sparse_teacher2", "permutation", "fp32"),
    ("single_layer", (64, 3), 2, 5, 16, 0.1, 2, 200, "gauss_linear", "sequential", "fp32"),
    ("sgd_n1_lam1", (50, 70, 4), 1, 1, 130, 0.05, 3, 300, "gauss_linear", "sequential", "fp32"),
    ("wide_tiles", (96, 300, 300, 12), 5, 2, 70, 0.05, 2, 1000, "sparse_teacher2", "permutation", "fp32"),
    ("batch_of_one", (16, 8, 2), 2, 3, 1, 0.1, 3, 10, "gauss_linear", "permutation", "fp32"),
    # the largest sizes the library accepts: AGN_MAX_LAYERS weight layers, and
    # AGN_MAX_WORKERS workers (commit orders over 256 workers, staleness up
    # to 255)
    ("max_layers", (24, 20, 18, 22, 16, 20, 24, 18, 16, 20, 22, 18, 16, 20, 24, 18, 6), 2, 2, 12, 0.05, 2, 200,
     "gauss_linear", "permutation", "fp32"),
    ("max_workers", (20, 16, 5), 256, 2, 8, 0.05, 2, 256 * 40, "gauss_linear", "permutation", "fp32"),
    # output-layer paths: many classes (separate logits product + softmax kernel),
    # a hidden width beyond the fused kernel's reach, and a fused kernel whose
    # LDS-resident output weights exceed 64 KB
    ("many_classes", (60, 50, 40), 3, 2, 24, 0.1, 2, 300, "gauss_linear", "permutation", "fp32"),
    ("wide_hidden", (30, 2100, 10), 2, 2, 8, 0.02, 2, 64, "gauss_linear", "permutation", "fp32"),
    ("big_head_lds", (50, 2000, 12), 2, 2, 16, 0.02, 2, 96, "gauss_linear", "permutation", "fp32"),
    # 32-class fused kernel over a width whose LDS rows are trimmed to the
    # width (1104 floats, not the 2048 its lanes span) to fit
    ("head_32_classes_wide", (40, 1102, 30), 2, 2, 16, 0.05, 2, 96, "gauss_linear", "permutation", "fp32"),
    ("head_trimmed_ragged", (50, 1502, 10), 3, 2, 16, 0.05, 2, 120, "gauss_linear", "permutation", "fp32"),
    # the fused output layer with each row's columns split over two waves
    # (width > 256): rows that do not allow 16-byte accesses, and the output
    # layer fed by the gathered data rows directly (with and without them)
    ("head_split_unaligned", (45, 301, 10), 3, 2, 20, 0.05, 2, 200, "gauss_linear", "permutation", "fp32"),
    ("head_split_gather", (301, 10), 2, 3, 16, 0.05, 2, 150, "gauss_linear", "permutation", "fp32"),
    ("head_split_gather_vec", (300, 7), 2, 3, 16, 0.05, 2, 150, "sparse_teacher2", "permutation", "fp32"),
    # bf16 products (bf16 operands, float32 accumulation and master weights)
    ("bf16_ragged", (200, 130, 70, 10), 3, 3, 40, 0.05, 3, 650, "gauss_linear", "permutation", "bf16"),
    ("bf16_many_classes", (256, 300, 300, 100), 4, 2, 70, 0.01, 2, 1000, "gauss_linear", "permutation", "bf16"),
    ("bf16_unaligned_d0", (37, 29, 5), 4, 2, 9, 0.1, 3, 101, "sparse_teacher2", "permutation", "bf16"),
    ("bf16_sgd_n1_lam1", (64, 150, 3), 1, 1, 130, 0.05, 3, 300, "gauss_linear", "sequential", "bf16"),
    # direct-load products with ragged 64-tiles: the persistent weight-gradient
    # schedule needs K = m >= 97 (four K steps) and widths divisible by 4
    ("dl_ragged", (100, 200, 136, 10), 3, 3, 100, 0.05, 3, 650, "sparse_teacher2", "permutation", "fp32"),
    ("bf16_dl_ragged", (100, 200, 136, 10), 3, 3, 100, 0.05, 2, 650, "sparse_teacher2", "permutation", "bf16"),
    # bf16 direct-load products on every layer but the output layer's
    # backward: ragged 128-tiles, a K tail (m = 100), the first layer's
    # weight gradient over gathered rows whose mini-batch wraps round the
    # shard's end (S = 216: steps at offsets 0, 100, 200)
    ("bf16_dl_gather", (136, 264, 200, 10), 3, 3, 100, 0.05, 2, 650, "sparse_teacher2", "permutation", "bf16"),
    # 256 x 256 forward tiles (a whole 256-row mini-batch per workgroup,
    # used from 256 tiles on): a hidden layer with a K tail, and the logits.
    # (Sparse inputs: with dense Gaussian ones some of the 16M hidden
    # pre-activations sit within rounding distance of zero, and the ReLU
    # mask they flip moves a committed delta by 2 % of its largest entry
    # between the oracle's own float32 and float64 products.)
    ("bf16_big_tiles", (520, 4096, 10), 16, 2, 256, 0.05, 1, 8192, "sparse_teacher2", "permutation", "bf16"),
    ("bf16_big_logits", (64, 264, 4096), 16, 2, 256, 0.05, 1, 8192, "gauss_linear", "permutation", "bf16"),
    # (Adam through the same kernels, at small widths: Adam's first step is
    # +-eta times the sign of the gradient, and on wider layers some
    # component's gradient cancels to the rounding level, where even the
    # oracle's float32 and float64 products disagree on its sign)
    ("bf16_dl_adam", (40, 48, 16, 10), 3, 3, 100, 0.002, 2, 650, "gauss_linear", "permutation", "bf16",
     True, ADAM),
    # without the normalization step (Section 2: DOWNPOUR with local
    # exploration): the committed delta is the accumulated update itself
    ("accumulated_ragged", (200, 130, 70, 10), 3, 3, 40, 0.02, 3, 650, "gauss_linear", "permutation", "fp32",
     False),
    ("accumulated_dl", (100, 200, 136, 10), 3, 3, 100, 0.02, 2, 650, "sparse_teacher2", "permutation", "fp32",
     False),
    # (one round: the bf16 rounding cascade grows with the lambda-times larger
    # commits; the commit rule is exercised in full by round 1)
    ("bf16_accumulated", (200, 130, 70, 10), 3, 3, 40, 0.02, 1, 650, "gauss_linear", "permutation", "bf16",
     False),
    # Adam as the local rule (moments kept across pulls)
    ("adam_ragged", (200, 130, 70, 10), 3, 3, 40, 0.002, 3, 650, "gauss_linear", "permutation", "fp32",
     True, ADAM),
    ("adam_dl_shape", (100, 200, 136, 10), 3, 3, 100, 0.002, 2, 650, "sparse_teacher2", "permutation", "fp32",
     True, ADAM),
    ("adam_many_classes", (60, 50, 40), 3, 2, 24, 0.002, 2, 300, "gauss_linear", "permutation", "fp32", True, ADAM),
    ("bf16_adam", (200, 130, 70, 10), 3, 3, 40, 0.002, 2, 650, "gauss_linear", "permutation", "bf16", True, ADAM),
    # staleness-scaled commits (Section 4's DynSGD comparison): with the
    # normalized delta, and DynSGD-style with the accumulated update
    ("stale_scaled_ragged", (200, 130, 70, 10), 3, 3, 40, 0.05, 3, 650, "gauss_linear", "permutation", "fp32",
     True, None, True),
    ("dynsgd_accumulated_dl", (100, 200, 136, 10), 4, 3, 100, 0.02, 3, 900, "sparse_teacher2", "permutation",
     "fp32", False, None, True),
    ("dynsgd_sequential", (64, 48, 10), 5, 2, 16, 0.05, 4, 400, "gauss_linear", "sequential", "fp32",
     False, None, True),
    ("bf16_dynsgd", (200, 130, 70, 10), 3, 3, 40, 0.02, 2, 650, "gauss_linear", "permutation", "bf16",
     False, None, True),
]


def delta_err(got, disp, start, dims, div, tol):
    """A committed delta against the oracle's displacement
    (theta_lambda - theta_0) / div, per tensor: the error allowed is tol
    relative to the delta, or 32 float32 ulps of the tensor's parameter scale
    (divided by div), whichever is larger.  The path stores the displacement
    of float32 parameters, so a rounding-level difference in theta_lambda is
    an error of a few ulps of theta in the delta, however small the delta
    is.  Returns (max over tensors of error / allowed, worst tensor)."""
    worst, where = 0.0, None
    got = got.astype(np.float64)
    for name, a, b in tensor_slices(dims):
        ref = disp[a:b]
        scale = np.max(np.abs(start[a:b]))
        ulp = 2.0 ** (np.floor(np.log2(scale)) - 23) if scale > 0 else 0.0
        allowed = max(tol * np.max(np.abs(ref)), 32 * ulp / div, 1e-30)
        e = np.max(np.abs(got[a:b] - ref)) / allowed
        if e > worst:
            worst, where = e, name
    return worst, where


def run_parity(wl, tol1, tolN, check_workers=True, normalize=True, adam=None, staleness_scaled=False):
    agn = _agn()
    import torch
    X, y = W.make_data(wl)
    orders = W.commit_orders(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, dtype=wl.dtype, normalize=normalize, adam=adam,
                staleness_scaled=staleness_scaled)
    o = AGNOracle(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, bf16=wl.dtype == "bf16",
                  normalize=normalize, adam=adam, staleness_scaled=staleness_scaled)
    # the initial central variable (same generator on both sides)
    init_err, _ = rel_err(g.central().cpu().numpy(), o.central_flat(), wl.dims)
    assert init_err <= 1e-7, f"init mismatch {init_err}"
    start = o.central_flat().astype(np.float64)   # every worker's round-1 start
    for r, order in enumerate(orders, start=1):
        g.round(xd, yd, order)
        o.round(X, y, order)
        tol = tol1 if r == 1 else tolN
        assert g.staleness() == o.staleness[-1]     # integer bookkeeping: exact
        err, where = rel_err(g.central().cpu().numpy(), o.central_flat(), wl.dims)
        print(f"{wl.name} round {r}: central rel err {err:.3e} ({where})", flush=True)
        assert err <= tol, (r, where, err)
        gl = g.loss().cpu().numpy()
        np.testing.assert_allclose(gl, o.last_loss, rtol=max(tol, 1e-5), atol=1e-6)
        if r == 1:   # the committed deltas (Eq. 1), from the same start
            div = wl.lam if normalize else 1
            # Adam's step depends on the ratio of a component's successive
            # gradients, not on their size: a component whose gradient is a
            # cancellation of larger terms carries the relative rounding
            # error of that gradient (bounded by the terms, not by the sum)
            # into its step.  The deltas are gated at 1e-2 (0.1 in bf16, the
            # per-worker bf16 gate); the central variable keeps the stated
            # bound
            dtol = tol if adam is None else (1e-2 if wl.dtype == "fp32" else 0.1)
            for k in range(wl.n):
                disp = (flat_params(o.last_finals[k]).astype(np.float64) - start) / div
                e, w = delta_err(g.delta(k).cpu().numpy(), disp, start, wl.dims, div, dtol)
                assert e <= 1.0, (r, k, w, e)
        if check_workers:
            for k in range(wl.n):
                e, w = rel_err(g.worker_params(k).cpu().numpy(), o.worker_flat(k), wl.dims)
                assert e <= tol, (r, k, w, e)
    torch.cuda.synchronize()
    g.close()


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_small_shapes(case):
    name, dims, n, lam, m, eta, R, N, data, order, dtype = case[:11]
    normalize = case[11] if len(case) > 11 else True
    adam = case[12] if len(case) > 12 else None
    scaled = case[13] if len(case) > 13 else False
    wl = W.small_workload(name, dims, n, lam, m, eta, R, N, data=data, order=order, dtype=dtype)
    tol1, tolN = (FP32_TOL_1, FP32_TOL_N) if dtype == "fp32" else (BF16_TOL, BF16_TOL)
    run_parity(wl, tol1, tolN, normalize=normalize, adam=adam, staleness_scaled=scaled)


@pytest.mark.timeout(300)
def test_adam_persistent_weight_gradient():
    """Adam as the local rule on the persistent direct-load weight-gradient
    kernels: the first layer's (with the output layer's folded in) and the
    combined backward launch of the hidden layer, 40 workers of
    128-256-256-10, so that each workgroup walks several tiles (the Adam
    variant runs one workgroup per compute unit).  Round 1 under the gates of
    check_adam_round1 (the commit bit for bit, every delta component within
    Adam's step bound, the median worker within 1e-4); round 2's commit bit
    for bit."""
    agn = _agn()
    from tests.test_gpu_fullsize import check_adam_round1, check_commit_prefix_sums
    wl = W.small_workload("adam_persistent", (128, 256, 256, 10), 40, 3, 128, 0.002, 2, 40 * 256,
                          data="sparse_teacher2", order="permutation")
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, adam=ADAM)
    o = AGNOracle(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, adam=ADAM)
    orders = W.commit_orders(wl)
    check_adam_round1(g, o, wl, X, y, xd, yd, orders[0], ADAM)
    start = g.central().cpu().numpy()
    g.round(xd, yd, orders[1])
    check_commit_prefix_sums(start, [g.delta(k).cpu().numpy() for k in range(wl.n)],
                             [g.worker_params(k).cpu().numpy() for k in range(wl.n)], g.central().cpu().numpy(),
                             orders[1], "adam_persistent round 2")
    g.close()


def test_downpour_lambda1_rules_coincide():
    """With lambda = 1 the normalized and the accumulated commit are the same
    rule (DOWNPOUR, Section 3 footnote to Eq. 1): bitwise equal results."""
    agn = _agn()
    wl = W.small_workload("dp", (100, 200, 136, 10), 4, 1, 100, 0.05, 3, 650, data="gauss_linear",
                          order="permutation")
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    res = []
    for normalize in (True, False):
        g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, normalize=normalize)
        for order in W.commit_orders(wl):
            g.round(xd, yd, order)
        res.append(g.central().cpu().numpy())
        g.close()
    np.testing.assert_array_equal(res[0], res[1])


def test_staleness_scaling_one_worker_is_plain():
    """n = 1: every commit has staleness 0, its scale is exactly 1, and the
    scaled commit is bitwise the plain one."""
    agn = _agn()
    wl = W.small_workload("s1", (100, 200, 136, 10), 1, 3, 100, 0.05, 3, 400, data="gauss_linear",
                          order="sequential")
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    res = []
    for scaled in (False, True):
        g = agn.AGN(wl.dims, 1, wl.lam, wl.eta, wl.m, seed=wl.seed, staleness_scaled=scaled)
        for order in W.commit_orders(wl):
            g.round(xd, yd, order)
            assert g.staleness() == [0]
        res.append(g.central().cpu().numpy())
        g.close()
    np.testing.assert_array_equal(res[0], res[1])


def test_set_staleness_scaling_errors():
    agn = _agn()
    g = agn.AGN((20, 16, 6), 2, 1, 0.05, 8, seed=1)
    assert agn.load_library().agn_set_staleness_scaling(g.ctx, 2) == -1   # (the binding passes a bool)
    with pytest.raises(agn.AGNError) as ei:
        g.staleness()
    assert ei.value.code == -4
    wl = W.small_workload("se", (20, 16, 6), 2, 1, 8, 0.05, 1, 64)
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g.round(xd, yd, [1, 0])
    assert g.staleness() == [0, 1]
    with pytest.raises(agn.AGNError) as ei:
        agn.agn_set_staleness_scaling(g.ctx, True)
    assert ei.value.code == -4
    g.close()


def test_set_optimizer_errors():
    """Bad hyperparameters: AGN_EINVAL; after the first round: AGN_ESTATE."""
    agn = _agn()
    wl = W.small_workload("opt", (20, 12, 4), 3, 2, 5, 0.1, 1, 60)
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=4)
    for args in [(2, 0.9, 0.999, 1e-8), (1, 1.0, 0.999, 1e-8), (1, 0.9, -0.1, 1e-8), (1, 0.9, 0.999, 0.0)]:
        with pytest.raises(agn.AGNError) as ei:
            agn.agn_set_optimizer(g.ctx, *args)
        assert ei.value.code == -1
    agn.agn_set_optimizer(g.ctx, agn.AGN_OPT_ADAM)
    g.round(xd, yd, [0, 1, 2])
    with pytest.raises(agn.AGNError) as ei:
        agn.agn_set_optimizer(g.ctx, agn.AGN_OPT_SGD)
    assert ei.value.code == -4
    g.close()


def test_set_normalization_errors():
    """Only 0 or 1, and only before the first round (AGN_EINVAL / AGN_ESTATE)."""
    agn = _agn()
    wl = W.small_workload("nrm", (20, 12, 4), 3, 2, 5, 0.1, 1, 60)
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=4)
    assert agn.load_library().agn_set_normalization(g.ctx, 2) == -1
    agn.agn_set_normalization(g.ctx, False)
    g.round(xd, yd, [0, 1, 2])
    with pytest.raises(agn.AGNError) as ei:
        agn.agn_set_normalization(g.ctx, True)
    assert ei.value.code == -4
    g.close()


def test_tiny_workload_full_size():
    run_parity(W.workload("tiny"), FP32_TOL_1, FP32_TOL_1)


def test_batch_indices_bit_exact():
    agn = _agn()
    for (N, n, m) in [(4096, 2, 32), (60000, 8, 128), (60000, 20, 128), (120000, 40, 128),
                      (262144, 32, 256), (101, 4, 9), (10, 2, 1)]:
        g = agn.AGN((8, 2), n, 1, 0.1, m, seed=1)
        S = N // n
        for k in sorted({0, n // 2, n - 1}):
            for t in (0, 1, 7, 58, 449, 10 ** 7 + 3):
                got = g.batch_indices(k, t, N).cpu().numpy()
                np.testing.assert_array_equal(got, batch_indices(k, t, m, S))
        g.close()


def test_init_matches_oracle_generator():
    agn = _agn()
    for dims, seed in [((784, 1000, 1000, 10), 20171002), ((3072, 2048, 100), 5), ((7, 3, 2), 2 ** 63 + 11)]:
        g = agn.AGN(dims, 2, 1, 0.1, 4, seed=seed)
        got = g.central().cpu().numpy()
        ref = flat_params(he_normal_init(dims, seed))
        diff = got.view(np.int32).astype(np.int64) - ref.view(np.int32).astype(np.int64)
        assert np.max(np.abs(diff)) <= 1, "more than 1 ulp apart"
        assert np.mean(diff == 0) > 0.999
        g.close()


def test_determinism_bitwise():
    agn = _agn()
    wl = W.small_workload("det", (96, 300, 300, 12), 5, 3, 70, 0.05, 2, 1000)
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    res = []
    for _ in range(2):
        g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed)
        for order in W.commit_orders(wl):
            g.round(xd, yd, order)
        res.append((g.central().cpu().numpy(), g.loss().cpu().numpy()))
        g.close()
    np.testing.assert_array_equal(res[0][0], res[1][0])
    np.testing.assert_array_equal(res[0][1], res[1][1])


def test_set_central_and_eta_zero_fixed_point():
    agn = _agn()
    import torch
    wl = W.small_workload("fix", (40, 24, 6), 3, 2, 8, 0.0, 2, 120)
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(wl.dims, wl.n, wl.lam, 0.0, wl.m, seed=3)
    v = torch.linspace(-1, 1, g.P, device="cuda", dtype=torch.float32)
    g.set_central(v)
    g.round(xd, yd, [2, 0, 1])
    assert torch.equal(g.central(), v)
    for k in range(wl.n):
        assert torch.equal(g.worker_params(k), v)
    with pytest.raises(agn.AGNError):          # only before the first round
        g.set_central(v)
    g.close()


def test_errors_leave_state_unchanged():
    agn = _agn()
    wl = W.small_workload("err", (20, 12, 4), 3, 2, 5, 0.1, 1, 60)
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=4)
    c0 = g.central().cpu().numpy()
    for bad in ([0, 0, 1], [0, 1, 3], [2, 2, 2], [-1, 0, 1]):
        with pytest.raises(agn.AGNError) as ei:
            agn.agn_round(g.ctx, xd, yd, X.shape[0], bad)
        assert ei.value.code == -1
    with pytest.raises(agn.AGNError):
        agn.agn_round(g.ctx, xd, yd, X.shape[0], [0, 1, 2], x_dtype=1)
    with pytest.raises(agn.AGNError):
        agn.agn_round(g.ctx, xd, yd, 2, [0, 1, 2])       # fewer samples than workers
    with pytest.raises(agn.AGNError) as ei:
        g.loss()                                          # no round yet
    assert ei.value.code == -4
    np.testing.assert_array_equal(g.central().cpu().numpy(), c0)
    g.round(xd, yd, [1, 2, 0])
    with pytest.raises(agn.AGNError):
        agn.agn_round(g.ctx, xd, yd, X.shape[0] - 1, [0, 1, 2])   # N changed
    g.close()


def test_rounds_on_a_caller_stream_match_the_null_stream():
    """A context bound to a stream the caller created (agn_set_stream, here a
    torch stream of default priority) records and replays its round graph on
    that stream: three rounds equal, bit for bit, the same rounds of a context
    on the null stream, and the per-worker losses too."""
    agn = _agn()
    import torch
    wl = W.small_workload("stream", (100, 70, 60, 10), 4, 3, 20, 0.05, 3, 400, order="permutation")
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    orders = W.commit_orders(wl)
    g0 = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed)
    for order in orders:
        g0.round(xd, yd, order)
    ref_c, ref_l = g0.central().cpu().numpy(), g0.loss().cpu().numpy()
    g0.close()
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        g1 = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed)
        for order in orders:
            g1.round(xd, yd, order)
        c1, l1 = g1.central(), g1.loss()
    s.synchronize()
    assert np.array_equal(c1.cpu().numpy(), ref_c)
    assert np.array_equal(l1.cpu().numpy(), ref_l)
    g1.close()


def test_interleaved_contexts_keep_their_own_state():
    """Two contexts in one process, a float32 and a bf16 one of different
    shapes, their rounds interleaved: each ends bit for bit where it ends
    when it runs alone (no state shared between contexts)."""
    agn = _agn()
    cases = [W.small_workload("ctx_a", (100, 70, 60, 10), 4, 3, 20, 0.05, 3, 400, order="permutation"),
             W.small_workload("ctx_b", (136, 264, 200, 10), 3, 2, 40, 0.05, 3, 650, data="sparse_teacher2",
                              order="permutation", dtype="bf16")]
    data = [W.make_data(wl) for wl in cases]
    dev = [to_device(X, y) for X, y in data]
    orders = [W.commit_orders(wl) for wl in cases]

    def make(wl):
        return agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, dtype=wl.dtype)

    alone = []
    for k, wl in enumerate(cases):
        g = make(wl)
        for order in orders[k]:
            g.round(*dev[k], order)
        alone.append(g.central().cpu().numpy())
        g.close()
    gs = [make(wl) for wl in cases]
    for r in range(3):
        for k in (1, 0):
            gs[k].round(*dev[k], orders[k][r])
    for k in range(2):
        assert np.array_equal(gs[k].central().cpu().numpy(), alone[k]), cases[k].name
        gs[k].close()


def test_divergent_learning_rate_is_reported_not_fatal():
    """A learning rate far too large for the model (eta = 1e5): the weights
    grow by orders of magnitude per round and overflow float32 within a few
    rounds, in the oracle as on the GPU.  The library keeps running (every
    round returns success), round 1 still matches the oracle, and the
    divergence shows where a caller looks for it: non-finite entries in the
    per-worker losses of agn_loss and in the central variable; agn_evaluate
    of the diverged central variable returns a non-finite mean loss and
    predictions inside the class range."""
    agn = _agn()
    wl = W.small_workload("diverge", (20, 12, 4), 3, 2, 5, 1e5, 4, 60)
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed)
    o = AGNOracle(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed)
    orders = W.commit_orders(wl)
    with np.errstate(all="ignore"):
        g.round(xd, yd, orders[0])
        o.round(X, y, orders[0])
        err, where = rel_err(g.central().cpu().numpy(), o.central_flat(), wl.dims)
        assert err <= FP32_TOL_1, (where, err)
        oracle_finite = [bool(np.isfinite(o.central_flat()).all())]
        for order in orders[1:]:
            g.round(xd, yd, order)
            o.round(X, y, order)
            oracle_finite.append(bool(np.isfinite(o.central_flat()).all()))
    assert not oracle_finite[-1], oracle_finite                 # the oracle diverged too
    c = g.central().cpu().numpy()
    assert not np.isfinite(c).all()
    assert not np.isfinite(g.loss().cpu().numpy()).all()
    loss, acc, correct = g.evaluate(xd, yd)
    assert not np.isfinite(loss) and 0 <= correct <= X.shape[0] and acc == correct / X.shape[0]
    _, rl, rp = g.evaluate(xd, yd, row_outputs=True)
    rp = rp.cpu().numpy()
    assert rp.min() >= 0 and rp.max() < wl.dims[-1]
    g.close()


@pytest.mark.parametrize("dims,folded", [((100, 200, 136, 10), True), ((100, 200, 136, 12), False),
                                         ((100, 200, 10), True)])
def test_output_layer_update_rides_in_first_layer_launch(dims, folded):
    """With at most 10 classes and the first layer's weight gradient on the
    direct-load path, the output layer's weight update runs inside that
    launch on every local step (the round's last one included, where it
    stores the normalized displacement); the class accounting follows, and
    the round still matches the oracle."""
    agn = _agn()
    wl = W.small_workload("fold", dims, 3, 2, 100, 0.05, 1, 650, data="sparse_teacher2", order="permutation")
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed)
    o = AGNOracle(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed)
    for c in agn.KERNEL_CLASSES.values():
        agn.agn_set_kernel_timing(g.ctx, c, True)
    order = W.commit_orders(wl)[0]
    g.round(xd, yd, order)
    o.round(X, y, order)
    _, n_out_dw = agn.agn_kernel_timing(g.ctx, agn.KERNEL_CLASSES["output_dw"])
    _, n_first = agn.agn_kernel_timing(g.ctx, agn.KERNEL_CLASSES["dw_first"])
    f_out_dw, _ = agn.agn_kernel_class_work(g.ctx, agn.KERNEL_CLASSES["output_dw"])
    f_first, _ = agn.agn_kernel_class_work(g.ctx, agn.KERNEL_CLASSES["dw_first"])
    mac = lambda l: dims[l] * dims[l + 1]
    rows = wl.n * wl.lam * wl.m
    assert n_first == wl.lam
    if folded:
        assert n_out_dw == 0 and f_out_dw == 0.0
        assert f_first == pytest.approx(2.0 * (mac(0) + mac(len(dims) - 2)) * rows, rel=1e-12)
    else:
        assert n_out_dw == wl.lam and f_out_dw == pytest.approx(2.0 * mac(len(dims) - 2) * rows, rel=1e-12)
        assert f_first == pytest.approx(2.0 * mac(0) * rows, rel=1e-12)
    err, where = rel_err(g.central().cpu().numpy(), o.central_flat(), wl.dims)
    assert err <= FP32_TOL_1, (where, err)
    for k in range(wl.n):
        e, w = rel_err(g.worker_params(k).cpu().numpy(), o.worker_flat(k), wl.dims)
        assert e <= FP32_TOL_1, (k, w, e)
    g.close()


def test_graph_replay_and_eager_launches_agree():
    """Rounds run eagerly (kernel timing on) and rounds replayed from the
    captured graph launch the same kernels: results are bitwise equal; the
    graph is re-captured when the data pointers change."""
    agn = _agn()
    import torch
    wl = W.small_workload("ge", (96, 300, 300, 12), 5, 3, 70, 0.05, 3, 1000)
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    orders = W.commit_orders(wl)
    res = []
    for eager in (False, True):
        g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed)
        if eager:
            for c in agn.KERNEL_CLASSES.values():
                agn.agn_set_kernel_timing(g.ctx, c, True)
        for r, order in enumerate(orders):
            if r == 2:   # new buffers with the same contents: a new binding
                xd, yd = xd.clone(), yd.clone()
            g.round(xd, yd, order)
        res.append((g.central().cpu().numpy(), g.loss().cpu().numpy()))
        if eager:
            g.evaluate(xd, yd)   # (the evaluation's class: not part of a round)
            for name, c in agn.KERNEL_CLASSES.items():
                ms, cnt = agn.agn_kernel_timing(g.ctx, c)
                assert cnt > 0 and ms > 0, name
        g.close()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(res[0][0], res[1][0])
    np.testing.assert_array_equal(res[0][1], res[1][1])
