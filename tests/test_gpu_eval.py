"""Evaluation of the central variable on the GPU (agn_evaluate) against the
oracle's evaluation, row by row, and the temporal efficiency (Eq. 4) of
curves measured on the GPU against the oracle's.

Per-row losses: float32 within 1e-4 of the oracle (relative to max(1,
|loss|)); bf16 normwise within 2e-2.  Predictions: a row's predicted class
must be a maximum of the oracle's logits up to the logit tolerance (the
same bound), so rows whose two largest logits are farther apart than that
must agree exactly; the correct count may differ from the oracle's only by
rows within that margin, and equals the count of the returned predictions
exactly.  The mean loss equals the float64 mean of the returned row losses.
"""
import math

import numpy as np
import pytest

import workloads as W
from oracle import AGNOracle, evaluate, temporal_efficiency, unflat_params
from tests.helpers import to_device, require_gpu

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-4
BF16_TOL = 2e-2


def _agn():
    require_gpu()
    import paper_1710_02368_amd as agn
    return agn


def check_rows(res, rl, rp, X, y, params, dims, dtype, tol):
    """Compare one GPU evaluation with the oracle's on (X, y) at params."""
    row_loss, pred, logits = evaluate(params, X, y, bf16=dtype == "bf16")
    rl = rl.cpu().numpy().astype(np.float64)
    rp = rp.cpu().numpy()
    N = len(y)
    assert rl.shape == (N,) and rp.shape == (N,)
    if dtype == "fp32":
        err = np.max(np.abs(rl - row_loss) / np.maximum(1.0, np.abs(row_loss)))
    else:
        err = np.linalg.norm(rl - row_loss) / max(np.linalg.norm(row_loss), 1e-30)
    assert err <= tol, err
    z = logits.astype(np.float64)
    zmax = z.max(axis=1)
    margin = tol * np.maximum(1.0, np.abs(zmax))
    chosen = z[np.arange(N), rp]
    assert np.all(chosen >= zmax - margin), np.flatnonzero(chosen < zmax - margin)[:10]
    zs = np.sort(z, axis=1)
    close = (zs[:, -1] - zs[:, -2]) <= margin        # rows whose prediction may differ
    assert np.array_equal(rp[~close], pred[~close])
    mean_loss, acc, correct = res
    assert correct == int(np.sum(rp == y))
    assert abs(correct - int(np.sum(pred == y))) <= int(close.sum())
    assert acc == correct / N
    assert mean_loss == pytest.approx(float(np.sum(rl) / N), rel=1e-12, abs=1e-300)
    return err, int(close.sum())


EVAL_CASES = [
    # name, dims, n, m, N rows, data, dtype
    ("head_ragged", (200, 130, 70, 10), 3, 40, 650, "gauss_linear", "fp32"),
    # output weights in LDS rows trimmed to the width (1502, not a multiple of 4)
    ("head_trimmed_rows", (40, 1502, 10), 2, 16, 300, "gauss_linear", "fp32"),
    ("unaligned_d0", (37, 29, 5), 4, 9, 101, "sparse_teacher2", "fp32"),
    ("many_classes", (60, 50, 40), 3, 24, 300, "gauss_linear", "fp32"),
    ("dl_shape", (100, 200, 136, 10), 3, 100, 1000, "sparse_teacher2", "fp32"),
    ("single_layer", (64, 3), 2, 16, 77, "gauss_linear", "fp32"),
    ("one_row", (50, 70, 4), 2, 30, 1, "gauss_linear", "fp32"),
    ("fewer_rows_than_chunk", (50, 70, 4), 2, 30, 41, "gauss_linear", "fp32"),
    ("bf16_ragged", (200, 130, 70, 10), 3, 40, 650, "gauss_linear", "bf16"),
    ("bf16_many_classes", (256, 300, 300, 100), 4, 70, 1000, "gauss_linear", "bf16"),
    ("bf16_unaligned_d0", (37, 29, 5), 4, 9, 101, "sparse_teacher2", "bf16"),
    # more rows than the 8192 the library evaluates at a time
    ("two_chunks", (200, 130, 70, 10), 3, 40, 8192 + 77, "gauss_linear", "fp32"),
    ("exact_chunk", (64, 48, 10), 2, 16, 8192, "gauss_linear", "fp32"),
    ("two_chunks_single_layer", (33, 7), 2, 16, 8193, "gauss_linear", "fp32"),
    ("two_chunks_many_classes", (60, 50, 40), 3, 24, 9000, "gauss_linear", "fp32"),
    ("bf16_two_chunks", (200, 130, 70, 10), 3, 40, 8192 + 555, "gauss_linear", "bf16"),
    # a full 8192-row chunk of a 2048-wide layer: 256 x 256 forward tiles
    ("bf16_big_tiles", (64, 2048, 10), 2, 16, 8192 + 300, "gauss_linear", "bf16"),
]


@pytest.mark.parametrize("case", EVAL_CASES, ids=[c[0] for c in EVAL_CASES])
@pytest.mark.parametrize("model", ["initial", "set"])
def test_evaluate_matches_oracle(case, model):
    """The initial model (same generator on both sides) and a seeded model
    set on both sides, over sets smaller and larger than the 8192 rows the
    library evaluates at a time, ragged at the tile and chunk edges."""
    agn = _agn()
    name, dims, n, m, N, data, dtype = case
    wl = W.small_workload(name, dims, n, 2, m, 0.05, 1, N, data=data, dtype=dtype)
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(dims, n, 2, 0.05, m, seed=wl.seed, dtype=dtype)
    if model == "set":
        import torch
        vec = W.random_params(dims, wl.seed, scale=2.0)
        g.set_central(torch.from_numpy(vec).cuda())
        params = unflat_params(vec, dims)
    else:
        params = AGNOracle(dims, n, 2, 0.05, m, seed=wl.seed, bf16=dtype == "bf16").central
    res, rl, rp = g.evaluate(xd, yd, row_outputs=True)
    tol = FP32_TOL if dtype == "fp32" else BF16_TOL
    err, close = check_rows(res, rl, rp, X, y, params, dims, dtype, tol)
    print(f"{name}/{model}: row loss err {err:.2e}, near-tie rows {close}, acc {res[1]:.4f}", flush=True)
    g.close()


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_evaluate_after_rounds(dtype):
    """Both sides train for 3 rounds, then each evaluates its own central
    variable on a held-out set (the validation accuracy of Section 4)."""
    agn = _agn()
    dims = (100, 200, 136, 10)
    wl = W.small_workload("after", dims, 3, 3, 100, 0.05, 3, 900, data="sparse_teacher2", dtype=dtype)
    X, y = W.make_data(wl)
    Xh, yh = W.make_heldout(wl, 700)
    xd, yd = to_device(X, y)
    xh, yh_d = to_device(Xh, yh)
    g = agn.AGN(dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, dtype=dtype)
    o = AGNOracle(dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, bf16=dtype == "bf16")
    for order in W.commit_orders(wl):
        g.round(xd, yd, order)
        o.round(X, y, order)
    res, rl, rp = g.evaluate(xh, yh_d, row_outputs=True)
    # the central variables agree to the round parity bound, so the logits
    # agree to about that bound times their scale
    tol = 1e-3 if dtype == "fp32" else BF16_TOL
    check_rows(res, rl, rp, Xh, yh, o.central, dims, dtype, tol)
    g.close()


@pytest.mark.parametrize("dtype,lam", [("fp32", 3), ("bf16", 3), ("bf16", 1)])
def test_evaluate_leaves_training_unchanged(dtype, lam):
    """round, evaluate, round gives bitwise the same central variable, pulled
    copies and losses as round, round."""
    agn = _agn()
    dims = (200, 130, 70, 10)
    wl = W.small_workload("undisturbed", dims, 3, lam, 40, 0.05, 2, 650, dtype=dtype)
    X, y = W.make_data(wl)
    Xh, yh = W.make_heldout(wl, 333)
    xd, yd = to_device(X, y)
    xh, yh_d = to_device(Xh, yh)
    out = []
    for with_eval in (False, True):
        g = agn.AGN(dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, dtype=dtype)
        for r, order in enumerate(W.commit_orders(wl)):
            g.round(xd, yd, order)
            if with_eval:
                g.evaluate(xh, yh_d)
        out.append((g.central().cpu().numpy(), g.loss().cpu().numpy(),
                    [g.worker_params(k).cpu().numpy() for k in range(wl.n)]))
        g.close()
    np.testing.assert_array_equal(out[0][0], out[1][0])
    np.testing.assert_array_equal(out[0][1], out[1][1])
    for a, b in zip(out[0][2], out[1][2]):
        np.testing.assert_array_equal(a, b)


def test_evaluate_is_deterministic():
    agn = _agn()
    dims = (100, 200, 136, 10)
    wl = W.small_workload("det", dims, 3, 2, 100, 0.05, 1, 2345, data="sparse_teacher2")
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    g = agn.AGN(dims, 3, 2, 0.05, 100, seed=wl.seed)
    a = g.evaluate(xd, yd, row_outputs=True)
    b = g.evaluate(xd, yd, row_outputs=True)
    assert a[0] == b[0]
    assert np.array_equal(a[1].cpu().numpy(), b[1].cpu().numpy())
    assert np.array_equal(a[2].cpu().numpy(), b[2].cpu().numpy())
    g.close()


def test_evaluate_non_finite_logits():
    """A NaN output bias makes that class's logit NaN on every row: the
    oracle's argmax picks it (NumPy's rule), the library's too, and every
    row's loss is NaN on both sides.  An infinite bias gives a NaN loss
    (inf - inf in the log-sum-exp) and predicts that class."""
    agn = _agn()
    import torch
    dims = (20, 16, 6)
    wl = W.small_workload("nan", dims, 2, 1, 8, 0.05, 1, 50)
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    for bad, cls in ((np.nan, 4), (np.inf, 2)):
        vec = W.random_params(dims, 7)
        vec[-dims[-1] + cls] = bad
        g = agn.AGN(dims, 2, 1, 0.05, 8, seed=1)
        g.set_central(torch.from_numpy(vec).cuda())
        res, rl, rp = g.evaluate(xd, yd, row_outputs=True)
        row_loss, pred, _ = evaluate(unflat_params(vec, dims), X, y)
        assert np.all(np.isnan(row_loss)) and np.all(np.isnan(rl.cpu().numpy()))
        np.testing.assert_array_equal(pred, cls)
        np.testing.assert_array_equal(rp.cpu().numpy(), cls)
        assert math.isnan(res[0]) and res[2] == int(np.sum(y == cls))
        g.close()


def test_evaluate_label_out_of_range():
    """A label outside [0, C) reads no logit: that row's loss is NaN and it
    does not count as correct; the prediction is still given."""
    agn = _agn()
    import torch
    dims = (20, 16, 6)
    wl = W.small_workload("lbl", dims, 2, 1, 8, 0.05, 1, 40)
    X, y = W.make_data(wl)
    y_bad = y.copy()
    y_bad[[3, 17]] = [6, -1]
    xd, yd = to_device(X, y_bad)
    g = agn.AGN(dims, 2, 1, 0.05, 8, seed=wl.seed)
    res, rl, rp = g.evaluate(xd, yd, row_outputs=True)
    rl = rl.cpu().numpy()
    rp = rp.cpu().numpy()
    assert np.isnan(rl[3]) and np.isnan(rl[17])
    assert np.all(np.isfinite(np.delete(rl, [3, 17])))
    assert np.all((rp >= 0) & (rp < 6))
    assert res[2] == int(np.sum(rp == y_bad))
    g.close()
    del torch


def test_evaluate_errors():
    agn = _agn()
    import torch
    dims = (20, 16, 6)
    g = agn.AGN(dims, 2, 1, 0.05, 8, seed=1)
    x = torch.zeros((10, 20), dtype=torch.float32, device="cuda")
    y = torch.zeros(10, dtype=torch.int32, device="cuda")
    with pytest.raises(agn.AGNError) as ei:
        agn.agn_evaluate(g.ctx, x, y, 0)
    assert ei.value.code == -1 and "num_samples" in str(ei.value)
    with pytest.raises(agn.AGNError) as ei:
        agn.agn_evaluate(g.ctx, x, y, 10, x_dtype=1)
    assert ei.value.code == -1 and "x_dtype" in str(ei.value)
    # still usable after rejected calls
    assert agn.agn_evaluate(g.ctx, x, y, 10)[2] >= 0
    g.close()


def test_temporal_efficiency_of_gpu_curves():
    """Accuracy curves of AGN and of DOWNPOUR with accumulated updates
    (the un-normalized commit), measured on the GPU and in the oracle
    against worker-samples processed; Eq. 4 from the library on the GPU
    curves agrees with the oracle's Eq. 4 on the oracle's curves."""
    agn = _agn()
    dims = (100, 200, 136, 10)
    wl = W.small_workload("te", dims, 4, 5, 100, 0.02, 4, 2000, data="sparse_teacher2")
    X, y = W.make_data(wl)
    Xh, yh = W.make_heldout(wl, 1000)
    xd, yd = to_device(X, y)
    xh, yh_d = to_device(Xh, yh)
    curves_g, curves_o = {}, {}
    for normalize in (True, False):
        g = agn.AGN(dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, normalize=normalize)
        o = AGNOracle(dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, normalize=normalize)
        t, fg, fo = [0.0], [g.evaluate(xh, yh_d)[1]], [float(np.mean(evaluate(o.central, Xh, yh)[1] == yh))]
        for r, order in enumerate(W.commit_orders(wl), start=1):
            g.round(xd, yd, order)
            o.round(X, y, order)
            t.append(float(r * wl.worker_samples_per_round))
            fg.append(g.evaluate(xh, yh_d)[1])
            fo.append(float(np.mean(evaluate(o.central, Xh, yh)[1] == yh)))
        curves_g[normalize] = (t, fg)
        curves_o[normalize] = (t, fo)
        g.close()
        # the accuracies agree up to rows within rounding of a tie
        assert np.max(np.abs(np.array(fg) - np.array(fo))) <= 0.01, (fg, fo)
    e_gpu = agn.agn_temporal_efficiency(*curves_g[True], *curves_g[False])
    e_ora = temporal_efficiency(*curves_o[True], *curves_o[False])
    # accuracies that differ by at most d move each area by at most d * T,
    # so E by at most (d * T / area_b) * (1 + E)
    d = max(np.max(np.abs(np.array(curves_g[k][1]) - np.array(curves_o[k][1]))) for k in (True, False))
    T = curves_o[True][0][-1]
    area_b = T * float(np.mean(curves_o[False][1]))   # (equal spacing: trapezoid ~ mean)
    bound = d * T / (0.5 * area_b) * (1 + e_ora) + 1e-12
    print(f"E(AGN, accumulated DOWNPOUR): GPU {e_gpu:.5f}, oracle {e_ora:.5f}, bound {bound:.2e}", flush=True)
    assert abs(e_gpu - e_ora) <= bound


@pytest.mark.parametrize("name,rows,rounds", [("mlp1000_n8", W.HELDOUT_ROWS, 1), ("wide_bf16", 2048, 0)])
def test_evaluate_full_size(name, rows, rounds):
    """The benchmark's evaluation: the central variable of a full-size
    workload on its held-out set, after `rounds` rounds on both sides."""
    agn = _agn()
    wl = W.workload(name)
    Xh, yh = W.make_heldout(wl, rows)
    xh, yh_d = to_device(Xh, yh)
    g = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, dtype=wl.dtype)
    o = AGNOracle(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, bf16=wl.dtype == "bf16")
    if rounds:
        X, y = W.make_data(wl)
        xd, yd = to_device(X, y)
        for order in W.commit_orders(wl, rounds):
            g.round(xd, yd, order)
            o.round(X, y, order)
    res, rl, rp = g.evaluate(xh, yh_d, row_outputs=True)
    tol = (FP32_TOL if rounds == 0 else 1e-3) if wl.dtype == "fp32" else BF16_TOL
    err, close = check_rows(res, rl, rp, Xh, yh, o.central, wl.dims, wl.dtype, tol)
    print(f"{name}: rows {rows}, row loss err {err:.2e}, near-tie rows {close}, "
          f"loss {res[0]:.5f}, acc {res[1]:.4f}", flush=True)
    g.close()


def test_accumulated_commits_fail_to_converge_where_agn_does():
    """The paper's motivating contrast (Section 2, the accumulated-gradient
    DOWNPOUR divergence figure) on the library itself: the same workers,
    learning rate, local steps and commit orders, once with the normalized
    commit (Eq. 2 with Eq. 1's delta / lambda) and once committing the
    accumulated update.  The central variable's loss, measured by
    agn_evaluate after every round, falls in every round under AGN, and under
    accumulated commits it does not, ending well above AGN's.  The same
    workload pins the oracle's trajectories in test_oracle_pins.py; here each
    measured loss is also held to the oracle's evaluation of the oracle's
    central variable after the same round."""
    agn = _agn()
    dims, n, lam, eta, m, R = (20, 16, 4), 8, 10, 0.1, 16, 6
    wl = W.small_workload("dv", dims, n, lam, m, eta, R, 4096, data="gauss_linear", order="permutation")
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    xe, ye = to_device(X[:1024], y[:1024])
    traj = {}
    for normalize in (True, False):
        g = agn.AGN(dims, n, lam, eta, m, seed=wl.seed, normalize=normalize)
        o = AGNOracle(dims, n, lam, eta, m, seed=wl.seed, normalize=normalize)
        losses = []
        for order in W.commit_orders(wl):
            g.round(xd, yd, order)
            o.round(X, y, order)
            loss, _, _ = g.evaluate(xe, ye)
            ref = evaluate(unflat_params(o.central_flat(), dims), X[:1024], y[:1024])[0].mean()
            assert abs(loss - ref) <= 1e-3 * max(1.0, abs(ref)), (normalize, len(losses), loss, ref)
            losses.append(loss)
        g.close()
        traj[normalize] = np.array(losses)
    agn_l, acc_l = traj[True], traj[False]
    assert np.all(np.diff(agn_l) < 0), agn_l
    assert not np.all(np.diff(acc_l) < 0), acc_l
    assert acc_l[-1] > 1.5 * agn_l[-1] and acc_l.mean() > 1.5 * agn_l.mean(), (agn_l, acc_l)
