"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: finite
differences, closed forms, a hand computation, an independent textbook SGD
loop driven by torch autograd, library routines (torch, scipy), published
generator test vectors, brute force, and the queueing invariants of the
parameter server.  A plausible mistake in the oracle (a dropped term, a
wrong sign or index, a transposed operand, a missing normalization, a
wrong commit/pull order) fails at least one of them.
"""
import math
import os

import numpy as np
import pytest
import scipy.special
import scipy.stats

from oracle import agn_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand_params(dims, rng, dtype=np.float64, scale=0.7):
    return [(rng.standard_normal((dims[l + 1], dims[l])).astype(dtype) * scale,
             rng.standard_normal(dims[l + 1]).astype(dtype) * 0.3)
            for l in range(len(dims) - 1)]


def f64prec():
    return O._Prec(np.float64, False)


# --------------------------------------------------------------------------
# P1: finite differences on tiny MLPs (the gradient term of Eq. 1)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("dims", [(5, 4, 3), (6, 3), (4, 5, 4, 3)])
def test_p1_finite_differences(dims):
    rng = np.random.default_rng(7)
    params = rand_params(dims, rng)
    m = 3
    xb = rng.standard_normal((m, dims[0]))
    yb = rng.integers(0, dims[-1], size=m)
    prec = f64prec()
    _, grads = O.loss_and_grads(params, xb, yb, prec)
    h = 1e-6

    def loss_at(ps):
        return O.loss_and_grads(ps, xb, yb, prec)[0]

    for l in range(len(params)):
        for which in (0, 1):
            base = params[l][which]
            num = np.zeros_like(base)
            for idx in np.ndindex(base.shape):
                for sgn in (+1, -1):
                    ps = [(W.copy(), b.copy()) for W, b in params]
                    ps[l][which][idx] += sgn * h
                    num[idx] += sgn * loss_at(ps) / (2 * h)
            ana = grads[l][which]
            err = np.max(np.abs(num - ana)) / max(np.max(np.abs(ana)), 1e-12)
            assert err < 1e-6, (l, which, err)


def test_loss_at_zero_weights_is_log_c():
    """Uniform logits give a cross-entropy of ln C exactly."""
    dims = (7, 5)
    params = [(np.zeros((5, 7)), np.zeros(5))]
    xb = np.random.default_rng(1).standard_normal((4, 7))
    loss, _ = O.loss_and_grads(params, xb, np.array([0, 1, 4, 2]), f64prec())
    assert abs(loss - math.log(5)) < 1e-15


def test_loss_matches_torch_cross_entropy():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(3)
    dims = (6, 9, 4)
    params = rand_params(dims, rng)
    xb = rng.standard_normal((8, 6))
    yb = rng.integers(0, 4, 8)
    loss, _ = O.loss_and_grads(params, xb, yb, f64prec())
    x = torch.tensor(xb)
    h = torch.relu(x @ torch.tensor(params[0][0]).T + torch.tensor(params[0][1]))
    z = h @ torch.tensor(params[1][0]).T + torch.tensor(params[1][1])
    ref = torch.nn.functional.cross_entropy(z, torch.tensor(yb)).item()
    assert abs(loss - ref) < 1e-13


# --------------------------------------------------------------------------
# P8: softmax regression (one layer) has a closed-form gradient
# --------------------------------------------------------------------------
def test_p8_softmax_regression_closed_form():
    rng = np.random.default_rng(11)
    d, C, m = 13, 6, 17
    W = rng.standard_normal((C, d))
    b = rng.standard_normal(C)
    X = rng.standard_normal((m, d))
    y = rng.integers(0, C, m)
    _, grads = O.loss_and_grads([(W, b)], X, y, f64prec())
    P = scipy.special.softmax(X @ W.T + b, axis=1)
    Y = np.eye(C)[y]
    np.testing.assert_allclose(grads[0][0], (P - Y).T @ X / m, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(grads[0][1], (P - Y).sum(0) / m, rtol=1e-12, atol=1e-14)


# --------------------------------------------------------------------------
# Mini-batch indices: brute-force cursor walk over each contiguous shard
# --------------------------------------------------------------------------
@pytest.mark.parametrize("N,n,m,steps", [(4096, 2, 32, 70), (60000, 8, 128, 40), (103, 4, 7, 19),
                                         (50, 5, 13, 9)])
def test_batch_indices_brute_force(N, n, m, steps):
    S = N // n
    for k in range(n):
        cursor = 0
        for t in range(steps):
            rows = []
            for _ in range(m):
                rows.append(k * S + cursor)
                cursor += 1
                if cursor == S:
                    cursor = 0
            got = O.batch_indices(k, t, m, S)
            assert got.dtype == np.int64
            assert list(got) == rows
            assert got.min() >= k * S and got.max() < (k + 1) * S


# --------------------------------------------------------------------------
# Generator and initialisation
# --------------------------------------------------------------------------
def test_splitmix64_published_vector():
    vals = [int(l) for l in open(os.path.join(GOLDEN, "splitmix64_seed1234567.txt"))
            if l.strip() and not l.startswith("#")]
    got = [int(v) for v in O.splitmix64(1234567, 0, 5)]
    assert got == vals
    # an offset window of the same stream agrees with the full stream
    assert [int(v) for v in O.splitmix64(1234567, 2, 3)] == vals[2:]


def test_he_normal_statistics():
    dims = (784, 1000, 10)
    params = O.he_normal_init(dims, seed=20171002)
    for l, (W, b) in enumerate(params):
        assert W.dtype == np.float32 and W.shape == (dims[l + 1], dims[l])
        assert np.all(b == 0)
        std = math.sqrt(2.0 / dims[l])
        z = W.astype(np.float64).ravel() / std
        nz = z.size
        assert abs(z.mean()) < 5 / math.sqrt(nz)
        assert abs(z.var() - 1) < 6 * math.sqrt(2 / nz)
        assert scipy.stats.kstest(z, "norm").pvalue > 1e-4
    # the two layers draw from disjoint parts of the stream: no repeated values
    assert not np.intersect1d(params[0][0].ravel()[:5000], params[1][0].ravel()).size


def test_he_normal_seed_dependence():
    a = O.he_normal_init((20, 5, 3), seed=1)
    b = O.he_normal_init((20, 5, 3), seed=1)
    c = O.he_normal_init((20, 5, 3), seed=2)
    assert all(np.array_equal(x[0], y[0]) for x, y in zip(a, b))
    assert not np.array_equal(a[0][0], c[0][0])


# --------------------------------------------------------------------------
# bf16 rounding: ties-to-even cases by hand, then torch's conversion
# --------------------------------------------------------------------------
def test_bf16_round_hand_cases():
    one = 1.0
    cases = {
        one: one,
        one + 2 ** -8: one,                       # halfway, round to even (down)
        one + 3 * 2 ** -8: one + 2 ** -6,         # halfway, round to even (up)
        one + 2 ** -8 + 2 ** -20: one + 2 ** -7,  # above halfway
        -(one + 2 ** -8 + 2 ** -20): -(one + 2 ** -7),
        0.0: 0.0,
    }
    x = np.array(list(cases.keys()), dtype=np.float32)
    np.testing.assert_array_equal(O.bf16_round(x), np.array(list(cases.values()), np.float32))


def test_bf16_round_matches_torch():
    torch = pytest.importorskip("torch")
    x = np.random.default_rng(5).standard_normal(100000).astype(np.float32) * 3
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(O.bf16_round(x), ref)


# --------------------------------------------------------------------------
# Helpers for the round-level pins
# --------------------------------------------------------------------------
def make_xy(N, d0, C, seed):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((N, d0)).astype(np.float32)
    y = rng.integers(0, C, N).astype(np.int32)
    return X, y


# --------------------------------------------------------------------------
# P2: lambda = 1, n = 1 is plain mini-batch SGD (footnote in Section 2:
# lambda = 1 generalises to DOWNPOUR; one worker has no asynchrony)
# --------------------------------------------------------------------------
def test_p2_lambda1_n1_is_textbook_sgd():
    torch = pytest.importorskip("torch")
    dims, m, eta, R, N = (10, 8, 6, 4), 5, 0.2, 6, 23
    X, y = make_xy(N, dims[0], dims[-1], 21)
    orc = O.AGNOracle(dims, n=1, lam=1, eta=eta, m=m, seed=99, dtype=np.float64)
    init = [(W.copy(), b.copy()) for W, b in orc.central]
    for r in range(R):
        orc.round(X, y, [0])

    # textbook loop: torch modules, autograd, optim.SGD, a plain cyclic cursor
    layers = []
    for W, b in init:
        lin = torch.nn.Linear(W.shape[1], W.shape[0]).double()
        with torch.no_grad():
            lin.weight.copy_(torch.from_numpy(W))
            lin.bias.copy_(torch.from_numpy(b))
        layers.append(lin)
    opt = torch.optim.SGD([p for lin in layers for p in lin.parameters()], lr=eta)
    cursor = 0
    for step in range(R):
        rows = [(cursor + j) % N for j in range(m)]
        cursor = (cursor + m) % N
        h = torch.from_numpy(X[rows].astype(np.float64))
        for i, lin in enumerate(layers):
            h = lin(h)
            if i < len(layers) - 1:
                h = torch.relu(h)
        loss = torch.nn.functional.cross_entropy(h, torch.from_numpy(y[rows]).long())
        opt.zero_grad()
        loss.backward()
        opt.step()
    for (W, b), lin in zip(orc.central, layers):
        np.testing.assert_allclose(W, lin.weight.detach().numpy(), rtol=0, atol=1e-13)
        np.testing.assert_allclose(b, lin.bias.detach().numpy(), rtol=0, atol=1e-13)


# --------------------------------------------------------------------------
# P3: the committed delta equals the worker's displacement divided by lambda
# (Algorithm 1 adds the same g to a and to theta, then divides a by lambda)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("dtype,tol", [(np.float64, 1e-12), (np.float32, 2e-5)])
def test_p3_displacement(dtype, tol):
    dims, n, lam, m = (12, 9, 5), 3, 6, 4
    X, y = make_xy(60, dims[0], dims[-1], 5)
    orc = O.AGNOracle(dims, n=n, lam=lam, eta=0.3, m=m, seed=3, dtype=dtype)
    for r in range(2):
        start = [orc.worker_flat(k).astype(np.float64) for k in range(n)]
        orc.round(X, y, np.random.default_rng(r).permutation(n))
        for k in range(n):
            a = O.flat_params(orc.last_deltas[k]).astype(np.float64)
            disp = (O.flat_params(orc.last_finals[k]).astype(np.float64) - start[k]) / lam
            assert np.max(np.abs(a - disp)) <= tol * np.max(np.abs(disp))
            assert np.max(np.abs(disp)) > 0


# --------------------------------------------------------------------------
# P4: sequential commit order, the central variable is the running sum of
# the deltas (Eq. 2) and each worker pulls the prefix sum after its commit
# --------------------------------------------------------------------------
def test_p4_hand_computed_two_workers():
    """Softmax regression with one input (x = 1), two classes, one sample
    per worker (label 0), zero init, eta = 0.1.  By hand: at theta = 0 the
    gradient is (-1/2, +1/2) for both W and b; at W = b = (c, -c) the logits
    are (2c, -2c) and the gradient is (sigma(4c) - 1, 1 - sigma(4c))."""
    eta = 0.1
    X = np.ones((2, 1), dtype=np.float64)
    y = np.zeros(2, dtype=np.int32)
    init = [(np.zeros((2, 1)), np.zeros(2))]
    sig = lambda v: 1.0 / (1.0 + math.exp(-v))

    # lambda = 1: both workers commit (0.05, -0.05)
    orc = O.AGNOracle((1, 2), n=2, lam=1, eta=eta, m=1, dtype=np.float64, init=init)
    orc.round(X, y, [0, 1])
    np.testing.assert_allclose(orc.worker_flat(0), [0.05, -0.05, 0.05, -0.05], atol=1e-16)
    np.testing.assert_allclose(orc.central_flat(), [0.1, -0.1, 0.1, -0.1], atol=1e-16)
    np.testing.assert_allclose(orc.worker_flat(1), orc.central_flat(), atol=0)

    # lambda = 2: second local step starts at c = 0.05
    orc = O.AGNOracle((1, 2), n=2, lam=2, eta=eta, m=1, dtype=np.float64, init=init)
    orc.round(X, y, [1, 0])
    d = (0.05 + eta * (1 - sig(4 * 0.05))) / 2
    np.testing.assert_allclose(orc.worker_flat(1), [d, -d, d, -d], rtol=1e-14)
    np.testing.assert_allclose(orc.central_flat(), [2 * d, -2 * d, 2 * d, -2 * d], rtol=1e-14)


def test_p4_sequential_prefix_sums_fp32_exact():
    dims, n, lam, m = (9, 7, 4), 5, 3, 6
    X, y = make_xy(90, dims[0], dims[-1], 8)
    orc = O.AGNOracle(dims, n=n, lam=lam, eta=0.1, m=m, seed=4)
    for r in range(3):
        c = orc.central_flat().copy()
        orc.round(X, y, list(range(n)))
        for k in range(n):
            c = (c + O.flat_params(orc.last_deltas[k])).astype(np.float32)  # left to right in fp32
            np.testing.assert_array_equal(orc.worker_flat(k), c)
        np.testing.assert_array_equal(orc.central_flat(), c)


# --------------------------------------------------------------------------
# P5: staleness of the FIFO queue (E[tau] = n - 1, Section 1)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("n", [2, 8, 20])
def test_p5_staleness(n):
    dims = (3, 2)
    X, y = make_xy(4 * n, 3, 2, 1)
    seq = O.AGNOracle(dims, n=n, lam=1, eta=0.0, m=1, seed=0)
    rnd = O.AGNOracle(dims, n=n, lam=1, eta=0.0, m=1, seed=0)
    rng = np.random.default_rng(n)
    orders = [rng.permutation(n) for _ in range(12)]
    for r in range(12):
        seq.round(X, y, range(n))
        rnd.round(X, y, orders[r])
    # round 1: the j-th commit has seen j earlier commits since the common pull
    assert seq.staleness[0] == list(range(n))
    assert rnd.staleness[0] == list(range(n))
    for r in range(1, 12):
        assert seq.staleness[r] == [n - 1] * n
        s = rnd.staleness[r]
        assert min(s) >= 0 and max(s) <= 2 * n - 2
        assert sum(s) == n * (n - 1)        # mean exactly n - 1 every round
        # closed form: tau = n - 1 + (position now) - (position last round)
        prev = {int(k): j for j, k in enumerate(orders[r - 1])}
        assert s == [n - 1 + j - prev[int(k)] for j, k in enumerate(orders[r])]


# --------------------------------------------------------------------------
# P6: eta = 0 is a fixed point
# --------------------------------------------------------------------------
def test_p6_eta_zero_fixed_point():
    dims, n = (11, 6, 3), 3
    X, y = make_xy(60, dims[0], dims[-1], 2)
    orc = O.AGNOracle(dims, n=n, lam=4, eta=0.0, m=5, seed=17)
    c0 = orc.central_flat().copy()
    orc.round(X, y, [2, 0, 1])
    orc.round(X, y, [0, 2, 1])
    np.testing.assert_array_equal(orc.central_flat(), c0)
    for k in range(n):
        np.testing.assert_array_equal(orc.worker_flat(k), c0)
    # the reported loss is the mean of the mini-batch losses at theta_0
    S = 60 // n
    ref = [np.mean([O.loss_and_grads(orc.central, X[O.batch_indices(k, 4 + i, 5, S)],
                                     y[O.batch_indices(k, 4 + i, 5, S)], orc.prec)[0]
                    for i in range(4)]) for k in range(n)]
    np.testing.assert_allclose(orc.last_loss, np.array(ref, np.float32), rtol=1e-6)


# --------------------------------------------------------------------------
# P7: identical shards give identical deltas; round 1 adds n equal deltas
# --------------------------------------------------------------------------
def test_p7_identical_shards():
    dims, n, lam, m = (8, 6, 3), 4, 3, 5
    Xs, ys = make_xy(15, dims[0], dims[-1], 9)
    X = np.concatenate([Xs] * n)
    y = np.concatenate([ys] * n)
    orc = O.AGNOracle(dims, n=n, lam=lam, eta=0.2, m=m, seed=5, dtype=np.float64)
    c0 = orc.central_flat().copy()
    orc.round(X, y, [3, 1, 0, 2])
    d = [O.flat_params(a) for a in orc.last_deltas]
    for k in range(1, n):
        np.testing.assert_array_equal(d[k], d[0])
    np.testing.assert_allclose(orc.central_flat(), c0 + n * d[0], rtol=1e-13, atol=1e-15)


# --------------------------------------------------------------------------
# P9: in round 1 every order gives the same central variable (up to
# rounding) but different pulled copies
# --------------------------------------------------------------------------
def test_p9_round1_order_invariance():
    dims, n = (10, 7, 4), 4
    X, y = make_xy(80, dims[0], dims[-1], 6)
    res = []
    for order in ([0, 1, 2, 3], [3, 2, 1, 0], [1, 3, 0, 2]):
        orc = O.AGNOracle(dims, n=n, lam=3, eta=0.2, m=6, seed=8, dtype=np.float64)
        orc.round(X, y, order)
        res.append((orc.central_flat(), [orc.worker_flat(k) for k in range(n)]))
    for c, w in res[1:]:
        np.testing.assert_allclose(c, res[0][0], rtol=1e-13, atol=1e-15)
        assert not np.allclose(w[0], res[0][1][0])
    # and later rounds do depend on the order (stale starting points differ)
    a = O.AGNOracle(dims, n=n, lam=3, eta=0.2, m=6, seed=8, dtype=np.float64)
    b = O.AGNOracle(dims, n=n, lam=3, eta=0.2, m=6, seed=8, dtype=np.float64)
    for order_a, order_b in (([0, 1, 2, 3], [3, 2, 1, 0]), ([0, 1, 2, 3], [0, 1, 2, 3])):
        a.round(X, y, order_a)
        b.round(X, y, order_b)
    assert np.max(np.abs(a.central_flat() - b.central_flat())) > 1e-8


# --------------------------------------------------------------------------
# lambda -> large (Section 3, Eq. 3): on a convex problem the normalized
# delta shrinks as lambda grows
# --------------------------------------------------------------------------
def test_normalized_delta_shrinks_with_lambda():
    X, y = make_xy(40, 6, 3, 12)
    norms = []
    for lam in (1, 10, 100, 1000):
        orc = O.AGNOracle((6, 3), n=1, lam=lam, eta=0.5, m=40, seed=2, dtype=np.float64)
        orc.round(X, y, [0])
        norms.append(np.linalg.norm(O.flat_params(orc.last_deltas[0])))
    assert norms[0] > norms[1] > norms[2] > norms[3]
    assert norms[3] < 0.05 * norms[0]


# --------------------------------------------------------------------------
# bf16 mode: within bf16 rounding of the float32 computation
# --------------------------------------------------------------------------
def test_bf16_mode_close_to_fp32():
    rng = np.random.default_rng(4)
    dims = (64, 48, 32, 10)
    params = [(W.astype(np.float32), b.astype(np.float32))
              for W, b in rand_params(dims, rng, scale=0.15)]
    xb = O.bf16_round(rng.standard_normal((16, 64)).astype(np.float32))
    yb = rng.integers(0, 10, 16)
    l32, g32 = O.loss_and_grads(params, xb, yb, O._Prec(np.float32, False))
    l16, g16 = O.loss_and_grads(params, xb, yb, O._Prec(np.float32, True))
    assert abs(l32 - l16) < 2e-2 * abs(l32)
    for (a, b_), (c, d) in zip(g32, g16):
        assert np.max(np.abs(a - c)) <= 3e-2 * np.max(np.abs(a))
        assert np.max(np.abs(b_ - d)) <= 3e-2 * np.max(np.abs(b_))
        assert not np.array_equal(a, c)     # the rounding is actually applied


def test_bad_order_rejected():
    orc = O.AGNOracle((3, 2), n=3, lam=1, eta=0.1, m=1)
    X, y = make_xy(9, 3, 2, 0)
    with pytest.raises(ValueError):
        orc.round(X, y, [0, 0, 1])


# --------------------------------------------------------------------------
# Without the normalization step (Section 2: DOWNPOUR with local
# exploration; Section 3 footnote to Eq. 1: lambda = 1 is DOWNPOUR)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("dtype,tol", [(np.float64, 1e-12), (np.float32, 2e-6)])
def test_accumulated_delta_is_displacement(dtype, tol):
    """Algorithm 1 adds every local step g to both a and theta, so the
    un-normalized commit is the displacement theta_lambda - theta_0."""
    dims, n, lam, m = (12, 9, 5), 3, 6, 4
    X, y = make_xy(60, dims[0], dims[-1], 5)
    orc = O.AGNOracle(dims, n=n, lam=lam, eta=0.3, m=m, seed=3, dtype=dtype, normalize=False)
    for r in range(2):
        start = [orc.worker_flat(k).astype(np.float64) for k in range(n)]
        orc.round(X, y, np.random.default_rng(r).permutation(n))
        for k in range(n):
            a = O.flat_params(orc.last_deltas[k]).astype(np.float64)
            disp = O.flat_params(orc.last_finals[k]).astype(np.float64) - start[k]
            assert np.max(np.abs(a - disp)) <= tol * np.max(np.abs(disp))
            assert np.max(np.abs(disp)) > 0


def test_accumulated_is_lambda_times_normalized():
    """From the same start the two rules commit a and a / lambda (fp64)."""
    dims, n, lam, m = (12, 9, 5), 3, 6, 4
    X, y = make_xy(60, dims[0], dims[-1], 5)
    a = O.AGNOracle(dims, n=n, lam=lam, eta=0.3, m=m, seed=3, dtype=np.float64, normalize=False)
    b = O.AGNOracle(dims, n=n, lam=lam, eta=0.3, m=m, seed=3, dtype=np.float64)
    a.round(X, y, [2, 0, 1])
    b.round(X, y, [2, 0, 1])
    for k in range(n):
        da = O.flat_params(a.last_deltas[k])
        db = O.flat_params(b.last_deltas[k])
        assert np.max(np.abs(da - lam * db)) <= 1e-13 * np.max(np.abs(da))
    # round 1: every worker starts from the same central variable, so the
    # central variable moves by the sum of the deltas under either rule
    c0 = O.flat_params(O.he_normal_init(dims, 3, dtype=np.float64))
    np.testing.assert_allclose(a.central_flat() - c0, lam * (b.central_flat() - c0), rtol=1e-10, atol=1e-14)


def test_lambda1_rules_coincide():
    """lambda = 1: normalized and accumulated commits are the same rule."""
    dims, n, m = (12, 9, 5), 4, 4
    X, y = make_xy(80, dims[0], dims[-1], 6)
    a = O.AGNOracle(dims, n=n, lam=1, eta=0.2, m=m, seed=8, normalize=False)
    b = O.AGNOracle(dims, n=n, lam=1, eta=0.2, m=m, seed=8)
    rng = np.random.default_rng(1)
    for r in range(3):
        order = rng.permutation(n)
        a.round(X, y, order)
        b.round(X, y, order)
    assert np.array_equal(a.central_flat(), b.central_flat())


def test_accumulated_commits_fail_to_converge_where_agn_does():
    """The paper's motivating observation (Section 2, the accumulated-
    gradient DOWNPOUR divergence figure): with the same workers, learning
    rate and local steps, committing accumulated updates makes the central
    variable oscillate at a high loss while AGN's loss falls every round.
    Synthetic stand-in: 20-16-4 MLP, n = 8, lambda = 10, eta = 0.1, m = 16."""
    import workloads as W
    dims, n, lam, eta, m, R = (20, 16, 4), 8, 10, 0.1, 16, 6
    wl = W.small_workload("dv", dims, n, lam, m, eta, R, 4096, data="gauss_linear", order="permutation")
    X, y = W.make_data(wl)
    prec = O._Prec(np.float32, False)
    traj = {}
    for normalize in (True, False):
        o = O.AGNOracle(dims, n, lam, eta, m, seed=wl.seed, normalize=normalize)
        losses = []
        for order in W.commit_orders(wl):
            o.round(X, y, order)
            losses.append(O.loss_and_grads(o.central, X[:1024], y[:1024], prec)[0])
        traj[normalize] = np.array(losses)
    agn, acc = traj[True], traj[False]
    assert np.all(np.diff(agn) < 0), agn
    assert not np.all(np.diff(acc) < 0), acc
    assert acc[-1] > 1.5 * agn[-1] and acc.mean() > 1.5 * agn.mean(), (agn, acc)


# --------------------------------------------------------------------------
# Adam as the local rule (Algorithm 1's gradient line; Kingma & Ba 2015).
# Reading: the worker's moment estimates and step counter run on across
# pulls, as Algorithm 1's t does.
# --------------------------------------------------------------------------
ADAM = (0.9, 0.999, 1e-8)


def torch_adam_trajectory(init, X, y, m, eta, steps, betas, eps):
    """Textbook loop: torch modules, autograd, one torch.optim.Adam, a plain
    cyclic cursor over the rows (one worker, shard = all N rows)."""
    import torch
    N = X.shape[0]
    layers = []
    for W, b in init:
        lin = torch.nn.Linear(W.shape[1], W.shape[0]).double()
        with torch.no_grad():
            lin.weight.copy_(torch.from_numpy(W))
            lin.bias.copy_(torch.from_numpy(b))
        layers.append(lin)
    opt = torch.optim.Adam([p for lin in layers for p in lin.parameters()], lr=eta, betas=betas, eps=eps)
    cursor = 0
    for _ in range(steps):
        rows = [(cursor + j) % N for j in range(m)]
        cursor = (cursor + m) % N
        h = torch.from_numpy(X[rows].astype(np.float64))
        for i, lin in enumerate(layers):
            h = lin(h)
            if i < len(layers) - 1:
                h = torch.relu(h)
        loss = torch.nn.functional.cross_entropy(h, torch.from_numpy(y[rows]).long())
        opt.zero_grad()
        loss.backward()
        opt.step()
    return [(lin.weight.detach().numpy(), lin.bias.detach().numpy()) for lin in layers]


@pytest.mark.parametrize("lam,normalize", [(1, True), (3, False)])
def test_adam_one_worker_is_textbook_adam(lam, normalize):
    """n = 1: with lambda = 1 (or without the normalization step) the worker
    pulls back its own parameters, so R rounds are lambda*R steps of plain
    Adam with one optimizer state, against torch.optim.Adam (fp64)."""
    pytest.importorskip("torch")
    dims, m, eta, R, N = (10, 8, 6, 4), 5, 0.01, 4, 23
    X, y = make_xy(N, dims[0], dims[-1], 21)
    orc = O.AGNOracle(dims, n=1, lam=lam, eta=eta, m=m, seed=99, dtype=np.float64, normalize=normalize,
                      adam=ADAM)
    init = [(W.copy(), b.copy()) for W, b in orc.central]
    for r in range(R):
        orc.round(X, y, [0])
    ref = torch_adam_trajectory(init, X, y, m, eta, lam * R, ADAM[:2], ADAM[2])
    for (W, b), (Wt, bt) in zip(orc.central, ref):
        np.testing.assert_allclose(W, Wt, rtol=0, atol=1e-12)
        np.testing.assert_allclose(b, bt, rtol=0, atol=1e-12)


def test_adam_first_step_closed_form():
    """From zero moments the first Adam step is -eta * g / (|g| + eps)
    (the bias corrections cancel (1 - beta) exactly)."""
    dims, m, eta, N = (10, 8, 6, 4), 5, 0.01, 23
    X, y = make_xy(N, dims[0], dims[-1], 22)
    orc = O.AGNOracle(dims, n=1, lam=1, eta=eta, m=m, seed=5, dtype=np.float64, adam=ADAM)
    theta0 = [(W.copy(), b.copy()) for W, b in orc.central]
    idx = O.batch_indices(0, 0, m, N)
    _, grads = O.loss_and_grads(theta0, X[idx], y[idx], O._Prec(np.float64, False))
    orc.round(X, y, [0])
    for (W0, b0), (gW, gb), (W1, b1) in zip(theta0, grads, orc.central):
        np.testing.assert_allclose(W1 - W0, -eta * gW / (np.abs(gW) + ADAM[2]), rtol=1e-12, atol=1e-16)
        np.testing.assert_allclose(b1 - b0, -eta * gb / (np.abs(gb) + ADAM[2]), rtol=1e-12, atol=1e-16)


def test_adam_moments_persist_across_pulls():
    """Two workers, sequential commits: round 2 must use each worker's own
    moments from round 1 (a fresh optimizer each round gives another
    result)."""
    dims, m, eta, N = (10, 8, 6, 4), 5, 0.01, 40
    X, y = make_xy(N, dims[0], dims[-1], 23)
    a = O.AGNOracle(dims, n=2, lam=2, eta=eta, m=m, seed=5, dtype=np.float64, adam=ADAM)
    a.round(X, y, [0, 1])
    mom = [[tuple(x.copy() for x in t) for t in w] for w in a.moments]
    assert all(np.max(np.abs(t[0])) > 0 for w in mom for t in w)
    a.round(X, y, [1, 0])
    # the same round 2 from zeroed moments differs
    b = O.AGNOracle(dims, n=2, lam=2, eta=eta, m=m, seed=5, dtype=np.float64, adam=ADAM)
    b.round(X, y, [0, 1])
    b.moments = [[tuple(np.zeros_like(x) for x in t) for t in w] for w in b.moments]
    b.round(X, y, [1, 0])
    assert np.max(np.abs(a.central_flat() - b.central_flat())) > 1e-6


# --------------------------------------------------------------------------
# Staleness-scaled commits (Section 4's DynSGD rule, read as 1 / (tau + 1))
# --------------------------------------------------------------------------
def test_staleness_scaling_one_worker_is_plain():
    """n = 1: every commit has staleness 0, so the scale is exactly 1."""
    dims = (12, 9, 5)
    X, y = make_xy(40, dims[0], dims[-1], 3)
    a = O.AGNOracle(dims, n=1, lam=3, eta=0.2, m=4, seed=5, staleness_scaled=True)
    b = O.AGNOracle(dims, n=1, lam=3, eta=0.2, m=4, seed=5)
    for r in range(3):
        a.round(X, y, [0])
        b.round(X, y, [0])
    assert np.array_equal(a.central_flat(), b.central_flat())


@pytest.mark.parametrize("n", [2, 4, 7])
def test_staleness_scaling_harmonic_first_round(n):
    """Every worker holds the same rows, so in round 1 (one common start)
    all n deltas equal the one-worker delta D, and the j-th commit has
    staleness j: the central variable moves by sum_j D / (j + 1) = H_n D
    (harmonic number; scales rounded to float32, float64 storage)."""
    dims, lam, m, S = (10, 8, 4), 3, 5, 23
    X1, y1 = make_xy(S, dims[0], dims[-1], 9)
    X, y = np.tile(X1, (n, 1)), np.tile(y1, n)
    one = O.AGNOracle(dims, n=1, lam=lam, eta=0.25, m=m, seed=2, dtype=np.float64)
    one.round(X1, y1, [0])
    c0 = O.flat_params(O.he_normal_init(dims, 2, dtype=np.float64))
    D = one.central_flat() - c0
    o = O.AGNOracle(dims, n=n, lam=lam, eta=0.25, m=m, seed=2, dtype=np.float64, staleness_scaled=True)
    o.round(X, y, np.random.default_rng(n).permutation(n))
    H = sum(1.0 / (j + 1) for j in range(n))
    np.testing.assert_allclose(o.central_flat() - c0, H * D, rtol=1e-7, atol=1e-15)


def test_staleness_scaling_uses_staleness_not_position():
    """n = 2, orders [0, 1] then [1, 0]: in round 2 worker 1 commits first
    with staleness 0 (it pulled the latest central variable) and worker 0
    second with staleness 2 (it pulled before worker 1's round-1 commit), so
    the scales are 1 and 1/3, not the positions' 1 and 1/2."""
    dims = (10, 8, 4)
    X, y = make_xy(40, dims[0], dims[-1], 4)
    o = O.AGNOracle(dims, n=2, lam=2, eta=0.25, m=5, seed=6, dtype=np.float64, staleness_scaled=True)
    o.round(X, y, [0, 1])
    c1 = o.central_flat().copy()
    o.round(X, y, [1, 0])
    assert o.staleness == [[0, 1], [0, 2]]
    d0 = O.flat_params(o.last_deltas[0])
    d1 = O.flat_params(o.last_deltas[1])
    want = c1 + d1 + np.float32(1.0 / 3.0) * d0
    np.testing.assert_allclose(o.central_flat(), want, rtol=1e-14, atol=1e-15)
    assert np.max(np.abs(o.central_flat() - (c1 + d1 + 0.5 * d0))) > 1e-6


def test_near_zero_units_flags_pre_activations_at_rounding_distance():
    """The parity tests' flip diagnostic: a hidden pre-activation that is
    zero up to rounding is flagged, with its layer and unit; one that is far
    from zero is not, whatever the magnitude of its terms."""
    prec = O._Prec(np.float64, False)
    W0 = np.array([[1.0, -1.0], [3.0, 1.0], [1e-3, 0.0]])
    b0 = np.zeros(3)
    W1 = np.array([[1.0, 1.0, -1.0], [0.5, 0.0, 1.0]])
    b1 = np.array([0.0, -2.0])
    W2 = np.ones((2, 2))
    b2 = np.zeros(2)
    x = np.array([[0.75, 0.75], [1.0, 0.0]])
    # layer 1: unit 0 is 0.75 - 0.75 = 0 for row 0; units 1 and 2 stay clear
    # layer 2 (from relu(layer 1)): row 0 -> (3 - 0.00075, 1.5 + 0.00075 - 2),
    # row 1 -> (1 + 3 - 0.001, 0.5 + 0.001 - 2): no zero
    near = O.near_zero_units([(W0, b0), (W1, b1), (W2, b2)], x, prec)
    assert [u.tolist() for u in near] == [[0], []]
    near = O.near_zero_units([(W0, b0 + 1e-3), (W1, b1), (W2, b2)], x, prec)
    assert [u.tolist() for u in near] == [[], []]
