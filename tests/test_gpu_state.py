"""Checkpoint and resume (agn_get_state / agn_set_state).

Algorithm 1 carries from one round to the next only the central variable,
each worker's last pulled copy, the workers' step counter (which picks the
mini-batches) and, for the staleness of each commit, how many commits each
worker has seen; with Adam also the workers' moment estimates.  A context
restored from a state taken after round r must therefore continue exactly
like the original: every round after the restore is compared bit for bit
(central variable, every pulled copy, the loss report and the staleness),
which also holds the kernels to run-to-run determinism.  The restored
context is created with another seed, so nothing of its own initial state
can leak into the comparison.  The state's documented layout (header, pull
counters, losses, packed vectors) is read back against agn_central,
agn_worker_params and agn_loss, and a state from another configuration, of
another size or with a broken magic is refused with the context unchanged.
"""
import numpy as np
import pytest

import workloads as W
from tests.helpers import to_device, require_gpu

pytestmark = pytest.mark.gpu

ADAM = (0.9, 0.999, 1e-8)

CASES = [
    # name, dims, n, lam, m, eta, N, data, dtype, options
    ("sgd_fp32", (100, 70, 60, 10), 4, 3, 20, 0.05, 400, "gauss_linear", "fp32", {}),
    ("accumulated_staleness_scaled", (100, 70, 60, 10), 5, 2, 20, 0.02, 500, "gauss_linear", "fp32",
     {"normalize": False, "staleness_scaled": True}),
    ("adam_fp32", (64, 48, 10), 3, 2, 16, 0.002, 300, "gauss_linear", "fp32", {"adam": ADAM}),
    ("bf16", (136, 264, 200, 10), 3, 3, 100, 0.05, 650, "sparse_teacher2", "bf16", {}),
    # 64 workers x 16 strips: both strip schedules of the float32 path
    ("strips", (96, 1000, 968, 12), 64, 2, 128, 0.02, 64 * 300, "sparse_teacher2", "fp32", {}),
]

HEADER = np.dtype([("magic", "S8"), ("version", "<i4"), ("L", "<i4"), ("m", "<i4"), ("n", "<i4"),
                   ("lam", "<i4"), ("dtype", "<i4"), ("optimizer", "<i4"), ("normalize", "<i4"),
                   ("staleness_scaling", "<i4"), ("dims", "<i4", (17,)), ("eta", "<f4"), ("beta1", "<f4"),
                   ("beta2", "<f4"), ("adam_eps", "<f4"), ("P", "<i8"), ("rounds", "<i8"), ("commits", "<i8"),
                   ("num_samples", "<i8"), ("last_committer", "<i8")], align=True)


def _context(agn, wl, opts, seed):
    return agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=seed, dtype=wl.dtype,
                   normalize=opts.get("normalize", True), adam=opts.get("adam"),
                   staleness_scaled=opts.get("staleness_scaled", False))


def _snapshot(g, n):
    """Everything a round leaves behind that the ABI reports (host copies)."""
    return {"central": g.central().cpu().numpy(),
            "workers": [g.worker_params(k).cpu().numpy() for k in range(n)],
            "loss": g.loss().cpu().numpy(),
            "staleness": np.asarray(g.staleness())}


def _assert_same(a, b, what):
    for key in ("central", "loss", "staleness"):
        assert np.array_equal(a[key], b[key]), f"{what}: {key} differs"
    for k, (x, y) in enumerate(zip(a["workers"], b["workers"])):
        assert np.array_equal(x, y), f"{what}: pulled copy of worker {k} differs"


@pytest.mark.timeout(600)
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_resume_continues_bit_for_bit(case):
    require_gpu()
    import paper_1710_02368_amd as agn
    name, dims, n, lam, m, eta, N, data, dtype, opts = case
    wl = W.small_workload(name, dims, n, lam, m, eta, 4, N, data=data, order="permutation", dtype=dtype)
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    orders = W.commit_orders(wl)
    g = _context(agn, wl, opts, wl.seed)
    for order in orders[:2]:
        g.round(xd, yd, order)
    saved = _snapshot(g, n)
    state = g.get_state()

    # the documented layout
    P = g.P
    hdr = np.frombuffer(state[:HEADER.itemsize].tobytes(), dtype=HEADER)[0]
    assert hdr["magic"] == b"AGNSTATE" and hdr["version"] == 1
    assert (hdr["n"], hdr["lam"], hdr["m"], hdr["P"]) == (n, lam, m, P)
    assert list(hdr["dims"][:len(dims)]) == list(dims) and hdr["L"] == len(dims) - 1
    assert (hdr["rounds"], hdr["commits"], hdr["num_samples"]) == (2, 2 * n, N)
    off = HEADER.itemsize
    pulls = np.frombuffer(state[off:off + 8 * n].tobytes(), dtype="<i8")
    assert pulls.min() >= n and pulls.max() <= 2 * n  # every worker pulled in round 2
    off += 16 * n
    losses = np.frombuffer(state[off:off + 4 * n * lam * m].tobytes(), dtype="<f4").reshape(n, lam * m)
    np.testing.assert_allclose(losses.astype(np.float64).mean(axis=1), saved["loss"], rtol=1e-5)
    off += 4 * n * lam * m
    vecs = np.frombuffer(state[off:].tobytes(), dtype="<f4").reshape(-1, P)
    assert vecs.shape[0] == 1 + n * (3 if "adam" in opts else 1)
    assert np.array_equal(vecs[0], saved["central"])
    for k in range(n):
        assert np.array_equal(vecs[1 + k], saved["workers"][k])

    # the original continues ...
    after = []
    for order in orders[2:4]:
        g.round(xd, yd, order)
        after.append(_snapshot(g, n))
    g.close()

    # ... and so does a context restored from the state (another seed)
    h = _context(agn, wl, opts, wl.seed + 99)
    h.set_state(state)
    assert np.array_equal(h.central().cpu().numpy(), saved["central"])
    assert np.array_equal(h.loss().cpu().numpy(), saved["loss"])
    assert np.array_equal(np.asarray(h.staleness()), saved["staleness"])
    with pytest.raises(agn.AGNError) as ei:
        h.delta(0)
    assert ei.value.code == agn.AGN_ESTATE
    for r, order in enumerate(orders[2:4]):
        h.round(xd, yd, order)
        _assert_same(_snapshot(h, n), after[r], f"{name}: round {3 + r} after the restore")
    h.close()


def test_state_from_another_configuration_is_refused():
    require_gpu()
    import paper_1710_02368_amd as agn
    wl = W.small_workload("state_refused", (100, 70, 60, 10), 4, 3, 20, 0.05, 2, 400, order="permutation")
    X, y = W.make_data(wl)
    xd, yd = to_device(X, y)
    orders = W.commit_orders(wl)
    g = _context(agn, wl, {}, wl.seed)
    g.round(xd, yd, orders[0])
    state = g.get_state()
    h = _context(agn, wl, {}, wl.seed + 1)
    before = h.central().cpu().numpy()

    def refused(st, ctx, needle):
        with pytest.raises(agn.AGNError) as ei:
            ctx.set_state(st)
        assert ei.value.code == agn.AGN_EINVAL
        assert needle in str(ei.value)

    refused(state[:-4], h, "bytes")                       # another size
    bad = state.copy()
    bad[0] ^= 0xFF
    refused(bad, h, "magic")                              # not a state
    other_eta = agn.AGN(wl.dims, wl.n, wl.lam, 0.5, wl.m, seed=wl.seed)
    refused(state, other_eta, "eta")                      # another learning rate
    other_eta.close()
    adam = agn.AGN(wl.dims, wl.n, wl.lam, wl.eta, wl.m, seed=wl.seed, adam=ADAM)
    refused(state, adam, "bytes")                         # Adam's state is larger
    adam.close()
    bad = state.copy()
    commits = HEADER.fields["commits"][1]
    bad[commits:commits + 8] = np.frombuffer(np.int64(7).tobytes(), dtype=np.uint8)
    refused(bad, h, "counters")                           # inconsistent counters
    assert np.array_equal(h.central().cpu().numpy(), before)  # unchanged
    with pytest.raises(agn.AGNError) as ei:
        h.loss()                                          # still before its first round
    assert ei.value.code == agn.AGN_ESTATE
    h.set_state(state)                                    # the genuine state is accepted
    assert np.array_equal(h.central().cpu().numpy(), g.central().cpu().numpy())
    g.close()
    h.close()
