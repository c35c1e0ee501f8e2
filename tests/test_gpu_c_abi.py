"""The C ABI used from a plain C99 program (tests/c_abi/agn_c_round.c):
device buffers from the HIP runtime's C API, shapes, data and commit orders
as plain structs, pointers and sizes.  Its rounds must equal, bit for bit,
the same rounds driven through the Python binding in this process (one
library, deterministic kernels), and the oracle within the float32 bounds
(1e-4 after round 1, 1e-3 after the last)."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import workloads as W
from oracle import AGNOracle
from tests.helpers import rel_err, to_device, require_gpu

pytestmark = pytest.mark.gpu


def test_c_program_rounds_match_binding_and_oracle(tmp_path):
    require_gpu()
    if shutil.which("gcc") is None:
        pytest.skip("no C compiler")
    import paper_1710_02368_amd as agn
    from tests.c_abi import build as c_build
    dims, n, lam, m, eta, R, N = (100, 70, 60, 10), 4, 3, 20, 0.05, 3, 400
    wl = W.small_workload("c_abi", dims, n, lam, m, eta, R, N, data="gauss_linear", order="permutation")
    X, y = W.make_data(wl)
    orders = W.commit_orders(wl)
    inp, out = str(tmp_path / "in.bin"), str(tmp_path / "out.bin")
    with open(inp, "wb") as fh:
        fh.write(np.array([len(dims) - 1, *dims, m, n, lam], dtype="<i4").tobytes())
        fh.write(np.array([eta], dtype="<f4").tobytes())
        fh.write(np.array([wl.seed], dtype="<u8").tobytes())
        fh.write(np.array([N], dtype="<i8").tobytes())
        fh.write(np.array([R], dtype="<i4").tobytes())
        fh.write(np.ascontiguousarray(X, dtype="<f4").tobytes())
        fh.write(np.ascontiguousarray(y, dtype="<i4").tobytes())
        fh.write(np.ascontiguousarray(np.stack(orders), dtype="<i4").tobytes())
    exe = c_build.build(str(tmp_path))
    print("running the C program on", wl.name, flush=True)
    r = subprocess.run([exe, "run", inp, out], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr

    g = agn.AGN(dims, n, lam, eta, m, seed=wl.seed)
    o = AGNOracle(dims, n, lam, eta, m, seed=wl.seed)
    P = g.P
    res = np.fromfile(out, dtype="<f4")
    assert res.size == R * (P + n)
    res = res.reshape(R, P + n)
    xd, yd = to_device(X, y)
    for k, order in enumerate(orders):
        g.round(xd, yd, order)
        o.round(X, y, order)
        central, loss = res[k, :P], res[k, P:]
        assert np.array_equal(central, g.central().cpu().numpy()), f"round {k + 1}: central variable"
        assert np.array_equal(loss, g.loss().cpu().numpy()), f"round {k + 1}: losses"
        err, where = rel_err(central, o.central_flat(), dims)
        assert err <= (1e-4 if k == 0 else 1e-3), (k, where, err)
    g.close()
