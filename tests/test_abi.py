"""The C ABI: the library loads, exports every declared entry point, and
rejects bad arguments on the host before touching a GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_1710_02368_amd as agn

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "agn.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*[a-z_0-9 \*]+?\b(agn_[a-z_]+)\s*\(", text, flags=re.M)))


def test_header_declares_the_binding_functions():
    assert declared_functions() == sorted(agn.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = agn.load_library()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_exported_symbols_are_c_linkage():
    out = os.popen(f"nm -D --defined-only {agn.LIB_PATH}").read()
    for name in declared_functions():
        assert re.search(rf"\bT {name}$", out, flags=re.M), name


@pytest.mark.parametrize("kwargs,msg", [
    (dict(dims=(10, 5), batch=4, n=0, lam=1, eta=0.1), "n must be"),
    (dict(dims=(10, 5), batch=4, n=300, lam=1, eta=0.1), "n must be"),
    (dict(dims=(10, 5), batch=4, n=2, lam=0, eta=0.1), "lambda"),
    (dict(dims=(10, 5), batch=0, n=2, lam=1, eta=0.1), "batch"),
    (dict(dims=(10, 1), batch=4, n=2, lam=1, eta=0.1), "2 classes"),
    (dict(dims=(10, 0, 5), batch=4, n=2, lam=1, eta=0.1), "width"),
    (dict(dims=(10,), batch=4, n=2, lam=1, eta=0.1), "num_layers"),
    (dict(dims=(10, 5), batch=4, n=2, lam=1, eta=float("nan")), "eta"),
    (dict(dims=(10, 5), batch=4, n=2, lam=1, eta=float("inf")), "eta"),
    (dict(dims=(10, 5), batch=4, n=2, lam=1, eta=0.1, dtype=7), "dtype"),
    (dict(dims=tuple([4] * 18), batch=4, n=2, lam=1, eta=0.1), "num_layers"),
])
def test_create_rejects_bad_arguments(kwargs, msg):
    with pytest.raises(agn.AGNError) as ei:
        agn.agn_create(kwargs["dims"], kwargs["batch"], kwargs["n"], kwargs["lam"], kwargs["eta"], 1,
                       kwargs.get("dtype", 0))
    assert ei.value.code == -1
    assert msg in str(ei.value)
    assert msg in agn.agn_last_error(None)


def test_null_arguments_are_rejected():
    lib = agn.load_library()
    ctx = ctypes.c_void_p()
    assert lib.agn_create(None, 2, 1, ctypes.c_float(0.1), 1, ctypes.byref(ctx)) == -1
    assert lib.agn_num_params(None) == -1
    assert lib.agn_round(None, None, None) == -1
    assert lib.agn_central(None, None) == -1
    assert lib.agn_loss(None, None) == -1
    lib.agn_destroy(None)  # no-op
    assert isinstance(agn.agn_last_error(None), str)


def test_null_state_arguments_are_rejected():
    lib = agn.load_library()
    assert lib.agn_state_bytes(None) == -1
    assert lib.agn_get_state(None, None, 0) == -1
    assert lib.agn_set_state(None, None, 0) == -1
    assert "null context" in agn.agn_last_error(None)


def test_null_evaluate_arguments_are_rejected():
    lib = agn.load_library()
    assert lib.agn_evaluate(None, None, None, None, None) == -1
    assert lib.agn_temporal_efficiency(None, None, 0, None, None, 0, None) == -1


# --------------------------------------------------------------------------
# temporal efficiency (Eq. 4): host arithmetic in the library, checked
# against the oracle's independent implementation
# --------------------------------------------------------------------------
def _curve(rng, k, start=0.0):
    t = np.concatenate([[start], start + np.cumsum(rng.random(k - 1) + 1e-3)])
    return t, rng.random(k)


@pytest.mark.parametrize("seed", range(6))
def test_temporal_efficiency_matches_oracle(seed):
    from oracle import temporal_efficiency
    rng = np.random.default_rng(seed)
    ta, fa = _curve(rng, int(rng.integers(2, 60)))
    tb, fb = _curve(rng, int(rng.integers(2, 60)))
    got = agn.agn_temporal_efficiency(ta, fa, tb, fb)
    want = temporal_efficiency(ta, fa, tb, fb)
    assert got == pytest.approx(want, rel=1e-12)


def test_temporal_efficiency_closed_forms():
    # f_a = t on [0, 2] against f_b = 1 on [0, 1]: cut at 1, E = 1/2
    assert agn.agn_temporal_efficiency([0, 2], [0, 2], [0, 1], [1, 1]) == pytest.approx(0.5, rel=1e-15)
    # lines are integrated exactly: 0.3 t against 0.6 over m = 3 -> 3/4
    ta = [0.0, 0.13, 0.9, 1.05, 2.4, 4.0]
    assert agn.agn_temporal_efficiency(ta, [0.3 * t for t in ta], [0, 1.1, 3.0], [0.6] * 3) == \
        pytest.approx(0.75, rel=1e-14)


@pytest.mark.parametrize("ta,fa,tb,fb", [
    ([0.0], [1.0], [0, 1], [1, 1]),                 # one sample
    ([0.5, 1.0], [1, 1], [0, 1], [1, 1]),           # not starting at 0
    ([0.0, 1.0, 1.0], [1, 1, 1], [0, 1], [1, 1]),   # times not increasing
    ([0.0, 1.0], [1.0, float("inf")], [0, 1], [1, 1]),
    ([0.0, 1.0], [1, 1], [0, 1], [0, 0]),           # zero area of b
])
def test_temporal_efficiency_rejects_bad_curves(ta, fa, tb, fb):
    with pytest.raises(agn.AGNError) as ei:
        agn.agn_temporal_efficiency(ta, fa, tb, fb)
    assert ei.value.code == -1


def test_plain_c_program_uses_the_abi(tmp_path):
    """agn.h compiles as ISO C99 with every warning an error, a C program links
    against libagn.so, and the argument checks answer it as documented
    (AGN_EINVAL with no context and a message; NULL contexts refused; Eq. 4
    of two identical curves is 1).  No device is needed."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("no C compiler")
    agn.load_library()
    from tests.c_abi import build as c_build
    exe = c_build.build(str(tmp_path))
    r = subprocess.run([exe, "validate"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and "0 failure(s)" in r.stdout, r.stdout + r.stderr
