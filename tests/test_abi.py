"""The C ABI: the library loads, exports every declared entry point, and
rejects bad arguments on the host before touching a GPU."""
import ctypes
import os
import re

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
