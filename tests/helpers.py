"""Shared test utilities: the normwise parity metric and GPU data upload."""
import numpy as np


def tensor_slices(dims):
    """(name, start, stop) of every parameter tensor in the packed layout."""
    out, o = [], 0
    for l in range(len(dims) - 1):
        w = dims[l] * dims[l + 1]
        out.append((f"W{l}", o, o + w))
        o += w
        out.append((f"b{l}", o, o + dims[l + 1]))
        o += dims[l + 1]
    return out


def rel_err(got, ref, dims):
    """Parity metric: per parameter tensor ||got - ref||_inf / ||ref||_inf,
    maximum over the tensors (a tensor whose reference is all zero uses an
    absolute error)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    worst, where = 0.0, None
    for name, a, b in tensor_slices(dims):
        den = np.max(np.abs(ref[a:b]))
        err = np.max(np.abs(got[a:b] - ref[a:b])) / (den if den > 0 else 1.0)
        if err > worst:
            worst, where = err, name
    return worst, where


def to_device(X, y):
    import torch
    if X.dtype == np.uint16:
        xt = torch.from_numpy(np.ascontiguousarray(X).view(np.int16)).cuda()
    else:
        xt = torch.from_numpy(np.ascontiguousarray(X)).cuda()
    return xt, torch.from_numpy(np.ascontiguousarray(y, dtype=np.int32)).cuda()


def require_gpu():
    import torch
    assert torch.cuda.is_available(), "a ROCm GPU is required for this test"


def rel_fro(got, ref, dims):
    """Per parameter tensor ||got - ref||_2 / ||ref||_2 (Frobenius), maximum
    over the tensors.  Unlike the max-norm metric it is not dominated by the
    localized change one flipped ReLU derivative makes."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    worst, where = 0.0, None
    for name, a, b in tensor_slices(dims):
        den = np.linalg.norm(ref[a:b])
        err = np.linalg.norm(got[a:b] - ref[a:b]) / (den if den > 0 else 1.0)
        if err > worst:
            worst, where = err, name
    return worst, where


def parity_report(got, ref, dims):
    """The full-size parity metrics of the central variable:
    vec   ||got - ref||_inf / ||ref||_inf over the whole parameter vector
    W     max over weight tensors of the per-tensor max-norm relative error
    b     max over bias tensors of the per-tensor Frobenius relative error
    """
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    vec = np.max(np.abs(got - ref)) / np.max(np.abs(ref))
    w = b = 0.0
    for name, a0, a1 in tensor_slices(dims):
        d = got[a0:a1] - ref[a0:a1]
        if name[0] == "W":
            w = max(w, np.max(np.abs(d)) / max(np.max(np.abs(ref[a0:a1])), 1e-300))
        else:
            b = max(b, np.linalg.norm(d) / max(np.linalg.norm(ref[a0:a1]), 1e-300))
    return {"vec": vec, "W": w, "b": b}
