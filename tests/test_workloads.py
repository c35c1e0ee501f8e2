"""Synthetic workload generator: shapes, value distributions, determinism."""
import numpy as np
import pytest

import workloads as W


def test_five_workloads_match_their_stated_shapes():
    t = W.workload("tiny")
    assert t.dims == (784, 64, 10) and t.num_params == 50890 and t.shard == 2048
    a = W.workload("mlp1000_n8")
    assert a.num_params == 1796010 and a.shard == 7500 and a.worker_samples_per_round == 15360
    assert W.workload("mlp1000_n20").shard == 3000
    c = W.workload("mlp2000_n40")
    assert c.num_params == 9594010 and c.shard == 3000
    d = W.workload("wide_bf16")
    assert d.num_params == 14891108 and d.shard == 8192 and d.dtype == "bf16"
    # FLOPs per worker-sample per step: 6 * sum(d_l d_{l+1}) - 2 d_0 d_1
    assert a.flops_per_round // a.worker_samples_per_round == 9196000
    assert c.flops_per_round // c.worker_samples_per_round == 54392000


def test_tiny_data_gaussian_linear_teacher():
    wl = W.workload("tiny")
    X, y = W.make_data(wl)
    assert X.shape == (4096, 784) and X.dtype == np.float32 and y.dtype == np.int32
    assert abs(X.mean()) < 0.01 and abs(X.std() - 1) < 0.01
    assert y.min() >= 0 and y.max() < 10 and len(np.unique(y)) == 10
    X2, y2 = W.make_data(wl)
    assert W.data_digest(X, y) == W.data_digest(X2, y2)


def test_sparse_data_and_two_layer_teacher():
    wl = W.small_workload("s", (784, 32, 10), 4, 2, 16, 0.01, 1, N=20000, data="sparse_teacher2")
    X, y = W.make_data(wl)
    zeros = np.mean(X == 0)
    assert 0.78 < zeros < 0.82
    assert X.min() >= 0 and X.max() < 1
    counts = np.bincount(y, minlength=10)
    print("class histogram", counts)
    assert (counts > 0).sum() == 10 and counts.min() > 0.3 * counts.mean()


def test_config3_shares_config2_data():
    a, b = W.workload("mlp1000_n8"), W.workload("mlp1000_n20")
    assert (a.data_seed or a.seed) == (b.data_seed or b.seed)


def test_bf16_storage_round_trip():
    wl = W.small_workload("b", (96, 16, 12), 2, 2, 8, 0.01, 1, N=512, dtype="bf16")
    X, y = W.make_data(wl)
    assert X.dtype == np.uint16
    xf = W.f32_from_bf16_bits(X)
    assert abs(xf.std() - 1) < 0.05
    np.testing.assert_array_equal(W.bf16_bits_from_f32(xf), X)


def test_commit_orders():
    assert all((o == np.arange(8)).all() for o in W.commit_orders(W.workload("mlp1000_n8")))
    ords = W.commit_orders(W.workload("mlp1000_n20"))
    assert len(ords) == 10
    for o in ords:
        assert sorted(o.tolist()) == list(range(20)) and o.dtype == np.int32
    assert not all((o == ords[0]).all() for o in ords[1:])
    again = W.commit_orders(W.workload("mlp1000_n20"))
    assert all((a == b).all() for a, b in zip(ords, again))
