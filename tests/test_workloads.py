"""The seeded input generators: the published SplitMix64 sequence,
reproducibility, ranges, moments and one-hot labels."""

import numpy as np

from paper_1902_06714_amd import workloads as W


def test_splitmix64_published_sequence():
    # SplitMix64 started from state 0 (Steele, Lea and Flood 2014)
    expect = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    with np.errstate(over="ignore"):
        got = [int(W._mix(np.array([W.GOLDEN * np.uint64(i)], dtype=np.uint64))[0])
               for i in (1, 2, 3)]
    assert got == expect


def test_streams_reproducible_and_prefix_stable():
    a = W.uniform(3, 7, 1000)
    b = W.uniform(3, 7, 1000)
    assert np.array_equal(a, b)
    assert np.array_equal(W.uniform(3, 7, 100), a[:100])
    assert not np.array_equal(W.uniform(3, 8, 1000), a)
    assert not np.array_equal(W.uniform(4, 7, 1000), a)
    n1 = W.normal(1, 2, 999)
    assert np.array_equal(W.normal(1, 2, 999), n1)
    assert np.array_equal(W.normal(1, 2, 51), n1[:51])


def test_uniform_range_and_moments():
    u = W.uniform(0, 0, 1 << 20)
    assert u.dtype == np.float32 and u.min() >= 0.0 and u.max() < 1.0
    assert np.all(u * (1 << 24) == np.floor(u * (1 << 24)))
    assert abs(u.mean() - 0.5) < 2e-3 and abs(u.var() - 1 / 12) < 2e-3


def test_normal_moments():
    z = W.normal(0, 5, 1 << 20).astype(np.float64)
    assert abs(z.mean()) < 5e-3 and abs(z.std() - 1) < 5e-3
    assert abs(np.mean(z ** 3)) < 2e-2 and abs(np.mean(z ** 4) - 3) < 5e-2


def test_labels_and_one_hot():
    lbl = W.labels(0, 1, 100000)
    assert lbl.min() == 0 and lbl.max() == 9
    counts = np.bincount(lbl, minlength=10)
    assert np.all(np.abs(counts - 10000) < 500)
    y = W.one_hot(lbl[:1000])
    assert y.shape == (1000, 10) and np.all(y.sum(1) == 1) and np.all(np.argmax(y, 1) == lbl[:1000])


def test_workload_shapes_and_params():
    for name, w in W.WORKLOADS.items():
        assert len(w.acts) == w.n_layers
        assert w.n_samples == w.batch * w.steps
        assert w.batch % w.shards == 0
    w = W.WORKLOADS["c1"]
    p = W.make_params(w)
    assert p.shape == (w.param_count(),) and p.dtype == np.float32
    W1 = p[:784 * 30].astype(np.float64)
    assert abs(W1.std() * np.sqrt(784) - 1) < 0.05
    x, y = W.make_data(w, 200)
    assert x.shape == (200, 784) and y.shape == (200, 10)
    x2, _ = W.make_data(w, 100)
    assert np.array_equal(x2, x[:100])
    w4 = W.WORKLOADS["c4"]
    p4 = W.init_params((784, 1024), "he", 1)
    assert abs(p4[:784 * 1024].astype(np.float64).std() * np.sqrt(784 / 2) - 1) < 0.02
