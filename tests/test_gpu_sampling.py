"""Single-sample steps, random-window mini-batches and the accuracy count on
the GPU, against the CPU reference (sections 3.4 and 4 of the paper)."""

import numpy as np
import pytest

from oracle import mlp
from paper_1902_06714_amd import workloads as W

from . import parity
from .gpu_run import GpuNet, note, to_dev, torch_cuda

pytestmark = pytest.mark.gpu


def _problem(dims, seed, n):
    rng = np.random.default_rng(seed)
    parts = []
    for l in range(1, len(dims)):
        parts.append(rng.normal(0, 1.0 / np.sqrt(dims[l - 1]), dims[l] * dims[l - 1]))
        parts.append(rng.normal(0, 1, dims[l]))
    theta = np.concatenate(parts).astype(np.float32)
    X = rng.uniform(0, 1, (n, dims[0])).astype(np.float32)
    Y = np.eye(dims[-1], dtype=np.float32)[rng.integers(0, dims[-1], n)]
    return theta, X, Y


@pytest.mark.parametrize("dims,acts", [((784, 30, 10), ("sigmoid",)),
                                       ((37, 133, 65, 7), ("tanh", "sigmoid", "gaussian"))])
def test_train_single_matches_reference(dims, acts):
    acts_full = list(acts) * (len(dims) - 1) if len(acts) == 1 else list(acts)
    theta, X, Y = _problem(dims, 11, 6)
    note(f"train_single dims={dims}")
    ref = theta
    fails = []
    with GpuNet(dims, acts, theta) as net:
        for i in range(X.shape[0]):
            net.nf.nf_train_single(net.h, to_dev(X[i]), to_dev(Y[i]), 0.7)
            ref = mlp.train_single(ref, dims, acts_full, X[i].astype(np.float64),
                                   Y[i].astype(np.float64), 0.7)
            fails += [f"sample {i}: {m}" for m in parity.check_params(net.params(), ref, dims)]
    assert not fails, "\n".join(fails[:20])


@pytest.mark.parametrize("name,shards", [("c1", 1), ("c1", 4)])
def test_windows_match_reference(name, shards):
    w = W.WORKLOADS[name]
    X, Y = W.make_data(w)
    theta = W.make_params(w)
    pos = W.window_positions(w.data_seed, w.steps)
    note(f"train_windows {name} shards={shards} steps={w.steps}")
    with GpuNet(w.dims, w.acts, theta) as net:
        net.nf.nf_train_windows(net.h, to_dev(X), to_dev(Y), w.batch, pos, w.eta, shards)
        got = net.params()
    ref = mlp.train_windows(theta, w.dims, list(w.acts), X, Y, w.batch, pos, w.eta, shards)
    fails = parity.check_params(got, ref, w.dims)
    assert not fails, "\n".join(fails[:20])


def test_windows_general_path_unaligned_rows():
    dims, acts = (37, 133, 65, 7), ("tanh", "sigmoid", "gaussian")
    theta, X, Y = _problem(dims, 12, 301)
    pos = W.window_positions(5, 7)
    note("train_windows general path, 301 samples, batch 50")
    with GpuNet(dims, acts, theta) as net:
        net.nf.nf_train_windows(net.h, to_dev(X), to_dev(Y), 50, pos, 0.5, 2)
        got = net.params()
    ref = mlp.train_windows(theta, dims, list(acts), X, Y, 50, pos, 0.5, 2)
    fails = parity.check_params(got, ref, dims)
    assert not fails, "\n".join(fails[:20])


@pytest.mark.parametrize("dims", [(784, 30, 10), (37, 133, 65, 7)])
def test_back_to_back_windows_equal_one_epoch_bitwise(dims):
    theta, X, Y = _problem(dims, 13, 400)
    B = 100
    pos = np.array([(t * B + 0.5) / (400 - B + 1) for t in range(4)], dtype=np.float32)
    note(f"windows vs epoch dims={dims}")
    xd, yd = to_dev(X), to_dev(Y)
    with GpuNet(dims, ("sigmoid",), theta) as a, GpuNet(dims, ("sigmoid",), theta) as b:
        a.nf.nf_train_windows(a.h, xd, yd, B, pos, 2.0, 1)
        b.train_epoch(xd, yd, B, 2.0)
        assert np.array_equal(a.params(), b.params())


def test_window_arguments_rejected_before_any_step():
    from paper_1902_06714_amd import nf
    dims = (784, 30, 10)
    theta, X, Y = _problem(dims, 14, 200)
    xd, yd = to_dev(X), to_dev(Y)
    with GpuNet(dims, ("sigmoid",), theta) as net:
        before = net.params()
        for pos, batch, code in (([0.2, 1.0], 50, nf.NF_EINVAL), ([0.2, -0.1], 50, nf.NF_EINVAL),
                                 ([0.2, float("nan")], 50, nf.NF_EINVAL),
                                 ([0.2], 201, nf.NF_ESHAPE)):
            with pytest.raises(nf.NfError) as e:
                nf.nf_train_windows(net.h, xd, yd, batch, pos, 1.0)
            assert e.value.status == code
        assert np.array_equal(net.params(), before)
        nf.nf_train_windows(net.h, xd, yd, 50, [], 1.0)       # no steps: nothing changes
        assert np.array_equal(net.params(), before)


def _first_argmax_rows(a):
    """numpy's argmax takes the first of equal largest entries; NaN rows -1."""
    idx = np.argmax(a, axis=1)
    idx[np.isnan(a).any(axis=1)] = -1
    return idx


@pytest.mark.parametrize("d0", [3, 4])
def test_accuracy_worked_by_hand(d0):
    # sigmoid with W = I, b = 0 keeps the order of the inputs and their ties
    dims = (d0, d0)
    theta = np.concatenate([np.eye(d0).ravel(), np.zeros(d0)]).astype(np.float32)
    X = np.full((6, d0), -4.0, np.float32)
    X[:, :3] = [[0.9, 0.1, 0.2], [0.5, 0.5, 0.1], [0.0, 0.3, 0.7], [0.2, 0.8, 0.8],
                [0.1, 0.4, 0.9], [0.3, 0.3, 0.3]]
    Y = np.eye(d0, dtype=np.float32)[[0, 1, 2, 1, 2, 0]]
    Y[4, 0] = np.nan                                   # a NaN target never counts
    note(f"accuracy by hand d0={d0}")
    with GpuNet(dims, ("sigmoid",), theta) as net:
        assert net.nf.nf_accuracy(net.h, to_dev(X), to_dev(Y)) == 4


@pytest.mark.parametrize("dims,n", [((784, 30, 10), 40000), ((8, 100), 1001),
                                    ((37, 133, 65, 7), 5000)])
def test_accuracy_counts_the_gpu_outputs(dims, n):
    """Bit-exact against the count of the GPU's own fp32 outputs (the decision
    taken in the same precision), and equal to the reference's fp64 count up
    to rows whose two largest outputs are within rounding of each other."""
    theta, X, _ = _problem(dims, 15, n)
    rng = np.random.default_rng(16)
    Y = np.eye(dims[-1], dtype=np.float32)[rng.integers(0, dims[-1], n)]
    note(f"accuracy dims={dims} n={n}")
    xd = to_dev(X)
    with GpuNet(dims, ("sigmoid",), theta) as net:
        got = net.nf.nf_accuracy(net.h, xd, to_dev(Y))
        out = net.forward(xd)
    mine = int(np.sum(_first_argmax_rows(out) == np.argmax(Y, axis=1)))
    assert got == mine
    ref_out = mlp.output(theta, dims, ["sigmoid"] * (len(dims) - 1), X)
    ref = mlp.correct_count(ref_out, Y)
    top2 = np.sort(ref_out, axis=1)[:, -2:]
    near = int(np.sum(top2[:, 1] - top2[:, 0] <= 1e-5 * np.abs(top2[:, 1])))
    assert abs(got - ref) <= near, (got, ref, near)


def test_accuracy_after_training_c2_prefix():
    """The held-out count after a few steps of the 784-30-10 workload."""
    torch = torch_cuda()
    w = W.WORKLOADS["c2"]
    X, Y = W.make_data(w, n=5000)
    Xh, Yh = W.make_data(w, n=2000, heldout=True)
    theta = W.make_params(w)
    note("accuracy after 5 steps of c2")
    with GpuNet(w.dims, w.acts, theta) as net:
        net.train_epoch(to_dev(X), to_dev(Y), w.batch, w.eta)
        got = net.nf.nf_accuracy(net.h, to_dev(Xh), to_dev(Yh))
        out = net.forward(to_dev(Xh))
        torch.cuda.synchronize()
    assert got == int(np.sum(_first_argmax_rows(out) == np.argmax(Yh, axis=1)))
    assert 0 <= got <= 2000
