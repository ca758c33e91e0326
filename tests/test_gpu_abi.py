"""C ABI behaviour on the GPU: errors leave the net untouched, parameters
round-trip exactly, results are bitwise reproducible, and the shard count
changes only the rounding of the batch sum."""

import ctypes

import numpy as np
import pytest

from paper_1902_06714_amd import nf

from . import parity
from .gpu_run import GpuNet, note, to_dev

pytestmark = pytest.mark.gpu


def _setup(dims=(20, 33, 7), n=48, seed=3):
    rng = np.random.default_rng(seed)
    npar = sum(dims[l] * dims[l - 1] + dims[l] for l in range(1, len(dims)))
    theta = rng.normal(0, 0.3, npar).astype(np.float32)
    X = rng.uniform(0, 1, (n, dims[0])).astype(np.float32)
    Y = rng.uniform(0, 1, (n, dims[-1])).astype(np.float32)
    return dims, theta, X, Y


def test_params_round_trip_bitwise():
    dims, theta, _, _ = _setup()
    theta[::7] = np.float32(-0.0)
    theta[1] = np.float32(1e-40)  # subnormal
    note("round trip")
    with GpuNet(dims, ("tanh",), theta) as net:
        got = net.params()
        assert got.tobytes() == theta.tobytes()
        assert np.all(net.grads() == 0)


def test_errors_leave_state_unchanged():
    dims, theta, X, Y = _setup()
    lib = nf.raw()
    note("error paths")
    with GpuNet(dims, ("sigmoid",), theta) as net:
        xd, yd = to_dev(X), to_dev(Y)
        h = net.h
        bad = [
            lambda: lib.nf_train_batch(h, xd.data_ptr(), yd.data_ptr(), 48, 1.0, 5, None),  # 48 % 5
            lambda: lib.nf_train_batch(h, xd.data_ptr(), yd.data_ptr(), 48, 1.0, 0, None),
            lambda: lib.nf_train_batch(h, xd.data_ptr(), yd.data_ptr(), 0, 1.0, 1, None),
            lambda: lib.nf_train_batch(h, None, yd.data_ptr(), 48, 1.0, 1, None),
            lambda: lib.nf_train_batch(h, xd.data_ptr(), yd.data_ptr(), 48, float("nan"), 1, None),
            lambda: lib.nf_train_epoch(h, xd.data_ptr(), yd.data_ptr(), 50, 48, 1.0, 1, None),
            lambda: lib.nf_forward(h, xd.data_ptr(), -1, xd.data_ptr(), None),
        ]
        for i, call in enumerate(bad):
            st = call()
            assert st in (nf.NF_EINVAL, nf.NF_ESHAPE), (i, st)
            assert nf.nf_last_error()
        buf = np.zeros(nf.nf_param_count(h) + 1, np.float32)
        assert lib.nf_set_params(h, buf.ctypes.data, buf.size) == nf.NF_ESHAPE
        assert lib.nf_get_params(h, buf.ctypes.data, buf.size - 2) == nf.NF_ESHAPE
        assert net.params().tobytes() == theta.tobytes()


def test_bitwise_reproducible():
    dims, theta, X, Y = _setup((300, 257, 129, 10), 2000, 8)
    res = []
    for _ in range(2):
        with GpuNet(dims, ("tanh", "relu", "sigmoid"), theta) as net:
            xd, yd = to_dev(X), to_dev(Y)
            for t in range(4):
                net.train_batch(xd[t * 500:(t + 1) * 500], yd[t * 500:(t + 1) * 500], 0.5, 4)
            res.append((net.params().tobytes(), net.grads().tobytes()))
    assert res[0] == res[1]


def test_shard_count_only_changes_rounding():
    dims, theta, X, Y = _setup((100, 80, 10), 1600, 9)
    out = {}
    for s in (1, 2, 16, 1600):
        with GpuNet(dims, ("tanh", "sigmoid"), theta) as net:
            net.train_batch(to_dev(X), to_dev(Y), 0.5, s)
            out[s] = (net.params(), net.grads())
    for s in (2, 16, 1600):
        assert not parity.check_params(out[s][0], out[1][0], dims, tol=1e-6)
        assert not parity.check_params(out[s][1], out[1][1], dims, tol=1e-5, what="grads")


def test_nets_are_independent_and_reusable_across_batch_sizes():
    dims, theta, X, Y = _setup((16, 24, 4), 512, 10)
    with GpuNet(dims, ("sigmoid",), theta) as a, GpuNet(dims, ("sigmoid",), theta) as b:
        xd, yd = to_dev(X), to_dev(Y)
        a.train_batch(xd[:64], yd[:64], 1.0)
        a.train_batch(xd[:512], yd[:512], 1.0)     # grows the workspace
        a.train_batch(xd[:32], yd[:32], 1.0)
        b.train_batch(xd[:64], yd[:64], 1.0)
        b.train_batch(xd[:512], yd[:512], 1.0)
        b.train_batch(xd[:32], yd[:32], 1.0)
        assert a.params().tobytes() == b.params().tobytes()


def test_explicit_stream():
    import torch
    dims, theta, X, Y = _setup()
    s = torch.cuda.Stream()
    with GpuNet(dims, ("sigmoid",), theta) as ref, GpuNet(dims, ("sigmoid",), theta) as net:
        xd, yd = to_dev(X), to_dev(Y)
        torch.cuda.synchronize()
        ref.train_batch(xd, yd, 1.0)
        nf.nf_train_batch(net.h, xd, yd, 1.0, 1, stream=s)
        assert net.params().tobytes() == ref.params().tobytes()
