"""The fp64 variant (the paper's real64 kind, section 3.1) against the CPU
reference run with fp64 parameters.

Both sides then compute every quantity in fp64 and differ only in the order
of their sums, so the gate is far tighter than the fp32 one:

    |gpu - ref| <= F64_TOL * max(|ref|, rms(ref_t))   per tensor t, elementwise,

for parameters, tendencies and outputs alike.  F64_TOL = 1e-9 comes from the
arithmetic: a sum of K products carries a relative error of at most about
K u (u = 2^-53 = 1.1e-16), and the longest sums here are the batch sums of
the tendencies (K up to 10000), so one step agrees to ~1e-12; the gate leaves
three orders of magnitude for what the steps of a schedule add (a relu unit
within 1e-16 of its kink would be a legitimate exception; none occurs on
these inputs).
"""

import numpy as np
import pytest

from oracle import mlp
from paper_1902_06714_amd import workloads as W

from . import parity
from .gpu_run import note, torch_cuda

pytestmark = pytest.mark.gpu

F64_TOL = 1e-9


def to_dev64(a):
    torch = torch_cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64)).to("cuda")


class Net64:
    """An fp64 network on the GPU, owned for the duration of a with-block."""

    def __init__(self, dims, acts, theta):
        from paper_1902_06714_amd import nf
        self.nf = nf
        self.dims = list(dims)
        self.h = nf.nf_net_create(dims, list(acts), dtype=nf.NF_F64)
        nf.nf_set_params_f64(self.h, theta)

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.nf.nf_net_destroy(self.h)

    def params(self):
        return self.nf.nf_get_params_f64(self.h)

    def grads(self):
        return self.nf.nf_get_grads_f64(self.h)

    def forward(self, xd):
        torch = torch_cuda()
        out = torch.empty((xd.shape[0], self.dims[-1]), dtype=torch.float64, device="cuda")
        self.nf.nf_forward_f64(self.h, xd, out)
        torch.cuda.synchronize()
        return out.cpu().numpy()


def _check(got, ref, dims, what):
    fails = []
    for name, sl in parity.tensor_slices(dims):
        e, i = parity.floored_rel(got[sl], ref[sl])
        if not e <= F64_TOL:
            fails.append(f"{what} {name}: {e:.3e} at {i}")
    return fails


def _problem(dims, seed, n, x_lo=0.0):
    rng = np.random.default_rng(seed)
    parts = []
    for l in range(1, len(dims)):
        parts.append(rng.normal(0, 1.0 / np.sqrt(dims[l - 1]), dims[l] * dims[l - 1]))
        parts.append(rng.normal(0, 1, dims[l]))
    theta = np.concatenate(parts)
    X = rng.uniform(x_lo, 1.0, (n, dims[0]))
    Y = np.eye(dims[-1])[rng.integers(0, dims[-1], n)]
    return theta, X, Y


SMALL = [
    # dims, acts, batch, shards, eta, steps
    ((37, 133, 65, 7), ("tanh", "sigmoid", "gaussian"), 300, 1, 0.5, 3),
    ((37, 133, 65, 7), ("tanh", "sigmoid", "gaussian"), 300, 3, 0.5, 3),
    ((784, 30, 10), ("sigmoid",), 1000, 1, 3.0, 4),        # the paper's network
    ((64, 200, 10), ("sigmoid",), 257, 1, 3.0, 3),
    ((12, 300, 300, 5), ("tanh",), 1024, 8, 1.0, 2),
    ((64, 64, 8), ("sigmoid", "tanh"), 8192, 1, 1.0, 2),   # long batch: split and ordered fold
    ((3, 5, 2), ("tanh",), 1, 1, 0.3, 4),                  # the paper's [3, 5, 2] tanh network
    ((129, 1, 1), ("sigmoid",), 65, 5, 2.0, 3),
    ((200, 130, 70, 3), ("relu", "relu", "sigmoid"), 4000, 4, 1.0, 2),
]


@pytest.mark.parametrize("dims,acts,batch,shards,eta,steps", SMALL)
def test_f64_trajectory(dims, acts, batch, shards, eta, steps):
    acts_full = list(acts) * (len(dims) - 1) if len(acts) == 1 else list(acts)
    theta, X, Y = _problem(dims, 31, batch * steps)
    note(f"f64 trajectory dims={dims} batch={batch} shards={shards}")
    ref = theta
    fails = []
    with Net64(dims, acts, theta) as net:
        xd, yd = to_dev64(X), to_dev64(Y)
        for t in range(steps):
            sl = slice(t * batch, (t + 1) * batch)
            net.nf.nf_train_batch_f64(net.h, xd[sl], yd[sl], eta, shards)
            ref, G = mlp.train_batch(ref, dims, acts_full, X[sl], Y[sl], eta, shards,
                                     precision="f64")
            fails += [f"step {t}: {m}" for m in _check(net.params(), ref, dims, "params")]
            fails += [f"step {t}: {m}" for m in _check(net.grads(), G, dims, "grads")]
    assert not fails, "\n".join(fails[:20])


# narrow fp64 networks (every layer after the input <= 32 units, even input
# width) take the two-kernel step of csrc/nf_narrow64.hip (4-sample tiles up
# to 2048 samples, 16-sample tiles above); odd input widths and split batches
# take the medium per-sample kernel on the same padded layout
NARROW64 = [
    # dims, acts, batch, shards
    ((4, 3), ("sigmoid",), 1, 1),
    ((8, 32), ("tanh",), 2, 1),
    ((60, 7, 2), ("sigmoid", "tanh"), 3, 1),
    ((64, 32, 31, 1), ("gaussian", "tanh", "sigmoid"), 17, 1),
    ((66, 20, 20, 20, 20), ("tanh",), 33, 1),
    ((1026, 30, 10), ("sigmoid",), 2049, 1),         # above 2048: 16-sample tiles
    ((1090, 30, 10), ("sigmoid",), 37, 1),           # 4-sample tiles, two rounds of input steps
    ((2050, 5), ("tanh",), 6, 1),                     # three rounds, a ragged last tile
    ((65536, 30, 10), ("sigmoid",), 5, 1),           # the widest input: 2048 input steps
    ((12, 32, 32, 32, 32), ("relu", "tanh", "tanh", "sigmoid"), 100, 1),
    ((7, 9, 4), ("tanh", "sigmoid"), 40, 1),          # odd input width: medium kernel
    ((64, 32, 10), ("sigmoid",), 96, 4),              # split batch: medium kernel
]


# the fp64 per-sample kernel (csrc/nf_medium.hip, 16-sample tiles): more
# layer-1 pieces than are loaded ahead, 2 to 4 layers with ragged widths,
# several rounds of tiles per workgroup, weights near the fp64 LDS limit, and
# one network just past it (the contraction kernels)
MEDIUM64 = [
    # dims, acts, batch, shards
    ((300, 120, 10), ("sigmoid",), 5, 1),
    ((784, 100, 100, 10), ("tanh", "tanh", "sigmoid"), 100, 4),
    ((20, 17, 31, 45, 7), ("tanh", "sigmoid", "gaussian", "sigmoid"), 5000, 2),
    ((40, 96, 64, 48, 16), ("gaussian", "tanh", "sigmoid", "tanh"), 700, 1),
    ((50, 128, 100, 10), ("tanh", "sigmoid", "sigmoid"), 300, 3),   # past the LDS limit
    ((1, 1, 1), ("tanh",), 33, 1),
]


@pytest.mark.parametrize("dims,acts,batch,shards", MEDIUM64)
def test_f64_medium(dims, acts, batch, shards):
    acts_full = list(acts) * (len(dims) - 1) if len(acts) == 1 else list(acts)
    theta, X, Y = _problem(dims, 3 * sum(dims) + batch, batch * 2)
    note(f"f64 medium dims={dims} batch={batch} shards={shards}")
    ref = theta
    fails = []
    with Net64(dims, acts, theta) as net:
        xd, yd = to_dev64(X), to_dev64(Y)
        for t in range(2):
            sl = slice(t * batch, (t + 1) * batch)
            net.nf.nf_train_batch_f64(net.h, xd[sl], yd[sl], 0.5, shards)
            ref, G = mlp.train_batch(ref, dims, acts_full, X[sl], Y[sl], 0.5, shards,
                                     precision="f64")
            fails += [f"step {t}: {m}" for m in _check(net.params(), ref, dims, "params")]
            fails += [f"step {t}: {m}" for m in _check(net.grads(), G, dims, "grads")]
    assert not fails, "\n".join(fails[:20])


# the fp64 skinny tendency kernel: unit counts over every combination of
# 32- and 16-row segments (1, 10, 16, 33, 49, 97, 100, 113, 127, 128), input
# tiles of 32 with one- and two-block tails (20, 36, 49, 97, 113, 788), shards
# of a few samples, and a check that the launches take that kernel
SKINNY64 = [
    ((20, 113, 49, 10), ("tanh", "sigmoid", "sigmoid"), 500, 4),
    ((36, 128, 97, 33), ("sigmoid", "tanh", "gaussian"), 333, 3),
    ((788, 100, 16, 1), ("tanh", "sigmoid", "sigmoid"), 1000, 8),
    ((100, 127, 64), ("sigmoid",), 160, 16),
]


@pytest.mark.parametrize("dims,acts,batch,shards", SKINNY64)
def test_f64_skinny_tendencies(dims, acts, batch, shards):
    acts_full = list(acts) * (len(dims) - 1) if len(acts) == 1 else list(acts)
    theta, X, Y = _problem(dims, 7 * sum(dims) + batch, batch * 2)
    note(f"f64 skinny dims={dims} batch={batch} shards={shards}")
    ref = theta
    fails = []
    with Net64(dims, acts, theta) as net:
        xd, yd = to_dev64(X), to_dev64(Y)
        for t in range(2):
            sl = slice(t * batch, (t + 1) * batch)
            net.nf.nf_profile(net.h, 1)
            net.nf.nf_train_batch_f64(net.h, xd[sl], yd[sl], 0.5, shards)
            names = {k["name"]: k["launches"] for k in net.nf.nf_profile_read(net.h)}
            net.nf.nf_profile(net.h, 0)
            assert names.get("dw64_skinny") == 1, names
            assert not any("dw_partial" in k for k in names), names
            ref, G = mlp.train_batch(ref, dims, acts_full, X[sl], Y[sl], 0.5, shards,
                                     precision="f64")
            fails += [f"step {t}: {m}" for m in _check(net.params(), ref, dims, "params")]
            fails += [f"step {t}: {m}" for m in _check(net.grads(), G, dims, "grads")]
    assert not fails, "\n".join(fails[:20])


@pytest.mark.parametrize("dims,acts,batch,shards", NARROW64)
def test_f64_narrow(dims, acts, batch, shards):
    acts_full = list(acts) * (len(dims) - 1) if len(acts) == 1 else list(acts)
    theta, X, Y = _problem(dims, 5 * sum(dims) + batch, batch * 2, x_lo=-1.0)
    note(f"f64 narrow dims={dims} batch={batch} shards={shards}")
    ref = theta
    fails = []
    with Net64(dims, acts, theta) as net:
        xd, yd = to_dev64(X), to_dev64(Y)
        for t in range(2):
            sl = slice(t * batch, (t + 1) * batch)
            net.nf.nf_train_batch_f64(net.h, xd[sl], yd[sl], 1.0, shards)
            ref, G = mlp.train_batch(ref, dims, acts_full, X[sl], Y[sl], 1.0, shards,
                                     precision="f64")
            fails += [f"step {t}: {m}" for m in _check(net.params(), ref, dims, "params")]
            fails += [f"step {t}: {m}" for m in _check(net.grads(), G, dims, "grads")]
        out = net.forward(xd)
    e, i = parity.floored_rel(out, mlp.output(ref, dims, acts_full, X))
    if e > F64_TOL:
        fails.append(f"inference: {e:.3e} at {i}")
    assert not fails, "\n".join(fails[:20])


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,steps", [("c1", 10), ("c2", 60), ("c3", 6), ("c4", 16), ("c5", 4)])
def test_f64_workloads(name, steps):
    """Each workload's network, data and whole schedule in fp64, free-running
    from the seeded parameters."""
    w = W.WORKLOADS[name]
    acts = list(w.acts)
    X, Y = W.make_data(w, w.batch * steps)
    X, Y = X.astype(np.float64), Y.astype(np.float64)
    theta = W.make_params(w).astype(np.float64)
    note(f"f64 {name}: {w.dims} batch={w.batch} shards={w.shards} steps={steps}")
    ref = theta
    worst_p = worst_g = 0.0
    fails = []
    with Net64(w.dims, acts, theta) as net:
        xd, yd = to_dev64(X), to_dev64(Y)
        for t in range(steps):
            sl = slice(t * w.batch, (t + 1) * w.batch)
            net.nf.nf_train_batch_f64(net.h, xd[sl], yd[sl], w.eta, w.shards)
            ref, G = mlp.train_batch(ref, w.dims, acts, X[sl], Y[sl], w.eta, w.shards,
                                     precision="f64")
            p, g = net.params(), net.grads()
            fails += [f"step {t}: {m}" for m in _check(p, ref, w.dims, "params")]
            fails += [f"step {t}: {m}" for m in _check(g, G, w.dims, "grads")]
            for nm, sl2 in parity.tensor_slices(w.dims):
                worst_p = max(worst_p, parity.floored_rel(p[sl2], ref[sl2])[0])
                worst_g = max(worst_g, parity.floored_rel(g[sl2], G[sl2])[0])
    print(f"[parity f64] {name}: worst param error {worst_p:.2e}, worst tendency error "
          f"{worst_g:.2e}", flush=True)
    assert not fails, "\n".join(fails[:20])


@pytest.mark.parametrize("dims,acts,n", [
    ((784, 30, 10), ("sigmoid",), 10000),
    ((37, 133, 65, 7), ("tanh", "relu", "gaussian"), 1001),
])
def test_f64_inference(dims, acts, n):
    acts_full = list(acts) * (len(dims) - 1) if len(acts) == 1 else list(acts)
    theta, X, _ = _problem(dims, 32, n, x_lo=-1.0)
    note(f"f64 inference dims={dims} n={n}")
    with Net64(dims, acts, theta) as net:
        out = net.forward(to_dev64(X))
    ref = mlp.output(theta, dims, acts_full, X)
    e, i = parity.floored_rel(out, ref)
    assert e <= F64_TOL, (e, i)


def test_f64_single_windows_and_accuracy():
    dims, acts = (784, 30, 10), ["sigmoid", "sigmoid"]
    theta, X, Y = _problem(dims, 33, 500)
    pos = W.window_positions(9, 6).astype(np.float64)
    note("f64 train_single, train_windows, accuracy")
    with Net64(dims, acts, theta) as net:
        xd, yd = to_dev64(X), to_dev64(Y)
        net.nf.nf_train_single_f64(net.h, xd[0], yd[0], 0.8)
        ref = mlp.train_single(theta, dims, acts, X[0], Y[0], 0.8, precision="f64")
        fails = _check(net.params(), ref, dims, "single")
        net.nf.nf_train_windows_f64(net.h, xd, yd, 100, pos, 3.0)
        ref = mlp.train_windows(ref, dims, acts, X, Y, 100, pos, 3.0, precision="f64")
        fails += _check(net.params(), ref, dims, "windows")
        got = net.nf.nf_accuracy_f64(net.h, xd, yd)
        out = net.forward(xd)
    assert not fails, "\n".join(fails)
    assert got == int(np.sum(np.argmax(out, axis=1) == np.argmax(Y, axis=1)))
    ref_out = mlp.output(ref, dims, acts, X)
    top2 = np.sort(ref_out, axis=1)[:, -2:]
    near = int(np.sum(top2[:, 1] - top2[:, 0] <= 1e-12 * np.abs(top2[:, 1])))
    assert abs(got - mlp.correct_count(ref_out, Y)) <= near


def test_precision_families_do_not_mix():
    from paper_1902_06714_amd import nf
    torch = torch_cuda()
    dims = (8, 5, 3)
    theta, X, Y = _problem(dims, 34, 16)
    note("fp32 calls on an fp64 net and the reverse")
    with Net64(dims, ["tanh", "sigmoid"], theta) as net:
        assert nf.nf_net_dtype(net.h) == nf.NF_F64
        before = net.params()
        x32 = torch.from_numpy(X.astype(np.float32)).cuda()
        y32 = torch.from_numpy(Y.astype(np.float32)).cuda()
        for call in (lambda: nf.nf_train_batch(net.h, x32, y32, 1.0),
                     lambda: nf.nf_get_params(net.h),
                     lambda: nf.nf_set_params(net.h, theta.astype(np.float32))):
            with pytest.raises(nf.NfError) as e:
                call()
            assert e.value.status == nf.NF_EINVAL
        assert np.array_equal(net.params(), before)
    h = nf.nf_net_create(dims, ["tanh", "sigmoid"])
    try:
        assert nf.nf_net_dtype(h) == nf.NF_F32
        with pytest.raises(nf.NfError) as e:
            nf.nf_train_batch_f64(h, to_dev64(X), to_dev64(Y), 1.0)
        assert e.value.status == nf.NF_EINVAL
    finally:
        nf.nf_net_destroy(h)


def test_f64_and_f32_agree_to_fp32_rounding():
    """The same step in both precisions: the fp32 result is the fp64 one to
    within fp32 rounding (the gate of the fp32 path)."""
    from .gpu_run import GpuNet, to_dev
    dims, acts = (784, 100, 10), ("tanh", "sigmoid")
    theta, X, Y = _problem(dims, 35, 2000)
    theta32 = theta.astype(np.float32)
    note("f64 vs f32 on one step")
    with Net64(dims, acts, theta32.astype(np.float64)) as a, GpuNet(dims, acts, theta32) as b:
        a.nf.nf_train_batch_f64(a.h, to_dev64(X.astype(np.float32)), to_dev64(Y), 1.0, 4)
        b.train_batch(to_dev(X), to_dev(Y), 1.0, 4)
        assert not parity.check_params(b.params(), a.params(), dims)
