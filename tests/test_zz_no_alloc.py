"""nf_train_batch_noalloc, the training step for callers that cannot allocate,
against nf_train_batch on the same net state and inputs: two calls in a row
on each path (the second with a smaller batch, so the shared scratch array
holds the first call's leftovers), compared bit for bit, which is stricter
than the parity gates (both calls run the same kernels in the same order).
The networks take the three kernel families: the narrow two-kernel step
(784-30-10), the medium per-sample kernel with 16 shards (784-100-100-10),
and the contraction kernels with split batches (relu, 4 shards).  A step
that needs more scratch than the array holds is refused before anything is
enqueued, and the net is left as it was."""

import numpy as np
import pytest

from paper_1902_06714_amd import workloads as W

from .gpu_run import note, to_dev

pytestmark = pytest.mark.gpu


def _problem(dims, seed, n):
    rng = np.random.default_rng(seed)
    parts = []
    for l in range(1, len(dims)):
        parts.append(rng.normal(0, 1.0 / np.sqrt(dims[l - 1]), dims[l] * dims[l - 1]))
        parts.append(rng.normal(0, 1, dims[l]))
    theta = np.concatenate(parts).astype(np.float32)
    X = rng.uniform(0, 1, (n, dims[0])).astype(np.float32)
    Y = np.zeros((n, dims[-1]), np.float32)
    Y[np.arange(n), rng.integers(0, dims[-1], n)] = 1.0
    return theta, X, Y


CASES = [
    # dims, acts, (batch of the first call, batch of the second), shards, eta
    ((784, 30, 10), ("sigmoid",), (1000, 300), 1, 3.0),
    ((784, 100, 100, 10), ("tanh", "tanh", "sigmoid"), (10000, 2000), 16, 1.0),
    ((300, 257, 129, 10), ("tanh", "relu", "sigmoid"), (2000, 500), 4, 0.5),
]


@pytest.mark.parametrize("dims,acts,batches,shards,eta", CASES)
def test_noalloc_step_equals_train_batch(dims, acts, batches, shards, eta):
    from paper_1902_06714_amd import nf
    theta, X, Y = _problem(dims, sum(dims), sum(batches))
    xd, yd = to_dev(X), to_dev(Y)
    a = nf.nf_net_create(dims, list(acts))
    b = nf.nf_net_create(dims, list(acts))
    try:
        nf.nf_set_params(a, theta)
        nf.nf_set_params(b, theta)
        off = 0
        for i, B in enumerate(batches):
            note(f"noalloc dims={dims} call {i} batch={B} shards={shards}")
            sl = slice(off, off + B)
            off += B
            nf.nf_train_batch(a, xd[sl], yd[sl], eta, shards)
            nf.nf_train_batch_noalloc(b, xd[sl], yd[sl], eta, shards)
            pa, pb = nf.nf_get_params(a), nf.nf_get_params(b)
            ga, gb = nf.nf_get_grads(a), nf.nf_get_grads(b)
            assert np.all(np.isfinite(pa)) and np.all(np.isfinite(ga))
            assert np.array_equal(pa, pb), f"call {i}: parameters differ"
            assert np.array_equal(ga, gb), f"call {i}: tendencies differ"
        # the net's own workspace still works after borrowing the scratch
        note(f"noalloc dims={dims} own path after")
        nf.nf_train_batch(b, xd[:batches[1]], yd[:batches[1]], eta, shards)
        nf.nf_train_batch(a, xd[:batches[1]], yd[:batches[1]], eta, shards)
        assert np.array_equal(nf.nf_get_params(a), nf.nf_get_params(b))
    finally:
        nf.nf_net_destroy(a)
        nf.nf_net_destroy(b)


def test_noalloc_refuses_steps_beyond_the_scratch():
    """784-1024^3-10 at 4096 samples needs about 150 MB of per-sample buffers:
    refused with NF_ESHAPE, nothing run, the net unchanged."""
    from paper_1902_06714_amd import nf
    w = W.WORKLOADS["c4"]
    theta = W.make_params(w)
    X, Y = W.make_data(w, w.batch)
    xd, yd = to_dev(X), to_dev(Y)
    h = nf.nf_net_create(w.dims, list(w.acts))
    try:
        nf.nf_set_params(h, theta)
        note("noalloc refused at 784-1024^3-10 batch 4096")
        with pytest.raises(nf.NfError) as err:
            nf.nf_train_batch_noalloc(h, xd, yd, w.eta, 1)
        assert err.value.status == nf.NF_ESHAPE
        assert "scratch" in str(err.value)
        assert np.array_equal(nf.nf_get_params(h), theta)
        assert not np.any(nf.nf_get_grads(h))
        # the same net then trains through the scratch on a batch that fits
        note("noalloc 784-1024^3-10 batch 256")
        nf.nf_train_batch_noalloc(h, xd[:256], yd[:256], w.eta, 1)
        assert np.all(np.isfinite(nf.nf_get_params(h)))
    finally:
        nf.nf_net_destroy(h)


def test_noalloc_rejects_fp64_nets():
    from paper_1902_06714_amd import nf
    dims = (8, 6, 3)
    h = nf.nf_net_create(dims, ["sigmoid"], dtype=nf.NF_F64)
    try:
        x = to_dev(np.zeros((4, 8), np.float32))
        y = to_dev(np.zeros((4, 3), np.float32))
        with pytest.raises(nf.NfError) as err:
            nf.nf_train_batch_noalloc(h, x, y, 1.0, 1)
        assert err.value.status == nf.NF_EINVAL
    finally:
        nf.nf_net_destroy(h)
