"""Saving a network to a file and creating one from it: the file follows the
layout include/nf.h documents (read back here by the test's own parser), and
a loaded net holds the saved parameters bit for bit and trains on exactly as
the original."""

import struct

import numpy as np
import pytest

from .gpu_run import note, torch_cuda

pytestmark = pytest.mark.gpu


def _parse(path):
    b = open(path, "rb").read()
    assert b[:8] == b"NFNET01\n"
    dtype, nd = struct.unpack_from("<ii", b, 8)
    dims = struct.unpack_from(f"<{nd}i", b, 16)
    acts = struct.unpack_from(f"<{nd - 1}i", b, 16 + 4 * nd)
    off = 16 + 4 * nd + 4 * (nd - 1)
    (n,) = struct.unpack_from("<q", b, off)
    off += 8
    el = np.float64 if dtype == 1 else np.float32
    params = np.frombuffer(b, dtype=el, count=n, offset=off)
    off += n * np.dtype(el).itemsize
    (h,) = struct.unpack_from("<Q", b, off)
    assert off + 8 == len(b)
    ref = 1469598103934665603
    for byte in b[:off]:
        ref = ((ref ^ byte) * 1099511628211) & 0xFFFFFFFFFFFFFFFF
    assert h == ref
    return dtype, list(dims), list(acts), params


@pytest.mark.parametrize("dims,acts,f64", [
    ((784, 30, 10), ("sigmoid", "sigmoid"), False),
    ((37, 133, 65, 7), ("tanh", "sigmoid", "gaussian"), False),
    ((37, 133, 65, 7), ("tanh", "relu", "gaussian"), True),
])
def test_save_load_round_trip(tmp_path, dims, acts, f64):
    from paper_1902_06714_amd import nf
    torch = torch_cuda()
    rng = np.random.default_rng(41)
    n = sum(dims[l] * dims[l - 1] + dims[l] for l in range(1, len(dims)))
    el, tdt = (np.float64, torch.float64) if f64 else (np.float32, torch.float32)
    theta = (rng.normal(size=n) * 0.1).astype(el)
    X = torch.from_numpy(rng.uniform(size=(200, dims[0])).astype(el)).cuda()
    Y = torch.from_numpy(np.eye(dims[-1])[rng.integers(0, dims[-1], 200)].astype(el)).cuda()
    sfx = "_f64" if f64 else ""
    setp, getp = getattr(nf, "nf_set_params" + sfx), getattr(nf, "nf_get_params" + sfx)
    train = getattr(nf, "nf_train_batch" + sfx)
    path = str(tmp_path / "net.bin")
    note(f"save/load dims={dims} f64={f64}")
    a = nf.nf_net_create(dims, list(acts), dtype=nf.NF_F64 if f64 else nf.NF_F32)
    b = None
    try:
        setp(a, theta)
        train(a, X[:100], Y[:100], 0.5)
        nf.nf_save(a, path)
        saved = getp(a)
        dtype, fdims, facts, fparams = _parse(path)
        assert dtype == (1 if f64 else 0)
        assert fdims == list(dims)
        assert facts == [nf.ACT_CODES[x] for x in acts]
        assert np.array_equal(fparams, saved)
        b = nf.nf_load(path)
        assert nf.nf_net_dtype(b) == dtype
        assert nf.nf_param_count(b) == n
        assert np.array_equal(getp(b), saved)
        # both nets take the same next step
        train(a, X[100:], Y[100:], 0.5)
        train(b, X[100:], Y[100:], 0.5)
        assert np.array_equal(getp(a), getp(b))
    finally:
        nf.nf_net_destroy(a)
        if b is not None:
            nf.nf_net_destroy(b)


def test_load_a_file_written_elsewhere(tmp_path):
    """A file assembled by the test from the documented layout loads into a
    net with exactly those parameters."""
    from paper_1902_06714_amd import nf
    from .test_abi_cpu import _net_file
    params = [float(i) / 8 for i in range(3 * 2 + 2)]
    path = tmp_path / "net.bin"
    path.write_bytes(_net_file(dtype=0, dims=(3, 2), acts=(4,), params=params))
    note("load a file written by the test")
    h = nf.nf_load(str(path))
    try:
        assert np.array_equal(nf.nf_get_params(h), np.array(params, np.float32))
        assert nf.nf_net_dtype(h) == nf.NF_F32
    finally:
        nf.nf_net_destroy(h)
