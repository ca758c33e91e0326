"""The C ABI library on a machine without a GPU: it loads, exports every
function include/nf.h declares, rejects bad arguments before touching the
device, and reports a missing device as an error instead of falling back."""

import ctypes
import os

import pytest

from paper_1902_06714_amd import nf


def _gpu_present() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def test_every_declared_function_is_exported():
    names = nf.declared_functions()
    assert {"nf_net_create", "nf_net_destroy", "nf_param_count", "nf_set_params",
            "nf_get_params", "nf_get_grads", "nf_forward", "nf_train_batch",
            "nf_train_epoch", "nf_profile", "nf_profile_read", "nf_last_error"} <= set(names)
    lib = nf.raw()
    for n in names:
        assert hasattr(lib, n), f"{n} declared in nf.h but not exported"


def test_header_is_plain_c():
    import subprocess
    res = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-fsyntax-only", "-x", "c",
                          nf.HEADER], capture_output=True, text=True)
    assert res.returncode == 0, res.stderr


def _create(dims, acts):
    d = (ctypes.c_int32 * max(1, len(dims)))(*dims)
    a = (ctypes.c_int32 * max(1, len(acts)))(*acts)
    out = ctypes.c_void_p(12345)
    st = nf.raw().nf_net_create(d if dims else None, len(dims), a if acts else None, len(acts),
                                ctypes.byref(out))
    return st, out.value


@pytest.mark.parametrize("dims,acts,expect", [
    ([784], [], nf.NF_ESHAPE),                       # no output layer
    ([], [], nf.NF_EINVAL),                          # NULL dims
    ([4, 0, 2], [], nf.NF_ESHAPE),                   # empty layer
    ([4, -3, 2], [], nf.NF_ESHAPE),
    ([4, 70000, 2], [], nf.NF_ESHAPE),               # layer too wide
    ([4, 3, 2], [2, 2, 2], nf.NF_ESHAPE),            # n_acts neither 0, 1 nor n_dims - 1
    ([4, 3, 2], [7], nf.NF_EINVAL),                  # unknown activation
    ([4, 3, 2], [-1, 2], nf.NF_EINVAL),
])
def test_create_rejects_bad_arguments(dims, acts, expect):
    st, handle = _create(dims, acts)
    assert st == expect, nf.nf_last_error()
    assert handle == 12345, "out must not be written on error"
    assert nf.nf_last_error() != ""


@pytest.mark.parametrize("dtype,expect", [(2, nf.NF_EINVAL), (-1, nf.NF_EINVAL)])
def test_create_ex_rejects_unknown_dtype(dtype, expect):
    d = (ctypes.c_int32 * 3)(4, 3, 2)
    out = ctypes.c_void_p(12345)
    assert nf.raw().nf_net_create_ex(d, 3, None, 0, dtype, ctypes.byref(out)) == expect
    assert out.value == 12345


def test_create_null_out():
    d = (ctypes.c_int32 * 2)(3, 2)
    assert nf.raw().nf_net_create(d, 2, None, 0, None) == nf.NF_EINVAL


def test_null_net_calls():
    lib = nf.raw()
    assert lib.nf_param_count(None) == -1
    assert lib.nf_net_destroy(None) == nf.NF_OK
    buf = (ctypes.c_float * 4)()
    assert lib.nf_set_params(None, buf, 4) == nf.NF_EINVAL
    assert lib.nf_get_params(None, buf, 4) == nf.NF_EINVAL
    assert lib.nf_get_grads(None, buf, 4) == nf.NF_EINVAL
    assert lib.nf_forward(None, buf, 1, buf, None) == nf.NF_EINVAL
    assert lib.nf_train_batch(None, buf, buf, 1, 1.0, 1, None) == nf.NF_EINVAL
    assert lib.nf_train_epoch(None, buf, buf, 1, 1, 1.0, 1, None) == nf.NF_EINVAL
    assert lib.nf_train_single(None, buf, buf, 1.0, None) == nf.NF_EINVAL
    assert lib.nf_train_windows(None, buf, buf, 4, 1, buf, 1, 1.0, 1, None) == nf.NF_EINVAL
    cnt = ctypes.c_int64()
    assert lib.nf_accuracy(None, buf, buf, 1, ctypes.byref(cnt), None) == nf.NF_EINVAL
    assert lib.nf_net_dtype(None) == -1
    dbuf = (ctypes.c_double * 4)()
    assert lib.nf_set_params_f64(None, dbuf, 4) == nf.NF_EINVAL
    assert lib.nf_get_params_f64(None, dbuf, 4) == nf.NF_EINVAL
    assert lib.nf_get_grads_f64(None, dbuf, 4) == nf.NF_EINVAL
    assert lib.nf_forward_f64(None, dbuf, 1, dbuf, None) == nf.NF_EINVAL
    assert lib.nf_train_batch_f64(None, dbuf, dbuf, 1, 1.0, 1, None) == nf.NF_EINVAL
    assert lib.nf_train_epoch_f64(None, dbuf, dbuf, 1, 1, 1.0, 1, None) == nf.NF_EINVAL
    assert lib.nf_train_single_f64(None, dbuf, dbuf, 1.0, None) == nf.NF_EINVAL
    assert lib.nf_train_windows_f64(None, dbuf, dbuf, 4, 1, dbuf, 1, 1.0, 1, None) == nf.NF_EINVAL
    assert lib.nf_accuracy_f64(None, dbuf, dbuf, 1, ctypes.byref(cnt), None) == nf.NF_EINVAL


@pytest.mark.skipif(_gpu_present(), reason="checks the behaviour without a GPU")
def test_no_device_is_an_error_not_a_fallback():
    st, _ = _create([784, 30, 10], [])
    assert st == nf.NF_EDEVICE
    assert "device" in nf.nf_last_error().lower()


def test_one_hip_runtime_per_process():
    """The binding loads the library after torch, so both share one HIP runtime
    (two runtimes in one process collide on the device)."""
    import subprocess
    import sys
    code = ("import paper_1902_06714_amd.nf, torch\n"
            "maps = open('/proc/self/maps').read().split('\\n')\n"
            "print(len({l.split()[-1] for l in maps if 'libamdhip64' in l}))\n")
    res = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                         cwd=__import__("os").path.dirname(nf.LIB_PATH) + "/..")
    assert res.returncode == 0, res.stderr
    assert res.stdout.strip() == "1"


def _net_file(dtype=0, dims=(3, 2), acts=(2,), params=None, magic=b"NFNET01\n", count=None,
              corrupt_hash=False, extra=b""):
    """A network file written by the test itself, following the layout
    include/nf.h documents."""
    import struct
    n = sum(dims[l] * dims[l - 1] + dims[l] for l in range(1, len(dims)))
    params = [0.5] * n if params is None else params
    body = magic + struct.pack("<ii", dtype, len(dims)) + struct.pack(f"<{len(dims)}i", *dims)
    body += struct.pack(f"<{len(acts)}i", *acts) + struct.pack("<q", n if count is None else count)
    body += struct.pack(f"<{len(params)}{'d' if dtype else 'f'}", *params)
    h = 1469598103934665603
    for b in body:
        h = ((h ^ b) * 1099511628211) & 0xFFFFFFFFFFFFFFFF
    if corrupt_hash:
        h ^= 1
    return body + struct.pack("<Q", h) + extra


@pytest.mark.parametrize("case", ["missing", "magic", "count", "hash", "trailing", "truncated",
                                  "dtype", "layers"])
def test_load_rejects_bad_files(tmp_path, case):
    path = tmp_path / "net.bin"
    if case == "magic":
        path.write_bytes(_net_file(magic=b"NFNET02\n"))
    elif case == "count":
        path.write_bytes(_net_file(count=7))
    elif case == "hash":
        path.write_bytes(_net_file(corrupt_hash=True))
    elif case == "trailing":
        path.write_bytes(_net_file(extra=b"\0"))
    elif case == "truncated":
        path.write_bytes(_net_file()[:-3])
    elif case == "dtype":
        path.write_bytes(_net_file(dtype=5))
    elif case == "layers":
        path.write_bytes(_net_file(dims=(3,), acts=()))
    out = ctypes.c_void_p(12345)
    st = nf.raw().nf_load(str(path).encode(), ctypes.byref(out))
    assert st == nf.NF_EINVAL, nf.nf_last_error()
    assert out.value == 12345
    assert nf.nf_last_error() != ""


@pytest.mark.skipif(_gpu_present(), reason="checks the behaviour without a GPU")
def test_load_of_a_valid_file_needs_a_device(tmp_path):
    path = tmp_path / "net.bin"
    path.write_bytes(_net_file())
    out = ctypes.c_void_p(12345)
    assert nf.raw().nf_load(str(path).encode(), ctypes.byref(out)) == nf.NF_EDEVICE


def test_save_rejects_null():
    assert nf.raw().nf_save(None, b"/tmp/x") == nf.NF_EINVAL


C_PROGRAM = r"""
#include <stdio.h>
#include "nf.h"
int main(void) {
  int32_t bad[2] = {784, 0};
  nf_net* net = NULL;
  if (nf_net_create(bad, 2, NULL, 0, &net) != NF_ESHAPE || net != NULL) return 1;
  if (nf_last_error()[0] == '\0') return 2;
  int32_t dims[3] = {784, 30, 10};
  nf_status st = nf_net_create(dims, 3, NULL, 0, &net);
  if (st == NF_OK) {
    if (nf_param_count(net) != 784 * 30 + 30 + 30 * 10 + 10) return 3;
    nf_net_destroy(net);
    puts("created");
    return 0;
  }
  if (st == NF_EDEVICE) {
    puts("no device");
    return 0;
  }
  return 4;
}
"""


def test_plain_c_program_links_and_calls_the_library(tmp_path):
    """The ABI used from C, without Python: a program built with gcc against
    include/nf.h and linked to the library validates a bad net, then creates
    one (or reports the missing device) through the same entry points."""
    import subprocess
    src = tmp_path / "prog.c"
    src.write_text(C_PROGRAM)
    exe = tmp_path / "prog"
    libdir = os.path.dirname(nf.LIB_PATH)
    res = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.dirname(nf.HEADER),
                          str(src), "-L", libdir, "-lnf", f"-Wl,-rpath,{libdir}", "-o", str(exe)],
                         capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, (run.returncode, run.stdout, run.stderr)
    assert run.stdout.strip() in ("created", "no device")
