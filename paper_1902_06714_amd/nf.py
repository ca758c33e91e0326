"""ctypes binding of include/nf.h: the same entry points, argument marshalling
only.  Every step of the computation runs in the HIP library; there is no
other implementation behind these functions.  Importing this module fails
loudly when the library has not been built.

Device buffers are passed as torch CUDA (HIP) tensors, which supply the device
pointer; streams default to torch's current stream.  Tensors must be
contiguous on the net's device, fp32 for the plain entry points and fp64 for
their _f64 twins (nets created with dtype NF_F64).
"""

from __future__ import annotations

import ctypes
import os
import re
from typing import Optional, Sequence, Union

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libnf.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "nf.h")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build the HIP library first "
        "(python -m paper_1902_06714_amd.build, or __graft_entry__.build())")

try:
    # load torch's HIP runtime first so that the library shares it (one HIP
    # runtime per process; see build.py)
    import torch  # noqa: F401
except ImportError:
    pass

_lib = ctypes.CDLL(LIB_PATH)

NF_GAUSSIAN, NF_RELU, NF_SIGMOID, NF_STEP, NF_TANH = 0, 1, 2, 3, 4
ACT_CODES = {"gaussian": NF_GAUSSIAN, "relu": NF_RELU, "sigmoid": NF_SIGMOID,
             "step": NF_STEP, "tanh": NF_TANH}
NF_OK, NF_EINVAL, NF_ESHAPE, NF_ENOMEM, NF_EDEVICE = 0, -1, -2, -3, -4
NF_F32, NF_F64 = 0, 1
STATUS_NAMES = {0: "NF_OK", -1: "NF_EINVAL", -2: "NF_ESHAPE", -3: "NF_ENOMEM", -4: "NF_EDEVICE"}

_c_i32p = ctypes.POINTER(ctypes.c_int32)
_c_f32p = ctypes.POINTER(ctypes.c_float)
_net_p = ctypes.c_void_p

class nf_kernel_stat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 64), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("bytes", ctypes.c_double),
                ("flops", ctypes.c_double), ("min_ms", ctypes.c_double),
                ("max_ms", ctypes.c_double)]


_sig = {
    "nf_net_create": (ctypes.c_int, [_c_i32p, ctypes.c_int32, _c_i32p, ctypes.c_int32,
                                     ctypes.POINTER(ctypes.c_void_p)]),
    "nf_net_create_ex": (ctypes.c_int, [_c_i32p, ctypes.c_int32, _c_i32p, ctypes.c_int32,
                                        ctypes.c_int32, ctypes.POINTER(ctypes.c_void_p)]),
    "nf_net_dtype": (ctypes.c_int32, [_net_p]),
    "nf_net_destroy": (ctypes.c_int, [_net_p]),
    "nf_param_count": (ctypes.c_int64, [_net_p]),
    "nf_set_params": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_int64]),
    "nf_get_params": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_int64]),
    "nf_get_grads": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_int64]),
    "nf_forward": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                  ctypes.c_void_p]),
    "nf_train_batch": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                      ctypes.c_float, ctypes.c_int32, ctypes.c_void_p]),
    "nf_train_batch_noalloc": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_int64, ctypes.c_float, ctypes.c_int32,
                                              ctypes.c_void_p]),
    "nf_train_epoch": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                      ctypes.c_int64, ctypes.c_float, ctypes.c_int32,
                                      ctypes.c_void_p]),
    "nf_train_single": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_float,
                                       ctypes.c_void_p]),
    "nf_train_windows": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                        ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                        ctypes.c_float, ctypes.c_int32, ctypes.c_void_p]),
    "nf_accuracy": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                   ctypes.POINTER(ctypes.c_int64), ctypes.c_void_p]),
    "nf_set_params_f64": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_int64]),
    "nf_get_params_f64": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_int64]),
    "nf_get_grads_f64": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_int64]),
    "nf_get_fprime": (ctypes.c_int, [_net_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64]),
    "nf_get_fprime_f64": (ctypes.c_int, [_net_p, ctypes.c_int32, ctypes.c_void_p,
                                         ctypes.c_int64]),
    "nf_forward_f64": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                      ctypes.c_void_p]),
    "nf_train_batch_f64": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_int64, ctypes.c_double, ctypes.c_int32,
                                          ctypes.c_void_p]),
    "nf_train_epoch_f64": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_int64, ctypes.c_int64, ctypes.c_double,
                                          ctypes.c_int32, ctypes.c_void_p]),
    "nf_train_single_f64": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_double, ctypes.c_void_p]),
    "nf_train_windows_f64": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                            ctypes.c_int64, ctypes.c_double, ctypes.c_int32,
                                            ctypes.c_void_p]),
    "nf_accuracy_f64": (ctypes.c_int, [_net_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                       ctypes.POINTER(ctypes.c_int64), ctypes.c_void_p]),
    "nf_save": (ctypes.c_int, [_net_p, ctypes.c_char_p]),
    "nf_load": (ctypes.c_int, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_void_p)]),
    "nf_profile": (ctypes.c_int, [_net_p, ctypes.c_int32]),
    "nf_profile_read": (ctypes.c_int, [_net_p, ctypes.POINTER(nf_kernel_stat), ctypes.c_int32,
                                       ctypes.POINTER(ctypes.c_int32)]),
    "nf_calib_read": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.POINTER(ctypes.c_double)]),
    "nf_calib_copy": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                     ctypes.c_void_p, ctypes.POINTER(ctypes.c_double)]),
    "nf_calib_mfma": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.POINTER(ctypes.c_double),
                                     ctypes.POINTER(ctypes.c_double),
                                     ctypes.POINTER(ctypes.c_double)]),
    "nf_calib_spin": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_double]),
    "nf_last_error": (ctypes.c_char_p, []),
}
for _name, (_res, _args) in _sig.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args


def declared_functions() -> list:
    """Names of the functions include/nf.h declares."""
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(nf_[a-z_]+)\s*\(", text)))


class NfError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = _lib.nf_last_error().decode(errors="replace")
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def _check(status: int, where: str) -> None:
    if status != NF_OK:
        raise NfError(status, where)


def _dev_ptr(t, name: str, f64: bool = False) -> int:
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor on the GPU")
    want = torch.float64 if f64 else torch.float32
    if t.dtype != want or not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {want} GPU tensor")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream or None
    if isinstance(stream, int):
        return stream or None
    return stream.cuda_stream or None


def nf_net_create(dims: Sequence[int], acts: Union[None, str, Sequence[str], Sequence[int]] = None,
                  dtype: int = NF_F32):
    """Returns an opaque handle (int).  acts: None (sigmoid everywhere), one
    name, or one per layer after the input.  dtype NF_F64 creates an fp64 net
    (nf_net_create_ex), driven with the _f64 functions."""
    d = (ctypes.c_int32 * len(dims))(*[int(v) for v in dims])
    if acts is None:
        codes = []
    elif isinstance(acts, str):
        codes = [ACT_CODES[acts]]
    else:
        codes = [ACT_CODES[a] if isinstance(a, str) else int(a) for a in acts]
    a = (ctypes.c_int32 * max(1, len(codes)))(*codes)
    out = ctypes.c_void_p()
    if dtype == NF_F32:
        _check(_lib.nf_net_create(d, len(dims), a if codes else None, len(codes),
                                  ctypes.byref(out)), "nf_net_create")
    else:
        _check(_lib.nf_net_create_ex(d, len(dims), a if codes else None, len(codes), int(dtype),
                                     ctypes.byref(out)), "nf_net_create_ex")
    return out.value


def nf_net_dtype(net) -> int:
    return int(_lib.nf_net_dtype(net))


def nf_net_destroy(net) -> None:
    _check(_lib.nf_net_destroy(net), "nf_net_destroy")


def nf_param_count(net) -> int:
    return int(_lib.nf_param_count(net))


def nf_set_params(net, params: np.ndarray) -> None:
    p = np.ascontiguousarray(params, dtype=np.float32)
    _check(_lib.nf_set_params(net, p.ctypes.data, p.size), "nf_set_params")


def nf_get_params(net) -> np.ndarray:
    out = np.empty(nf_param_count(net), dtype=np.float32)
    _check(_lib.nf_get_params(net, out.ctypes.data, out.size), "nf_get_params")
    return out


def nf_get_grads(net) -> np.ndarray:
    out = np.empty(nf_param_count(net), dtype=np.float32)
    _check(_lib.nf_get_grads(net, out.ctypes.data, out.size), "nf_get_grads")
    return out


def nf_get_fprime(net, layer: int, batch: int, width: int) -> np.ndarray:
    """f'(z_layer) [batch][width] of the last training step (width = d_layer)."""
    out = np.empty((batch, width), dtype=np.float32)
    _check(_lib.nf_get_fprime(net, layer, out.ctypes.data, batch), "nf_get_fprime")
    return out


def nf_forward(net, x, out, stream=None) -> None:
    """x: [batch][d_0] GPU tensor, out: [batch][d_L] GPU tensor."""
    _check(_lib.nf_forward(net, _dev_ptr(x, "x"), x.shape[0], _dev_ptr(out, "out"),
                           _stream(stream)), "nf_forward")


def nf_train_batch(net, x, y, eta: float, n_shards: int = 1, stream=None) -> None:
    _check(_lib.nf_train_batch(net, _dev_ptr(x, "x"), _dev_ptr(y, "y"), x.shape[0], float(eta),
                               int(n_shards), _stream(stream)), "nf_train_batch")


NF_NOALLOC_SCRATCH_BYTES = 48 << 20


def nf_train_batch_noalloc(net, x, y, eta: float, n_shards: int = 1, stream=None) -> None:
    """nf_train_batch on the library's scratch array (allocates nothing)."""
    _check(_lib.nf_train_batch_noalloc(net, _dev_ptr(x, "x"), _dev_ptr(y, "y"), x.shape[0],
                                       float(eta), int(n_shards), _stream(stream)),
           "nf_train_batch_noalloc")


def nf_train_epoch(net, x, y, batch: int, eta: float, n_shards: int = 1, stream=None) -> None:
    _check(_lib.nf_train_epoch(net, _dev_ptr(x, "x"), _dev_ptr(y, "y"), x.shape[0], int(batch),
                               float(eta), int(n_shards), _stream(stream)), "nf_train_epoch")


def nf_train_single(net, x, y, eta: float, stream=None) -> None:
    """x: [d_0] (or [1][d_0]), y: [d_L] GPU tensors."""
    _check(_lib.nf_train_single(net, _dev_ptr(x, "x"), _dev_ptr(y, "y"), float(eta),
                                _stream(stream)), "nf_train_single")


def nf_train_windows(net, x, y, batch: int, pos, eta: float, n_shards: int = 1,
                     stream=None) -> None:
    """One step per entry of pos (uniform numbers in [0, 1), host array) on
    the window of `batch` samples it places in (x, y)."""
    p = np.ascontiguousarray(pos, dtype=np.float32)
    _check(_lib.nf_train_windows(net, _dev_ptr(x, "x"), _dev_ptr(y, "y"), x.shape[0], int(batch),
                                 p.ctypes.data if p.size else None, p.size, float(eta),
                                 int(n_shards), _stream(stream)), "nf_train_windows")


def nf_accuracy(net, x, y, stream=None) -> int:
    """Number of samples whose output and target peak at the same index."""
    c = ctypes.c_int64()
    _check(_lib.nf_accuracy(net, _dev_ptr(x, "x"), _dev_ptr(y, "y"), x.shape[0], ctypes.byref(c),
                            _stream(stream)), "nf_accuracy")
    return int(c.value)


def nf_set_params_f64(net, params: np.ndarray) -> None:
    p = np.ascontiguousarray(params, dtype=np.float64)
    _check(_lib.nf_set_params_f64(net, p.ctypes.data, p.size), "nf_set_params_f64")


def nf_get_params_f64(net) -> np.ndarray:
    out = np.empty(nf_param_count(net), dtype=np.float64)
    _check(_lib.nf_get_params_f64(net, out.ctypes.data, out.size), "nf_get_params_f64")
    return out


def nf_get_grads_f64(net) -> np.ndarray:
    out = np.empty(nf_param_count(net), dtype=np.float64)
    _check(_lib.nf_get_grads_f64(net, out.ctypes.data, out.size), "nf_get_grads_f64")
    return out


def nf_get_fprime_f64(net, layer: int, batch: int, width: int) -> np.ndarray:
    out = np.empty((batch, width), dtype=np.float64)
    _check(_lib.nf_get_fprime_f64(net, layer, out.ctypes.data, batch), "nf_get_fprime_f64")
    return out


def nf_forward_f64(net, x, out, stream=None) -> None:
    _check(_lib.nf_forward_f64(net, _dev_ptr(x, "x", True), x.shape[0], _dev_ptr(out, "out", True),
                               _stream(stream)), "nf_forward_f64")


def nf_train_batch_f64(net, x, y, eta: float, n_shards: int = 1, stream=None) -> None:
    _check(_lib.nf_train_batch_f64(net, _dev_ptr(x, "x", True), _dev_ptr(y, "y", True), x.shape[0],
                                   float(eta), int(n_shards), _stream(stream)),
           "nf_train_batch_f64")


def nf_train_epoch_f64(net, x, y, batch: int, eta: float, n_shards: int = 1, stream=None) -> None:
    _check(_lib.nf_train_epoch_f64(net, _dev_ptr(x, "x", True), _dev_ptr(y, "y", True), x.shape[0],
                                   int(batch), float(eta), int(n_shards), _stream(stream)),
           "nf_train_epoch_f64")


def nf_train_single_f64(net, x, y, eta: float, stream=None) -> None:
    _check(_lib.nf_train_single_f64(net, _dev_ptr(x, "x", True), _dev_ptr(y, "y", True),
                                    float(eta), _stream(stream)), "nf_train_single_f64")


def nf_train_windows_f64(net, x, y, batch: int, pos, eta: float, n_shards: int = 1,
                         stream=None) -> None:
    p = np.ascontiguousarray(pos, dtype=np.float64)
    _check(_lib.nf_train_windows_f64(net, _dev_ptr(x, "x", True), _dev_ptr(y, "y", True),
                                     x.shape[0], int(batch), p.ctypes.data if p.size else None,
                                     p.size, float(eta), int(n_shards), _stream(stream)),
           "nf_train_windows_f64")


def nf_accuracy_f64(net, x, y, stream=None) -> int:
    c = ctypes.c_int64()
    _check(_lib.nf_accuracy_f64(net, _dev_ptr(x, "x", True), _dev_ptr(y, "y", True), x.shape[0],
                                ctypes.byref(c), _stream(stream)), "nf_accuracy_f64")
    return int(c.value)


def nf_save(net, path: str) -> None:
    _check(_lib.nf_save(net, os.fsencode(path)), "nf_save")


def nf_load(path: str):
    """Returns the handle of a new net created from the file."""
    out = ctypes.c_void_p()
    _check(_lib.nf_load(os.fsencode(path), ctypes.byref(out)), "nf_load")
    return out.value


def nf_profile(net, repeats: int) -> None:
    """0: off; R >= 1: record, running every launch R times between its events."""
    _check(_lib.nf_profile(net, int(repeats)), "nf_profile")


def nf_profile_read(net, cap: int = 64) -> list:
    """[{name, launches, total_ms, bytes, flops, min_ms, max_ms}], largest
    total time first."""
    buf = (nf_kernel_stat * cap)()
    n = ctypes.c_int32()
    _check(_lib.nf_profile_read(net, buf, cap, ctypes.byref(n)), "nf_profile_read")
    return [{"name": buf[i].name.decode(), "launches": buf[i].launches,
             "total_ms": buf[i].total_ms, "bytes": buf[i].bytes, "flops": buf[i].flops,
             "min_ms": buf[i].min_ms, "max_ms": buf[i].max_ms}
            for i in range(n.value)]


NF_CALIB_SINK_BYTES = 1 << 20


def nf_calib_read(src, sink, stream=None) -> float:
    """ms of one streaming read of the GPU tensor src (sink: a GPU tensor of at
    least NF_CALIB_SINK_BYTES bytes)."""
    ms = ctypes.c_double()
    _check(_lib.nf_calib_read(src.data_ptr(), src.numel() * src.element_size(), sink.data_ptr(),
                              _stream(stream), ctypes.byref(ms)), "nf_calib_read")
    return ms.value


def nf_calib_copy(dst, src, stream=None) -> float:
    ms = ctypes.c_double()
    _check(_lib.nf_calib_copy(dst.data_ptr(), src.data_ptr(), src.numel() * src.element_size(),
                              _stream(stream), ctypes.byref(ms)), "nf_calib_copy")
    return ms.value


def nf_calib_mfma(dtype: int, iters: int, sink, stream=None):
    """(ms, flops, shader clock GHz) of the matrix-core loop."""
    ms, fl, ghz = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(_lib.nf_calib_mfma(dtype, iters, sink.data_ptr(), _stream(stream), ctypes.byref(ms),
                              ctypes.byref(fl), ctypes.byref(ghz)), "nf_calib_mfma")
    return ms.value, fl.value, ghz.value


def nf_calib_spin(us: float, stream=None) -> None:
    """Hold the stream for `us` microseconds (returns at once)."""
    _check(_lib.nf_calib_spin(_stream(stream), float(us)), "nf_calib_spin")


def nf_last_error() -> str:
    return _lib.nf_last_error().decode(errors="replace")


def raw():
    """The loaded library, for calls with raw pointers."""
    return _lib
