"""Drive the GPU library through its ctypes binding for the parity tests."""

from __future__ import annotations

import sys
from typing import Callable, List, Optional, Sequence

import numpy as np


def note(msg: str) -> None:
    """Name the case about to run on the GPU (flushed, so it survives a crash)."""
    print(f"[gpu] {msg}", file=sys.stderr, flush=True)


def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a visible HIP device")
    return torch


def to_dev(a: np.ndarray):
    torch = torch_cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda")


class GpuNet:
    """A network on the GPU, owned for the duration of a with-block."""

    def __init__(self, dims: Sequence[int], acts, theta: np.ndarray):
        from paper_1902_06714_amd import nf
        self.nf = nf
        self.dims = list(dims)
        self.h = nf.nf_net_create(dims, list(acts))
        nf.nf_set_params(self.h, theta)

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.nf.nf_net_destroy(self.h)

    def params(self) -> np.ndarray:
        return self.nf.nf_get_params(self.h)

    def grads(self) -> np.ndarray:
        return self.nf.nf_get_grads(self.h)

    def train_batch(self, xd, yd, eta, shards=1):
        self.nf.nf_train_batch(self.h, xd, yd, eta, shards)

    def train_epoch(self, xd, yd, batch, eta, shards=1):
        self.nf.nf_train_epoch(self.h, xd, yd, batch, eta, shards)

    def forward(self, xd) -> np.ndarray:
        torch = torch_cuda()
        out = torch.empty((xd.shape[0], self.dims[-1]), dtype=torch.float32, device="cuda")
        self.nf.nf_forward(self.h, xd, out)
        torch.cuda.synchronize()
        return out.cpu().numpy()


def trajectory(dims, acts, theta0, X, Y, batch, eta, shards, steps,
               each: Optional[Callable] = None):
    """Train on consecutive batches on the GPU, calling each(t, params, grads,
    net) after every step.  Returns the final parameters."""
    xd, yd = to_dev(X[:batch * steps]), to_dev(Y[:batch * steps])
    with GpuNet(dims, acts, theta0) as net:
        for t in range(steps):
            net.train_batch(xd[t * batch:(t + 1) * batch], yd[t * batch:(t + 1) * batch], eta,
                            shards)
            if each is not None:
                each(t, net.params(), net.grads(), net)
        return net.params()
