"""Seeded synthetic workloads for mini-batch MLP training.

This module only draws numbers: it holds the network shapes, the training
schedules and a counter-based generator for inputs, labels and initial
parameters. It contains none of the method's arithmetic (no forward pass,
no gradient, no update), so both the GPU path and the CPU reference can take
their inputs from it without sharing any computation.

Generator (documented so that any side can reproduce it bit for bit):

* bit source: SplitMix64 (Steele, Lea and Flood, "Fast splittable
  pseudorandom number generators", OOPSLA 2014).  A stream is keyed by
  ``key = mix(mix(seed) + stream)`` and its i-th 64-bit word is
  ``mix(key + (i + 1) * 0x9E3779B97F4A7C15)``, i.e. the SplitMix64 sequence
  started from state ``key``.
* uniform float in [0, 1): ``(u >> 40) * 2**-24`` (exact in fp32).
* normal: Box-Muller (Box and Muller, 1958) in fp64 on the word pair
  (2j, 2j + 1), giving normals 2j (cosine branch) and 2j + 1 (sine branch),
  each rounded to fp32 after any scaling.
* class label in {0..9}: ``((u >> 32) * 10) >> 32``.

Streams: 0 training inputs, 1 training labels, 3 held-out inputs,
4 held-out labels, 5 the uniform numbers that place random mini-batch
windows (one per step), 100 + 2l the weights of layer l (1-based), 101 + 2l the
biases of layer l.

The paper trains on MNIST (28x28 greyscale digits scaled to [0, 1], one-hot
labels over 10 classes, section 4).  That dataset is not available here; the
uniform [0, 1) 784-vectors with one-hot labels below stand in for it with the
same shapes and value range.  No MNIST item is reproduced.
"""

from __future__ import annotations

import dataclasses
from typing import List, Sequence, Tuple

import numpy as np

GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

STREAM_X_TRAIN = 0
STREAM_Y_TRAIN = 1
STREAM_X_HELDOUT = 3
STREAM_Y_HELDOUT = 4
STREAM_WINDOWS = 5

# activation names, in the order of the C enum nf_act
ACTIVATIONS = ("gaussian", "relu", "sigmoid", "step", "tanh")

_CHUNK = 1 << 22


def _mix(z: np.ndarray) -> np.ndarray:
    """SplitMix64 output function on a uint64 array (wrapping arithmetic)."""
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        return z ^ (z >> np.uint64(31))


def stream_key(seed: int, stream: int) -> np.uint64:
    s = _mix(np.array([seed & 0xFFFFFFFFFFFFFFFF], dtype=np.uint64))
    with np.errstate(over="ignore"):
        s = s + np.uint64(stream & 0xFFFFFFFFFFFFFFFF)
    return _mix(s)[0]


def words(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """64-bit words start .. start+count-1 of stream (seed, stream)."""
    key = stream_key(seed, stream)
    idx = np.arange(start + 1, start + count + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return _mix(key + idx * GOLDEN)


def uniform(seed: int, stream: int, n: int) -> np.ndarray:
    """n fp32 values in [0, 1), a multiple of 2**-24."""
    out = np.empty(n, dtype=np.float32)
    for s in range(0, n, _CHUNK):
        c = min(_CHUNK, n - s)
        u = words(seed, stream, s, c)
        out[s:s + c] = (u >> np.uint64(40)).astype(np.float64) * (2.0 ** -24)
    return out


def normal(seed: int, stream: int, n: int, scale: float = 1.0) -> np.ndarray:
    """n fp32 normals N(0, scale**2): Box-Muller in fp64, scaled, rounded once."""
    out = np.empty(n, dtype=np.float32)
    npairs = (n + 1) // 2
    step = _CHUNK // 2
    for p0 in range(0, npairs, step):
        pc = min(step, npairs - p0)
        w = words(seed, stream, 2 * p0, 2 * pc)
        u1 = ((w[0::2] >> np.uint64(11)).astype(np.float64) + 1.0) * (2.0 ** -53)
        u2 = (w[1::2] >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)
        r = np.sqrt(-2.0 * np.log(u1))
        t = 2.0 * np.pi * u2
        z = np.empty(2 * pc, dtype=np.float64)
        z[0::2] = r * np.cos(t)
        z[1::2] = r * np.sin(t)
        lo, hi = 2 * p0, min(n, 2 * (p0 + pc))
        out[lo:hi] = (z[:hi - lo] * scale).astype(np.float32)
    return out


def labels(seed: int, stream: int, n: int, classes: int = 10) -> np.ndarray:
    out = np.empty(n, dtype=np.int64)
    for s in range(0, n, _CHUNK):
        c = min(_CHUNK, n - s)
        u = words(seed, stream, s, c)
        with np.errstate(over="ignore"):
            out[s:s + c] = ((u >> np.uint64(32)) * np.uint64(classes)) >> np.uint64(32)
    return out


def window_positions(seed: int, n_steps: int) -> np.ndarray:
    """The uniform numbers in [0, 1) that place the mini-batch window of each
    of n_steps random-window steps."""
    return uniform(seed, STREAM_WINDOWS, n_steps)


def one_hot(lbl: np.ndarray, classes: int = 10) -> np.ndarray:
    y = np.zeros((lbl.shape[0], classes), dtype=np.float32)
    y[np.arange(lbl.shape[0]), lbl] = 1.0
    return y


@dataclasses.dataclass(frozen=True)
class Workload:
    """One training configuration: network shape, data recipe and schedule."""

    name: str
    dims: Tuple[int, ...]
    acts: Tuple[str, ...]          # one per layer after the input
    n_samples: int
    batch: int
    steps: int
    eta: float
    shards: int
    input_dist: str                # "uniform" in [0,1) or "normal" N(0,1)
    init: str                      # "fan_in": N(0,1)/sqrt(fan_in); "he": N(0, 2/fan_in)
    data_seed: int
    param_seed: int
    heldout: int = 0               # held-out samples for batched inference

    @property
    def n_layers(self) -> int:
        return len(self.dims) - 1

    def param_count(self) -> int:
        return sum(self.dims[l] * self.dims[l - 1] + self.dims[l]
                   for l in range(1, len(self.dims)))


WORKLOADS = {
    # 784-30-10 sigmoid, the paper's MNIST network (section 4), small case
    "c1": Workload("c1", (784, 30, 10), ("sigmoid", "sigmoid"), 1000, 100, 10,
                   3.0, 1, "uniform", "fan_in", 0, 0),
    # same network, one epoch of 60 batches of 1000 plus inference on 10000
    "c2": Workload("c2", (784, 30, 10), ("sigmoid", "sigmoid"), 60000, 1000, 60,
                   3.0, 1, "uniform", "fan_in", 0, 0, heldout=10000),
    # two tanh hidden layers, batch split into 16 shards summed in order
    "c3": Workload("c3", (784, 100, 100, 10), ("tanh", "tanh", "sigmoid"), 60000,
                   10000, 6, 1.0, 16, "uniform", "fan_in", 0, 0),
    # three 1024-wide relu hidden layers
    "c4": Workload("c4", (784, 1024, 1024, 1024, 10),
                   ("relu", "relu", "relu", "sigmoid"), 65536, 4096, 16, 0.1, 1,
                   "uniform", "he", 0, 1),
    # three 4096-wide relu hidden layers on N(0,1) inputs
    "c5": Workload("c5", (4096, 4096, 4096, 4096, 10),
                   ("relu", "relu", "relu", "sigmoid"), 32768, 8192, 4, 0.01, 1,
                   "normal", "he", 0, 1),
}


def init_params(dims: Sequence[int], init: str, seed: int) -> np.ndarray:
    """Initial parameters in canonical order: for l = 1..L, W_l row-major
    [d_l][d_{l-1}], then b_l[d_l].  Weights are N(0,1) times 1/sqrt(fan_in)
    ("fan_in") or sqrt(2/fan_in) ("he"); biases are N(0,1) as in the paper's
    layer constructor (section 3.1)."""
    parts: List[np.ndarray] = []
    for l in range(1, len(dims)):
        fan_in, fan_out = dims[l - 1], dims[l]
        if init == "fan_in":
            scale = 1.0 / np.sqrt(fan_in)
        elif init == "he":
            scale = np.sqrt(2.0 / fan_in)
        else:
            raise ValueError(f"unknown init {init!r}")
        parts.append(normal(seed, 100 + 2 * l, fan_out * fan_in, scale))
        parts.append(normal(seed, 101 + 2 * l, fan_out, 1.0))
    return np.concatenate(parts).astype(np.float32, copy=False)


def inputs(dist: str, seed: int, stream: int, n: int, dim: int) -> np.ndarray:
    if dist == "uniform":
        return uniform(seed, stream, n * dim).reshape(n, dim)
    if dist == "normal":
        return normal(seed, stream, n * dim).reshape(n, dim)
    raise ValueError(f"unknown input distribution {dist!r}")


def make_data(w: Workload, n: int | None = None, heldout: bool = False):
    """(X [n][d_0] fp32, Y [n][d_L] fp32 one-hot) for the training set, or the
    held-out set.  ``n`` truncates to the first n samples (same values)."""
    if heldout:
        n = w.heldout if n is None else n
        xs, ys = STREAM_X_HELDOUT, STREAM_Y_HELDOUT
    else:
        n = w.n_samples if n is None else n
        xs, ys = STREAM_X_TRAIN, STREAM_Y_TRAIN
    x = inputs(w.input_dist, w.data_seed, xs, n, w.dims[0])
    y = one_hot(labels(w.data_seed, ys, n, w.dims[-1]), w.dims[-1])
    return x, y


def make_params(w: Workload) -> np.ndarray:
    return init_params(w.dims, w.init, w.param_seed)
