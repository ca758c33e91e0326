"""CPU reference ("oracle") for mini-batch training of a fully connected
feed-forward network, written from Curcic, "A parallel Fortran framework for
neural networks and deep learning" (arXiv:1902.06714).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the tests, the smoke check in ``__graft_entry__``
and the CPU-baseline leg of ``bench.py`` use it.  It shares no code with the
GPU library; both sides take their inputs from the seeded generators.

Arithmetic: every quantity is computed in fp64 from the stored values.  The
network state (weights and biases) is stored in fp32, the paper's default
``real32`` kind (section 3.1, layer definition), so ``precision="f32"``
rounds the parameters to fp32 once after each update; ``precision="f64"``
keeps them in fp64 (the paper's ``real64`` kind) and is used by the
finite-difference and invariant checks.

Notation: the network has L = len(dims) - 1 layers after the input.  Layer l
(1-based in the text, index l-1 in the Python lists) holds W_l with shape
[d_l][d_{l-1}] and b_l with shape [d_l].  The paper keeps w(this, next) on the
source layer in column-major order (section 3.1); that array has the same
bytes as row-major W_l[d_l][d_{l-1}].  The canonical flat layout is, for
l = 1..L, W_l row-major followed by b_l; the input layer's bias and the last
layer's weights of the paper's layer objects are never used and are not
stored.

Readings of points the paper leaves open (each is listed in the design notes):

* update scale: the tendencies summed over a mini-batch of B samples are
  applied as theta <- theta - (eta / B) * sum, with B the whole mini-batch
  (also when the batch is split into shards).  The paper omits the body of its
  update and of train_batch (section 3.3 and 3.4); the mean step is the one
  for which eta = 3 with B = 1000 trains the 784-30-10 sigmoid network
  (section 4).  A batch of B copies of one sample then gives exactly the
  single-sample step with the same eta.
* cost: C = sum over samples of 1/2 ||a_L - y||^2, whose output delta is
  (a_L - y) * f'(z_L) (backprop listing, section 3.3).
* activations: only the sigmoid is written out in the paper (section 3.1);
  the others named in section 2 are read as tanh(x) with 1 - tanh(x)^2,
  max(0, x) with derivative 1 for x > 0 else 0, exp(-x^2) with -2x exp(-x^2),
  and the step 1 for x > 0 else 0 with derivative 0.
* one activation per layer (the paper uses one for the whole network; a list
  with equal entries is the paper's case).
* shards: the batch is split into S equal contiguous pieces; piece k holds
  samples [k B/S, (k+1) B/S) and the per-piece tendencies are summed in the
  order k = 0, 1, ..., S-1 (the collective sum of section 3.5).
"""

from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np

ACT_NAMES = ("gaussian", "relu", "sigmoid", "step", "tanh")


# ---------------------------------------------------------------------------
# activation functions and their derivatives (section 2 lists them; section
# 3.1 defines the sigmoid); all in fp64
# ---------------------------------------------------------------------------

def _sigmoid(z: np.ndarray) -> np.ndarray:
    # 1 / (1 + exp(-z)), evaluated without overflow for either sign of z
    e = np.exp(-np.abs(z))
    return np.where(z >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def act(name: str, z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, dtype=np.float64)
    if name == "sigmoid":
        return _sigmoid(z)
    if name == "tanh":
        return np.tanh(z)
    if name == "relu":
        return np.where(z > 0, z, 0.0)
    if name == "gaussian":
        return np.exp(-z * z)
    if name == "step":
        return np.where(z > 0, 1.0, 0.0)
    raise ValueError(f"unknown activation {name!r}")


def act_prime(name: str, z: np.ndarray) -> np.ndarray:
    """Derivative of the activation, evaluated at the pre-activation z (the
    paper applies activation_prime to the stored z, backprop listing)."""
    z = np.asarray(z, dtype=np.float64)
    if name == "sigmoid":
        # sigma'(z) = sigma(z) (1 - sigma(z)) = sigma(z) sigma(-z)
        return _sigmoid(z) * _sigmoid(-z)
    if name == "tanh":
        # 1 - tanh(z)^2 = 1 / cosh(z)^2
        with np.errstate(over="ignore"):
            c = np.cosh(z)
        return 1.0 / (c * c)
    if name == "relu":
        return np.where(z > 0, 1.0, 0.0)
    if name == "gaussian":
        return -2.0 * z * np.exp(-z * z)
    if name == "step":
        return np.zeros_like(z)
    raise ValueError(f"unknown activation {name!r}")


# ---------------------------------------------------------------------------
# parameters
# ---------------------------------------------------------------------------

def param_count(dims: Sequence[int]) -> int:
    return sum(dims[l] * dims[l - 1] + dims[l] for l in range(1, len(dims)))


def unpack(theta: np.ndarray, dims: Sequence[int]) -> List[Tuple[np.ndarray, np.ndarray]]:
    """Flat canonical vector -> [(W_1, b_1), ..., (W_L, b_L)] in fp64."""
    theta = np.asarray(theta)
    if theta.shape != (param_count(dims),):
        raise ValueError("parameter vector has the wrong length")
    out, off = [], 0
    for l in range(1, len(dims)):
        n, k = dims[l], dims[l - 1]
        W = theta[off:off + n * k].astype(np.float64).reshape(n, k)
        off += n * k
        b = theta[off:off + n].astype(np.float64)
        off += n
        out.append((W, b))
    return out


def pack(layers: Sequence[Tuple[np.ndarray, np.ndarray]]) -> np.ndarray:
    return np.concatenate([np.concatenate([W.ravel(), b.ravel()]) for W, b in layers])


def _check_acts(acts: Sequence[str], dims: Sequence[int]) -> List[str]:
    acts = list(acts)
    if len(acts) == 1:
        acts = acts * (len(dims) - 1)
    if len(acts) != len(dims) - 1:
        raise ValueError("need one activation per layer after the input")
    for a in acts:
        if a not in ACT_NAMES:
            raise ValueError(f"unknown activation {a!r}")
    return acts


def _round(theta: np.ndarray, precision: str) -> np.ndarray:
    if precision == "f32":
        return theta.astype(np.float32)
    if precision == "f64":
        return theta.astype(np.float64)
    raise ValueError(precision)


# ---------------------------------------------------------------------------
# one sample at a time: forward propagation, back-propagation, single-sample
# training (sections 3.2, 3.3 and 3.4)
# ---------------------------------------------------------------------------

def fwdprop(theta, dims, acts, x):
    """Forward propagation of one sample (Eq. 1-2, section 3.2).
    Returns (z, a): z[l] and a[l] for l = 0..L; a[0] = x, z[0] unused."""
    acts = _check_acts(acts, dims)
    layers = unpack(theta, dims)
    a = [np.asarray(x, dtype=np.float64)]
    z = [None]
    for l, (W, b) in enumerate(layers):
        zl = W @ a[-1] + b            # weighted sum of the previous activations plus bias
        z.append(zl)
        a.append(act(acts[l], zl))
    return z, a


def backprop(theta, dims, acts, z, a, y):
    """Tendencies of one sample (section 3.3): the output delta
    (a_L - y) f'(z_L); each hidden delta is the transposed weights of the
    next layer times the next delta, times f'(z_l); the weight tendency of
    layer l is the outer product of its delta with the previous activation and
    the bias tendency is the delta itself.  Nothing is modified.
    Returns (dW, db), lists indexed like the layers."""
    acts = _check_acts(acts, dims)
    layers = unpack(theta, dims)
    L = len(layers)
    y = np.asarray(y, dtype=np.float64)
    dW: List[np.ndarray] = [None] * L
    db: List[np.ndarray] = [None] * L
    delta = (a[L] - y) * act_prime(acts[L - 1], z[L])
    for l in range(L - 1, -1, -1):          # layer l+1 in 1-based notation
        db[l] = delta
        dW[l] = np.outer(delta, a[l])
        if l > 0:
            W = layers[l][0]                # weights into layer l+1 (pre-update)
            delta = (W.T @ delta) * act_prime(acts[l - 1], z[l])
    return dW, db


def sample_gradient(theta, dims, acts, x, y) -> np.ndarray:
    """Flat canonical fp64 vector of one sample's tendencies."""
    z, a = fwdprop(theta, dims, acts, x)
    dW, db = backprop(theta, dims, acts, z, a, y)
    return pack(list(zip(dW, db)))


def train_single(theta, dims, acts, x, y, eta, precision="f32") -> np.ndarray:
    """fwdprop, backprop, update for one sample (section 3.4)."""
    g = sample_gradient(theta, dims, acts, x, y)
    return _round(np.asarray(theta, dtype=np.float64) - eta * g, precision)


# ---------------------------------------------------------------------------
# a mini-batch: the same per-sample steps for every sample, stacked as rows
# ---------------------------------------------------------------------------

def forward(theta, dims, acts, X):
    """Forward propagation of every row of X [B][d_0] (each row is one
    sample's Eq. 2).  Returns (Z, A) lists of [B][d_l] fp64 arrays."""
    acts = _check_acts(acts, dims)
    layers = unpack(theta, dims)
    A = [np.asarray(X, dtype=np.float64)]
    Z = [None]
    for l, (W, b) in enumerate(layers):
        Zl = A[-1] @ W.T + b
        Z.append(Zl)
        A.append(act(acts[l], Zl))
    return Z, A


def output(theta, dims, acts, X) -> np.ndarray:
    """Network output for every row of X, storing nothing (the pure output
    function used for inference, section 3.2)."""
    return forward(theta, dims, acts, X)[1][-1]


def cost(theta, dims, acts, X, Y) -> float:
    """Quadratic cost summed over the samples: sum_s 1/2 ||a_L(x_s) - y_s||^2."""
    d = output(theta, dims, acts, X) - np.asarray(Y, dtype=np.float64)
    return 0.5 * float(np.sum(d * d))


def _kink_side(name: str, Z: np.ndarray, fp: np.ndarray, kink_tol: float) -> np.ndarray:
    """The other admissible derivative for relu units whose pre-activation lies
    within kink_tol * rms(z of the layer) of the kink at zero: a computation
    that rounds z may land on either side, and both results are correct."""
    if kink_tol <= 0.0 or name != "relu":
        return fp
    near = kink_band(Z, kink_tol)
    return np.where(near, 1.0 - fp, fp)


def kink_band(Z: np.ndarray, kink_tol: float) -> np.ndarray:
    """Mask of the units of one layer's pre-activations Z [B][d] that lie
    within kink_tol * rms(Z) of the relu kink (see _kink_side)."""
    Z = np.asarray(Z, dtype=np.float64)
    return np.abs(Z) <= kink_tol * np.sqrt(np.mean(Z * Z))


def piece_gradient(theta, dims, acts, X, Y, kink_tol: float = 0.0, sides=None) -> np.ndarray:
    """Tendencies summed over the samples of one piece of a batch: for each
    layer, sum over samples s of delta_s (outer) a_s, and sum of delta_s.
    The delta recurrences are the single-sample ones, applied to each row.
    kink_tol > 0 takes the other side of the relu kink for units within that
    relative distance of it (used to measure how much a result depends on
    those undetermined decisions); kink_tol = 0 is the method itself.
    sides[l-1], where given (rows like X), is the relu derivative to use for
    layer l in place of the method's own (see batch_gradient)."""
    acts = _check_acts(acts, dims)
    layers = unpack(theta, dims)
    L = len(layers)
    sides = list(sides) if sides is not None else [None] * L
    Z, A = forward(theta, dims, acts, X)
    Yd = np.asarray(Y, dtype=np.float64)

    def fprime(l):                      # f' of layer l (1-based)
        if sides[l - 1] is not None:
            return np.asarray(sides[l - 1], dtype=np.float64)
        return _kink_side(acts[l - 1], Z[l], act_prime(acts[l - 1], Z[l]), kink_tol)

    parts: List[Tuple[np.ndarray, np.ndarray]] = [None] * L
    D = (A[L] - Yd) * fprime(L)
    for l in range(L - 1, -1, -1):
        parts[l] = (D.T @ A[l], D.sum(axis=0))              # sum_s delta_s a_s^T, sum_s delta_s
        if l > 0:
            W = layers[l][0]
            D = (D @ W) * fprime(l)
    return pack(parts)


def kink_sides(theta, dims, acts, X, kink_tol: float, given) -> list:
    """The relu derivative of every layer when the units within kink_tol *
    rms(z of the layer over the batch) of the kink take the sides in given
    (given[l-1]: rows like X, nonzero where the unit counts as above the
    kink; None keeps the method's own decisions for that layer).  Units
    outside that band keep the method's own decision 1[z > 0].  Entries are
    None for layers whose activation is not relu."""
    acts = _check_acts(acts, dims)
    Z, _ = forward(theta, dims, acts, X)
    out = []
    for l, a in enumerate(acts):
        if a != "relu":
            out.append(None)
            continue
        own = Z[l + 1] > 0
        if given is not None and given[l] is not None:
            own = np.where(kink_band(Z[l + 1], kink_tol), np.asarray(given[l]) > 0, own)
        out.append(own.astype(np.float64))
    return out


def batch_gradient(theta, dims, acts, X, Y, shards: int = 1, kink_tol: float = 0.0,
                   kink_given=None) -> np.ndarray:
    """Tendencies summed over the whole mini-batch.  The batch is split into
    `shards` equal contiguous pieces whose sums are added in piece order, the
    single-process picture of the collective sum of section 3.5.  With
    kink_given, relu units within kink_tol * rms(z) of the kink (rms over the
    whole batch) take the sides given for them (kink_sides); without it,
    kink_tol > 0 takes the other side for them (piece_gradient)."""
    X = np.asarray(X)
    B = X.shape[0]
    if shards < 1 or B % shards != 0:
        raise ValueError("the batch must split evenly into the shards")
    per = B // shards
    sides = kink_sides(theta, dims, acts, X, kink_tol, kink_given) if kink_given is not None else None
    total = None
    for k in range(shards):
        rows = slice(k * per, (k + 1) * per)
        if sides is None:
            gk = piece_gradient(theta, dims, acts, X[rows], Y[rows], kink_tol)
        else:
            gk = piece_gradient(theta, dims, acts, X[rows], Y[rows], 0.0,
                                [None if sd is None else sd[rows] for sd in sides])
        total = gk if total is None else total + gk
    return total


def train_batch(theta, dims, acts, X, Y, eta, shards: int = 1, precision="f32",
                kink_tol: float = 0.0, kink_given=None):
    """One SGD step on a mini-batch: theta - (eta / B) * (summed tendencies).
    Returns (new theta, summed tendencies in fp64)."""
    B = np.asarray(X).shape[0]
    g = batch_gradient(theta, dims, acts, X, Y, shards, kink_tol, kink_given)
    new = np.asarray(theta, dtype=np.float64) - (eta / B) * g
    return _round(new, precision), g


def train_epoch(theta, dims, acts, X, Y, batch, eta, shards=1, precision="f32",
                callback=None):
    """Consecutive mini-batches [t B, (t+1) B) of (X, Y), one step each.
    ``callback(t, theta, grad)`` is called after every step."""
    n = np.asarray(X).shape[0]
    if batch <= 0 or n % batch != 0:
        raise ValueError("the sample count must be a multiple of the batch")
    for t in range(n // batch):
        theta, g = train_batch(theta, dims, acts, X[t * batch:(t + 1) * batch],
                               Y[t * batch:(t + 1) * batch], eta, shards, precision)
        if callback is not None:
            callback(t, theta, g)
    return theta


def window_start(pos: float, n: int, batch: int, precision: str = "f32") -> int:
    """Start of the mini-batch window drawn by the example program of section
    4: the integer part of pos * (n - batch + 1), with pos uniform in [0, 1).
    The product is taken in the real kind of the run: fp32 (the paper's
    default) or fp64 (its real64 kind); a product that rounds up to
    n - batch + 1 is kept inside the sample set."""
    if not 0.0 <= pos < 1.0:
        raise ValueError("pos must lie in [0, 1)")
    if batch > n:
        raise ValueError("the window is longer than the sample set")
    if precision == "f32":
        prod = np.float32(pos) * np.float32(n - batch + 1)
    else:
        prod = np.float64(pos) * np.float64(n - batch + 1)
    return min(int(prod), n - batch)


def train_windows(theta, dims, acts, X, Y, batch, pos, eta, shards=1, precision="f32"):
    """One mini-batch step per entry of pos, in order, each on the window of
    ``batch`` samples that window_start places (section 4)."""
    n = np.asarray(X).shape[0]
    for p in pos:
        s = window_start(float(p), n, batch, precision)
        theta, _ = train_batch(theta, dims, acts, X[s:s + batch], Y[s:s + batch], eta, shards,
                               precision)
    return theta


def _first_argmax(v: np.ndarray) -> int:
    """Index of the first largest entry of v (Fortran's maxloc), or -1 when v
    holds a NaN."""
    best = 0
    for j in range(1, v.shape[0]):
        if np.isnan(v[j]):
            return -1
        if v[j] > v[best]:
            best = j
    return -1 if np.isnan(v[0]) else best


def correct_count(out, Y) -> int:
    """Number of rows whose output and one-hot target peak at the same index
    (section 4's accuracy before dividing by the sample count); a row with a
    NaN counts as incorrect."""
    n = 0
    for o, y in zip(np.asarray(out), np.asarray(Y)):
        i, j = _first_argmax(o), _first_argmax(y)
        n += int(i >= 0 and i == j)
    return n


def accuracy(theta, dims, acts, X, labels) -> float:
    """Fraction of samples whose largest output (first index among ties) is
    the label."""
    out = output(theta, dims, acts, X)
    return float(np.mean(np.argmax(out, axis=1) == np.asarray(labels)))
