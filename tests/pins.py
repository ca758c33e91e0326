"""Checks that pin the CPU reference to facts outside itself.

Each check takes the reference module as an argument and returns a list of
failure messages (empty when the check passes), so that the mutation tests
can run the same checks against copies of the reference with a planted
mistake and show that at least one check catches it.
"""

from __future__ import annotations

import ast
import json
import math
import operator
import os
from typing import Callable, List

import numpy as np

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

_CONST = {"ln2": math.log(2.0), "ln3": math.log(3.0), "e": math.e}
_OPS = {ast.Add: operator.add, ast.Sub: operator.sub, ast.Mult: operator.mul,
        ast.Div: operator.truediv, ast.Pow: operator.pow, ast.USub: operator.neg,
        ast.UAdd: operator.pos}


def expr(s: str) -> float:
    """Evaluate a fixture expression: numbers, + - * / **, ln2, ln3, e."""
    def ev(n):
        if isinstance(n, ast.Expression):
            return ev(n.body)
        if isinstance(n, ast.Constant) and isinstance(n.value, (int, float)):
            return float(n.value)
        if isinstance(n, ast.Name) and n.id in _CONST:
            return _CONST[n.id]
        if isinstance(n, ast.BinOp) and type(n.op) in _OPS:
            return _OPS[type(n.op)](ev(n.left), ev(n.right))
        if isinstance(n, ast.UnaryOp) and type(n.op) in _OPS:
            return _OPS[type(n.op)](ev(n.operand))
        raise ValueError(f"unsupported fixture expression {s!r}")
    return ev(ast.parse(s, mode="eval"))


def arr(v) -> np.ndarray:
    if isinstance(v, str):
        return np.array(expr(v))
    return np.array([arr(x) for x in v], dtype=np.float64)


def load_hand_worked():
    with open(os.path.join(GOLDEN, "hand_worked.json")) as f:
        return json.load(f)["cases"]


def _close(a, b, tol) -> bool:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return a.shape == b.shape and bool(np.all(np.abs(a - b) <= tol * (1.0 + np.abs(b))))


def check_hand_worked(m) -> List[str]:
    """Forward outputs, cost, summed tendencies and updated parameters of the
    hand-worked tiny networks."""
    fails = []
    for c in load_hand_worked():
        dims, acts = c["dims"], c["acts"]
        theta = arr(c["params"])
        X, Y = arr(c["x"]), arr(c["y"])
        eta = float(expr(c["eta"]))
        if not _close(m.output(theta, dims, acts, X), arr(c["out"]), 1e-14):
            fails.append(f"{c['name']}: output")
        if not _close(m.cost(theta, dims, acts, X, Y), expr(c["cost"]), 1e-14):
            fails.append(f"{c['name']}: cost")
        for s in c["shards"]:
            g = m.batch_gradient(theta, dims, acts, X, Y, s)
            if not _close(g, arr(c["grad"]), 1e-14):
                fails.append(f"{c['name']}: gradient (shards={s})")
            new, _ = m.train_batch(theta, dims, acts, X, Y, eta, s, precision="f64")
            if not _close(new, arr(c["new_params"]), 1e-14):
                fails.append(f"{c['name']}: updated parameters (shards={s})")
        if X.shape[0] == 1:
            new1 = m.train_single(theta, dims, acts, X[0], Y[0], eta, precision="f64")
            if not _close(new1, arr(c["new_params"]), 1e-14):
                fails.append(f"{c['name']}: train_single")
    return fails


def check_activation_values(m) -> List[str]:
    """Values the functions take at points where they have closed forms."""
    l2, l3 = math.log(2.0), math.log(3.0)
    cases = [
        ("sigmoid", 0.0, 0.5, 0.25), ("sigmoid", l3, 0.75, 3.0 / 16.0),
        ("sigmoid", -l3, 0.25, 3.0 / 16.0),
        ("tanh", 0.0, 0.0, 1.0), ("tanh", l2, 0.6, 16.0 / 25.0), ("tanh", -l2, -0.6, 16.0 / 25.0),
        ("gaussian", 0.0, 1.0, 0.0), ("gaussian", 1.0, math.exp(-1.0), -2.0 * math.exp(-1.0)),
        ("gaussian", -1.0, math.exp(-1.0), 2.0 * math.exp(-1.0)),
        ("relu", -2.0, 0.0, 0.0), ("relu", 2.5, 2.5, 1.0), ("relu", 0.0, 0.0, 0.0),
        ("relu", -0.0, 0.0, 0.0),
        ("step", -2.0, 0.0, 0.0), ("step", 2.5, 1.0, 0.0), ("step", 0.0, 0.0, 0.0),
    ]
    fails = []
    for name, z, f, fp in cases:
        got_f = float(m.act(name, np.array([z]))[0])
        got_fp = float(m.act_prime(name, np.array([z]))[0])
        if abs(got_f - f) > 1e-15 * (1 + abs(f)):
            fails.append(f"{name}({z}) = {got_f}, expected {f}")
        if abs(got_fp - fp) > 1e-15 * (1 + abs(fp)):
            fails.append(f"{name}'({z}) = {got_fp}, expected {fp}")
    # saturated sigmoid: sigma'(z) = e^-|z| / (1 + e^-|z|)^2 -> e^-|z| (1 - 2 e^-|z|)
    for z in (30.0, -30.0, 60.0):
        got = float(m.act_prime("sigmoid", np.array([z]))[0])
        if abs(got / math.exp(-abs(z)) - 1.0) > 1e-12:
            fails.append(f"sigmoid'({z}) loses relative accuracy: {got}")
    # saturated tanh: 1 - tanh^2(z) = 4 e^-2|z| / (1 + e^-2|z|)^2 -> 4 e^-2|z|
    for z in (20.0, -25.0):
        got = float(m.act_prime("tanh", np.array([z]))[0])
        if abs(got / (4.0 * math.exp(-2.0 * abs(z))) - 1.0) > 1e-12:
            fails.append(f"tanh'({z}) loses relative accuracy: {got}")
    return fails


def check_activation_fd(m) -> List[str]:
    """Each derivative against a central difference of its function."""
    rng = np.random.default_rng(11)
    z = rng.uniform(-4.0, 4.0, 400)
    z = z[np.abs(z) > 1e-2]                # away from the relu / step kink
    h = 1e-6
    fails = []
    for name in ("sigmoid", "tanh", "gaussian", "relu", "step"):
        fd = (m.act(name, z + h) - m.act(name, z - h)) / (2 * h)
        an = m.act_prime(name, z)
        err = np.max(np.abs(fd - an))
        if err > 1e-8:
            fails.append(f"{name}': central difference disagrees by {err:.3e}")
    return fails


FD_NETS = [
    # the paper's own example network, [3, 5, 2] with tanh (section 3.1)
    ((3, 5, 2), ("tanh",)),
    ((4, 3, 3, 2), ("sigmoid",)),
    ((4, 3, 3, 2), ("tanh",)),
    ((4, 3, 3, 2), ("gaussian",)),
    ((4, 3, 3, 2), ("relu",)),
    ((5, 4, 3, 3), ("tanh", "relu", "sigmoid")),
]


def _fd_problem(dims, seed, batch=3):
    rng = np.random.default_rng(seed)
    n = sum(dims[l] * dims[l - 1] + dims[l] for l in range(1, len(dims)))
    theta = rng.normal(0.0, 0.7, n)
    X = rng.uniform(-1.0, 1.0, (batch, dims[0]))
    Y = rng.uniform(0.0, 1.0, (batch, dims[-1]))
    return theta, X, Y


def check_gradient_fd(m) -> List[str]:
    """The summed tendencies are the gradient of the summed quadratic cost:
    central differences of the cost, parameter by parameter, in fp64."""
    fails = []
    for i, (dims, acts) in enumerate(FD_NETS):
        theta, X, Y = _fd_problem(dims, 100 + i)
        acts_full = list(acts) * (len(dims) - 1) if len(acts) == 1 else list(acts)
        if "relu" in acts_full:
            # keep every relu pre-activation away from the kink
            Z, _ = m.forward(theta, dims, acts_full, X)
            if min(np.min(np.abs(z)) for z in Z[1:]) < 1e-3:
                fails.append(f"{dims}: fd problem too close to a relu kink")
                continue
        g = m.batch_gradient(theta, dims, acts_full, X, Y)
        h = 1e-6
        fd = np.empty_like(theta)
        for j in range(theta.size):
            tp, tm = theta.copy(), theta.copy()
            tp[j] += h
            tm[j] -= h
            fd[j] = (m.cost(tp, dims, acts_full, X, Y) - m.cost(tm, dims, acts_full, X, Y)) / (2 * h)
        err = np.max(np.abs(fd - g)) / max(1e-3, np.max(np.abs(fd)))
        if not err < 1e-6:
            fails.append(f"{dims} {acts}: finite-difference gradient off by {err:.3e}")
    return fails


def check_gradient_autograd(m) -> List[str]:
    """The summed tendencies against torch.autograd (fp64, CPU) of the summed
    quadratic cost of the same network, built from torch's own layers."""
    import torch
    fails = []
    act_fn: dict = {
        "sigmoid": torch.sigmoid, "tanh": torch.tanh, "relu": torch.relu,
        "gaussian": lambda t: torch.exp(-t * t),
    }
    for i, (dims, acts) in enumerate(FD_NETS):
        theta, X, Y = _fd_problem(dims, 200 + i, batch=7)
        acts_full = list(acts) * (len(dims) - 1) if len(acts) == 1 else list(acts)
        params, off = [], 0
        for l in range(1, len(dims)):
            n, k = dims[l], dims[l - 1]
            W = torch.tensor(theta[off:off + n * k].reshape(n, k), dtype=torch.float64,
                             requires_grad=True)
            off += n * k
            b = torch.tensor(theta[off:off + n], dtype=torch.float64, requires_grad=True)
            off += n
            params += [W, b]
        h = torch.tensor(X, dtype=torch.float64)
        for l in range(len(dims) - 1):
            h = act_fn[acts_full[l]](torch.nn.functional.linear(h, params[2 * l], params[2 * l + 1]))
        loss = 0.5 * torch.sum((h - torch.tensor(Y, dtype=torch.float64)) ** 2)
        loss.backward()
        ref = torch.cat([p.grad.reshape(-1) for p in params]).numpy()
        g = m.batch_gradient(theta, dims, acts_full, X, Y)
        err = np.max(np.abs(ref - g)) / max(1e-12, np.max(np.abs(ref)))
        if not err < 1e-12:
            fails.append(f"{dims} {acts}: autograd disagrees by {err:.3e}")
    return fails


def check_sum_of_samples(m) -> List[str]:
    """The batch tendencies equal the sum of the single-sample tendencies."""
    fails = []
    for i, (dims, acts) in enumerate(FD_NETS):
        theta, X, Y = _fd_problem(dims, 300 + i, batch=6)
        acts_full = list(acts) * (len(dims) - 1) if len(acts) == 1 else list(acts)
        g = m.batch_gradient(theta, dims, acts_full, X, Y)
        s = sum(m.sample_gradient(theta, dims, acts_full, X[j], Y[j]) for j in range(X.shape[0]))
        if np.max(np.abs(g - s)) > 1e-12 * (1 + np.max(np.abs(s))):
            fails.append(f"{dims}: batch != sum of samples")
    return fails


def check_partition(m) -> List[str]:
    """Any partition of the batch sums to the full-batch tendencies, and the
    shard count changes nothing but rounding."""
    fails = []
    rng = np.random.default_rng(5)
    dims, acts = (6, 5, 4), ("tanh", "sigmoid")
    theta, X, Y = _fd_problem(dims, 400, batch=12)
    full = m.piece_gradient(theta, dims, acts, X, Y)
    for S in (1, 2, 3, 4, 6, 12):
        g = m.batch_gradient(theta, dims, acts, X, Y, S)
        if np.max(np.abs(g - full)) > 1e-12 * (1 + np.max(np.abs(full))):
            fails.append(f"shards={S} differs from the whole batch")
    perm = rng.permutation(12)
    cuts = [0, 5, 7, 12]
    parts = sum(m.piece_gradient(theta, dims, acts, X[perm[a:b]], Y[perm[a:b]])
                for a, b in zip(cuts[:-1], cuts[1:]))
    if np.max(np.abs(parts - full)) > 1e-12 * (1 + np.max(np.abs(full))):
        fails.append("an uneven shuffled partition does not sum to the batch")
    return fails


def check_replicated_sample(m) -> List[str]:
    """A batch of B copies of one sample takes exactly the single-sample step
    with the same eta (the eta/B reading of the update)."""
    fails = []
    dims, acts = (4, 3, 2), ("sigmoid",)
    theta, X, Y = _fd_problem(dims, 500, batch=1)
    one = m.train_single(theta, dims, acts, X[0], Y[0], 0.7, precision="f64")
    for B in (2, 5, 16):
        many, _ = m.train_batch(theta, dims, acts, np.repeat(X, B, 0), np.repeat(Y, B, 0), 0.7,
                                precision="f64")
        if np.max(np.abs(many - one)) > 1e-12:
            fails.append(f"B={B} copies differ from the single-sample step")
    return fails


def check_uniform_acts(m) -> List[str]:
    """One activation name means that activation on every layer."""
    dims = (4, 3, 3, 2)
    theta, X, Y = _fd_problem(dims, 600)
    a = m.batch_gradient(theta, dims, ["tanh"], X, Y)
    b = m.batch_gradient(theta, dims, ["tanh"] * 3, X, Y)
    return [] if np.array_equal(a, b) else ["a single activation is not applied to all layers"]


def check_accuracy(m) -> List[str]:
    """Accuracy counts samples whose largest output (first index among equal
    ones) is the label: a one-layer identity-like network worked by hand."""
    # dims [3, 3], relu, W = I, b = 0: the output equals the (non-negative) input
    theta = np.concatenate([np.eye(3).ravel(), np.zeros(3)])
    X = np.array([[0.9, 0.1, 0.2],     # argmax 0
                  [0.5, 0.5, 0.1],     # tie: first index, 0
                  [0.0, 0.3, 0.7],     # argmax 2
                  [0.2, 0.8, 0.8]])    # tie: 1
    labels = np.array([0, 1, 2, 1])
    got = m.accuracy(theta, (3, 3), ["relu"], X, labels)
    return [] if got == 0.75 else [f"accuracy {got}, expected 3/4"]


def check_kink_side(m) -> List[str]:
    """The other side of the relu kink, worked by hand: x = 1, W1 = 1, b1 = -1
    puts z1 exactly at the kink; W2 = 2, b2 = 1, y = 0 (relu output, z2 = 1).
    The method: relu'(0) = 0, so the tendencies are dW1 = db1 = dW2 = 0 and
    db2 = 1.  Taking the other side: delta1 = 2, so dW1 = db1 = 2."""
    theta = np.array([1.0, -1.0, 2.0, 1.0])
    X, Y = np.array([[1.0]]), np.array([[0.0]])
    fails = []
    g0 = m.batch_gradient(theta, (1, 1, 1), ["relu"], X, Y)
    g1 = m.batch_gradient(theta, (1, 1, 1), ["relu"], X, Y, kink_tol=1e-5)
    if not np.array_equal(g0, [0.0, 0.0, 0.0, 1.0]):
        fails.append(f"tendencies at the kink {g0}")
    if not np.array_equal(g1, [2.0, 2.0, 0.0, 1.0]):
        fails.append(f"tendencies on the other side of the kink {g1}")
    # sides given for the units in the band: "above" gives the other side,
    # "below" the method's own; a given side outside the band is ignored
    # (b1 = -0.5: z1 = 0.5, a1 = 0.5, z2 = 2, delta2 = 2, delta1 = 4)
    up, down = [np.array([[1.0]]), None], [np.array([[0.0]]), None]
    g_up = m.batch_gradient(theta, (1, 1, 1), ["relu"], X, Y, kink_tol=1e-5, kink_given=up)
    g_dn = m.batch_gradient(theta, (1, 1, 1), ["relu"], X, Y, kink_tol=1e-5, kink_given=down)
    if not np.array_equal(g_up, [2.0, 2.0, 0.0, 1.0]):
        fails.append(f"given side above the kink {g_up}")
    if not np.array_equal(g_dn, [0.0, 0.0, 0.0, 1.0]):
        fails.append(f"given side below the kink {g_dn}")
    clear = np.array([1.0, -0.5, 2.0, 1.0])
    g_cl = m.batch_gradient(clear, (1, 1, 1), ["relu"], X, Y, kink_tol=1e-5, kink_given=down)
    if not np.array_equal(g_cl, [4.0, 4.0, 1.0, 2.0]):
        fails.append(f"a given side outside the band changed the tendencies {g_cl}")
    # two samples, one at the kink and one clear of it, in one or two shards:
    # the band is taken over the whole batch and each shard gets its rows
    X2, Y2 = np.array([[1.0], [1.5]]), np.array([[0.0], [0.0]])
    given2 = [np.array([[1.0], [0.0]]), None]
    g_1 = m.batch_gradient(theta, (1, 1, 1), ["relu"], X2, Y2, 1, kink_tol=1e-5, kink_given=given2)
    g_2 = m.batch_gradient(theta, (1, 1, 1), ["relu"], X2, Y2, 2, kink_tol=1e-5, kink_given=given2)
    # sample 2: z1 = 0.5, a1 = 0.5, z2 = 2, delta2 = 2, delta1 = 4, x = 1.5
    want2 = np.array([2.0 + 6.0, 2.0 + 4.0, 0.0 + 1.0, 1.0 + 2.0])
    if not (np.array_equal(g_1, want2) and np.array_equal(g_2, want2)):
        fails.append(f"given sides over shards {g_1} {g_2}, expected {want2}")
    return fails


def check_window_starts(m) -> List[str]:
    """The window start of section 4 is the integer part of pos * (n - B + 1):
    exact on a grid of pos = k / 64 (products exact in fp32), 0 at pos = 0,
    the last window n - B at the largest fp32 below 1, and every start in
    0 .. n - B reached, none outside."""
    fails = []
    for n in range(1, 41):
        for b in range(1, n + 1):
            span = n - b + 1
            seen = set()
            for k in range(64):
                got = m.window_start(k / 64.0, n, b)
                if got != (k * span) // 64:
                    fails.append(f"n={n} B={b} pos={k}/64: start {got}, expected {(k * span) // 64}")
                    return fails
                seen.add(got)
            if span <= 64 and seen != set(range(span)):
                fails.append(f"n={n} B={b}: starts {sorted(seen)} do not cover 0..{span - 1}")
                return fails
    top = float(np.nextafter(np.float32(1.0), np.float32(0.0)))
    for span in (1, 2, 3, 1000, 59001, (1 << 23) + 1, (1 << 24) - 1):
        got = m.window_start(top, span + 99, 100)
        if got != span - 1:
            fails.append(f"span {span}: start at the top of [0,1) is {got}, expected {span - 1}")
    # the real64 kind: the same grid, and the largest double below 1
    for n, b in ((40, 7), (1000, 100), (60000, 1000)):
        span = n - b + 1
        for k in range(64):
            got = m.window_start(k / 64.0, n, b, "f64")
            if got != (k * span) // 64:
                fails.append(f"f64 n={n} B={b} pos={k}/64: start {got}")
                return fails
    top64 = float(np.nextafter(1.0, 0.0))
    for span in (1, 3, 59001, (1 << 24) - 1, (1 << 40) + 1):
        got = m.window_start(top64, span + 99, 100, "f64")
        if got != span - 1:
            fails.append(f"f64 span {span}: start at the top of [0,1) is {got}, expected {span - 1}")
    return fails


def check_windows_sequential(m) -> List[str]:
    """Windows placed back to back (pos_t = (t B + 1/2) / (n - B + 1)) are the
    consecutive mini-batches of one epoch, taken in the same order: the two
    training loops give identical parameters."""
    rng = np.random.default_rng(7)
    dims, acts = (3, 4, 2), ["sigmoid", "sigmoid"]
    theta = rng.normal(size=m.param_count(dims))
    X, Y = rng.uniform(size=(12, 3)), rng.uniform(size=(12, 2))
    B = 3
    pos = [(t * B + 0.5) / (12 - B + 1) for t in range(4)]
    a = m.train_windows(theta, dims, acts, X, Y, B, pos, 0.5, precision="f64")
    e = m.train_epoch(theta, dims, acts, X, Y, B, 0.5, precision="f64")
    fails = [] if np.array_equal(a, e) else ["back-to-back windows differ from one epoch"]
    rev = m.train_windows(theta, dims, acts, X, Y, B, pos[::-1], 0.5, precision="f64")
    if np.array_equal(rev, e):
        fails.append("the order of the windows has no effect")
    return fails


def check_correct_count(m) -> List[str]:
    """Outputs against one-hot targets, worked by hand: the first index among
    equal largest outputs is the prediction, and a NaN row never counts."""
    out = np.array([[0.9, 0.1, 0.2],        # predicts 0, target 0: correct
                    [0.5, 0.5, 0.1],        # tie, predicts 0, target 1: wrong
                    [0.0, 0.3, 0.7],        # predicts 2, target 2: correct
                    [0.2, 0.8, 0.8],        # tie, predicts 1, target 1: correct
                    [0.1, np.nan, 0.9],     # NaN: wrong
                    [0.3, 0.3, 0.3]])       # all equal, predicts 0, target 0: correct
    Y = np.eye(3)[[0, 1, 2, 1, 2, 0]]
    got = m.correct_count(out, Y)
    return [] if got == 4 else [f"correct count {got}, expected 4"]


ALL_CHECKS: List[Callable] = [
    check_hand_worked, check_activation_values, check_activation_fd, check_gradient_fd,
    check_gradient_autograd, check_sum_of_samples, check_partition, check_replicated_sample,
    check_uniform_acts, check_accuracy, check_kink_side, check_window_starts,
    check_windows_sequential, check_correct_count,
]
