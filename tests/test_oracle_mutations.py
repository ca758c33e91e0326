"""Plant one mistake at a time in a copy of the CPU reference and show that
the pins catch it.  This runs on the CPU only; the reference itself is not
modified."""

import importlib.util
import inspect
import types

import pytest

from oracle import mlp

from . import pins

MUTATIONS = {
    "bias dropped from the forward pass": [
        ("zl = W @ a[-1] + b", "zl = W @ a[-1]"),
        ("Zl = A[-1] @ W.T + b", "Zl = A[-1] @ W.T"),
    ],
    "output delta sign flipped": [
        ("(a[L] - y) *", "(y - a[L]) *"),
        ("(A[L] - Yd) *", "(Yd - A[L]) *"),
    ],
    "derivative taken with the next layer's activation": [
        ("act_prime(acts[l - 1], z[l])", "act_prime(acts[l], z[l])"),
        ("act_prime(acts[l - 1], Z[l])", "act_prime(acts[l], Z[l])"),
    ],
    "derivative taken at the activation instead of z": [
        ("act_prime(acts[l - 1], z[l])", "act_prime(acts[l - 1], a[l])"),
        ("act_prime(acts[l - 1], Z[l])", "act_prime(acts[l - 1], A[l])"),
    ],
    "update uses eta instead of eta / B": [
        ("(eta / B) * g", "eta * g"),
    ],
    "last shard dropped from the sum": [
        ("for k in range(shards):", "for k in range(max(1, shards - 1)):"),
    ],
    "bias tendency averaged instead of summed": [
        ("D.sum(axis=0)", "D.mean(axis=0)"),
    ],
    "sigmoid derivative squared": [
        ("return _sigmoid(z) * _sigmoid(-z)", "return _sigmoid(z) * _sigmoid(z)"),
    ],
    "tanh derivative off by a factor": [
        ("return 1.0 / (c * c)", "return 1.0 / c"),
    ],
    "relu derivative true at zero": [
        ('if name == "relu":\n        return np.where(z > 0, 1.0, 0.0)',
         'if name == "relu":\n        return np.where(z >= 0, 1.0, 0.0)'),
    ],
    "cost without the one half": [
        ("return 0.5 * float(np.sum(d * d))", "return float(np.sum(d * d))"),
    ],
    "window span without the last start": [
        ("np.float32(n - batch + 1)", "np.float32(n - batch)"),
    ],
    "window start rounded instead of truncated": [
        ("return min(int(prod), n - batch)", "return min(int(np.rint(prod)), n - batch)"),
    ],
    "equal largest outputs resolved to the last index": [
        ("if v[j] > v[best]:", "if v[j] >= v[best]:"),
    ],
    "weight tendency built from z instead of the activation": [
        ("dW[l] = np.outer(delta, a[l])", "dW[l] = np.outer(delta, z[l] if l > 0 else a[l])"),
        ("(D.T @ A[l], D.sum(axis=0))", "(D.T @ (Z[l] if l > 0 else A[l]), D.sum(axis=0))"),
    ],
}


def _mutant(edits):
    src = inspect.getsource(mlp)
    for old, new in edits:
        assert old in src, f"mutation anchor not found: {old!r}"
        src = src.replace(old, new)
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src, "oracle_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(name):
    mutant = _mutant(MUTATIONS[name])
    caught = []
    for check in pins.ALL_CHECKS:
        try:
            fails = check(mutant)
        except Exception as e:  # a crash also counts as caught
            fails = [f"raised {type(e).__name__}"]
        if fails:
            caught.append(check.__name__)
    assert caught, f"no pin catches: {name}"
