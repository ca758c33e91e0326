"""CPU reference for mini-batch MLP training (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package; the GPU library never does.
"""
from . import mlp  # noqa: F401
