"""The CPU reference against facts outside itself: hand-worked networks,
closed forms of the activations, finite differences, torch.autograd, and the
invariants of the batch sum (sections 3.2-3.5 of the paper)."""

import pytest

from oracle import mlp

from . import pins


@pytest.mark.parametrize("check", pins.ALL_CHECKS, ids=lambda c: c.__name__)
def test_pin(check):
    fails = check(mlp)
    assert not fails, "\n".join(fails)
